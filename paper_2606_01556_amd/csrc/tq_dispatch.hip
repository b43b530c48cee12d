// Kernel selection for the fused layer by token count: the decode kernel for
// m <= 16 (bound by the weight bytes and by H's K-long chain), the mid kernel
// (32-token blocks, H formed per block) up to 512 tokens, then the large
// kernel (128 x 256 blocks, 16 wavefronts), or for r > 64 once its blocks
// take more than one round over the CUs the prefill kernel (H shared by runs
// of column blocks).
#include <stdlib.h>

#include "tq_kernels.hpp"

namespace tq {

hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s) {
  // the activation code format follows the same token-count split
  if (a.m <= 16) return launch_dual_gemm_decode(a, s);
  if (!act_codes_fp8(a.m)) return launch_dual_gemm_mid(a, s);
  // 128 x 256 blocks: the large kernel (16 wavefronts, H formed in the main
  // loop of every block) is faster while its blocks fit in one round over the
  // 256 CUs, and for ranks up to 64 at any size (its H share is then at most a
  // quarter of a block's work); beyond, the prefill kernel forms H once per
  // run of column blocks
  const int blocks = (a.m + 127) / 128 * ((a.geo.n_pad + 255) / 256);
  int large = blocks <= 256 || a.geo.r_pad32 <= 64;
  // TQ_LARGE=0|1 forces either kernel (the tests run both on the same shapes)
  if (const char *lenv = getenv("TQ_LARGE")) large = atoi(lenv);
  if (large) return launch_dual_gemm_large(a, s);
  return launch_dual_gemm_prefill(a, s);
}

}  // namespace tq
