// Kernel selection for the fused layer by token count: the decode kernel for
// m <= 16 (bound by the weight bytes and by H's K-long chain), the mid kernel
// (32-token blocks, H formed per block) up to a few hundred tokens, the
// prefill kernel (128-token blocks) beyond.
#include <stdlib.h>

#include "tq_kernels.hpp"

namespace tq {

hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s) {
  const char *env = getenv("TQ_MID_MAX");   // crossover override for tuning sweeps
  const int mid_max = env ? atoi(env) : 512;
  if (a.m <= 16) return launch_dual_gemm_decode(a, s);
  if (a.m <= mid_max) return launch_dual_gemm_mid(a, s);
  return launch_dual_gemm_prefill(a, s);
}

}  // namespace tq
