// Kernel selection for the fused layer by token count: the decode kernel for
// m <= 16 (bound by the weight bytes and by H's K-long chain), the prefill
// kernel otherwise (bound by the matrix cores and the vector ALU).
#include "tq_kernels.hpp"

namespace tq {

hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s) {
  if (a.m <= 16) return launch_dual_gemm_decode(a, s);
  return launch_dual_gemm_prefill(a, s);
}

}  // namespace tq
