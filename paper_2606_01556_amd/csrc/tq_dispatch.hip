// Kernel selection for the fused layer by token count: the decode kernel for
// m <= 16 (bound by the weight bytes; H formed in every work-group), the mid kernel
// (32-token blocks, H formed per block) up to 512 tokens, then the large
// kernel (128 x 256 blocks, 16 wavefronts), or once its blocks take more
// than one round over the CUs the prefill kernel (H shared by runs of column
// blocks) -- for r <= 64 only where a run is long enough to carry its H pass;
// past 512 tokens the mid kernel again where the large kernel's blocks would
// leave most CUs idle.
#include "tq_kernels.hpp"

namespace tq {

// one round of large-kernel blocks in the mid kernel's cost units, for 64-
// and 128-wide groups (fitted to measured mid and large times: 164 layer
// shapes with K 4096-28672, N 1024-14336, r 0-128, M 576-4096, and the
// LLaMA3 shapes of both group widths)
constexpr int kLargeRound64 = 34, kLargeRound128 = 28;
// K-groups per prefill work-group run from which it beats the large kernel at r <= 64
constexpr int kPrefillMinRun = 256;

int choose_kernel(const GemmArgs &a) {
  if (a.force_kernel >= 0) return a.force_kernel;   // validated by the caller
  // the activation code format follows the same token-count split
  if (a.m <= kDecodeMaxTokens && decode_fits(a.m, a.geo.k)) return kKernelDecode;
  if (!act_codes_fp8(a.m)) return kKernelMid;
  // 128 x 256 blocks: the large kernel (16 wavefronts, H formed in the main
  // loop of every block) is faster while its blocks fit in one round over the
  // 256 CUs; beyond, the prefill kernel forms H once per run of column blocks
  // (one work-group per CU).  For ranks up to 64 the large kernel's H share
  // is at most a quarter of a block's work, so the prefill kernel wins only
  // where its run (cpw column blocks of KG groups each) is long -- at least
  // kPrefillMinRun groups -- for its H pass and per-block fills to amortize.
  const int m_tiles = (a.m + 127) / 128, n_tiles = (a.geo.n_pad + 255) / 256;
  const int blocks = m_tiles * n_tiles;
  const int runs = m_tiles >= 256 ? 1 : 256 / m_tiles;
  const int cpw = (n_tiles + runs - 1) / runs;
  const bool long_run = cpw * (a.geo.k / 64) >= kPrefillMinRun;   // 64-wide K-groups
  // With 128-wide groups the large kernel chains two dependent products per H
  // tile in its main loop, and the prefill kernel applies half the scale
  // products per K block: the prefill kernel wins past one round of blocks
  // at every rank but 0.
  const bool prefill_wins = a.geo.gk == 1 ? a.geo.r_pad32 > 64 || long_run : a.geo.r_pad32 > 0;
  const bool large = blocks <= 256 || !prefill_wins;
  // Few large blocks leave most CUs idle (a round of them costs about as much
  // as kLargeRound64 / kLargeRound128 tile-group units of the mid kernel,
  // whose 32-token blocks fill the CUs at these sizes too): take the cheaper
  // of the two.
  const int rounds = (blocks + 255) / 256;
  const int large_round = a.geo.gk == 1 ? kLargeRound64 : kLargeRound128;
  const bool mid = large && dual_gemm_mid_cost(a) < rounds * large_round;
  if (mid) return kKernelMid;
  return large ? kKernelLarge : kKernelPrefill;
}

hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s) {
  switch (choose_kernel(a)) {
    case kKernelDecode: return launch_dual_gemm_decode(a, nullptr, s);
    case kKernelMid: return launch_dual_gemm_mid(a, s);
    case kKernelLarge: return launch_dual_gemm_large(a, s);
    default: return launch_dual_gemm_prefill(a, s);
  }
}

}  // namespace tq
