// Host-side launch interface of the TwinQuant kernels (internal to libtq).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tq {

// Largest supported rank; token counts served by the decode kernel.
constexpr int kMaxRank = 128;
constexpr int kDecodeMaxTokens = 16;

// Token counts up to kMidMaxTokens run the decode and mid kernels, which take
// the activation codes as TQ4 nibbles (k / 2 bytes per token).  Larger counts
// run the large and prefill kernels, which are bound by vector-ALU work and
// take the codes already expanded to their fp8 operand bytes (k bytes per
// token), so none of their wavefronts unpacks an activation operand.
constexpr int kMidMaxTokens = 512;
inline bool act_codes_fp8(int m) { return m > kMidMaxTokens; }
inline size_t act_codes_bytes(int m, int k) {
  const size_t m32 = (size_t)(m + 31) / 32 * 32;
  return act_codes_fp8(m) ? m32 * (size_t)k : m32 * (size_t)k / 2;
}

// Geometry shared by the packing, export and GEMM kernels.
//  W_res codes: [n_pad/32][k/64] blocks of 1 KiB; block lane L (16 bytes,
//               4 TQ4 words) holds column 32*t + L%32, k in [32*(L/32), +32)
//               of the group.  Scales: [k/64][n_pad] fp16.
//  L1 codes:    the same block format with the rank index as the column:
//               [r_pad32/32][k/64] blocks.  Scales: [k/64][r_pad32] fp16.
//  L2 codes:    [n_pad/32][r_pad64/64] blocks, the rank index as the
//               reduction axis (zero past r).  Scales: [r/group_r][n_pad].
struct Geometry {
  int n, k, r, gr, n_pad, r_pad32, r_pad64;
  int gk;   // 64-wide K blocks per quantization group (group / 64: 1 or 2)
  uint64_t off_w, off_ws, off_l1, off_l1s, off_l2, off_l2s;
};

struct GemmArgs {
  const uint8_t *packed;
  Geometry geo;
  const uint32_t *xc;   // [m32/32][k/64] activation tiles (matrix-core lane order):
                        // 1 KiB of TQ4 nibbles, or 2 KiB of fp8 bytes if act_codes_fp8(m)
  const uint16_t *xs;   // [k/64][ms] fp16
  int ms;               // row stride of xs: m rounded up to a multiple of 32 (= m32)
  void *y;              // [m][n]
  int m;
  int bf16_out;
  float *dbg_h;         // optional [m][r]
  float *dbg_sh;        // optional [m][r/gr]
  int8_t *dbg_qh;       // optional [m][r]
  int force_kernel;     // -1: chosen by choose_kernel; else a kKernel* value (tests)
  int mid_ct;           // 0: chosen by the mid kernel's cost model; else 1, 2 or 4 (tests)
};

// gk: 64-wide K blocks per quantization group (1 or 2)
hipError_t launch_quant_act(const uint16_t *x, int m, int k, int gk, uint32_t *codes,
                            uint16_t *scales, hipStream_t s);
hipError_t launch_pack(const Geometry &g, const uint16_t *w, const uint16_t *l1,
                       const uint16_t *l2, uint8_t *packed, hipStream_t s);
hipError_t launch_export_canonical(const Geometry &g, const uint8_t *packed, uint8_t *wq, uint16_t *ws,
                                   uint8_t *l1q, uint16_t *l1s, uint8_t *l2q, uint16_t *l2s,
                                   hipStream_t s);
hipError_t launch_act_canonical(const uint8_t *x_codes, const uint16_t *x_scales, int m, int k, int gk,
                                uint8_t *out_q, uint16_t *out_s, hipStream_t s);
hipError_t launch_export(const Geometry &g, const uint8_t *packed, uint32_t *wc, uint16_t *ws,
                         uint32_t *l1c, uint16_t *l1s, uint32_t *l2c, uint16_t *l2s,
                         hipStream_t s);
hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s);
// m <= kDecodeMaxTokens; xh = NULL: codes from a.xc / a.xs, else fp16
// activations [m][k] quantized inside the kernel
hipError_t launch_dual_gemm_decode(const GemmArgs &a, const uint16_t *xh, hipStream_t s);
// whether the decode kernel's LDS holds the activation codes of m tokens
bool decode_fits(int m, int k);
// the kernel launch_dual_gemm runs (values of tq_kernel in the C header)
constexpr int kKernelDecode = 0, kKernelMid = 1, kKernelLarge = 2, kKernelPrefill = 3;
int choose_kernel(const GemmArgs &a);
hipError_t launch_dual_gemm_mid(const GemmArgs &a, hipStream_t s);      // mid sizes
// relative time of the mid kernel's launch: rounds of work-groups over the
// CUs x tile-groups per work-group and chunk (+3 for its fixed latency)
int dual_gemm_mid_cost(const GemmArgs &a);
hipError_t launch_dual_gemm_prefill(const GemmArgs &a, hipStream_t s);  // prefill sizes
hipError_t launch_dual_gemm_large(const GemmArgs &a, hipStream_t s);    // large token counts
// the layer without fusion (comparison baseline): residual GEMM, stage 1 to
// global H, re-quantization, stage 2 added to the residual output
size_t unfused_scratch_bytes(int m, const Geometry &g);
hipError_t launch_dual_gemm_unfused(const GemmArgs &a, void *scratch, hipStream_t s);

}  // namespace tq
