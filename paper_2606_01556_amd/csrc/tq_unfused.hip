// The layer without kernel fusion, as the comparison baseline of the paper's
// kernel profile (Appendix, Kernel Profile): the residual 4-bit GEMM, the
// stage-1 product H written to global memory, its re-quantization in a kernel
// of its own (Q_H and s_H to global memory), and stage 2 adding Q_H Q(L2) to
// the residual output -- four launches where the fused layer takes one
// (Sec. 4.3 describes the intermediate traffic and launches that fusion
// removes).  The arithmetic is the fused layer's: H accumulates one fma per
// K-group in ascending order and is bit-identical to it, s_H = max|H| / 7 in
// fp32 with IEEE division, and Q_H rounds half to even; only Y differs, by
// the fp16 rounding of the residual output before the low-rank part is added.
//
// Scratch (caller-owned, tq_unfused_scratch_bytes):
//   H   fp32 [m32][r_pad32]           (row-major by token)
//   Q_H fp8 code bytes [m32][r_pad64] (ranks past r are zero)
//   s_H fp32 [r / group_r][m32]
#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

// activation operand of token tile t, group g (both activation formats)
template <bool FP8>
__device__ __forceinline__ v8i act_operand(const uint8_t *xc, int KG, int t, int g, int lane) {
  if constexpr (FP8) {
    const uint8_t *b = xc + ((int64_t)t * KG + g) * 2048 + lane * 16;
    const u32x4 lo = *reinterpret_cast<const u32x4 *>(b);
    const u32x4 hi = *reinterpret_cast<const u32x4 *>(b + 1024);
    return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
  } else {
    return unpack32(*reinterpret_cast<const u32x4 *>(xc + (((int64_t)t * KG + g) * 64 + lane) * 16));
  }
}

// Stage 1: one work-group of eight wavefronts per 32-token x 32-rank tile of
// H.  K runs in chunks of up to 32 groups: wavefront w forms the exact
// integer sums of groups w, w + 8, w + 16 and w + 24 of the chunk (one
// matrix-core product each, with the next chunk's operands already in
// flight) and stores them and the group scales in LDS; then each wavefront
// takes two of the tile's sixteen accumulator registers and runs the
// ascending-group chain over the chunk, one fma per group with the exact
// fp32 scale product s_x s_L1.
constexpr int kS1Waves = 8, kS1Gpw = 4, kS1Chunk = kS1Waves * kS1Gpw;
constexpr int kS1Lds = kS1Chunk * 16 * 64 * 4 + 2 * kS1Chunk * 32 * 4;

template <bool FP8>
__global__ __launch_bounds__(64 * kS1Waves) void unfused_stage1_kernel(GemmArgs a,
                                                                        float *__restrict__ h) {
  extern __shared__ __attribute__((aligned(16))) float s1_lds[];
  float *CS = s1_lds;                              // [chunk group][v][lane]
  float *SX = s1_lds + kS1Chunk * 16 * 64;         // [chunk group][32 tokens]
  float *SL = SX + kS1Chunk * 32;                  // [chunk group][32 ranks]
  const Geometry &geo = a.geo;
  const int t = blockIdx.x, rt = blockIdx.y, tid = threadIdx.x, lane = tid & 63, l32 = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KG = geo.k / kGroup;
  const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
  const uint8_t *l1 = a.packed + geo.off_l1 + (int64_t)rt * KG * 1024 + lane * 16;
  const uint16_t *l1s = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l1s);
  v8i av[kS1Gpw];
  u32x4 lraw[kS1Gpw];
  uint32_t sc[kS1Gpw];   // lanes 0-31: token scale, lanes 32-63: rank scale
  const int gk = geo.gk;   // 64-wide blocks per quantization group: scale row g / gk
  auto load = [&](int i, int g) {
    av[i] = act_operand<FP8>(xc, KG, t, g, lane);
    lraw[i] = *reinterpret_cast<const u32x4 *>(l1 + (int64_t)g * 1024);
    sc[i] = lane < 32 ? a.xs[(int64_t)(g / gk) * a.ms + 32 * t + l32]
                      : l1s[(int64_t)(g / gk) * geo.r_pad32 + 32 * rt + l32];
  };
#pragma unroll
  for (int i = 0; i < kS1Gpw; i++)
    if (i * kS1Waves + w < KG) load(i, i * kS1Waves + w);
  float acc0 = 0.0f, acc1 = 0.0f;
  const int v0 = 2 * w, row0 = row_of_32x32(lane, v0), row1 = row_of_32x32(lane, v0 + 1);
  for (int c0 = 0; c0 < KG; c0 += kS1Chunk) {
#pragma unroll
    for (int i = 0; i < kS1Gpw; i++) {
      const int gl = i * kS1Waves + w;
      if (c0 + gl < KG) {
        const v16f c = mfma_codes_32x32x64(av[i], unpack32(lraw[i]));
#pragma unroll
        for (int v = 0; v < 16; v++) CS[(gl * 16 + v) * 64 + lane] = c[v];
        const float sv = half_bits_to_float((uint16_t)sc[i]);
        if (lane < 32) SX[gl * 32 + l32] = sv;
        else SL[gl * 32 + l32] = sv;
      }
      if (c0 + kS1Chunk + gl < KG) load(i, c0 + kS1Chunk + gl);
    }
    __syncthreads();
    const int ng = min(kS1Chunk, KG - c0);
    // one step per quantization group: a 128-wide group adds its two blocks'
    // exact integer sums first (chunks start on group boundaries)
    for (int gl = 0; gl < ng; gl += gk) {
      const float sl = SL[gl * 32 + l32];
      float c0v = CS[(gl * 16 + v0) * 64 + lane], c1v = CS[(gl * 16 + v0 + 1) * 64 + lane];
      if (gk == 2) {
        c0v += CS[((gl + 1) * 16 + v0) * 64 + lane];
        c1v += CS[((gl + 1) * 16 + v0 + 1) * 64 + lane];
      }
      acc0 = fmaf(c0v, SX[gl * 32 + row0] * sl, acc0);
      acc1 = fmaf(c1v, SX[gl * 32 + row1] * sl, acc1);
    }
    __syncthreads();
  }
  h[(int64_t)(32 * t + row0) * geo.r_pad32 + 32 * rt + l32] = acc0;
  h[(int64_t)(32 * t + row1) * geo.r_pad32 + 32 * rt + l32] = acc1;
}

// Re-quantization: one lane per element of H; a wavefront covers 64 ranks of
// one token (a rank group is gr <= 64 consecutive lanes: its max comes from a
// butterfly over those lanes).  A 128-rank group: one wavefront per token,
// two ranks per lane (j and j + 64).
__global__ __launch_bounds__(256) void unfused_requant_kernel(const float *__restrict__ h, int m,
                                                              int m32, int r, int gr, int r_pad32,
                                                              int r_pad64, uint8_t *__restrict__ qh,
                                                              float *__restrict__ sh) {
  const int lane = threadIdx.x & 63;
  const int64_t wv = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);   // (token, 64-rank block)
  if (gr > 64) {
    if (wv >= m32) return;
    const int row = (int)wv;
    float hv[2];
    float amax = 0.0f;
    for (int b = 0; b < 2; b++) {
      const int j = 64 * b + lane;
      hv[b] = row < m && j < r ? h[(int64_t)row * r_pad32 + j] : 0.0f;
      amax = fmaxf(amax, fabsf(hv[b]));
    }
    for (int msk = 1; msk < 64; msk <<= 1) amax = fmaxf(amax, __shfl_xor(amax, msk));
    const float s = amax / 7.0f;
    for (int b = 0; b < 2; b++) {
      int q = 0;
      if (row < m && s != 0.0f) {
        float tq = __builtin_rintf(hv[b] / s);
        tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
        q = (int)tq;
      }
      qh[(int64_t)row * r_pad64 + 64 * b + lane] = (uint8_t)code_to_fp8(q);
    }
    if (lane == 0) sh[row] = row < m ? s : 0.0f;
    return;
  }
  const int RB = r_pad64 / 64;
  if (wv >= (int64_t)m32 * RB) return;
  const int row = (int)(wv / RB), j = (int)(wv % RB) * 64 + lane;
  const bool live = row < m && j < r;
  const float hv = live ? h[(int64_t)row * r_pad32 + j] : 0.0f;
  float amax = fabsf(hv);
  for (int msk = 1; msk < gr; msk <<= 1) amax = fmaxf(amax, __shfl_xor(amax, msk));
  const float s = amax / 7.0f;   // IEEE division; s_H stays fp32
  int q = 0;
  if (live && s != 0.0f) {
    float tq = __builtin_rintf(hv / s);
    tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
    q = (int)tq;
  }
  qh[(int64_t)row * r_pad64 + j] = (uint8_t)code_to_fp8(q);   // padding ranks get 0
  if (j < r && j % gr == 0) sh[(int64_t)(j / gr) * m32 + row] = row < m ? s : 0.0f;
}

// Stage 2 and the sum: one wavefront per 32 x 32 output tile, four column
// tiles per work-group; Y = round(Y_res + sum over rank groups of
// Q_H Q(L2) s_H s_L2), Y_res read back from y.
__global__ __launch_bounds__(256) void unfused_stage2_kernel(GemmArgs a, const uint8_t *__restrict__ qh,
                                                             const float *__restrict__ sh) {
  const Geometry &geo = a.geo;
  const int t = blockIdx.x, lane = threadIdx.x & 63, l32 = lane & 31;
  const int ct = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (ct >= geo.n_pad / 32) return;
  const int RB = geo.r_pad64 / 64;
  const uint16_t *l2s = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  v16f ylr = v16f{0};
  for (int rb = 0; rb < RB; rb++) {
    const uint8_t *qrow = qh + (int64_t)(32 * t + l32) * geo.r_pad64 + rb * 64 + (lane >> 5) * 32;
    const u32x4 lo = *reinterpret_cast<const u32x4 *>(qrow);
    const u32x4 hi = *reinterpret_cast<const u32x4 *>(qrow + 16);
    const v8i qa = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    const v8i lb = unpack32(*reinterpret_cast<const u32x4 *>(
        a.packed + geo.off_l2 + (((int64_t)ct * RB + rb) * 64 + lane) * 16));
    const int hg = rb * 64 / geo.gr;   // rank group of this 64-rank block (gr >= 64 when RB > 1)
    const float sl2 = half_bits_to_float(l2s[(int64_t)hg * geo.n_pad + ct * 32 + l32]);
    const v16f cbv = mfma_codes_32x32x64(qa, lb);
#pragma unroll
    for (int v = 0; v < 16; v++)
      ylr[v] = fmaf(cbv[v], sh[(int64_t)hg * a.ms + 32 * t + row_of_32x32(lane, v)] * sl2, ylr[v]);
  }
  asm volatile("" : "+v"(ylr));
  const int col = ct * 32 + l32;
  if (col < geo.n) {
    uint16_t *y = reinterpret_cast<uint16_t *>(a.y);
#pragma unroll
    for (int v = 0; v < 16; v++) {
      const int row = 32 * t + row_of_32x32(lane, v);
      if (row < a.m) {
        const int64_t i = (int64_t)row * geo.n + col;
        const float yres = a.bf16_out ? bf16_bits_to_float(y[i]) : half_bits_to_float(y[i]);
        const float yv = yres + ylr[v];
        y[i] = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
      }
    }
  }
}

}  // namespace

size_t unfused_scratch_bytes(int m, const Geometry &g) {
  const size_t m32 = (size_t)(m + 31) / 32 * 32;
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  if (g.r == 0) return 256;
  return up(m32 * g.r_pad32 * 4) + up(m32 * g.r_pad64) + up((size_t)(g.r / g.gr) * m32 * 4);
}

hipError_t launch_dual_gemm_unfused(const GemmArgs &a, void *scratch, hipStream_t s) {
  // 1. residual 4-bit GEMM: the fused layer's kernels with the rank-0 view of
  //    the same packed weights (their residual part has the same offsets)
  GemmArgs ra = a;
  ra.geo.r = 0;
  ra.geo.gr = 0;
  ra.geo.r_pad32 = 0;
  ra.geo.r_pad64 = 0;
  ra.dbg_h = nullptr;
  ra.dbg_sh = nullptr;
  ra.dbg_qh = nullptr;
  hipError_t e = launch_dual_gemm(ra, s);
  if (e != hipSuccess || a.geo.r == 0) return e;
  const Geometry &g = a.geo;
  const int m32 = a.ms, tiles = m32 / 32;
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  uint8_t *base = static_cast<uint8_t *>(scratch);
  float *h = reinterpret_cast<float *>(base);
  uint8_t *qh = base + up((size_t)m32 * g.r_pad32 * 4);
  float *sh = reinterpret_cast<float *>(qh + up((size_t)m32 * g.r_pad64));
  // 2. stage 1: H to global memory
  auto s1 = act_codes_fp8(a.m) ? unfused_stage1_kernel<true> : unfused_stage1_kernel<false>;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(s1),
                          hipFuncAttributeMaxDynamicSharedMemorySize, kS1Lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(s1, dim3(tiles, g.r_pad32 / 32), dim3(64 * kS1Waves), kS1Lds, s, a, h);
  // 3. re-quantization: Q_H and s_H to global memory
  const int64_t waves = (int64_t)m32 * (g.gr > 64 ? 1 : g.r_pad64 / 64);
  hipLaunchKernelGGL(unfused_requant_kernel, dim3((unsigned)((waves + 3) / 4)), dim3(256), 0, s, h,
                     a.m, m32, g.r, g.gr, g.r_pad32, g.r_pad64, qh, sh);
  // 4. stage 2 added to the residual output
  hipLaunchKernelGGL(unfused_stage2_kernel, dim3(tiles, (g.n_pad / 32 + 3) / 4), dim3(256), 0, s, a, qh,
                     sh);
  return hipGetLastError();
}

}  // namespace tq
