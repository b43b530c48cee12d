// Fused dual-component layer for decode-sized token counts (m <= 16).
//
// Same computation as the tile kernel (paper Sec. 4.3), shaped for the
// memory-bound regime: a workgroup owns NC 16-column output tiles and all
// m <= 16 tokens; the 16x16x128 fp8 matrix-core instruction covers two K
// groups per operand load (operand lanes 0-31 hold group g, lanes 32-63 group
// g+1), and two instructions with complementary halves of the activation
// operand zeroed give the two groups' exact integer sums separately.
//
//  * Stage 1 (H, all r ranks): the 16-rank column tiles of H are spread over
//    the four wavefronts; each wavefront runs the whole K loop for its tiles
//    in ascending group order, so H (and therefore Q_H) is bit-identical to
//    the tile kernel's and the oracle's.
//  * Residual: with SPLITK the K loop of the NC column tiles is split over
//    the four wavefronts (group pair p goes to wavefront p mod 4) and the
//    partial sums are added in LDS in a fixed order; without SPLITK each
//    wavefront owns one of NC = 4 column tiles and accumulates it in order.
//  * After the K loop: H is re-quantized in LDS, stage 2 (Q_H Q(L2)) runs
//    per column tile, and one epilogue stores Y.
// Every operand fragment and scale is loaded straight from global memory
// into a per-wavefront register ring four group pairs deep; nothing goes
// through LDS in the K loop and the K loop has no barrier.
#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {

namespace {

// operand fragment (16 bytes) of a 16-column slice of a packed 32-column
// block pair: lane l = (q, c), q = l / 16 picks group g + q / 2 and the
// 32-code half q % 2, c = l % 16 the column inside the slice.
__device__ __forceinline__ u32x4 load_slice(const uint8_t *blocks, int64_t kblocks, int col16,
                                            int g, int kgroups, int lane) {
  const int q = lane >> 4, c = lane & 15;
  const int gg = g + (q >> 1);
  if (gg >= kgroups) return u32x4{0, 0, 0, 0};
  const int64_t blk = (int64_t)(col16 >> 1) * kblocks + gg;
  const int L = (q & 1) * 32 + (col16 & 1) * 16 + c;
  return *reinterpret_cast<const u32x4 *>(blocks + (blk * 64 + L) * 16);
}

__device__ __forceinline__ v8i zero_v8i() { return v8i{0, 0, 0, 0, 0, 0, 0, 0}; }

}  // namespace

template <int NC, int RT16, bool SPLITK>
__global__ __launch_bounds__(256) void dual_gemm_small_kernel(GemmArgs a) {
  constexpr int HT = (RT16 + 3) / 4;          // H tiles (16 ranks) per wavefront
  constexpr int RB = (RT16 + 3) / 4;          // 64-rank blocks (= rank groups)
  constexpr int RP = RT16 * 16;               // padded rank
  constexpr int HSTR = RP + 1;
  constexpr int QSTR = (RB > 0 ? RB : 1) * 64 + 16;
  static_assert(SPLITK || NC == 4, "without split-K each wavefront owns one column tile");
  constexpr int RT_W = SPLITK ? NC : 1;       // residual tiles per wavefront

  __shared__ float RES[SPLITK ? 4 : 1][NC][4][64];
  __shared__ float HS[16 * (RP > 0 ? HSTR : 1)];
  __shared__ __attribute__((aligned(16))) uint8_t QS[16 * QSTR];
  __shared__ float SHS[16 * (RB > 0 ? RB : 1)];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int q = lane >> 4, c16 = lane & 15;
  const Geometry &geo = a.geo;
  const int KG = geo.k / kGroup, NP = (KG + 1) / 2;
  const int m = a.m;
  const int col0 = blockIdx.x * NC;             // first 16-column tile of this workgroup
  const int ctiles16 = geo.n_pad / 16;
  const uint8_t *wcodes = a.packed + geo.off_w;
  const uint16_t *wscales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_ws);
  const uint8_t *l1codes = a.packed + geo.off_l1;
  const uint16_t *l1scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l1s);
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const int64_t xwords = geo.k / 8;
  const int xrow = c16;                          // activation row held by this lane
  const int orow0 = 4 * q;                       // output rows 4q..4q+3 held by this lane

  // residual tiles handled by this wavefront
  auto res_tile = [&](int j) { return SPLITK ? col0 + j : col0 + w; };

  v4f acc[RT_W];
  v4f hacc[HT > 0 ? HT : 1];
#pragma unroll
  for (int j = 0; j < RT_W; j++) acc[j] = v4f{0, 0, 0, 0};
#pragma unroll
  for (int h = 0; h < (HT > 0 ? HT : 1); h++) hacc[h] = v4f{0, 0, 0, 0};

  // one group pair of operand slices and scales; a ring of D pairs per
  // wavefront keeps D pairs of loads in flight (no LDS, no barriers)
  struct Frag {
    u32x4 x, l[HT > 0 ? HT : 1], wv[RT_W];
    uint16_t sx1[4], sx2[4], sl1[HT > 0 ? HT : 1][2], sw[RT_W][2];
  };
  auto load_pair = [&](int p, Frag &f) {
    const int g = 2 * p;
    const int gg = g + (q >> 1);
    const bool two = g + 1 < KG;
    f.x = u32x4{0, 0, 0, 0};
    if (xrow < m && gg < KG)
      f.x = *reinterpret_cast<const u32x4 *>(a.xc + xrow * xwords + gg * 8 + (q & 1) * 4);
#pragma unroll
    for (int v = 0; v < 4; v++) {
      const int row = orow0 + v;
      f.sx1[v] = row < m ? a.xs[(int64_t)g * a.ms + row] : (uint16_t)0;
      f.sx2[v] = (row < m && two) ? a.xs[(int64_t)(g + 1) * a.ms + row] : (uint16_t)0;
    }
#pragma unroll
    for (int h = 0; h < HT; h++) {
      const int t16 = w + 4 * h;
      f.l[h] = u32x4{0, 0, 0, 0};
      f.sl1[h][0] = f.sl1[h][1] = 0;
      if (t16 < RT16) {
        f.l[h] = load_slice(l1codes, KG, t16, g, KG, lane);
        const int rk = t16 * 16 + c16;
        f.sl1[h][0] = l1scales[(int64_t)g * geo.r_pad32 + rk];
        if (two) f.sl1[h][1] = l1scales[(int64_t)(g + 1) * geo.r_pad32 + rk];
      }
    }
    const bool mine = SPLITK ? ((p & 3) == w) : true;
#pragma unroll
    for (int j = 0; j < RT_W; j++) {
      const int ct = res_tile(j);
      f.wv[j] = u32x4{0, 0, 0, 0};
      f.sw[j][0] = f.sw[j][1] = 0;
      if (mine && ct < ctiles16) {
        f.wv[j] = load_slice(wcodes, KG, ct, g, KG, lane);
        const int col = ct * 16 + c16;
        f.sw[j][0] = wscales[(int64_t)g * geo.n_pad + col];
        if (two) f.sw[j][1] = wscales[(int64_t)(g + 1) * geo.n_pad + col];
      }
    }
  };

  auto compute_pair = [&](int p, const Frag &f) {
    const int g = 2 * p;
    const bool two = g + 1 < KG;
    const v8i xa = unpack32(f.x);
    const v8i x1 = q < 2 ? xa : zero_v8i();     // group g only
    const v8i x2 = q < 2 ? zero_v8i() : xa;     // group g + 1 only
    float sx1[4], sx2[4];
#pragma unroll
    for (int v = 0; v < 4; v++) {
      sx1[v] = half_bits_to_float(f.sx1[v]);
      sx2[v] = half_bits_to_float(f.sx2[v]);
    }
    // ---- stage 1: H tiles of this wavefront, ascending groups ----
#pragma unroll
    for (int h = 0; h < HT; h++) {
      const int t16 = w + 4 * h;
      if (t16 < RT16) {
        const v8i lb = unpack32(f.l[h]);
        const float s1 = half_bits_to_float(f.sl1[h][0]);
        const v4f c1 = mfma_codes_16x16x128(x1, lb);
#pragma unroll
        for (int v = 0; v < 4; v++) hacc[h][v] = fmaf(c1[v], sx1[v] * s1, hacc[h][v]);
        if (two) {
          const float s2 = half_bits_to_float(f.sl1[h][1]);
          const v4f c2 = mfma_codes_16x16x128(x2, lb);
#pragma unroll
          for (int v = 0; v < 4; v++) hacc[h][v] = fmaf(c2[v], sx2[v] * s2, hacc[h][v]);
        }
      }
    }
    // ---- residual ----
    const bool mine = SPLITK ? ((p & 3) == w) : true;
    if (mine) {
#pragma unroll
      for (int j = 0; j < RT_W; j++) {
        const int ct = res_tile(j);
        if (ct < ctiles16) {
          const v8i wb = unpack32(f.wv[j]);
          const float s1 = half_bits_to_float(f.sw[j][0]);
          const v4f c1 = mfma_codes_16x16x128(x1, wb);
#pragma unroll
          for (int v = 0; v < 4; v++) acc[j][v] = fmaf(c1[v], sx1[v] * s1, acc[j][v]);
          if (two) {
            const float s2 = half_bits_to_float(f.sw[j][1]);
            const v4f c2 = mfma_codes_16x16x128(x2, wb);
#pragma unroll
            for (int v = 0; v < 4; v++) acc[j][v] = fmaf(c2[v], sx2[v] * s2, acc[j][v]);
          }
        }
      }
    }
  };

  constexpr int D = 4;
  Frag ring[D];
#pragma unroll
  for (int i = 0; i < D; i++)
    if (i < NP) load_pair(i, ring[i]);
  for (int p0 = 0; p0 < NP; p0 += D) {
#pragma unroll
    for (int i = 0; i < D; i++) {
      const int p = p0 + i;
      if (p < NP) {
        compute_pair(p, ring[i]);
        if (p + D < NP) load_pair(p + D, ring[i]);
      }
    }
  }

  // ---- partial sums and H to LDS ----
#pragma unroll
  for (int j = 0; j < RT_W; j++)
#pragma unroll
    for (int v = 0; v < 4; v++) RES[SPLITK ? w : 0][SPLITK ? j : w][v][lane] = acc[j][v];
  if constexpr (RT16 > 0) {
#pragma unroll
    for (int h = 0; h < HT; h++) {
      const int t16 = w + 4 * h;
      if (t16 < RT16)
#pragma unroll
        for (int v = 0; v < 4; v++) HS[(orow0 + v) * HSTR + t16 * 16 + c16] = hacc[h][v];
    }
    const int r = geo.r;
    if (r < RB * 64)
      for (int idx = tid; idx < 16 * RB * 64; idx += 256) {
        const int row = idx / (RB * 64), j = idx % (RB * 64);
        if (j >= r) QS[row * QSTR + j] = 0;
      }
  }
  __syncthreads();

  // ---- requantize H per token and rank group (s_H stays fp32) ----
  if constexpr (RT16 > 0) {
    const int r = geo.r, gr = geo.gr, rg = r / gr;
    const int subs = gr / 8;
    const int work = 16 * rg * subs;        // <= 256
    const bool dbg = a.dbg_h != nullptr && blockIdx.x == 0;
    const int idx = tid;
    const bool valid = idx < work;
    const int pair = idx / subs, sub = idx % subs;
    const int row = pair / rg, hg = pair % rg;
    const int j0 = hg * gr + sub * 8;
    float hv[8];
    float amax = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; e++) {
      hv[e] = valid ? HS[row * HSTR + j0 + e] : 0.0f;
      amax = fmaxf(amax, fabsf(hv[e]));
    }
    for (int msk = 1; msk < subs; msk <<= 1) amax = fmaxf(amax, __shfl_xor(amax, msk));
    const float s = amax / 7.0f;
    if (valid) {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        int qv = 0;
        if (s != 0.0f) {
          float tq = __builtin_rintf(hv[e] / s);
          tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
          qv = (int)tq;
        }
        const uint32_t b = code_to_fp8(qv);
        if (e < 4) w0 |= b << (8 * e); else w1 |= b << (8 * (e - 4));
        if (dbg && row < m) {
          a.dbg_h[(int64_t)row * r + j0 + e] = hv[e];
          a.dbg_qh[(int64_t)row * r + j0 + e] = (int8_t)qv;
        }
      }
      *reinterpret_cast<uint32_t *>(QS + row * QSTR + j0) = w0;
      *reinterpret_cast<uint32_t *>(QS + row * QSTR + j0 + 4) = w1;
      if (sub == 0) {
        SHS[row * RB + hg] = s;
        if (dbg && row < m) a.dbg_sh[(int64_t)row * rg + hg] = s;
      }
    }
    __syncthreads();
  }

  // ---- stage 2 and the single epilogue: wavefront j < NC stores tile j ----
  for (int j = w; j < NC; j += 4) {
    const int ct = col0 + j;
    if (ct >= ctiles16) continue;
    v4f ylr = v4f{0, 0, 0, 0};
    if constexpr (RT16 > 0) {
      // rank blocks in pairs: lanes q < 2 carry block rb, lanes q >= 2 block rb + 1
      for (int rb = 0; rb < RB; rb += 2) {
        const int rbq = rb + (q >> 1);
        v8i qa = zero_v8i();
        u32x4 lraw = u32x4{0, 0, 0, 0};
        if (rbq < RB) {
          const uint8_t *qrow = QS + c16 * QSTR + rbq * 64 + (q & 1) * 32;
          const u32x4 q0 = *reinterpret_cast<const u32x4 *>(qrow);
          const u32x4 q1 = *reinterpret_cast<const u32x4 *>(qrow + 16);
          qa = v8i{(int)q0.x, (int)q0.y, (int)q0.z, (int)q0.w, (int)q1.x, (int)q1.y, (int)q1.z, (int)q1.w};
          lraw = load_slice(l2codes, RB, ct, rb, RB, lane);
        }
        const v8i lb = unpack32(lraw);
        const v8i qa1 = q < 2 ? qa : zero_v8i();
        const v8i qa2 = q < 2 ? zero_v8i() : qa;
        const int col = ct * 16 + c16;
        {
          const float sl2 = half_bits_to_float(l2scales[(int64_t)rb * geo.n_pad + col]);
          const v4f cb = mfma_codes_16x16x128(qa1, lb);
#pragma unroll
          for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[(orow0 + v) * RB + rb] * sl2, ylr[v]);
        }
        if (rb + 1 < RB) {
          const float sl2 = half_bits_to_float(l2scales[(int64_t)(rb + 1) * geo.n_pad + col]);
          const v4f cb = mfma_codes_16x16x128(qa2, lb);
#pragma unroll
          for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[(orow0 + v) * RB + rb + 1] * sl2, ylr[v]);
        }
      }
    }
    const int col = ct * 16 + c16;
    if (col < geo.n) {
#pragma unroll
      for (int v = 0; v < 4; v++) {
        const int row = orow0 + v;
        if (row < m) {
          float yres;
          if (SPLITK)
            yres = ((RES[0][j][v][lane] + RES[1][j][v][lane]) + RES[2][j][v][lane]) + RES[3][j][v][lane];
          else
            yres = RES[0][j][v][lane];
          const float yv = yres + ylr[v];
          const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
          reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
        }
      }
    }
  }
}

template <int NC, bool SPLITK>
static hipError_t launch_small_nc(const GemmArgs &a, hipStream_t s) {
  const int tiles16 = a.geo.n_pad / 16;
  const dim3 grid((tiles16 + NC - 1) / NC);
  switch ((a.geo.r + 15) / 16) {
    case 0: hipLaunchKernelGGL((dual_gemm_small_kernel<NC, 0, SPLITK>), grid, dim3(256), 0, s, a); break;
    case 1: hipLaunchKernelGGL((dual_gemm_small_kernel<NC, 1, SPLITK>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((dual_gemm_small_kernel<NC, 2, SPLITK>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((dual_gemm_small_kernel<NC, 4, SPLITK>), grid, dim3(256), 0, s, a); break;
    case 8: hipLaunchKernelGGL((dual_gemm_small_kernel<NC, 8, SPLITK>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_dual_gemm_small(const GemmArgs &a, hipStream_t s) {
  // aim at >= 256 workgroups (one per CU); own whole column tiles (exact
  // accumulation order) only when that still fills the GPU
  const int tiles16 = a.geo.n_pad / 16;
  if (tiles16 >= 4 * 256) return launch_small_nc<4, false>(a, s);
  if (tiles16 >= 2 * 256) return launch_small_nc<2, true>(a, s);
  return launch_small_nc<1, true>(a, s);
}

}  // namespace tq
