// Fused dual-component W4A4 layer (paper Sec. 4.3): one kernel computes the
// residual 4-bit GEMM and the two-stage low-rank branch over the same
// quantized activation tile, keeps the low-rank intermediate H on chip,
// re-quantizes it on the fly, and merges both branches in one epilogue.
//
// Work decomposition (one workgroup = 4 wavefronts, one per SIMD):
//  * a workgroup owns BM tokens and a run of consecutive BN-column tiles;
//  * during the K loop of its first column tile it also accumulates the
//    stage-1 product H = Q(X) Q(L1) for its BM tokens (all r ranks), then
//    re-quantizes H into LDS; later column tiles reuse Q_H and s_H from LDS,
//    so H is formed once per workgroup and never leaves the chip;
//  * per 64-wide K group, 16-byte slices of packed codes are staged through
//    double-buffered LDS in matrix-core fragment order, expanded to fp8 with
//    three bit operations per 8 codes, and multiplied exactly on the matrix
//    cores (v_mfma_scale_f32_32x32x64_f8f6f4); the exact integer group sums
//    are scaled by s_x * s_w and accumulated with one fma per group, in
//    ascending group order (the same order for H, whose codes depend on it).
#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {

template <int WM, int WN, int TM, int TN, int RT>
struct TileCfg {
  static_assert(WM * WN == 4, "four wavefronts per workgroup");
  static constexpr int BM = WM * TM * 32;
  static constexpr int BN = WN * TN * 32;
  static constexpr int A_CH = BM * 2;        // 16-byte chunks of one K group
  static constexpr int B_CH = BN * 2;
  static constexpr int L_CH = RT * 64;
  static constexpr int RB = (RT + 1) / 2;    // 64-rank blocks (= rank groups)
  static constexpr int HT = (RT + WN - 1) / WN;  // H column tiles per wave
  // LDS layout of one pipeline stage
  static constexpr int OFF_A = 0;
  static constexpr int OFF_B = OFF_A + A_CH * 16;
  static constexpr int OFF_L = OFF_B + B_CH * 16;
  static constexpr int OFF_SX = OFF_L + L_CH * 16;
  static constexpr int OFF_SW = OFF_SX + BM * 4;
  static constexpr int OFF_SL = OFF_SW + BN * 4;
  static constexpr int STAGE = OFF_SL + RT * 32 * 4;
  // after the first K loop the stage buffers hold H in fp32
  static constexpr int HSTR = RT * 32 + 1;
  static constexpr int H_BYTES = RT > 0 ? BM * HSTR * 4 : 0;
  static constexpr int UNION = (2 * STAGE > H_BYTES ? 2 * STAGE : H_BYTES);
  static constexpr int QSTR = RB * 64 + 16;  // bytes per token row of Q_H (fp8)
  static constexpr int OFF_Q = (UNION + 15) / 16 * 16;
  static constexpr int OFF_SH = OFF_Q + (RT > 0 ? BM * QSTR : 0);
  static constexpr int LDS = OFF_SH + (RT > 0 ? BM * RB * 4 : 0);
};

template <int WM, int WN, int TM, int TN, int RT>
__global__ __launch_bounds__(256, 1) void dual_gemm_tile_kernel(GemmArgs a, int m_tiles,
                                                                int n_tiles, int tiles_per_wg) {
  using C = TileCfg<WM, WN, TM, TN, RT>;
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wy = wave / WN, wx = wave % WN;
  const Geometry &geo = a.geo;
  const int KG = geo.k / kGroup;
  const int m = a.m;
  const int ctiles = geo.n_pad / 32;

  // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
  // contiguous range of logical ids so that workgroups sharing weight columns
  // share one L2.
  int logical;
  {
    const int nwg = gridDim.x, per = nwg / 8, rem = nwg % 8;
    const int x = blockIdx.x % 8, s = blockIdx.x / 8;
    logical = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + s;
  }
  const int m_tile = logical % m_tiles;
  const int chunk = logical / m_tiles;
  const int m0 = m_tile * C::BM;
  const int t_begin = chunk * tiles_per_wg;
  const int t_end = min(t_begin + tiles_per_wg, n_tiles);

  const uint8_t *wcodes = a.packed + geo.off_w;
  const uint16_t *wscales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_ws);
  const uint8_t *l1codes = a.packed + geo.off_l1;
  const uint16_t *l1scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l1s);
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const int64_t xwords = geo.k / 8;

  constexpr int A_PER = (C::A_CH + 255) / 256;
  constexpr int B_PER = (C::B_CH + 255) / 256;

  for (int t = t_begin; t < t_end; t++) {
    const int n0 = t * C::BN;
    const bool do_h = (RT > 0) && (t == t_begin);

    v16f acc[TM][TN];
    v16f hacc[TM][C::HT > 0 ? C::HT : 1];
#pragma unroll
    for (int i = 0; i < TM; i++) {
#pragma unroll
      for (int j = 0; j < TN; j++) acc[i][j] = v16f{0};
#pragma unroll
      for (int h = 0; h < (C::HT > 0 ? C::HT : 1); h++) hacc[i][h] = v16f{0};
    }

    // ---- global -> register staging of one K group ----
    u32x4 ra[A_PER], rb[B_PER], rl = {0, 0, 0, 0};
    uint16_t rsx = 0, rsw[(C::BN + 255) / 256], rsl = 0;
    auto load_group = [&](int g) {
#pragma unroll
      for (int p = 0; p < A_PER; p++) {
        const int c = tid + p * 256;
        ra[p] = u32x4{0, 0, 0, 0};
        if (c < C::A_CH) {
          const int row = m0 + (c >> 6) * 32 + (c & 31);
          const int khalf = (c >> 5) & 1;
          if (row < m)
            ra[p] = *reinterpret_cast<const u32x4 *>(a.xc + row * xwords + g * 8 + khalf * 4);
        }
      }
#pragma unroll
      for (int p = 0; p < B_PER; p++) {
        const int c = tid + p * 256;
        rb[p] = u32x4{0, 0, 0, 0};
        if (c < C::B_CH) {
          const int ct = n0 / 32 + (c >> 6);
          if (ct < ctiles)
            rb[p] = *reinterpret_cast<const u32x4 *>(wcodes + (((int64_t)ct * KG + g) * 64 + (c & 63)) * 16);
        }
      }
      if (do_h && tid < C::L_CH)
        rl = *reinterpret_cast<const u32x4 *>(l1codes + (((int64_t)(tid >> 6) * KG + g) * 64 + (tid & 63)) * 16);
      rsx = 0;
      if (tid < C::BM && m0 + tid < m) rsx = a.xs[(int64_t)g * m + m0 + tid];
#pragma unroll
      for (int p = 0; p < (C::BN + 255) / 256; p++) {
        const int j = tid + p * 256;
        rsw[p] = 0;
        if (j < C::BN && n0 + j < geo.n_pad) rsw[p] = wscales[(int64_t)g * geo.n_pad + n0 + j];
      }
      if (do_h && tid < RT * 32) rsl = l1scales[(int64_t)g * geo.r_pad32 + tid];
    };
    auto store_group = [&](int stage) {
      uint8_t *st = smem + stage * C::STAGE;
#pragma unroll
      for (int p = 0; p < A_PER; p++) {
        const int c = tid + p * 256;
        if (c < C::A_CH) *reinterpret_cast<u32x4 *>(st + C::OFF_A + c * 16) = ra[p];
      }
#pragma unroll
      for (int p = 0; p < B_PER; p++) {
        const int c = tid + p * 256;
        if (c < C::B_CH) *reinterpret_cast<u32x4 *>(st + C::OFF_B + c * 16) = rb[p];
      }
      if (do_h && tid < C::L_CH) *reinterpret_cast<u32x4 *>(st + C::OFF_L + tid * 16) = rl;
      if (tid < C::BM) reinterpret_cast<float *>(st + C::OFF_SX)[tid] = half_bits_to_float(rsx);
#pragma unroll
      for (int p = 0; p < (C::BN + 255) / 256; p++) {
        const int j = tid + p * 256;
        if (j < C::BN) reinterpret_cast<float *>(st + C::OFF_SW)[j] = half_bits_to_float(rsw[p]);
      }
      if (do_h && tid < RT * 32) reinterpret_cast<float *>(st + C::OFF_SL)[tid] = half_bits_to_float(rsl);
    };

    load_group(0);
    store_group(0);
    __syncthreads();

    for (int g = 0; g < KG; g++) {
      if (g + 1 < KG) load_group(g + 1);
      const uint8_t *st = smem + (g & 1) * C::STAGE;
      const float *sxl = reinterpret_cast<const float *>(st + C::OFF_SX);
      const float *swl = reinterpret_cast<const float *>(st + C::OFF_SW);
      v8i af[TM], bf[TN];
      float sxv[TM][16];
#pragma unroll
      for (int i = 0; i < TM; i++) {
        const int ti = wy * TM + i;
        af[i] = unpack32(*reinterpret_cast<const u32x4 *>(st + C::OFF_A + (ti * 64 + lane) * 16));
#pragma unroll
        for (int q = 0; q < 4; q++) {
          const v4f s4 = *reinterpret_cast<const v4f *>(sxl + ti * 32 + 8 * q + 4 * (lane >> 5));
          sxv[i][4 * q + 0] = s4.x; sxv[i][4 * q + 1] = s4.y;
          sxv[i][4 * q + 2] = s4.z; sxv[i][4 * q + 3] = s4.w;
        }
      }
      float swv[TN];
#pragma unroll
      for (int j = 0; j < TN; j++) {
        const int tj = wx * TN + j;
        bf[j] = unpack32(*reinterpret_cast<const u32x4 *>(st + C::OFF_B + (tj * 64 + lane) * 16));
        swv[j] = swl[tj * 32 + (lane & 31)];
      }
#pragma unroll
      for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) {
          const v16f cg = mfma_codes_32x32x64(af[i], bf[j]);
#pragma unroll
          for (int v = 0; v < 16; v++) acc[i][j][v] = fmaf(cg[v], sxv[i][v] * swv[j], acc[i][j][v]);
        }
      if constexpr (RT > 0) {
        if (do_h) {
          const float *sll = reinterpret_cast<const float *>(st + C::OFF_SL);
#pragma unroll
          for (int h = 0; h < C::HT; h++) {
            const int rt = wx + h * WN;
            if (rt < RT) {
              const v8i lf = unpack32(*reinterpret_cast<const u32x4 *>(st + C::OFF_L + (rt * 64 + lane) * 16));
              const float sl = sll[rt * 32 + (lane & 31)];
#pragma unroll
              for (int i = 0; i < TM; i++) {
                const v16f cg = mfma_codes_32x32x64(af[i], lf);
#pragma unroll
                for (int v = 0; v < 16; v++) hacc[i][h][v] = fmaf(cg[v], sxv[i][v] * sl, hacc[i][h][v]);
              }
            }
          }
        }
      }
      if (g + 1 < KG) store_group((g + 1) & 1);
      __syncthreads();
    }

    if constexpr (RT > 0) {
      float *HS = reinterpret_cast<float *>(smem);
      uint8_t *QS = smem + C::OFF_Q;
      float *SHS = reinterpret_cast<float *>(smem + C::OFF_SH);
      const int r = geo.r, gr = geo.gr, rg = r / gr;
      if (do_h) {
        // ---- H -> LDS (fp32), then per-token, per-rank-group requantization ----
#pragma unroll
        for (int h = 0; h < C::HT; h++) {
          const int rt = wx + h * WN;
          if (rt < RT) {
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
              for (int v = 0; v < 16; v++) {
                const int row = (wy * TM + i) * 32 + row_of_32x32(lane, v);
                HS[row * C::HSTR + rt * 32 + (lane & 31)] = hacc[i][h][v];
              }
          }
        }
        // zero the fp8 padding ranks [r, 64*RB) of Q_H once
        if (r < C::RB * 64) {
          for (int idx = tid; idx < C::BM * C::RB * 64; idx += 256) {
            const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
            if (j >= r) QS[row * C::QSTR + j] = 0;
          }
        }
        __syncthreads();
        const int subs = gr / 8;               // lanes per (token, rank group): 1, 2, 4 or 8
        const int work = C::BM * rg * subs;
        const bool dbg = a.dbg_h != nullptr && chunk == 0;
        for (int base = 0; base < work; base += 256) {
          const int idx = base + tid;
          const bool valid = idx < work;
          const int pair = idx / subs, sub = idx % subs;
          const int row = pair / rg, hg = pair % rg;
          const int j0 = hg * gr + sub * 8;
          float hv[8];
          float amax = 0.0f;
#pragma unroll
          for (int e = 0; e < 8; e++) {
            hv[e] = valid ? HS[row * C::HSTR + j0 + e] : 0.0f;
            amax = fmaxf(amax, fabsf(hv[e]));
          }
          for (int msk = 1; msk < subs; msk <<= 1) amax = fmaxf(amax, __shfl_xor(amax, msk));
          const float s = amax / 7.0f;  // s_H stays fp32
          if (valid) {
            uint32_t w0 = 0, w1 = 0;
#pragma unroll
            for (int e = 0; e < 8; e++) {
              int q = 0;
              if (s != 0.0f) {
                float tq = __builtin_rintf(hv[e] / s);
                tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
                q = (int)tq;
              }
              const uint32_t b = code_to_fp8(q);
              if (e < 4) w0 |= b << (8 * e); else w1 |= b << (8 * (e - 4));
              if (dbg && m0 + row < m) {
                a.dbg_h[(int64_t)(m0 + row) * r + j0 + e] = hv[e];
                a.dbg_qh[(int64_t)(m0 + row) * r + j0 + e] = (int8_t)q;
              }
            }
            *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0) = w0;
            *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0 + 4) = w1;
            if (sub == 0) {
              SHS[row * C::RB + hg] = s;
              if (dbg && m0 + row < m) a.dbg_sh[(int64_t)(m0 + row) * rg + hg] = s;
            }
          }
        }
        __syncthreads();
      }
    }

    // ---- stage 2 (Q_H Q(L2)) and the single epilogue ----
#pragma unroll
    for (int i = 0; i < TM; i++) {
      const int trow = (wy * TM + i) * 32;
#pragma unroll
      for (int j = 0; j < TN; j++) {
        const int ct = n0 / 32 + wx * TN + j;
        const bool cvalid = ct < ctiles;
        v16f ylr = v16f{0};
        if constexpr (RT > 0) {
          const uint8_t *QS = smem + C::OFF_Q;
          const float *SHS = reinterpret_cast<const float *>(smem + C::OFF_SH);
#pragma unroll
          for (int rbk = 0; rbk < C::RB; rbk++) {
            const uint8_t *qrow = QS + (trow + (lane & 31)) * C::QSTR + rbk * 64 + (lane >> 5) * 32;
            const u32x4 q0 = *reinterpret_cast<const u32x4 *>(qrow);
            const u32x4 q1 = *reinterpret_cast<const u32x4 *>(qrow + 16);
            const v8i qa = {(int)q0.x, (int)q0.y, (int)q0.z, (int)q0.w,
                            (int)q1.x, (int)q1.y, (int)q1.z, (int)q1.w};
            v8i lb = {0, 0, 0, 0, 0, 0, 0, 0};
            float sl2 = 0.0f;
            if (cvalid) {
              lb = unpack32(*reinterpret_cast<const u32x4 *>(l2codes + (((int64_t)ct * C::RB + rbk) * 64 + lane) * 16));
              sl2 = half_bits_to_float(l2scales[(int64_t)rbk * geo.n_pad + ct * 32 + (lane & 31)]);
            }
            const v16f cb = mfma_codes_32x32x64(qa, lb);
#pragma unroll
            for (int v = 0; v < 16; v++) {
              const float sh = SHS[(trow + row_of_32x32(lane, v)) * C::RB + rbk];
              ylr[v] = fmaf(cb[v], sh * sl2, ylr[v]);
            }
          }
        }
        const int col = ct * 32 + (lane & 31);
        if (cvalid && col < geo.n) {
#pragma unroll
          for (int v = 0; v < 16; v++) {
            const int row = m0 + trow + row_of_32x32(lane, v);
            if (row < m) {
              const float yv = acc[i][j][v] + ylr[v];
              const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
              reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
            }
          }
        }
      }
    }
    // the next column tile overwrites the stage buffers
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
template <int WM, int WN, int TM, int TN, int RT>
static hipError_t launch_tile(const GemmArgs &a, hipStream_t s, int target_wgs) {
  using C = TileCfg<WM, WN, TM, TN, RT>;
  const int m_tiles = (a.m + C::BM - 1) / C::BM;
  const int n_tiles = (a.geo.n_pad + C::BN - 1) / C::BN;
  int chunks = (target_wgs + m_tiles - 1) / m_tiles;
  if (chunks > n_tiles) chunks = n_tiles;
  if (chunks < 1) chunks = 1;
  const int tiles_per_wg = (n_tiles + chunks - 1) / chunks;
  chunks = (n_tiles + tiles_per_wg - 1) / tiles_per_wg;
  auto kern = dual_gemm_tile_kernel<WM, WN, TM, TN, RT>;
  // more than 64 KiB of dynamic LDS must be enabled per kernel (and device)
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(m_tiles * chunks), dim3(256), C::LDS, s, a, m_tiles, n_tiles,
                     tiles_per_wg);
  return hipGetLastError();
}

template <int WM, int WN, int TM, int TN>
static hipError_t launch_rt(const GemmArgs &a, hipStream_t s, int target_wgs) {
  switch (a.geo.r_pad32 / 32) {
    case 0: return launch_tile<WM, WN, TM, TN, 0>(a, s, target_wgs);
    case 1: return launch_tile<WM, WN, TM, TN, 1>(a, s, target_wgs);
    case 2: return launch_tile<WM, WN, TM, TN, 2>(a, s, target_wgs);
    case 4: return launch_tile<WM, WN, TM, TN, 4>(a, s, target_wgs);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_dual_gemm(const GemmArgs &a, hipStream_t s) {
  if (a.m <= 32) return launch_rt<1, 4, 1, 1>(a, s, 512);
  if (a.m <= 64) return launch_rt<1, 4, 2, 1>(a, s, 512);
  return launch_rt<2, 2, 2, 2>(a, s, 256);
}

}  // namespace tq
