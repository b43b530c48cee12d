// Fused dual-component W4A4 layer (paper Sec. 4.3) for prefill-sized token
// counts, with free-running wavefronts: the residual 4-bit GEMM, the stage-1
// product H = Q(X) Q(L1) kept on chip, its on-the-fly re-quantization,
// stage 2 Q_H Q(L2) and one epilogue, in one kernel.
//
// Work decomposition.  A workgroup of 8 wavefronts (two per SIMD) owns 64
// tokens and a run of 512-column passes; each wavefront computes all 64 tokens
// x 64 columns of a pass (four 32x32 tiles).  During the first pass,
// wavefront h < 2 r / 32 also accumulates H tile h (32 tokens x 32 ranks);
// after it the workgroup re-quantizes H into LDS, and later passes reuse Q_H
// and s_H, so H is formed once per workgroup.
//
// K pipeline: no workgroup barrier in the K loop.  Every wavefront streams
// its own operands -- the activation rows of its tiles, its weight columns,
// its L1 ranks and all their scales -- with direct global->LDS loads
// (global_load_lds_dwordx4) three K-groups ahead into a private 3-slot LDS
// ring, waits for its own loads by count (they complete in order), reads a
// group back into registers, expands the 4-bit codes to fp8 and runs the
// group's products.  The two wavefronts of a SIMD drift apart, so the matrix
// core of one overlaps the fp32 rescaling fmas of the other.
//
// Arithmetic per 32x32 tile and group (Eq. 2): the exact integer group sum of
// code products comes from v_mfma_scale_f32_32x32x64_f8f6f4 (codes as fp8
// subnormals; block scales 2^8 and 2^9 return half of the integer sum), the
// exact scale product from v_mfma_f32_32x32x8f16 with both scale operands
// repeated in k = 0 and k = 4 (twice the product), and one fma adds their
// product -- exactly I * s_x * s_w -- to the fp32 accumulator in ascending
// group order, the order of the oracle for H and for the residual.
#include <stdio.h>
#include <stdlib.h>

#include <type_traits>

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int SBM = 64;      // tokens per workgroup (two 32-row tiles)
constexpr int SNW = 8;       // wavefronts per workgroup
constexpr int SPASS = 512;   // output columns per pass (8 wavefronts x 64)
constexpr int SD = 3;        // ring slots per wavefront = load distance in K-groups
// one slot: 2 activation blocks, 2 weight blocks, 1 L1 block (1 KiB each, in
// matrix-core lane order) and one 1 KiB scale block (activation scales of the
// 64 tokens at 0, the wavefront's 64 weight scales at 128, its 32 L1 scales at
// 256; the remaining lanes load duplicates)
constexpr int S_A = 0, S_B = 2048, S_L = 4096, S_S = 5120, SSLOT = 6144;
constexpr int SRING = SD * SSLOT;

template <int RT>
struct SCfg {
  static constexpr int HTILES = 2 * RT;   // 32x32 H tiles: wavefront h owns tile h
  static constexpr int HSTR = RT * 32 + 1;
  static constexpr int RB = (RT + 1) / 2;  // 64-rank blocks
  static constexpr int QSTR = RB * 64 + 16;
  static constexpr int OFF_Q = SNW * SRING;
  static constexpr int OFF_SH = OFF_Q + (RT > 0 ? SBM * QSTR : 0);
  static constexpr int LDS = OFF_SH + (RT > 0 ? SBM * RB * 4 : 0);
  static_assert(HTILES <= SNW, "one H tile per wavefront");
  static_assert(SBM * HSTR * 4 <= SNW * SRING, "H staging fits in the rings");
  static_assert(LDS <= 160 * 1024, "fits the 160 KiB LDS of a CU");
};

// exact scale products of a 32x32 tile: lane l carries s[l % 32] in k = 0
// (lanes 0-31) and k = 4 (lanes 32-63) of both operands, so the result is
// 2 * s_row * s_col
__device__ __forceinline__ v16f outer2(uint32_t sa, uint32_t sb) {
  const v16f z = {0};
  const u32x2 a2 = {sa, 0u}, b2 = {sb, 0u};
  return __builtin_amdgcn_mfma_f32_32x32x8f16(__builtin_bit_cast(v4h, a2),
                                              __builtin_bit_cast(v4h, b2), z, 0, 0, 0);
}

// half of the exact integer group sum of a 32x32 tile of code products
__device__ __forceinline__ v16f codes_half(v8i a, v8i b) {
  const v16f z = {0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, z, 0, 0, 0, kScale2p9 - 1, 0,
                                                         kScale2p9);
}

__device__ __forceinline__ void fma16(v16f &acc, const v16f &c, const v16f &p) {
#pragma unroll
  for (int v = 0; v < 16; v++) acc[v] = fmaf(c[v], p[v], acc[v]);
}

__device__ __forceinline__ v8i join(u32x4 lo, u32x4 hi) {
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// s_waitcnt vmcnt(n): at most n of this wavefront's loads in flight
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N < 64, "vmcnt has 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// direct global -> LDS load of 16 bytes per lane: scalar base + 32-bit lane
// offset, or a full 64-bit lane address
__device__ __forceinline__ void dma_s(uint32_t voff, const uint8_t *sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase),
               "s"(lds)
               : "memory");
}
__device__ __forceinline__ void dma_v(const uint8_t *addr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(addr), "s"(lds)
               : "memory");
}

// The loads of one wavefront: activation rows, weight columns (and L1 ranks)
// of its tiles with a scalar base per group, and one scale load with a
// per-lane address that advances by a per-lane stride per group.
struct SPlan {
  const uint8_t *a_base;    // activation codes of row m0, group 0
  uint32_t a_off[2];        // lane offsets of the two row tiles
  const uint8_t *b_base[2]; // weight blocks of the two column tiles, group 0
  const uint8_t *l_base;    // L1 blocks of the H tile, group 0
  const uint8_t *s_ptr;     // this lane's scale address for the next group to load
  uint32_t s_inc;           // its stride per group (bytes)
};

template <bool H>
__device__ __forceinline__ void s_issue(SPlan &P, int g, uint32_t slot_lds, int lane) {
  dma_s(P.a_off[0], P.a_base + (uint64_t)g * 32, slot_lds + S_A);
  dma_s(P.a_off[1], P.a_base + (uint64_t)g * 32, slot_lds + S_A + 1024);
  dma_s(lane * 16, P.b_base[0] + (uint64_t)g * 1024, slot_lds + S_B);
  dma_s(lane * 16, P.b_base[1] + (uint64_t)g * 1024, slot_lds + S_B + 1024);
  if constexpr (H) dma_s(lane * 16, P.l_base + (uint64_t)g * 1024, slot_lds + S_L);
  dma_v(P.s_ptr, slot_lds + S_S);
}

template <int RT>
__global__ __launch_bounds__(64 * SNW, 1) void dual_gemm_stream_kernel(GemmArgs a, int m_tiles,
                                                                       int n_chunks,
                                                                       int passes_per_wg,
                                                                       int band) {
  using C = SCfg<RT>;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KG = geo.k / kGroup;
  const int m = a.m, ms = a.ms;
  const int ctiles = geo.n_pad / 32;
  const int n_passes = (geo.n_pad + SPASS - 1) / SPASS;
  uint8_t *ring = smem + wave * SRING;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)ring);

  // Workgroups go round-robin over the 8 XCDs: give each XCD a contiguous run
  // of logical ids, and order logical ids in bands of `band` token tiles,
  // column chunk by column chunk, so an XCD's workgroups share both their
  // activation rows and their weight columns in its L2.
  int logical;
  {
    const int nwg = gridDim.x, per = nwg / 8, rem = nwg % 8;
    const int x = blockIdx.x % 8, s = blockIdx.x / 8;
    logical = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + s;
  }
  const int bsz = band * n_chunks;
  const int bidx = logical / bsz, brem = logical % bsz;
  const int rows_in_band = min(band, m_tiles - bidx * band);
  const int chunk = brem / rows_in_band;
  const int m_tile = bidx * band + brem % rows_in_band;
  const int m0 = m_tile * SBM;
  const int p_begin = chunk * passes_per_wg;
  const int p_end = min(p_begin + passes_per_wg, n_passes);

  const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
  const int64_t xrow = geo.k / 2;
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const bool hmine = RT > 0 && wave < C::HTILES;   // wave-uniform
  const int h_row = wave & 1, h_rt = min(wave, C::HTILES > 0 ? C::HTILES - 1 : 0) >> 1;

  for (int p = p_begin; p < p_end; p++) {
    const int n0 = p * SPASS;
    const int nw0 = n0 + 64 * wave;   // this wavefront's 64 columns
    const bool do_h = RT > 0 && p == p_begin;
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xf << 8));   // earlier stores drained (vmcnt(0))

    // ---- load plan ----
    SPlan P;
    P.a_base = xc + (int64_t)m0 * xrow;
#pragma unroll
    for (int i = 0; i < 2; i++) {
      const int row = min(m0 + 32 * i + l32, m - 1);
      P.a_off[i] = (uint32_t)((row - m0) * xrow + (lane >> 5) * 16);
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int ct = min(nw0 / 32 + j, ctiles - 1);
      P.b_base[j] = a.packed + geo.off_w + (int64_t)ct * KG * 1024;
    }
    P.l_base = a.packed + geo.off_l1 + (int64_t)h_rt * KG * 1024;
    if (lane >= 8 && lane < 16) {          // weight scales of the wavefront's 64 columns
      P.s_ptr = a.packed + geo.off_ws + (int64_t)min(nw0 + 8 * (lane - 8), geo.n_pad - 8) * 2;
      P.s_inc = (uint32_t)geo.n_pad * 2;
    } else if (RT > 0 && lane >= 16 && lane < 20) {   // L1 scales of the H tile's 32 ranks
      P.s_ptr = a.packed + geo.off_l1s + (int64_t)(h_rt * 32 + 8 * (lane - 16)) * 2;
      P.s_inc = (uint32_t)geo.r_pad32 * 2;
    } else {                               // activation scales of the 64 tokens
      const int l8 = lane < 8 ? lane : 0;
      P.s_ptr = reinterpret_cast<const uint8_t *>(a.xs) + (int64_t)min(m0 + 8 * l8, ms - 8) * 2;
      P.s_inc = (uint32_t)ms * 2;
    }

    v16f acc[2][2];
    v16f hacc = v16f{0};
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
      for (int j = 0; j < 2; j++) acc[i][j] = v16f{0};

    // one K loop; H rides along on the first pass of the H wavefronts
    auto k_loop = [&](auto HC) {
      constexpr bool H = decltype(HC)::value;
      constexpr int NL = H ? 6 : 5;
      auto issue = [&](int g, int slot) {
        s_issue<H>(P, min(g, KG - 1), ring_lds + slot * SSLOT, lane);
        P.s_ptr += g < KG - 1 ? P.s_inc : 0;   // stop at the last group
      };
      issue(0, 0);
      issue(1, 1);
      issue(2, 2);
      auto step = [&](int g, int slot) {
        wait_vm<(SD - 1) * NL>();            // group g has landed
        const uint8_t *S = ring + slot * SSLOT;
        const u32x4 ra0 = *reinterpret_cast<const u32x4 *>(S + S_A + lane * 16);
        const u32x4 ra1 = *reinterpret_cast<const u32x4 *>(S + S_A + 1024 + lane * 16);
        const u32x4 rb0 = *reinterpret_cast<const u32x4 *>(S + S_B + lane * 16);
        const u32x4 rb1 = *reinterpret_cast<const u32x4 *>(S + S_B + 1024 + lane * 16);
        const uint32_t sa0 = *reinterpret_cast<const uint16_t *>(S + S_S + l32 * 2);
        const uint32_t sa1 = *reinterpret_cast<const uint16_t *>(S + S_S + (32 + l32) * 2);
        const uint32_t sb0 = *reinterpret_cast<const uint16_t *>(S + S_S + 128 + l32 * 2);
        const uint32_t sb1 = *reinterpret_cast<const uint16_t *>(S + S_S + 128 + (32 + l32) * 2);
        u32x4 rl = u32x4{0, 0, 0, 0};
        uint32_t sl = 0;
        if constexpr (H) {
          rl = *reinterpret_cast<const u32x4 *>(S + S_L + lane * 16);
          sl = *reinterpret_cast<const uint16_t *>(S + S_S + 256 + l32 * 2);
        }
        // the slot is consumed: refill it with group g + SD
        __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
        issue(g + SD, slot);
        const v8i a0 = unpack32(ra0), a1 = unpack32(ra1);
        const v8i b0 = unpack32(rb0), b1 = unpack32(rb1);
        fma16(acc[0][0], codes_half(a0, b0), outer2(sa0, sb0));
        fma16(acc[0][1], codes_half(a0, b1), outer2(sa0, sb1));
        fma16(acc[1][0], codes_half(a1, b0), outer2(sa1, sb0));
        fma16(acc[1][1], codes_half(a1, b1), outer2(sa1, sb1));
        if constexpr (H) {
          const v8i lb = unpack32(rl);
          if (h_row) fma16(hacc, codes_half(a1, lb), outer2(sa1, sl));
          else fma16(hacc, codes_half(a0, lb), outer2(sa0, sl));
        }
      };
      for (int g = 0; g < KG; g += SD) {
        step(g, 0);
        if (g + 1 < KG) step(g + 1, 1);
        if (g + 2 < KG) step(g + 2, 2);
      }
      wait_vm<0>();   // the refills past the end are drained before the ring is reused
    };
    if (do_h && hmine) k_loop(std::true_type{});
    else k_loop(std::false_type{});
    __syncthreads();   // every wavefront is done with its ring

    if constexpr (RT > 0) {
      float *HS = reinterpret_cast<float *>(smem);
      uint8_t *QS = smem + C::OFF_Q;
      float *SHS = reinterpret_cast<float *>(smem + C::OFF_SH);
      const int r = geo.r, gr = geo.gr, rg = r / gr;
      if (do_h) {
        // ---- H -> LDS (fp32), then per-token, per-rank-group requantization ----
        if (hmine) {
#pragma unroll
          for (int v = 0; v < 16; v++) {
            const int row = 32 * h_row + row_of_32x32(lane, v);
            HS[row * C::HSTR + h_rt * 32 + l32] = hacc[v];
          }
        }
        if (r < C::RB * 64) {   // zero the fp8 padding ranks [r, 64 RB) of Q_H
          for (int idx = tid; idx < SBM * C::RB * 64; idx += 64 * SNW) {
            const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
            if (j >= r) QS[row * C::QSTR + j] = 0;
          }
        }
        __syncthreads();
        const int subs = gr / 8;               // lanes per (token, rank group): 1, 2, 4 or 8
        const int work = SBM * rg * subs;
        const bool dbg = a.dbg_h != nullptr && chunk == 0;
        for (int base = 0; base < work; base += 64 * SNW) {
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
    for (int i = 0; i < 2; i++) {
      const int trow = 32 * i;
#pragma unroll
      for (int j = 0; j < 2; j++) {
        const int ct = nw0 / 32 + j;
        const bool cvalid = ct < ctiles;
        v16f ylr = v16f{0};
        if constexpr (RT > 0) {
          const uint8_t *QS = smem + C::OFF_Q;
          const float *SHS = reinterpret_cast<const float *>(smem + C::OFF_SH);
#pragma unroll
          for (int rbk = 0; rbk < C::RB; rbk++) {
            const uint8_t *qrow = QS + (trow + l32) * C::QSTR + rbk * 64 + (lane >> 5) * 32;
            const v8i qa = join(*reinterpret_cast<const u32x4 *>(qrow),
                                *reinterpret_cast<const u32x4 *>(qrow + 16));
            v8i lb = {0, 0, 0, 0, 0, 0, 0, 0};
            float sl2 = 0.0f;
            if (cvalid) {
              lb = unpack32(*reinterpret_cast<const u32x4 *>(
                  l2codes + (((int64_t)ct * C::RB + rbk) * 64 + lane) * 16));
              sl2 = half_bits_to_float(l2scales[(int64_t)rbk * geo.n_pad + ct * 32 + l32]);
            }
            const v16f cb = mfma_codes_32x32x64(qa, lb);
#pragma unroll
            for (int v = 0; v < 16; v++) {
              const float sh = SHS[(trow + row_of_32x32(lane, v)) * C::RB + rbk];
              ylr[v] = fmaf(cb[v], sh * sl2, ylr[v]);
            }
          }
        }
        const int col = ct * 32 + l32;
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
    __syncthreads();   // the next pass refills the rings
  }
}

template <int RT>
hipError_t launch_stream(const GemmArgs &a, hipStream_t s) {
  using C = SCfg<RT>;
  const int m_tiles = (a.m + SBM - 1) / SBM;
  const int n_passes = (a.geo.n_pad + SPASS - 1) / SPASS;
  int ppw = 0, band = 0;
  if (const char *env = getenv("TQ_STREAM")) sscanf(env, "%d:%d", &ppw, &band);
  if (ppw <= 0) {
    ppw = (m_tiles * n_passes) / 256;
    if (ppw < 1) ppw = 1;
  }
  if (ppw > n_passes) ppw = n_passes;
  const int n_chunks = (n_passes + ppw - 1) / ppw;
  if (band <= 0) band = 16;
  if (band > m_tiles) band = m_tiles;
  auto kern = dual_gemm_stream_kernel<RT>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(m_tiles * n_chunks), dim3(64 * SNW), C::LDS, s, a, m_tiles,
                     n_chunks, ppw, band);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dual_gemm_stream(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.r_pad32 / 32) {
    case 0: return launch_stream<0>(a, s);
    case 1: return launch_stream<1>(a, s);
    case 2: return launch_stream<2>(a, s);
    case 4: return launch_stream<4>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tq
