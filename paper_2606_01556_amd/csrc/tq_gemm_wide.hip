// Fused dual-component W4A4 layer (paper Sec. 4.3) for prefill-sized token
// counts: the residual 4-bit GEMM, the stage-1 product H = Q(X) Q(L1) kept on
// chip, its on-the-fly re-quantization, stage 2 Q_H Q(L2) and one epilogue,
// in one kernel.
//
// Work decomposition.  A workgroup of 4 wavefronts (one per SIMD) owns 64
// tokens and a run of 256-column passes; each wavefront computes all 64
// tokens x 64 columns of a pass (four 32x32 tiles).  The activation operand of
// a K-group is therefore shared by the four wavefronts: it is expanded from
// 4-bit codes to fp8 once per workgroup, into LDS, while every wavefront
// expands its own weight columns in registers.  During the first pass the
// workgroup also accumulates H for its 64 tokens (2 r / 32 tiles of 32x32,
// spread over the wavefronts), then re-quantizes H into LDS; later passes
// reuse Q_H and s_H, so H is formed once per workgroup.
//
// K pipeline (one K-group of 64 per step, one workgroup barrier per step):
//   * every global byte arrives by direct global->LDS loads
//     (global_load_lds_dwordx4: scalar base + per-lane offset), four groups
//     ahead, into a 4-slot ring; every step of every wavefront issues the same
//     number of loads (the last groups repeat the final group), so waiting
//     for a group is one constant s_waitcnt, and the barrier then publishes
//     the group to the workgroup;
//   * two groups ahead, the workgroup expands the shared activation and L1
//     codes into fp8 matrix-core operands (4-slot LDS buffer);
//   * one group ahead, each wavefront reads its next operands into a second
//     register set while the current group's products run;
//   * within a step the matrix-core products of all tiles are issued before
//     the fp32 rescaling fmas, so the matrix core and the vector ALU overlap
//     inside each wavefront (one wavefront per SIMD, 512 registers).
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

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int WBM = 64;     // tokens per workgroup (two 32-row tiles)
constexpr int NWAVE = 4;    // wavefronts per workgroup
constexpr int WPASS = 256;  // output columns per pass (4 wavefronts x 64)
constexpr int WST = 4;      // raw ring slots (= load distance in K-groups)
constexpr int WUN = 4;      // expanded-operand slots

template <int RT>
struct WCfg {
  static constexpr int HTILES = 2 * RT;                  // 32x32 H tiles of a workgroup
  static constexpr int HT = (HTILES + NWAVE - 1) / NWAVE;  // per wavefront: tiles w + 4 hh
  static constexpr int HT1 = HT > 0 ? HT : 1;
  // shared loads of a group: activation blocks (2), L1 blocks (RT, first
  // pass), activation scales, weight scales, L1 scales (first pass); item q
  // is loaded by wavefront q % 4 as its load 2 + q / 4 (loads 0 and 1 are its
  // own weight blocks); the other wavefronts pad with a dummy load
  static constexpr int NSH_H = 2 + RT + 3;
  static constexpr int NSH_R = 4;
  static constexpr int NL_H = 2 + (NSH_H + NWAVE - 1) / NWAVE;
  static constexpr int NL_R = 2 + (NSH_R + NWAVE - 1) / NWAVE;
  static constexpr int NL_MAX = NL_H > NL_R ? NL_H : NL_R;
  // raw slot: codes in matrix-core lane order, 1 KiB per 32-row/column block
  static constexpr int R_A = 0;                  // 2 activation blocks
  static constexpr int R_L = 2048;               // RT L1 blocks
  static constexpr int R_B = R_L + RT * 1024;    // 8 weight blocks (2 per wavefront)
  static constexpr int R_SA = R_B + 8192;        // 64 activation scales (first 128 B)
  static constexpr int R_SL = R_SA + 1024;       // 32 RT L1 scales
  static constexpr int R_SW = R_SL + 1024;       // 256 weight scales (first 512 B)
  static constexpr int R_D = R_SW + 1024;        // dummy-load target
  static constexpr int SLOT = R_D + 1024;
  // expanded slot: fp8 operands [block][half][lane][16 B]
  static constexpr int U_L = 4096;
  static constexpr int USLOT = U_L + RT * 2048;
  static constexpr int OFF_UNP = WST * SLOT;
  static constexpr int LOOP_LDS = OFF_UNP + WUN * USLOT;
  // after the first pass: H in fp32 (aliases the ring), then Q_H and s_H,
  // which later passes read, outside the ring
  static constexpr int HSTR = RT * 32 + 1;
  static constexpr int RB = (RT + 1) / 2;        // 64-rank blocks
  static constexpr int QSTR = RB * 64 + 16;
  static constexpr int OFF_Q = LOOP_LDS;
  static constexpr int OFF_SH = OFF_Q + (RT > 0 ? WBM * QSTR : 0);
  static constexpr int LDS = OFF_SH + (RT > 0 ? WBM * RB * 4 : 0);
  static_assert(HT <= 2, "at most two H tiles per wavefront");
  static_assert(WBM * HSTR * 4 <= LOOP_LDS, "H staging fits in the ring");
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

template <int RT>
struct WKernel {
  using C = WCfg<RT>;

  struct Ctx {
    uint8_t *smem;
    uint32_t lds0;   // LDS address of smem (wave-uniform)
    int tid, lane, wave, KG;
  };

  // This wavefront's loads of one group: load s reads 16 bytes per lane from
  // sb[s] + g * inc[s] + voff[s] into slot offset loff[s] (sb, inc, loff
  // wave-uniform).
  struct Plan {
    const uint8_t *sb[C::NL_MAX];
    uint32_t inc[C::NL_MAX];
    uint32_t voff[C::NL_MAX];
    uint32_t loff[C::NL_MAX];
  };

  template <bool H>
  __device__ __forceinline__ static void plan(const GemmArgs &a, const Ctx &c, int m0, int n0,
                                              Plan &P) {
    const Geometry &geo = a.geo;
    const int KG = c.KG, lane = c.lane, wave = c.wave;
    const int ctiles = geo.n_pad / 32;
    const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
    const uint8_t *xs = reinterpret_cast<const uint8_t *>(a.xs);
    const int64_t xrow = geo.k / 2;
    constexpr int NL = H ? C::NL_H : C::NL_R;
    // the two weight blocks of this wavefront (clamped past the last column
    // tile: such tiles are computed and never stored)
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int ct = min(n0 / 32 + 2 * wave + j, ctiles - 1);
      P.sb[j] = a.packed + geo.off_w + (int64_t)ct * KG * 1024;
      P.inc[j] = 1024;
      P.voff[j] = lane * 16;
      P.loff[j] = C::R_B + (2 * wave + j) * 1024;
    }
    auto a_block = [&](int s, int q) {   // activation rows 32 q + lane % 32 (clamped to m - 1)
      const int row = min(m0 + 32 * q + (lane & 31), a.m - 1);
      P.sb[s] = xc + (int64_t)m0 * xrow;
      P.inc[s] = 32;
      P.voff[s] = (uint32_t)((row - m0) * xrow + (lane >> 5) * 16);
    };
#pragma unroll
    for (int s = 2; s < NL; s++) {
      int q = (s - 2) * NWAVE + wave;
      if (q < 2) {
        a_block(s, q);
        P.loff[s] = C::R_A + q * 1024;
        continue;
      }
      q -= 2;
      if (H && q < RT) {
        P.sb[s] = a.packed + geo.off_l1 + (int64_t)q * KG * 1024;
        P.inc[s] = 1024;
        P.voff[s] = lane * 16;
        P.loff[s] = C::R_L + q * 1024;
        continue;
      }
      if (H) q -= RT;
      if (q == 0) {                        // activation scales of the 64 tokens
        P.sb[s] = xs + (int64_t)m0 * 2;
        P.inc[s] = (uint32_t)a.ms * 2;
        P.voff[s] = (uint32_t)min(16 * lane, (a.ms - m0 - 8) * 2);
        P.loff[s] = C::R_SA;
      } else if (q == 1) {                 // weight scales of the pass
        P.sb[s] = a.packed + geo.off_ws;
        P.inc[s] = (uint32_t)geo.n_pad * 2;
        P.voff[s] = (uint32_t)min(n0 + 8 * lane, geo.n_pad - 8) * 2;
        P.loff[s] = C::R_SW;
      } else if (H && q == 2) {            // L1 scales
        P.sb[s] = a.packed + geo.off_l1s;
        P.inc[s] = (uint32_t)geo.r_pad32 * 2;
        P.voff[s] = (uint32_t)min(16 * lane, (geo.r_pad32 - 8) * 2);
        P.loff[s] = C::R_SL;
      } else {                             // padding load
        a_block(s, 0);
        P.loff[s] = C::R_D;
      }
    }
  }

  template <bool H>
  __device__ __forceinline__ static void issue(const Ctx &c, const Plan &P, int g, int slot) {
    constexpr int NL = H ? C::NL_H : C::NL_R;
    const uint32_t base = c.lds0 + slot * C::SLOT;
#pragma unroll
    for (int s = 0; s < NL; s++) {
      const uint8_t *sb = P.sb[s] + (uint64_t)g * P.inc[s];
      asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(P.voff[s]),
                   "s"(sb), "s"(base + P.loff[s])
                   : "memory");
    }
  }

  // s_waitcnt vmcnt(n): at most n of this wavefront's loads in flight
  template <int N>
  __device__ __forceinline__ static void wait_vm() {
    static_assert(N < 64, "vmcnt has 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
  }

  // expand the shared activation (and L1) codes of a raw slot into fp8
  template <bool H>
  __device__ __forceinline__ static void expand(const Ctx &c, int slot, int uslot) {
    constexpr int NCH = 64 * (2 + (H ? RT : 0));
    const uint8_t *raw = c.smem + slot * C::SLOT + C::R_A;
    uint8_t *dst = c.smem + C::OFF_UNP + uslot * C::USLOT;
#pragma unroll
    for (int ch0 = 0; ch0 < NCH; ch0 += 64 * NWAVE) {
      const int ch = ch0 + c.tid;
      if (NCH % (64 * NWAVE) == 0 || ch < NCH) {
        const v8i u = unpack32(*reinterpret_cast<const u32x4 *>(raw + ch * 16));
        uint8_t *d = dst + (ch >> 6) * 2048 + (ch & 63) * 16;
        *reinterpret_cast<u32x4 *>(d) = u32x4{(uint32_t)u[0], (uint32_t)u[1], (uint32_t)u[2], (uint32_t)u[3]};
        *reinterpret_cast<u32x4 *>(d + 1024) =
            u32x4{(uint32_t)u[4], (uint32_t)u[5], (uint32_t)u[6], (uint32_t)u[7]};
      }
    }
  }

  // one group's operands for this wavefront
  struct Frags {
    v8i a[2];              // activation rows 0-31, 32-63 (fp8)
    u32x4 braw[2];         // this wavefront's two weight column tiles (codes)
    v8i b[2];              // ... expanded
    v8i ah;                // activation rows of this wavefront's H tiles (fp8)
    v8i l[C::HT1];         // L1 ranks of its H tiles (fp8)
    uint32_t sa[2], sb[2], sah, sl[C::HT1];   // scale operands (fp16 in the low half)
  };

  template <bool H>
  __device__ __forceinline__ static void read_frags(const Ctx &c, int slot, int uslot, Frags &F) {
    const uint8_t *R = c.smem + slot * C::SLOT;
    const uint8_t *U = c.smem + C::OFF_UNP + uslot * C::USLOT;
    const int lane = c.lane, l32 = lane & 31;
#pragma unroll
    for (int i = 0; i < 2; i++) {
      F.a[i] = join(*reinterpret_cast<const u32x4 *>(U + i * 2048 + lane * 16),
                    *reinterpret_cast<const u32x4 *>(U + i * 2048 + 1024 + lane * 16));
      F.sa[i] = *reinterpret_cast<const uint16_t *>(R + C::R_SA + (32 * i + l32) * 2);
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      F.braw[j] = *reinterpret_cast<const u32x4 *>(R + C::R_B + (2 * c.wave + j) * 1024 + lane * 16);
      F.sb[j] = *reinterpret_cast<const uint16_t *>(R + C::R_SW + (64 * c.wave + 32 * j + l32) * 2);
    }
    if constexpr (H && RT > 0) {
      // H tiles w + 4 hh: row tile w % 2 (the same for both), rank tile
      // (w + 4 hh) / 2, clamped for the wavefronts without one (never stored)
      const int i = c.wave & 1;
      F.ah = join(*reinterpret_cast<const u32x4 *>(U + i * 2048 + lane * 16),
                  *reinterpret_cast<const u32x4 *>(U + i * 2048 + 1024 + lane * 16));
      F.sah = *reinterpret_cast<const uint16_t *>(R + C::R_SA + (32 * i + l32) * 2);
#pragma unroll
      for (int hh = 0; hh < C::HT; hh++) {
        const int rt = min(c.wave + NWAVE * hh, C::HTILES - 1) >> 1;
        F.l[hh] = join(*reinterpret_cast<const u32x4 *>(U + C::U_L + rt * 2048 + lane * 16),
                       *reinterpret_cast<const u32x4 *>(U + C::U_L + rt * 2048 + 1024 + lane * 16));
        F.sl[hh] = *reinterpret_cast<const uint16_t *>(R + C::R_SL + (32 * rt + l32) * 2);
      }
    }
  }

  __device__ __forceinline__ static void expand_b(Frags &F) {
    F.b[0] = unpack32(F.braw[0]);
    F.b[1] = unpack32(F.braw[1]);
  }

  // One K-group g (ph = g % 4): wait for group g + 2, barrier, start the loads
  // of group g + 4; issue the products of group g (operands in F), expand
  // group g + 2 and read group g + 1's operands into N while they run, then
  // apply the fmas of group g.
  template <bool H, int ph>
  __device__ __forceinline__ static void step(const Ctx &c, const Plan &P, int g, const Frags &F,
                                              Frags &N, v16f (&acc)[2][2], v16f (&hacc)[C::HT1],
                                              bool hmine) {
    constexpr int NL = H ? C::NL_H : C::NL_R;
    const int KG = c.KG;
    wait_vm<NL>();                           // only group g + 3's loads may be in flight
    __builtin_amdgcn_s_waitcnt(0xc07f);      // lgkmcnt(0): this wavefront's LDS reads are done
    __syncthreads();
    issue<H>(c, P, min(g + WST, KG - 1), ph);
    const v16f c00 = codes_half(F.a[0], F.b[0]), p00 = outer2(F.sa[0], F.sb[0]);
    const v16f c01 = codes_half(F.a[0], F.b[1]), p01 = outer2(F.sa[0], F.sb[1]);
    const v16f c10 = codes_half(F.a[1], F.b[0]), p10 = outer2(F.sa[1], F.sb[0]);
    const v16f c11 = codes_half(F.a[1], F.b[1]), p11 = outer2(F.sa[1], F.sb[1]);
    expand<H>(c, (ph + 2) & 3, (ph + 2) & 3);
    read_frags<H>(c, (ph + 1) & 3, (ph + 1) & 3, N);
    fma16(acc[0][0], c00, p00);
    fma16(acc[0][1], c01, p01);
    if constexpr (H && RT > 0) {
      if (hmine) {
        const v16f ch0 = codes_half(F.ah, F.l[0]), ph0 = outer2(F.sah, F.sl[0]);
        fma16(acc[1][0], c10, p10);
        fma16(acc[1][1], c11, p11);
        if constexpr (C::HT > 1) {
          const v16f ch1 = codes_half(F.ah, F.l[1]), ph1 = outer2(F.sah, F.sl[1]);
          fma16(hacc[0], ch0, ph0);
          expand_b(N);
          fma16(hacc[1], ch1, ph1);
        } else {
          expand_b(N);
          fma16(hacc[0], ch0, ph0);
        }
        return;
      }
    }
    fma16(acc[1][0], c10, p10);
    expand_b(N);
    fma16(acc[1][1], c11, p11);
  }

  template <bool H>
  __device__ __forceinline__ static void k_loop(const Ctx &c, const Plan &P, v16f (&acc)[2][2],
                                                v16f (&hacc)[C::HT1], bool hmine) {
    constexpr int NL = H ? C::NL_H : C::NL_R;
    const int KG = c.KG;
#pragma unroll
    for (int j = 0; j < WST; j++) issue<H>(c, P, min(j, KG - 1), j);
    wait_vm<2 * NL>();                       // groups 0 and 1 have landed
    __syncthreads();
    expand<H>(c, 0, 0);
    expand<H>(c, 1, 1);
    __syncthreads();
    Frags F0, F1;
    read_frags<H>(c, 0, 0, F0);
    expand_b(F0);
    for (int g = 0; g < KG; g += 4) {
      step<H, 0>(c, P, g, F0, F1, acc, hacc, hmine);
      if (g + 1 < KG) step<H, 1>(c, P, g + 1, F1, F0, acc, hacc, hmine);
      if (g + 2 < KG) step<H, 2>(c, P, g + 2, F0, F1, acc, hacc, hmine);
      if (g + 3 < KG) step<H, 3>(c, P, g + 3, F1, F0, acc, hacc, hmine);
    }
    wait_vm<0>();
    __syncthreads();   // every wavefront is done with the ring
  }
};

template <int RT>
__global__ __launch_bounds__(64 * NWAVE, 1) void dual_gemm_wide_kernel(GemmArgs a, int m_tiles,
                                                                       int n_chunks,
                                                                       int passes_per_wg, int band) {
  using K_ = WKernel<RT>;
  using C = typename K_::C;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  typename K_::Ctx c;
  c.smem = smem;
  c.lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
  c.tid = threadIdx.x;
  c.lane = threadIdx.x & 63;
  c.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  c.KG = geo.k / kGroup;
  const int tid = c.tid, lane = c.lane, wave = c.wave;
  const int m = a.m;
  const int ctiles = geo.n_pad / 32;
  const int n_passes = (geo.n_pad + WPASS - 1) / WPASS;

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
  const int m0 = m_tile * WBM;
  const int p_begin = chunk * passes_per_wg;
  const int p_end = min(p_begin + passes_per_wg, n_passes);

  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const bool hmine = RT > 0 && wave < C::HTILES;

  for (int p = p_begin; p < p_end; p++) {
    const int n0 = p * WPASS;
    const bool do_h = RT > 0 && p == p_begin;
    __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xf << 8));   // earlier stores drained (vmcnt(0))

    v16f acc[2][2];
    v16f hacc[C::HT1];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
      for (int j = 0; j < 2; j++) acc[i][j] = v16f{0};
#pragma unroll
    for (int h = 0; h < C::HT1; h++) hacc[h] = v16f{0};
    typename K_::Plan P;
    if (do_h) {
      K_::template plan<true>(a, c, m0, n0, P);
      K_::template k_loop<true>(c, P, acc, hacc, hmine);
    } else {
      K_::template plan<false>(a, c, m0, n0, P);
      K_::template k_loop<false>(c, P, acc, hacc, hmine);
    }

    if constexpr (RT > 0) {
      float *HS = reinterpret_cast<float *>(smem);
      uint8_t *QS = smem + C::OFF_Q;
      float *SHS = reinterpret_cast<float *>(smem + C::OFF_SH);
      const int r = geo.r, gr = geo.gr, rg = r / gr;
      if (do_h) {
        // ---- H -> LDS (fp32), then per-token, per-rank-group requantization ----
        if (hmine) {
          const int i = wave & 1;
#pragma unroll
          for (int hh = 0; hh < C::HT; hh++) {
            const int h = wave + NWAVE * hh;
            if (h < C::HTILES) {
              const int rt = h >> 1;
#pragma unroll
              for (int v = 0; v < 16; v++) {
                const int row = 32 * i + row_of_32x32(lane, v);
                HS[row * C::HSTR + rt * 32 + (lane & 31)] = hacc[hh][v];
              }
            }
          }
        }
        if (r < C::RB * 64) {   // zero the fp8 padding ranks [r, 64 RB) of Q_H
          for (int idx = tid; idx < WBM * C::RB * 64; idx += 64 * NWAVE) {
            const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
            if (j >= r) QS[row * C::QSTR + j] = 0;
          }
        }
        __syncthreads();
        const int subs = gr / 8;               // lanes per (token, rank group): 1, 2, 4 or 8
        const int work = WBM * rg * subs;
        const bool dbg = a.dbg_h != nullptr && chunk == 0;
        for (int base = 0; base < work; base += 64 * NWAVE) {
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
        const int ct = n0 / 32 + 2 * wave + j;
        const bool cvalid = ct < ctiles;
        v16f ylr = v16f{0};
        if constexpr (RT > 0) {
          const uint8_t *QS = smem + C::OFF_Q;
          const float *SHS = reinterpret_cast<const float *>(smem + C::OFF_SH);
#pragma unroll
          for (int rbk = 0; rbk < C::RB; rbk++) {
            const uint8_t *qrow = QS + (trow + (lane & 31)) * C::QSTR + rbk * 64 + (lane >> 5) * 32;
            const v8i qa = join(*reinterpret_cast<const u32x4 *>(qrow),
                                *reinterpret_cast<const u32x4 *>(qrow + 16));
            v8i lb = {0, 0, 0, 0, 0, 0, 0, 0};
            float sl2 = 0.0f;
            if (cvalid) {
              lb = unpack32(*reinterpret_cast<const u32x4 *>(
                  l2codes + (((int64_t)ct * C::RB + rbk) * 64 + lane) * 16));
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
    __syncthreads();   // the next pass refills the ring
  }
}

template <int RT>
hipError_t launch_wide(const GemmArgs &a, hipStream_t s) {
  using C = WCfg<RT>;
  const int m_tiles = (a.m + WBM - 1) / WBM;
  const int n_passes = (a.geo.n_pad + WPASS - 1) / WPASS;
  // passes per workgroup: enough workgroups to fill the 256 CUs once, and
  // beyond that longer runs of passes (fewer recomputations of H)
  int ppw = 0, band = 0;
  if (const char *env = getenv("TQ_WIDE")) sscanf(env, "%d:%d", &ppw, &band);
  if (ppw <= 0) {
    ppw = (m_tiles * n_passes) / 256;
    if (ppw < 1) ppw = 1;
  }
  if (ppw > n_passes) ppw = n_passes;
  const int n_chunks = (n_passes + ppw - 1) / ppw;
  if (band <= 0) band = 16;
  if (band > m_tiles) band = m_tiles;
  auto kern = dual_gemm_wide_kernel<RT>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(m_tiles * n_chunks), dim3(64 * NWAVE), C::LDS, s, a, m_tiles,
                     n_chunks, ppw, band);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dual_gemm_wide(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.r_pad32 / 32) {
    case 0: return launch_wide<0>(a, s);
    case 1: return launch_wide<1>(a, s);
    case 2: return launch_wide<2>(a, s);
    case 4: return launch_wide<4>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tq
