// Fused dual-component W4A4 layer (paper Sec. 4.3) for decode-sized token
// counts (m <= 16): the residual 4-bit GEMM, the stage-1 product
// H = Q(X) Q(L1), its on-chip re-quantization, stage 2 Q_H Q(L2) and one
// epilogue, in one kernel.  Nothing of the layer leaves the chip but Y.
//
// Work decomposition.  One work-group of sixteen wavefronts per CU owns CT
// 16-column tiles of Y and streams their packed weights once.  H is small
// (m x r) and every work-group forms all of it in its own registers, so no
// work-group waits for another; the price is that each CU reads all of L1
// (from L2, where the first reader leaves it) in addition to its columns.
//  * Wavefront w < ceil(r / 16) owns rank tile w of H and walks every
//    K-group pair in ascending order, so its fp32 chain (one fma per K-group,
//    ascending, with the exact product I s_x) stays in registers and H is
//    bit-identical to the oracle's.
//  * The other wavefronts take the residual work: each owns one or two of
//    the column tiles and every NPH-th K-group pair (NPH wavefronts share a
//    tile group); their partial sums are added in a fixed order at the end
//    (the order of Y's fp32 accumulation is free; H's is not).
//  * Operands stream from global memory straight into registers through
//    per-wavefront rings of 8 to 10 pairs (the L1 bytes come from L2, at its
//    latency); there is no LDS staging and no barrier in the K loop.  The
//    activation codes (a few KiB at these sizes) are copied to LDS once, or,
//    for the fp16 entry point, quantized into LDS by the work-group itself
//    (Sec. 4.3: the activation tile is quantized once and reused by both
//    branches), with the same arithmetic as the quantizer kernel.
//
// Products.  v_mfma_scale_f32_16x16x128_f8f6f4 on codes as fp8 subnormals
// (block scales 2^9: exact integer sums).  A K-group pair spans the 128 K of
// one product, and the two groups need separate sums:
//  * up to 8 tokens, rows 0-7 take group A's codes in k < 64 and rows 8-15
//    group B's in k >= 64 (zeros elsewhere), so one product yields both
//    groups' sums; lanes 32-63 hold group B's and v_permlane32_swap brings
//    them to lanes 0-31 for the chain;
//  * up to 16 tokens, rows are tokens and two products take the pair's
//    groups in turn (the other group's half of the operand zero).
// Only the accumulator rows that hold real tokens (MV of the four per lane)
// are rescaled, so single-token decode spends one fma per group and output
// column, not sixteen.
#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

constexpr int DW = 16;                     // wavefronts per work-group
constexpr int kDecodeXBytes = 112 * 1024;  // LDS for the activation codes

// Token layouts: MODE 1 / 2 / 4 put two K-groups in one product (rows are
// (group, token) pairs, up to 8 tokens) with MV = MODE live accumulator rows
// per lane; MODE 16 takes up to 16 tokens, one group per product.
template <int MODE>
struct DMode {
  static constexpr bool TOK8 = MODE != 16;
  static constexpr int MV = MODE == 16 ? 4 : MODE;
  // LDS copy of the activation codes: fp8 operand bytes for one or two tokens,
  // TQ4 words (unpacked at use) otherwise; MX token slots per K-group
  static constexpr bool XFP8 = MODE <= 2;
  static constexpr int MX = MODE == 16 ? 16 : (MODE <= 2 ? MODE : 8);
  static constexpr int XB = XFP8 ? 64 : 32;   // bytes per (group, token)
  // pairs of operands in flight per stage-1 wavefront, and the residual
  // ring's budget in 16-byte fragments (what fits 128 registers unspilled)
  static constexpr int D1 = MODE == 16 ? 8 : (MODE == 1 ? 9 : 10);
  // one token: the two L1 scale rows of a pair arrive by one load (group A's
  // row in lanes 0-31, group B's in lanes 32-63)
  static constexpr bool MS = MODE == 1;
  static constexpr int RF = MODE == 1 ? 10 : 8;
};

// A residual wavefront owns CTW of the work-group's CT column tiles (TG
// tile groups) and keeps D2 pairs of their operands in flight.
template <int CT, int RF> struct DRes {
  static constexpr int CTW = CT == 1 ? 1 : 2;
  static constexpr int TG = CT / CTW;
  static constexpr int D2 = RF / CTW;
};

// LDS layout (bytes): region 0 holds the activation codes during the K loop
// and, aliased, the epilogue's residual partials, H, Q_H and s_H; the fp32
// activation scales follow it.
struct DLayout {
  int xa, epi_res, epi_h, epi_q, epi_sh, xs, total;
  static constexpr int HSTR = kMaxRank + 1;   // fp32 per H row
  static constexpr int QSTR = kMaxRank + 16;  // bytes per Q_H row
  // res_bytes: the residual partials [NPH][CT][16][16] fp32
  __host__ __device__ DLayout(int kg, int mx, int xb, int res_bytes) {
    const int kgp = (kg + 1) / 2 * 2;
    xa = kgp * mx * xb + 32;   // + a 32-byte zero pad
    epi_res = 0;
    epi_h = res_bytes;
    epi_q = epi_h + 16 * HSTR * 4;
    epi_sh = epi_q + 16 * QSTR;
    const int epi_end = epi_sh + 2 * 16 * 4;
    xs = ((xa > epi_end ? xa : epi_end) + 15) / 16 * 16;
    total = xs + kgp * mx * 4;
  }
};

__host__ __device__ inline int rank_tiles(int r) { return (r + 15) / 16; }

// The K-loop roles: wavefronts 0 .. R - 1 form H, the others the residual.
template <int MODE, int CT>
__host__ __device__ inline DLayout decode_layout(int kg, int r) {
  using DR = DRes<CT, DMode<MODE>::RF>;
  const int nph = (DW - rank_tiles(r)) / DR::TG;
  return DLayout(kg, DMode<MODE>::MX, DMode<MODE>::XB, nph * CT * 1024);
}

// max over runs of n = 8, 16 or 32 aligned lanes, in every lane of the run
__device__ __forceinline__ float dpp_max(float a, int ctrl_sel) {
  int b;
  switch (ctrl_sel) {
    case 0: b = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0xB1, 0xF, 0xF, false); break;
    case 1: b = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x4E, 0xF, 0xF, false); break;
    case 2: b = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x141, 0xF, 0xF, false); break;
    default: b = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, a), 0x140, 0xF, 0xF, false); break;
  }
  return fmaxf(a, __builtin_bit_cast(float, b));
}
__device__ __forceinline__ float run_max(float a, int n, int lane) {
  a = dpp_max(a, 0);   // lane ^ 1
  a = dpp_max(a, 1);   // lane ^ 2
  a = dpp_max(a, 2);   // half-row mirror: 8 lanes
  if (n >= 16) a = dpp_max(a, 3);   // row mirror: 16 lanes
  if (n >= 32) {
    const float r0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, a), 0));
    const float r1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, a), 16));
    const float r2 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, a), 32));
    const float r3 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, a), 48));
    a = lane < 32 ? fmaxf(r0, r1) : fmaxf(r2, r3);
  }
  return a;
}

// lanes 0-31 receive lanes 32-63 of v (lanes 32-63 get their own values back)
__device__ __forceinline__ float upper_half(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[1]);
}

__device__ __forceinline__ v8i lds_v8i(const uint8_t *p) {
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(p);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(p + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

__device__ __forceinline__ float lo_half(uint32_t w) { return half_bits_to_float((uint16_t)(w & 0xffffu)); }
__device__ __forceinline__ float hi_half(uint32_t w) { return half_bits_to_float((uint16_t)(w >> 16)); }

// Operands of one K-group pair: for a stage-1 wavefront the fragment of its
// rank tile with the L1 scales of both groups, for a residual wavefront the
// CT weight fragments with their scales.
struct S1Slot {
  u32x4 l1;
  // fp16 L1 scales of the lane's rank for groups A and B; for one token a
  // single load, the lane's own group's row (sla only)
  uint32_t sla, slb;
};
template <int CTW>
struct ResSlot {
  u32x4 w[CTW];
  uint32_t swa[CTW], swb[CTW];   // fp16 weight scales (TOK8: the lane's own group in swa)
};

// GK: 64-wide K blocks per quantization group (1 or 2, the layer's geo.gk),
// or 0: read from geo.gk at run time
template <int MODE, int CT, bool FQ, int GK>
__global__ __launch_bounds__(64 * DW) void dual_gemm_decode_kernel(GemmArgs a,
                                                                   const uint16_t *__restrict__ xh) {
  using MD = DMode<MODE>;
  constexpr int MX = MD::MX, MV = MD::MV, XB = MD::XB;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, c16 = lane & 15, qh = q & 1;
  const int KG = geo.k / kGroup, NP = (KG + 1) / 2;
  const int m = a.m;
  const int r = geo.r, R = rank_tiles(r);
  const int NS = R;   // stage-1 wavefronts
  const int NRES = DW - NS;
  const int ct16 = geo.n_pad / 16;
  const int c0 = blockIdx.x * CT;
  const DLayout LY = decode_layout<MODE, CT>(KG, r);
  uint8_t *XA = smem;
  float *XS = reinterpret_cast<float *>(smem + LY.xs);
  const uint8_t *wcodes = a.packed + geo.off_w;
  const uint16_t *wscales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_ws);
  const uint8_t *l1codes = a.packed + geo.off_l1;
  const uint16_t *l1scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l1s);
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);

  // ---- roles: wavefront w < R forms rank tile w of H over every pair; the
  // others are residual wavefronts: rslot = w - R owns tile group rslot % TG
  // and the pairs rslot / TG + i NPH ----
  using DR = DRes<CT, MD::RF>;
  constexpr int D1 = MD::D1;
  constexpr int CTW = DR::CTW, TG = DR::TG, D2 = DR::D2;
  const bool s1 = wave < NS;
  const int rslot = wave - NS;
  const int NPH = NRES / TG;
  const int tg = s1 ? 0 : rslot % TG, ph = s1 ? 0 : rslot / TG;
  const bool rbusy = !s1 && ph < NPH;
  const int nres_it = rbusy && ph < NP ? (NP - ph + NPH - 1) / NPH : 0;
  const int ctw0 = c0 + tg * CTW;   // first column tile of this residual wavefront

  // Ring loads are unconditional (a pair past the end reloads the last one),
  // so the compiler can count the outstanding loads and wait only for the
  // slot it uses.  Lane quarters q < 2 take group A = 2p, q >= 2 group B.
  // Addresses are a wave-uniform base (pair p) plus a fixed 32-bit lane
  // offset, kept to a few scalar operations per load: the scalar unit, which
  // all wavefronts of a CU share, is what a costlier form saturates first.
  // On an odd tail (group 2p + 1 == KG) the group-B lanes read the zero codes
  // and zero scale row that follow each section in the packed buffer.
  // (Section offsets fit 32 bits: the packed buffer is below 4 GiB.)
  const int gq = q >> 1;
  const uint32_t l1_lane = (uint32_t)(((wave >> 1) * KG * 64 + gq * 64 + qh * 32 + (wave & 1) * 16 + c16) * 16);
  const uint32_t l1s_lane = (uint32_t)(16 * wave + c16) * 2;
  // Scale rows: one per quantization group, so a pair of 64-wide blocks spans
  // two rows (64-wide groups) or one (128-wide groups, gk = 2), and group B's
  // row is the next one or the same.
  const int gk = GK ? GK : geo.gk;
  const uint32_t l1s_pair = (uint32_t)geo.r_pad32 * 4 / gk, ws_pair = (uint32_t)geo.n_pad * 4 / gk;
  const uint32_t l1s_b = gk == 1 ? (uint32_t)geo.r_pad32 * 2 : 0u, ws_b = gk == 1 ? (uint32_t)geo.n_pad * 2 : 0u;
  const uint8_t *l1sb = reinterpret_cast<const uint8_t *>(l1scales);
  const uint8_t *wsb = reinterpret_cast<const uint8_t *>(wscales);
  const uint32_t l1s_own = l1s_lane + gq * l1s_b;   // the lane's own group's row
  auto load_s1 = [&](S1Slot &S, int p) {
    S.l1 = *reinterpret_cast<const u32x4 *>(l1codes + (uint32_t)(p * 2048) + l1_lane);
    const uint8_t *sb = l1sb + (uint32_t)p * l1s_pair;
    if constexpr (MD::MS) {
      S.sla = *reinterpret_cast<const uint16_t *>(sb + l1s_own);
    } else {
      S.sla = *reinterpret_cast<const uint16_t *>(sb + l1s_lane);
      S.slb = *reinterpret_cast<const uint16_t *>(sb + l1s_b + l1s_lane);
    }
  };
  uint32_t w_lane[CTW], ws_lane[CTW];
  const uint32_t ws_gq = gq * ws_b;   // the lane's own block's group (TOK8)
#pragma unroll
  for (int j = 0; j < CTW; j++) {
    const int ct = min(ctw0 + j, ct16 - 1);
    w_lane[j] = (uint32_t)((((ct >> 1) * KG + gq) * 64 + qh * 32 + (ct & 1) * 16 + c16) * 16);
    ws_lane[j] = (uint32_t)(16 * ct + c16) * 2;
  }
  auto load_res = [&](ResSlot<CTW> &S, int p) {
    const uint8_t *sa = wsb + (uint32_t)p * ws_pair;
#pragma unroll
    for (int j = 0; j < CTW; j++) {
      S.w[j] = *reinterpret_cast<const u32x4 *>(wcodes + (uint32_t)(p * 2048) + w_lane[j]);
      if constexpr (MD::TOK8) {
        S.swa[j] = *reinterpret_cast<const uint16_t *>(sa + (ws_lane[j] + ws_gq));
      } else {
        S.swa[j] = *reinterpret_cast<const uint16_t *>(sa + ws_lane[j]);
        S.swb[j] = *reinterpret_cast<const uint16_t *>(sa + ws_b + ws_lane[j]);
      }
    }
  };

  // ---- the activation codes and scales into LDS (each wavefront runs this
  // once, after issuing the first loads of its own ring) ----
  const int KGP = 2 * NP;
  auto prologue = [&]() {
    if constexpr (FQ) {
      // eight lanes per (token, quantization group), eight values of each of
      // the group's gk 64-wide blocks; the steps are those of the quantizer
      // kernel, so the codes and scales are the same bits
      const int e = lane & 7;
      const int KQ = KG / gk;
      const int nitem = m * KQ;
      for (int it0 = 0; it0 < nitem; it0 += 64 * DW / 8) {
        const int it = it0 + tid / 8;
        const bool live = it < nitem;
        const int t = live ? it / KQ : 0, g0 = live ? it % KQ * gk : 0, g1 = g0 + gk - 1;
        const uint16_t *src = xh + (int64_t)t * geo.k + 8 * e;
        const u32x4 raw0 = *reinterpret_cast<const u32x4 *>(src + g0 * kGroup);
        u32x4 raw1 = raw0;
        if (gk == 2) raw1 = *reinterpret_cast<const u32x4 *>(src + g1 * kGroup);
        float v0[8], v1[8];
#pragma unroll
        for (int i = 0; i < 4; i++) {
          v0[2 * i] = half_bits_to_float((uint16_t)(raw0[i] & 0xffffu));
          v0[2 * i + 1] = half_bits_to_float((uint16_t)(raw0[i] >> 16));
          v1[2 * i] = half_bits_to_float((uint16_t)(raw1[i] & 0xffffu));
          v1[2 * i + 1] = half_bits_to_float((uint16_t)(raw1[i] >> 16));
        }
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; i++) amax = fmaxf(amax, fmaxf(fabsf(v0[i]), fabsf(v1[i])));
        amax = max8_dpp(amax);
        uint16_t s16;
        const float sc = q4_scale(amax, s16);
        const float y = sc == 0.0f ? 0.0f : __builtin_amdgcn_rcpf(sc);
#pragma unroll
        for (int b = 0; b < 2; b++) {
          if (b == 1 && gk == 1) break;
          uint32_t b0, b1;
          quant8_fp8(b == 0 ? v0 : v1, sc, y, b0, b1);
          const int g = b == 0 ? g0 : g1;
          if (live) {
            uint8_t *dst = XA + (g * MX + t) * XB;
            if constexpr (MD::XFP8)
              *reinterpret_cast<uint2 *>(dst + 8 * e) = make_uint2(b0, b1);
            else
              *reinterpret_cast<uint32_t *>(dst + 4 * e) = b0 | __builtin_amdgcn_alignbit(b1, b1, 28);
            if (e == 0) XS[g * MX + t] = sc;
          }
        }
      }
      for (int idx = tid; idx < KGP * MX; idx += 64 * DW)
        if (idx / MX >= KG || idx % MX >= m) XS[idx] = 0.0f;
    } else {
      // 16-byte fragments (group g, token t, half h) of tile 0's TQ4 blocks
      const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
      const int nfrag = KG * m * 2;
      for (int f = tid; f < nfrag; f += 64 * DW) {
        const int g = f / (2 * m), t = (f / 2) % m, h = f & 1;
        const u32x4 raw = *reinterpret_cast<const u32x4 *>(xc + ((int64_t)g * 64 + 32 * h + t) * 16);
        uint8_t *dst = XA + (g * MX + t) * XB;
        if constexpr (MD::XFP8) {
          const v8i o = unpack32(raw);
          *reinterpret_cast<u32x4 *>(dst + 32 * h) = u32x4{(uint32_t)o[0], (uint32_t)o[1], (uint32_t)o[2], (uint32_t)o[3]};
          *reinterpret_cast<u32x4 *>(dst + 32 * h + 16) = u32x4{(uint32_t)o[4], (uint32_t)o[5], (uint32_t)o[6], (uint32_t)o[7]};
        } else {
          *reinterpret_cast<u32x4 *>(dst + 16 * h) = raw;
        }
      }
      for (int idx = tid; idx < KGP * MX; idx += 64 * DW) {
        const int g = idx / MX, t = idx % MX;
        XS[idx] = g < KG && t < m ? half_bits_to_float(a.xs[(int64_t)(g / gk) * a.ms + t]) : 0.0f;
      }
    }
    // zero codes for the token slots past m, the odd tail group and the pad
    // that lanes outside the operand's live rows read
    for (int idx = tid; idx < KGP * MX * XB / 16 + 2; idx += 64 * DW) {
      const int e = idx * 16;
      const int g = e / (MX * XB), t = (e / XB) % MX;
      if (idx >= KGP * MX * XB / 16 || g >= KG || t >= m)
        *reinterpret_cast<u32x4 *>(XA + e) = u32x4{0u, 0u, 0u, 0u};
    }
    __syncthreads();
  };

  // activation operand of pair p: lanes outside the operand's live rows
  // (TOK8: group A lives in rows 0-7 of quarters 0-1, group B in rows 8-15
  // of quarters 2-3) or past the MX token slots read the zero pad after the
  // codes; the others read their (group 2p + gq, token, half) slot, zero
  // past m and past the last K-group
  const int arow = lane & 15;
  const int atok = MD::TOK8 ? (arow & 7) : arow;
  const bool alive = (MD::TOK8 ? ((arow < 8) == (q < 2)) : true) && atok < MX;
  const int xpad = KGP * MX * XB;
  const int abase = alive ? (gq * MX + atok) * XB + qh * (XB / 2) : xpad;
  const int astride = alive ? 2 * MX * XB : 0;
  auto act_op = [&](int p) -> v8i {
    const uint8_t *src = XA + abase + p * astride;
    if constexpr (MD::XFP8) return lds_v8i(src);
    else return unpack32(*reinterpret_cast<const u32x4 *>(src));
  };
  // token of accumulator row v of this lane, clamped into the LDS slots
  auto tok_of = [&](int v) {
    const int t = MD::TOK8 ? 4 * qh + v : 4 * q + v;
    return t < MX ? t : 0;
  };
  const v8i z8 = {0, 0, 0, 0, 0, 0, 0, 0};

  float hacc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  v4f acc[CTW];
#pragma unroll
  for (int j = 0; j < CTW; j++) acc[j] = v4f{0, 0, 0, 0};

  // the activation scales of this lane's accumulator rows for group g (the
  // rows are consecutive tokens, so one LDS read)
  auto xs_row = [&](int g) -> v4f {
    const float *p = XS + g * MX + tok_of(0);
    if constexpr (MV == 1) return v4f{p[0], 0.0f, 0.0f, 0.0f};
    else if constexpr (MV == 2) { const float2 t = *reinterpret_cast<const float2 *>(p); return v4f{t.x, t.y, 0.0f, 0.0f}; }
    else return *reinterpret_cast<const v4f *>(p);
  };

  // Stage 1, software-pipelined three deep so that no step waits on the one
  // before it: the LDS operands of pair i + 2 are read, the matrix product of
  // pair i + 1 is issued, and the chain step of pair i runs, in that order.
  // The chain is the ascending-group fma of rank tile `wave` (gb == KG on an
  // odd tail: zero codes and scales, so that step adds exactly nothing).
  struct S1Lds {
    v8i av;          // activation operand
    v4f sxa, sxb;    // activation scales of the lane's rows, groups A and B
  };
  struct S1Prod {
    v4f I;           // integer sums (TOK8: group A in lanes 0-31, B in 32-63)
    v4f I2;          // 16-token layout: group B's sums
    v4f sxa, sxb;
    uint32_t sla, slb;   // one token: the L1 scales of groups A and B for lanes 0-31
  };
  auto s1_lds = [&](int p) -> S1Lds {
    S1Lds r;
    r.av = act_op(p);
    r.sxa = xs_row(2 * p);
    r.sxb = xs_row(2 * p + 1);
    return r;
  };
  auto s1_mfma = [&](const S1Lds &A, const S1Slot &Sl) -> S1Prod {
    S1Prod r;
    const v8i b = unpack32(Sl.l1);
    if constexpr (MD::TOK8) {
      r.I = mfma_codes_16x16x128(A.av, b);
      r.I2 = v4f{0, 0, 0, 0};
    } else {
      r.I = mfma_codes_16x16x128(q < 2 ? A.av : z8, b);
      r.I2 = mfma_codes_16x16x128(q < 2 ? z8 : A.av, b);
    }
    r.sxa = A.sxa;
    r.sxb = A.sxb;
    // group B's scale comes from lanes 32-63, as its sums do (with 128-wide
    // groups both halves read the same row and only sla is used)
    r.sla = Sl.sla;
    r.slb = MD::MS && GK != 2 ? __builtin_bit_cast(uint32_t, upper_half(__builtin_bit_cast(float, Sl.sla))) : 0u;
    return r;
  };
  // One chain step per group: h = fma(I s_x, s_L1, h).  I s_x is exact in
  // fp32 (|I| < 2^12 times an 11-bit fp16 significand), so this rounds the
  // same exact value I s_x s_L1 + h once, as fma(I, s_x s_L1, h) does; the
  // fp16 scale enters the fma without a separate conversion.
  auto s1_chain = [&](const S1Prod &P, const S1Slot &Sl) {
    const _Float16 sla = __builtin_bit_cast(_Float16, (uint16_t)(MD::MS ? P.sla : Sl.sla));
    const _Float16 slb = __builtin_bit_cast(_Float16, (uint16_t)(MD::MS ? P.slb : Sl.slb));
#pragma unroll
    for (int v = 0; v < MV; v++) {
      const float ib = MD::TOK8 ? upper_half(P.I[v]) : P.I2[v];
      if constexpr (GK == 2) {
        // a 128-wide group: its two halves' sums add exactly (|I| < 2^13)
        // into the group's one step
        hacc[v] = fmaf((P.I[v] + ib) * P.sxa[v], (float)sla, hacc[v]);
      } else if constexpr (GK == 1) {
        hacc[v] = fmaf(P.I[v] * P.sxa[v], (float)sla, hacc[v]);
        hacc[v] = fmaf(ib * P.sxb[v], (float)slb, hacc[v]);
      } else {
        // the same, chosen at run time: for a 128-wide group the second step
        // adds +0, which leaves the (never negative-zero) h as is
        const float i1 = gk == 2 ? P.I[v] + ib : P.I[v];
        const float i2 = gk == 2 ? 0.0f : ib;
        hacc[v] = fmaf(i1 * P.sxa[v], (float)sla, hacc[v]);
        hacc[v] = fmaf(i2 * P.sxb[v], (float)slb, hacc[v]);
      }
    }
  };
  auto residual = [&](const ResSlot<CTW> &Sl, int p) {
    const int ga = 2 * p, gb = 2 * p + 1;
    const v8i av = act_op(p);
    const v4f sxa = xs_row(ga), sxb = xs_row(gb);
#pragma unroll
    for (int j = 0; j < CTW; j++) {
      const v8i b = unpack32(Sl.w[j]);
      if constexpr (MD::TOK8) {
        const v4f I = mfma_codes_16x16x128(av, b);
        const _Float16 sw = __builtin_bit_cast(_Float16, (uint16_t)Sl.swa[j]);
        const v4f sx = q < 2 ? sxa : sxb;   // the lane's own group
#pragma unroll
        for (int v = 0; v < MV; v++) acc[j][v] = fmaf(I[v] * sx[v], (float)sw, acc[j][v]);
      } else {
        const v4f I1 = mfma_codes_16x16x128(q < 2 ? av : z8, b);
        const v4f I2 = mfma_codes_16x16x128(q < 2 ? z8 : av, b);
        const _Float16 swa = __builtin_bit_cast(_Float16, (uint16_t)Sl.swa[j]);
        const _Float16 swb = __builtin_bit_cast(_Float16, (uint16_t)Sl.swb[j]);
#pragma unroll
        for (int v = 0; v < 4; v++) {
          acc[j][v] = fmaf(I1[v] * sxa[v], (float)swa, acc[j][v]);
          acc[j][v] = fmaf(I2[v] * sxb[v], (float)swb, acc[j][v]);
        }
      }
    }
  };

  // The two roles keep their rings in separate scopes, so their registers
  // overlap.  Each issues its first loads, then joins the prologue's barrier.
  if (s1) {
    S1Slot S1[D1];
#pragma unroll
    for (int s = 0; s < D1; s++) load_s1(S1[s], min(s, NP - 1));
    prologue();
    // slot s holds pair i0 + s; it is refilled after pair i's chain step
    S1Lds lds2 = s1_lds(min(1, NP - 1));
    S1Prod prod = s1_mfma(s1_lds(0), S1[0]);
    auto s1_step = [&](int i, int s) {
      const S1Lds lds_next = s1_lds(min(i + 2, NP - 1));
      const S1Prod prod_next = s1_mfma(lds2, S1[(s + 1) % D1]);
      s1_chain(prod, S1[s]);
      prod = prod_next;
      lds2 = lds_next;
    };
    int i0 = 0;
    if constexpr (MV <= 2) {
      // whole rounds of the ring with no per-pair test, so that the
      // pipeline's registers rotate by renaming inside a round (a per-pair
      // test splits the round into blocks joined by register copies), then
      // the last NP % D1 pairs.  (With four rows per lane the longer-lived
      // operands do not fit 128 registers that way: those layouts keep the
      // tested loop.)
      for (; i0 + D1 <= NP; i0 += D1) {
#pragma unroll
        for (int s = 0; s < D1; s++) {
          s1_step(i0 + s, s);
          load_s1(S1[s], min(i0 + s + D1, NP - 1));
        }
      }
    }
    for (; i0 < NP; i0 += D1) {
#pragma unroll
      for (int s = 0; s < D1; s++) {
        if (i0 + s < NP) s1_step(i0 + s, s);
        load_s1(S1[s], min(i0 + s + D1, NP - 1));
      }
    }
  } else {
    ResSlot<CTW> SR[D2];
    const int plast = nres_it > 0 ? ph + (nres_it - 1) * NPH : 0;
#pragma unroll
    for (int s = 0; s < D2; s++) load_res(SR[s], min(ph + s * NPH, plast));
    prologue();
    for (int i0 = 0; i0 < nres_it; i0 += D2) {
#pragma unroll
      for (int s = 0; s < D2; s++) {
        const int i = i0 + s;
        if (i < nres_it) residual(SR[s], ph + i * NPH);
        load_res(SR[s], min(ph + (i + D2) * NPH, plast));
      }
    }
  }
  __syncthreads();   // every wavefront is done with the activation codes

  // ---- epilogue: residual partials, H, re-quantization, stage 2, store ----
  float *RES = reinterpret_cast<float *>(smem + LY.epi_res);   // [NPH][CT][16 tokens][16 columns]
  float *HS = reinterpret_cast<float *>(smem + LY.epi_h);      // [16][HSTR]
  uint8_t *QS = smem + LY.epi_q;                                // [16][QSTR] fp8 codes
  float *SHS = reinterpret_cast<float *>(smem + LY.epi_sh);    // [2][16]
  constexpr int HSTR = DLayout::HSTR, QSTR = DLayout::QSTR;
  const bool store_lane = !MD::TOK8 || lane < 32;
  if (rbusy) {
#pragma unroll
    for (int j = 0; j < CTW; j++)
#pragma unroll
      for (int v = 0; v < MV; v++) {
        float val = acc[j][v];
        if constexpr (MD::TOK8) val += upper_half(val);   // group A + group B partials
        const int t = MD::TOK8 ? 4 * qh + v : 4 * q + v;
        if (store_lane) RES[((ph * CT + tg * CTW + j) * 16 + t) * 16 + c16] = val;
      }
  }
  if (s1) {
#pragma unroll
    for (int v = 0; v < MV; v++) {
      const int t = MD::TOK8 ? 4 * qh + v : 4 * q + v;
      if (store_lane) HS[t * HSTR + 16 * wave + c16] = hacc[v];
    }
  }
  const int RB = (r + 63) / 64;   // 64-rank blocks of stage 2 (<= 2)
  if (r > 0) {
    for (int idx = tid; idx < 16 * RB * 64; idx += 64 * DW) {
      const int row = idx / (RB * 64), j = idx % (RB * 64);
      if (j >= r) QS[row * QSTR + j] = 0;
    }
  }
  __syncthreads();

  if (r > 0) {
    // Re-quantize H per token and rank group (s_H stays fp32).  Half a
    // wavefront per token row (wavefront w < 8: rows 2w, 2w + 1); lane j of
    // the half takes ranks epl j .. epl j + epl - 1, so a rank group is a run
    // of gr / epl lanes and its max is a shuffle reduction over them.
    if (wave < 8) {
      const int gr = geo.gr, rg = r / gr;
      const int epl = r >= 32 ? r / 32 : 1;      // ranks per lane: 1, 2 or 4
      const int row = 2 * wave + (lane >> 5), j = lane & 31;
      const int lpg = gr / epl;                  // lanes per rank group (<= 32)
      const int hg = j / lpg;
      const bool valid = j * epl < r;
      const bool live = valid && row < m;
      const bool dbg = a.dbg_h != nullptr && blockIdx.x == 0;
      float hv[4];
      float amax = 0.0f;
#pragma unroll
      for (int e = 0; e < 4; e++) {
        hv[e] = live && e < epl ? HS[row * HSTR + j * epl + e] : 0.0f;
        amax = fmaxf(amax, fabsf(hv[e]));
      }
      amax = run_max(amax, lpg, lane);
      const float sh = amax / 7.0f;   // IEEE division
      if (valid) {
        uint32_t w = 0;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          if (e < epl) {
            int qv = 0;
            if (sh != 0.0f) {
              float tq = __builtin_rintf(hv[e] / sh);
              tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
              qv = (int)tq;
            }
            w |= code_to_fp8(qv) << (8 * e);
            if (dbg && row < m) {
              a.dbg_h[(int64_t)row * r + j * epl + e] = hv[e];
              a.dbg_qh[(int64_t)row * r + j * epl + e] = (int8_t)qv;
            }
          }
        }
        uint8_t *qd = QS + row * QSTR + j * epl;
        if (epl == 4) *reinterpret_cast<uint32_t *>(qd) = w;
        else if (epl == 2) *reinterpret_cast<uint16_t *>(qd) = (uint16_t)w;
        else *qd = (uint8_t)w;
        if (j % lpg == 0) {
          SHS[hg * 16 + row] = sh;
          if (dbg && row < m) a.dbg_sh[(int64_t)row * rg + hg] = sh;
        }
      }
    }
    __syncthreads();
  }

  // ---- stage 2 and the single epilogue: wavefront j < CT stores tile j ----
  if (wave < CT) {
    const int j = wave;
    const int ct = c0 + j;
    if (ct < ct16) {
      v4f ylr = v4f{0, 0, 0, 0};
      const int orow0 = 4 * q;   // output rows 4q .. 4q + 3 of this lane
      if (r > 0) {
        const int rbq = min(q >> 1, RB - 1);
        const int L = qh * 32 + (ct & 1) * 16 + c16;
        const u32x4 l2raw = *reinterpret_cast<const u32x4 *>(
            l2codes + (((int64_t)(ct >> 1) * (geo.r_pad64 / 64) + rbq) * 64 + L) * 16);
        const int col = ct * 16 + c16;
        const float s2a = half_bits_to_float(l2scales[col]);
        const int hg1 = 64 / geo.gr;   // rank group of the second 64-rank block (0 if gr = 128)
        const float s2b = RB > 1 ? half_bits_to_float(l2scales[(int64_t)hg1 * geo.n_pad + col]) : 0.0f;
        const v8i qa = lds_v8i(QS + c16 * QSTR + rbq * 64 + qh * 32);
        const v8i lb = unpack32(l2raw);
        {
          const v4f cb = mfma_codes_16x16x128(q < 2 ? qa : z8, lb);
#pragma unroll
          for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[orow0 + v] * s2a, ylr[v]);
        }
        if (RB > 1) {
          const v4f cb = mfma_codes_16x16x128(q < 2 ? z8 : qa, lb);
#pragma unroll
          for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[16 * hg1 + orow0 + v] * s2b, ylr[v]);
        }
      }
      // the matrix-core products above read operands from every lane: keep
      // them out of the per-lane store branch below
      asm volatile("" : "+v"(ylr));
      const int col = ct * 16 + c16;
      if (col < geo.n) {
#pragma unroll
        for (int v = 0; v < 4; v++) {
          const int row = orow0 + v;
          if (row < m) {
            float yres = 0.0f;
            for (int w2 = 0; w2 < NPH; w2++) yres += RES[((w2 * CT + j) * 16 + row) * 16 + c16];
            const float yv = yres + ylr[v];
            const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
            reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
          }
        }
      }
    }
  }
}

template <int MODE, int CT, bool FQ>
hipError_t launch_decode(const GemmArgs &a, const uint16_t *xh, hipStream_t s) {
  const DLayout LY = decode_layout<MODE, CT>(a.geo.k / kGroup, a.geo.r);
  const int tiles16 = a.geo.n_pad / 16;
  if (a.geo.gk != 1 && a.geo.gk != 2) return hipErrorInvalidValue;
  // the group width is a compile-time constant where the registers allow it
  // (64-wide groups up to two rows per lane, 128-wide groups at one row): the
  // chain then takes one or two steps per pair without a per-pair choice
  constexpr int MV = DMode<MODE>::MV;
  auto kern = a.geo.gk == 1 ? dual_gemm_decode_kernel<MODE, CT, FQ, MV <= 2 ? 1 : 0>
                            : dual_gemm_decode_kernel<MODE, CT, FQ, MV == 1 ? 2 : 0>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, LY.total);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((tiles16 + CT - 1) / CT), dim3(64 * DW), LY.total, s, a, xh);
  return hipGetLastError();
}

template <int MODE, bool FQ>
hipError_t launch_decode_mode(const GemmArgs &a, const uint16_t *xh, hipStream_t s) {
  // the fewest 16-column tiles per work-group that keep the grid within one
  // work-group per CU
  const int tiles16 = a.geo.n_pad / 16;
  if (tiles16 <= 256) return launch_decode<MODE, 1, FQ>(a, xh, s);
  if (tiles16 <= 512) return launch_decode<MODE, 2, FQ>(a, xh, s);
  if (tiles16 <= 1024) return launch_decode<MODE, 4, FQ>(a, xh, s);
  return launch_decode<MODE, 8, FQ>(a, xh, s);
}

int decode_mode(int m) { return m == 1 ? 1 : (m == 2 ? 2 : (m <= 8 ? 4 : 16)); }

}  // namespace

bool decode_fits(int m, int k) {
  if (m < 1 || m > kDecodeMaxTokens) return false;
  const int mode = decode_mode(m);
  const int mx = mode == 16 ? 16 : (mode <= 2 ? mode : 8);
  const int xb = mode <= 2 ? 64 : 32;
  const int64_t kgp = (int64_t)(k / kGroup + 1) / 2 * 2;
  return kgp * mx * xb <= kDecodeXBytes;
}

hipError_t launch_dual_gemm_decode(const GemmArgs &a, const uint16_t *xh, hipStream_t s) {
  const bool fq = xh != nullptr;
  switch (decode_mode(a.m)) {
    case 1: return fq ? launch_decode_mode<1, true>(a, xh, s) : launch_decode_mode<1, false>(a, xh, s);
    case 2: return fq ? launch_decode_mode<2, true>(a, xh, s) : launch_decode_mode<2, false>(a, xh, s);
    case 4: return fq ? launch_decode_mode<4, true>(a, xh, s) : launch_decode_mode<4, false>(a, xh, s);
    default: return fq ? launch_decode_mode<16, true>(a, xh, s) : launch_decode_mode<16, false>(a, xh, s);
  }
}

}  // namespace tq
