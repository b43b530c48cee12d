// Fused dual-component W4A4 layer (paper Sec. 4.3) for decode-sized token
// counts (m <= 16): the residual 4-bit GEMM, the stage-1 product
// H = Q(X) Q(L1), its re-quantization, stage 2 Q_H Q(L2) and one epilogue,
// in one kernel.  At these sizes the layer is bound by the bytes of the
// packed weights and by the latency of H's K-long chain (one fp32 fma per
// K-group, in ascending group order, so that Q_H is bit-exact).
//
// Work decomposition.  Forming H in every work-group would read all of L1
// (K x r codes) once per work-group and put the K-long chain in front of
// every tile, so H is formed once per call:
//  * Work-groups 0 .. ceil(r / 16) - 1 are H producers, one per 16-rank tile
//    of H.  Work-groups are dispatched in index order, so the producers are
//    running before any work-group that waits for them; they wait for nothing
//    themselves.  (The wait is bounded all the same: a work-group that gives
//    up sets an error word in the workspace instead of hanging.)
//  * Each producer writes its fp32 H tile to the caller's workspace and then
//    counts itself on a ready counter kept on up to 32 cache lines; column
//    work-group c polls line c mod 32 (so that few work-groups poll any one
//    line).
//  * Every other work-group owns CT 16-column tiles of Y.  It forms its
//    residual tiles, waits until every producer has counted, reads H,
//    re-quantizes it in LDS (per token and rank group, s_H in fp32; every
//    column work-group computes the same Q_H from the same H), runs stage 2
//    with its L2 columns and stores Y once.
//  * Flags and H are written with device-scope stores, which complete at the
//    device's point of coherence; a writer waits for its stores to complete
//    before it counts itself (no cache write-back, which would touch every
//    other work-group's lines).  Flags are polled with device-scope loads.  H
//    is read with ordinary loads: its lines are first touched in this launch
//    after the count is complete and every launch starts with invalidated
//    caches, so the column work-groups on one XCD share a fresh copy in L2.
//  * Column work-groups also count themselves on their line once they have
//    read H; the last one on a line clears the line's two counts, so every
//    call leaves the workspace as it found it (zero).
//
// Products.  16 x 16 x 128 fp8 MFMAs over a K-group pair (codes as fp8
// subnormals, block scales 2^9: exact integer sums); a group's own sum uses
// the other group's half of the activation operand as zeros.  The exact scale
// products s_x s_w (and s_x s_L1) come from a 16 x 16 x 16 f16 product with
// the scales in k = 0.  Wavefront w of a work-group takes the group pairs
// w, w + 8, w + 16, ... and fetches their operands from global memory straight
// into registers, four pairs ahead: there is no LDS staging and no barrier in
// the residual loop.  A producer stages the integer products of up to 64
// groups and their fp32 scales in LDS; four wavefronts (one for each of a
// lane's four outputs) then run the ascending-group fma chain over them,
// forming each scale product s_x s_L1 exactly in fp32 as they go.
#include <stdlib.h>

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int SW = 8;      // wavefronts per work-group
constexpr int SPD = 4;     // group pairs in flight per wavefront
constexpr int SCG = 64;    // K-groups per producer chunk

// Workspace layout (bytes; every counter on its own 128-byte line):
constexpr int WS_LINE = 128;
constexpr int WS_NL = 32;                              // flag / count copies
constexpr int WS_ERR = 0;                              // set when a wait gave up
constexpr int WS_READY = WS_LINE;   // line x: producers finished (word 0), column work-groups done (word 1)
constexpr int WS_H = WS_READY + WS_NL * WS_LINE;       // [16][kMaxRank] fp32 H
constexpr int WS_END = WS_H + 16 * kMaxRank * 4;
static_assert(WS_END <= (int)kWorkspaceBytes, "the workspace holds the layout");
constexpr int kSpinLimit = 1 << 20;   // polls (~1 s at most) before giving up

__device__ __forceinline__ uint32_t *ws_word(uint32_t *ws, int byte) {
  return reinterpret_cast<uint32_t *>(reinterpret_cast<uint8_t *>(ws) + byte);
}
__device__ __forceinline__ uint32_t ld_dev(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t add_dev(uint32_t *p) {
  return __hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void add_dev_nr(uint32_t *p) {   // result unused: no return trip
  (void)__hip_atomic_fetch_add(p, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// max over runs of n = 8, 16 or 32 lanes (aligned), in every lane of the run:
// quad permutes and row mirrors (DPP) within a row of 16, the two rows of a
// 32-lane half from scalar reads
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
__device__ __forceinline__ v8i lds_v8i(const uint8_t *p) {
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(p);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(p + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}
// Release for device-scope stores: every store the other work-groups read is a
// device-scope store, which completes at the device's point of coherence, so
// waiting for this wavefront's stores to complete orders them before a later
// flag.  (A release fence would also write back the whole L2, ~1 us.)
__device__ __forceinline__ void wait_dev_stores() {
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
}

template <int CT>
struct SCfg {
  // producer: integer products [4 outputs][SCG / 4][64 lanes][4 groups] fp32,
  // then scales [16 tokens][SSTR] and [16 ranks][SSTR] fp32 (groups
  // contiguous, so that the chain reads 4 groups per 16-byte load)
  static constexpr int SSTR = SCG + 4;
  static constexpr int P_C = 0;
  static constexpr int P_SX = SCG * 1024;
  static constexpr int P_SL = P_SX + 16 * SSTR * 4;
  static constexpr int P_END = P_SL + 16 * SSTR * 4;
  // column work-group (aliases the producer region)
  static constexpr int RES = SW * CT * 1024;                   // [SW][CT][4][64] fp32
  static constexpr int HSTR = kMaxRank + 1;
  static constexpr int E_HS = RES;                             // [16][HSTR] fp32
  static constexpr int QSTR = kMaxRank + 16;
  static constexpr int E_QS = E_HS + 16 * HSTR * 4;            // [16][QSTR] fp8 codes
  static constexpr int E_SH = E_QS + 16 * QSTR;                // [2][16] fp32
  static constexpr int E_END = E_SH + 2 * 16 * 4;
  static constexpr int LDS = P_END > E_END ? P_END : E_END;
  static_assert(LDS <= 80 * 1024, "two work-groups fit in the 160 KiB LDS of a CU");
};

// exact products s_a[row] * s_b[col] of a 16 x 16 tile (lanes 0-15 carry the
// fp16 scales in k = 0, every other operand element is zero)
__device__ __forceinline__ v4f outer16(uint32_t sa, uint32_t sb) {
  const v4f z = {0, 0, 0, 0};
  const u32x2 a2 = {sa, 0u}, b2 = {sb, 0u};
  return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(v4h, a2),
                                               __builtin_bit_cast(v4h, b2), z, 0, 0, 0);
}

// Operands of one group pair: raw activation codes (token c16, half q % 2 of
// group 2p + q / 2), NB raw weight (or L1) fragments of 16 columns, and the
// fp16 scales of both groups on lanes 0-15.
template <int NB>
struct PairOps {
  u32x4 x;
  u32x4 b[NB];
  uint32_t sx1, sx2;
  uint32_t sb1[NB], sb2[NB];
};

template <int CT>
__global__ __launch_bounds__(64 * SW, 4) void dual_gemm_decode_kernel(GemmArgs a, int nprod) {
  using C = SCfg<CT>;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, c16 = lane & 15;
  const int KG = geo.k / kGroup, NP = (KG + 1) / 2;
  const int m = a.m, ms = a.ms;
  const int ct16 = geo.n_pad / 16;
  const int r = geo.r;
  const int RB = (r + 63) / 64;   // 64-rank blocks of stage 2 (<= 2)
  uint32_t *ws = a.ws;
  uint8_t *wsb = reinterpret_cast<uint8_t *>(ws);
  const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
  const uint16_t *xs = a.xs;
  const uint8_t *wcodes = a.packed + geo.off_w;
  const uint16_t *wscales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_ws);
  const uint8_t *l1codes = a.packed + geo.off_l1;
  const uint16_t *l1scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l1s);
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const int wg = blockIdx.x;
  const bool producer = wg < nprod;

  // fetch the operands of pair p (p < NP) into o: activation fragment and NB
  // fragments of the 16-column blocks col16 + j of `blocks`, with their scales
  // (scale of column c, group g at scales[g * sstride + c])
  auto fetch = [&](auto &o, int p, const uint8_t *blocks, const uint16_t *scales, int sstride,
                   int col16, int ncol16) {
    constexpr int NB = sizeof(o.b) / sizeof(o.b[0]);
    const int g1 = 2 * p, g2 = min(2 * p + 1, KG - 1);
    const int gq = (q >> 1) ? g2 : g1;
    o.x = u32x4{0u, 0u, 0u, 0u};
    if (c16 < m) o.x = *reinterpret_cast<const u32x4 *>(xc + ((int64_t)gq * 64 + 32 * (q & 1) + c16) * 16);
    o.sx1 = 0u;
    o.sx2 = 0u;
    if (lane < 16) {
      o.sx1 = xs[(int64_t)g1 * ms + c16];
      o.sx2 = xs[(int64_t)g2 * ms + c16];
    }
#pragma unroll
    for (int j = 0; j < NB; j++) {
      const int cj = min(col16 + j, ncol16 - 1);
      const int L = (q & 1) * 32 + (cj & 1) * 16 + c16;
      o.b[j] = *reinterpret_cast<const u32x4 *>(blocks + (((int64_t)(cj >> 1) * KG + gq) * 64 + L) * 16);
      o.sb1[j] = 0u;
      o.sb2[j] = 0u;
      if (lane < 16) {
        o.sb1[j] = scales[(int64_t)g1 * sstride + cj * 16 + c16];
        o.sb2[j] = scales[(int64_t)g2 * sstride + cj * 16 + c16];
      }
    }
  };
  // products of pair p: f(j, g, codes, scale products) for both groups
  auto products = [&](const auto &o, int p, auto f) {
    constexpr int NB = sizeof(o.b) / sizeof(o.b[0]);
    const v8i av = unpack32(o.x);
    const v8i z = {0, 0, 0, 0, 0, 0, 0, 0};
    const v8i a1 = q < 2 ? av : z;
    const v8i a2 = q < 2 ? z : av;
#pragma unroll
    for (int j = 0; j < NB; j++) {
      const v8i b = unpack32(o.b[j]);
      const v4f m1 = mfma_codes_16x16x128(a1, b);
      const v4f o1 = outer16(o.sx1, o.sb1[j]);
      const v4f m2 = mfma_codes_16x16x128(a2, b);
      const v4f o2 = outer16(o.sx2, o.sb2[j]);
      f(j, 2 * p, m1, o1);
      if (2 * p + 1 < KG) f(j, 2 * p + 1, m2, o2);
    }
  };

  if (producer) {
    // ================= H producer: 16-rank tile `wg` =================
    const int p16 = wg;
    float *CV = reinterpret_cast<float *>(smem + C::P_C);
    float *SXL = reinterpret_cast<float *>(smem + C::P_SX);
    float *SLL = reinterpret_cast<float *>(smem + C::P_SL);
    const int nchunk = (KG + SCG - 1) / SCG;
    constexpr int PPC = SCG / 2 / SW;   // pairs per wavefront and chunk (= SPD)
    static_assert(PPC == SPD, "one chunk of pairs in flight");
    PairOps<1> F[SPD];
    // wavefront pair sequence i -> pair SW i + wave; chunk c holds i in [SPD c, SPD c + SPD)
    const int npw = SPD * nchunk;
#pragma unroll
    for (int s = 0; s < SPD; s++)
      if (SW * s + wave < NP) fetch(F[s], SW * s + wave, l1codes, l1scales, geo.r_pad32, p16, geo.r_pad32 / 16);
    float hacc = 0.0f;
    for (int c = 0; c < nchunk; c++) {
#pragma unroll
      for (int s = 0; s < SPD; s++) {
        const int i = SPD * c + s;
        const int p = SW * i + wave;
        if (p < NP) {
          const PairOps<1> &o = F[s];
          const v8i av = unpack32(o.x);
          const v8i z = {0, 0, 0, 0, 0, 0, 0, 0};
          const v8i b = unpack32(o.b[0]);
          const v4f m1 = mfma_codes_16x16x128(q < 2 ? av : z, b);
          const v4f m2 = mfma_codes_16x16x128(q < 2 ? z : av, b);
          const int gl1 = 2 * p - SCG * c, gl2 = gl1 + 1;
          auto cidx = [&](int v, int gl) { return ((v * (SCG / 4) + gl / 4) * 64 + lane) * 4 + gl % 4; };
#pragma unroll
          for (int v = 0; v < 4; v++) CV[cidx(v, gl1)] = m1[v];
          if (2 * p + 1 < KG) {
#pragma unroll
            for (int v = 0; v < 4; v++) CV[cidx(v, gl2)] = m2[v];
          }
          if (lane < 16) {
            SXL[c16 * C::SSTR + gl1] = half_bits_to_float((uint16_t)o.sx1);
            SXL[c16 * C::SSTR + gl2] = half_bits_to_float((uint16_t)o.sx2);
            SLL[c16 * C::SSTR + gl1] = half_bits_to_float((uint16_t)o.sb1[0]);
            SLL[c16 * C::SSTR + gl2] = half_bits_to_float((uint16_t)o.sb2[0]);
          }
        }
        const int pn = SW * (i + SPD) + wave;
        if (i + SPD < npw && pn < NP)
          fetch(F[s], pn, l1codes, l1scales, geo.r_pad32, p16, geo.r_pad32 / 16);
      }
      __syncthreads();   // the chunk's products and scales are in LDS
      if (wave < 4) {
        // output v = wave of every lane (token 4q + v, rank 16 p16 + c16),
        // groups in ascending order, in batches of 8 whose reads (six
        // 16-byte loads) go before their fmas
        const int row = 4 * q + wave;
        const int ng = min(SCG, KG - SCG * c);
        const float4 *CV4 = reinterpret_cast<const float4 *>(CV) + (wave * (SCG / 4)) * 64 + lane;
        const float4 *SX4 = reinterpret_cast<const float4 *>(SXL + row * C::SSTR);
        const float4 *SL4 = reinterpret_cast<const float4 *>(SLL + c16 * C::SSTR);
        int g0 = 0;
        for (; g0 + 8 <= ng; g0 += 8) {
          float4 cv[2], sv[2], lv[2];
#pragma unroll
          for (int e = 0; e < 2; e++) {
            cv[e] = CV4[(g0 / 4 + e) * 64];
            sv[e] = SX4[g0 / 4 + e];
            lv[e] = SL4[g0 / 4 + e];
          }
#pragma unroll
          for (int e = 0; e < 8; e++)   // s_x s_L1 is exact in fp32
            hacc = fmaf(cv[e / 4][e % 4], sv[e / 4][e % 4] * lv[e / 4][e % 4], hacc);
        }
        for (; g0 < ng; g0++) {
          const int gl = g0;
          hacc = fmaf(CV[((wave * (SCG / 4) + gl / 4) * 64 + lane) * 4 + gl % 4],
                      SXL[row * C::SSTR + gl] * SLL[c16 * C::SSTR + gl], hacc);
        }
      }
      __syncthreads();   // the chunk's products are consumed
    }
    // this tile of H -> workspace; each wavefront waits for its stores, the
    // barrier orders them before the count
    float *wsH = reinterpret_cast<float *>(wsb + WS_H);
    if (wave < 4)
      __hip_atomic_store(wsH + (4 * q + wave) * kMaxRank + 16 * p16 + c16, hacc, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    wait_dev_stores();
    __syncthreads();
    const int ncol = (int)gridDim.x - nprod;
    if (tid < WS_NL && tid < ncol) add_dev_nr(ws_word(ws, WS_READY + tid * WS_LINE));
  } else {
    // ================= column work-group =================
    const int c0 = (wg - nprod) * CT;   // first 16-column tile
    // stage-2 operands (wavefront j < CT, tile c0 + j), fetched before the
    // residual loop: rank blocks in pairs, lanes q < 2 carry block 0, lanes
    // q >= 2 block 1
    u32x4 l2raw = u32x4{0u, 0u, 0u, 0u};
    float s2a = 0.0f, s2b = 0.0f;
    if (nprod > 0 && wave < CT && c0 + wave < ct16) {
      const int ct = c0 + wave;
      const int rbq = min(q >> 1, RB - 1);
      const int L = (q & 1) * 32 + (ct & 1) * 16 + c16;
      l2raw = *reinterpret_cast<const u32x4 *>(
          l2codes + (((int64_t)(ct >> 1) * (geo.r_pad64 / 64) + rbq) * 64 + L) * 16);
      const int col = ct * 16 + c16;
      s2a = half_bits_to_float(l2scales[col]);
      if (RB > 1) s2b = half_bits_to_float(l2scales[(int64_t)geo.n_pad + col]);
    }
    v4f acc[CT];
#pragma unroll
    for (int j = 0; j < CT; j++) acc[j] = v4f{0, 0, 0, 0};
    {
      constexpr int PD = CT == 1 ? SPD : SPD / 2;   // pairs in flight (registers)
      PairOps<CT> F[PD];
      const int npw = (NP + SW - 1) / SW;
#pragma unroll
      for (int s = 0; s < PD; s++)
        if (s < npw && SW * s + wave < NP) fetch(F[s], SW * s + wave, wcodes, wscales, geo.n_pad, c0, ct16);
      for (int i0 = 0; i0 < npw; i0 += PD) {
#pragma unroll
        for (int s = 0; s < PD; s++) {
          const int i = i0 + s;
          const int p = SW * i + wave;
          if (i < npw && p < NP)
            products(F[s], p, [&](int j, int, const v4f &cv, const v4f &pv) {
#pragma unroll
              for (int v = 0; v < 4; v++) acc[j][v] = fmaf(cv[v], pv[v], acc[j][v]);
            });
          const int pn = SW * (i + PD) + wave;
          if (i + PD < npw && pn < NP) fetch(F[s], pn, wcodes, wscales, geo.n_pad, c0, ct16);
        }
      }
    }
    float *RES = reinterpret_cast<float *>(smem);
#pragma unroll
    for (int j = 0; j < CT; j++)
#pragma unroll
      for (int v = 0; v < 4; v++) RES[((wave * CT + j) * 4 + v) * 64 + lane] = acc[j][v];
    __syncthreads();

    float *HS = reinterpret_cast<float *>(smem + C::E_HS);
    uint8_t *QS = smem + C::E_QS;
    float *SHS = reinterpret_cast<float *>(smem + C::E_SH);
    if (nprod > 0) {
      // ---- wait for every producer's H tile ----
      if (wave == 0) {
        const uint32_t *cnt = ws_word(ws, WS_READY + ((wg - nprod) % WS_NL) * WS_LINE);
        int spins = 0;
        while (ld_dev(cnt) < (uint32_t)nprod) {
          __builtin_amdgcn_s_sleep(2);
          if (++spins > kSpinLimit) {
            st_dev(ws_word(ws, WS_ERR), 1u);
            break;
          }
        }
      }
      __syncthreads();
      // all of a thread's loads are issued before any is used
      const float *wsH = reinterpret_cast<const float *>(wsb + WS_H);
      const int rp = 16 * nprod;
      constexpr int HPT = 16 * kMaxRank / (64 * SW);   // H values per thread at most
      float hl[HPT];
#pragma unroll
      for (int e = 0; e < HPT; e++) {
        const int idx = tid + 64 * SW * e;
        const int row = idx / rp, j = idx % rp;
        hl[e] = idx < 16 * rp && row < m ? wsH[row * kMaxRank + j] : 0.0f;
      }
#pragma unroll
      for (int e = 0; e < HPT; e++) {
        const int idx = tid + 64 * SW * e;
        if (idx < 16 * rp) HS[(idx / rp) * C::HSTR + idx % rp] = hl[e];
      }
      for (int idx = tid; idx < 16 * RB * 64; idx += 64 * SW) {
        const int row = idx / (RB * 64), j = idx % (RB * 64);
        if (j >= r) QS[row * C::QSTR + j] = 0;
      }
      __syncthreads();

      // ---- re-quantize H per token and rank group (s_H stays fp32) ----
      // Half a wavefront per token row (wavefront w: rows 2w, 2w + 1); lane j
      // of the half takes ranks epl j .. epl j + epl - 1, so a rank group is a
      // run of gr / epl lanes and its max is a shuffle reduction over them.
      {
        const int gr = geo.gr, rg = r / gr;
        const int epl = r >= 32 ? r / 32 : 1;      // ranks per lane: 1, 2 or 4
        const int row = 2 * wave + (lane >> 5), j = lane & 31;
        const int lpg = gr / epl;                  // lanes per rank group (<= 32)
        const int hg = j / lpg;
        const bool valid = j * epl < r;
        const bool dbg = a.dbg_h != nullptr && wg == nprod;
        float hv[4];
        float amax = 0.0f;
#pragma unroll
        for (int e = 0; e < 4; e++) {
          hv[e] = valid && e < epl ? HS[row * C::HSTR + j * epl + e] : 0.0f;
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
          uint8_t *qd = QS + row * C::QSTR + j * epl;
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
        if (nprod > 0) {
          const int rbq = min(q >> 1, RB - 1);
          const v8i qa = lds_v8i(QS + c16 * C::QSTR + rbq * 64 + (q & 1) * 32);
          float sh0[4], sh1[4];
#pragma unroll
          for (int v = 0; v < 4; v++) {
            sh0[v] = SHS[orow0 + v];
            sh1[v] = RB > 1 ? SHS[16 + orow0 + v] : 0.0f;
          }
          const v8i lb = unpack32(l2raw);
          const v8i zero = {0, 0, 0, 0, 0, 0, 0, 0};
          const v8i qa1 = q < 2 ? qa : zero;
          const v8i qa2 = q < 2 ? zero : qa;
          {
            const v4f cb = mfma_codes_16x16x128(qa1, lb);
#pragma unroll
            for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], sh0[v] * s2a, ylr[v]);
          }
          if (RB > 1) {
            const v4f cb = mfma_codes_16x16x128(qa2, lb);
#pragma unroll
            for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], sh1[v] * s2b, ylr[v]);
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
              for (int w2 = 0; w2 < SW; w2++) yres += RES[((w2 * CT + j) * 4 + v) * 64 + lane];
              const float yv = yres + ylr[v];
              const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
              reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
            }
          }
        }
      }
    }
  }

  // ---- the last column work-group of a line clears the line ----
  if (nprod > 0 && !producer) {
    __syncthreads();   // every read of the line and of H is done
    if (tid == 0) {
      const int x = (wg - nprod) % WS_NL, ncol = (int)gridDim.x - nprod;
      const uint32_t per = (uint32_t)((ncol - x + WS_NL - 1) / WS_NL);   // column work-groups on line x
      if (add_dev(ws_word(ws, WS_READY + x * WS_LINE + 4)) == per - 1) {
        st_dev(ws_word(ws, WS_READY + x * WS_LINE), 0u);
        st_dev(ws_word(ws, WS_READY + x * WS_LINE + 4), 0u);
      }
    }
  }
}

template <int CT>
hipError_t launch_decode(const GemmArgs &a, hipStream_t s) {
  using C = SCfg<CT>;
  const int tiles16 = a.geo.n_pad / 16;
  const int ncol = (tiles16 + CT - 1) / CT;
  const int nprod = (a.geo.r + 15) / 16;
  auto kern = dual_gemm_decode_kernel<CT>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(nprod + ncol), dim3(64 * SW), C::LDS, s, a, nprod);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_dual_gemm_decode(const GemmArgs &a, hipStream_t s) {
  // two 16-column tiles per work-group once one tile per work-group would not
  // fit one round of resident work-groups (two per CU, 512 on the 256 CUs),
  // the H producers included: a second round for a few work-groups costs a
  // whole work-group's time (measured at N = 8192, r = 128, K = 28672: 68 us
  // with 520 work-groups, 47 us with 264)
  const int tiles16 = a.geo.n_pad / 16;
  const int nprod = (a.geo.r + 15) / 16;
  const int ct = tiles16 + nprod > 2 * 256 ? 2 : 1;
  return ct == 2 ? launch_decode<2>(a, s) : launch_decode<1>(a, s);
}

}  // namespace tq
