// Fused dual-component W4A4 layer (paper Sec. 4.3) for decode-sized token
// counts (m <= 16): the residual 4-bit GEMM, the stage-1 product
// H = Q(X) Q(L1) kept on chip, its on-the-fly re-quantization, stage 2
// Q_H Q(L2) and one epilogue, in one kernel.  The layer is bound by HBM
// bandwidth (the packed weights) and by the latency of H's K-long chain.
//
// Work decomposition.  A workgroup of 8 wavefronts owns CT output tiles of 16
// columns and all m <= 16 tokens.  Matrix-core products are 16 x 16 x 128
// fp8 (codes as fp8 subnormals, block scales 2^9: exact integer sums).  One
// instruction covers a K-group pair, so a group's own sum is taken with the
// other group's half of the activation operand read as zeros.  The exact
// scale products s_x s_w (and s_x s_L1) come from a 16 x 16 x 16 f16 product
// with the scales in k = 0.
//  * H wavefronts (one per 16-rank tile of H, r <= 64: wavefronts 0 .. r/16-1)
//    run the whole K loop for their tile in ascending group order, so H and
//    Q_H are bit-identical to the oracle's.
//  * residual wavefronts split the group pairs of every chunk of K among
//    themselves; their partial sums are added in a fixed order at the end
//    (only Y's fp32 summation order differs from the oracle's).  For r = 128
//    every wavefront does both.
//
// Data movement: direct global -> LDS loads with explicit wait counts only.
//  * K runs in chunks of 16 groups.  The chunk's raw activation codes and all
//    its scales arrive two chunks ahead in a 3-slot raw ring (loads spread
//    over the wavefronts); one chunk ahead the workgroup expands the codes to
//    fp8 operand bytes (2-slot buffer).  One workgroup barrier per chunk.
//  * Each wavefront streams its own weight (or L1) fragments -- one 1 KiB
//    wave load per group pair and tile -- through a private LDS ring one
//    chunk deep.
// Every wavefront issues the same loads in the same order every chunk, so
// each wait is one constant s_waitcnt.
#include <stdlib.h>

#include <type_traits>

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int DW = 8;       // wavefronts per workgroup
constexpr int DCG = 16;     // K-groups per chunk
constexpr int DCP = 8;      // group pairs per chunk
constexpr int DRAW = 3;     // raw chunk slots (two chunks in flight)

template <int RT16, int CT>
struct DCfg {
  static constexpr int NH = RT16;                         // H wavefronts (0, 2, 4 or 8)
  static constexpr bool SHARED = NH == DW;                // r = 128: every wavefront does both
  static constexpr int NR = SHARED ? DW : DW - NH;        // residual wavefronts
  static constexpr int RPAD = RT16 * 16;                  // ranks covered by the H tiles
  // raw chunk slot: codes of 16 groups (16 tokens x 2 halves x 16 B each),
  // then one 1 KiB region per scale item
  static constexpr int R_X = 0;                           // 8 KiB
  static constexpr int R_SX = 8192;                       // [16 groups][16 tokens] fp16
  static constexpr int R_SW = R_SX + 1024;                // [16 groups][16 CT cols] fp16
  static constexpr int NSL = RPAD > 0 ? (RPAD * 32 + 1023) / 1024 : 0;   // L1 scale regions
  static constexpr int R_SL = R_SW + 1024;                // [16 groups][RPAD ranks] fp16
  static constexpr int RSLOT = R_SL + NSL * 1024;
  // chunk items (1 KiB wave loads): 8 code pairs, activation scales, weight
  // scales, L1 scales; NCI per wavefront, padded with repeats
  static constexpr int NITEM = 8 + 1 + 1 + NSL;
  static constexpr int NCI = (NITEM + DW - 1) / DW;
  // expanded codes: [16 groups][2 halves][16 tokens] x 32 fp8 bytes
  static constexpr int XE = 16384;
  // per-wavefront fragment ring: H pairs (8) then residual pairs x CT
  static constexpr int OFF_RAW = 0;
  static constexpr int OFF_XE = OFF_RAW + DRAW * RSLOT;
  static constexpr int OFF_ZERO = OFF_XE + 2 * XE;        // 64 zero bytes
  static constexpr int OFF_RING = OFF_ZERO + 64;
  static constexpr int RES_PAIRS_MAX = SHARED ? 1 : (DCP + NR - 1) / NR;
  static constexpr int FH_MAX = NH > 0 ? DCP + (SHARED ? CT : 0) : 0;   // an H wavefront
  static constexpr int FR_MAX = RES_PAIRS_MAX * CT;                     // a residual wavefront
  static constexpr int FMAX = FH_MAX > FR_MAX ? FH_MAX : FR_MAX;
  static constexpr int RING = FMAX * 1024;
  static constexpr int LDS_LOOP = OFF_RING + DW * RING;
  // epilogue (aliases the raw ring and the expanded buffers)
  static constexpr int RB = (RT16 + 3) / 4;               // 64-rank blocks
  static constexpr int HSTR = RPAD + 1;
  static constexpr int QSTR = (RB > 0 ? RB : 1) * 64 + 16;
  static constexpr int E_HS = 0;                          // [16][HSTR] fp32
  static constexpr int E_QS = E_HS + 16 * HSTR * 4;       // [16][QSTR] fp8 codes
  static constexpr int E_SH = E_QS + 16 * QSTR;           // [RB][16] fp32
  static constexpr int E_RES = E_SH + (RB > 0 ? RB : 1) * 64;   // [NR][CT][4][64] fp32
  static constexpr int E_END = E_RES + NR * CT * 1024;
  static constexpr int LDS = LDS_LOOP > E_END ? LDS_LOOP : E_END;
  static_assert(LDS <= 160 * 1024, "fits the 160 KiB LDS of a CU");
  static_assert(E_END <= OFF_RING, "the epilogue fits below the fragment rings");
};

template <int N>
__device__ __forceinline__ void dwait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt has 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

__device__ __forceinline__ void ddma(const uint8_t *addr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(addr), "s"(lds)
               : "memory");
}

__device__ __forceinline__ v8i dlds_v8i(const uint8_t *p) {
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(p);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(p + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// exact products s_a[row] * s_b[col] of a 16 x 16 tile (lanes 0-15 carry the
// fp16 scales in k = 0, every other operand element is zero)
__device__ __forceinline__ v4f outer16(uint32_t sa, uint32_t sb) {
  const v4f z = {0, 0, 0, 0};
  const u32x2 a2 = {sa, 0u}, b2 = {sb, 0u};
  return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(v4h, a2),
                                               __builtin_bit_cast(v4h, b2), z, 0, 0, 0);
}

// A lane's load of one chunk item: 16 bytes at base + min(16 c + gl, KG - 1) * gs
struct DItem {
  const uint8_t *base;
  uint32_t gs;
  int gl;
  uint32_t lds;   // wave-uniform offset within a raw slot
};

template <int RT16, int CT>
__global__ __launch_bounds__(64 * DW, 1) void dual_gemm_decode_kernel(GemmArgs a) {
  using C = DCfg<RT16, CT>;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KG = geo.k / kGroup, NP = (KG + 1) / 2, NCH = (KG + DCG - 1) / DCG;
  const int m = a.m, ms = a.ms;
  const int c0 = blockIdx.x * CT;           // first 16-column tile
  const int ct16 = geo.n_pad / 16;
  const uint8_t *xc = reinterpret_cast<const uint8_t *>(a.xc);
  const uint8_t *xs = reinterpret_cast<const uint8_t *>(a.xs);
  const uint8_t *wcodes = a.packed + geo.off_w;
  const uint8_t *wscales = a.packed + geo.off_ws;
  const uint8_t *l1codes = a.packed + geo.off_l1;
  const uint8_t *l1scales = a.packed + geo.off_l1s;
  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);
  const int q = lane >> 4, c16 = lane & 15;

  // ---- this wavefront's chunk items ----
  DItem it[C::NCI];
#pragma unroll
  for (int t = 0; t < C::NCI; t++) {
    int k = wave + DW * t;
    if (k >= C::NITEM) k = wave;   // a repeat of item `wave` (same bytes, same place)
    DItem &d = it[t];
    if (k < 8) {                   // code pair k: groups 2k, 2k + 1 of the chunk
      // lane (group 2k + q / 2, half q % 2, token c16) of the first token tile
      d.base = xc + (int64_t)(32 * (q & 1) + min(c16, m - 1)) * 16;
      d.gs = 1024;
      d.gl = 2 * k + (q >> 1);
      d.lds = C::R_X + k * 1024;
    } else if (k == 8) {           // activation scales: lane (group l / 2, tokens 8 (l % 2) ..)
      const int l = lane & 31;
      d.base = xs + (int64_t)min(8 * (l & 1), ms - 8) * 2;
      d.gs = (uint32_t)ms * 2;
      d.gl = l >> 1;
      d.lds = C::R_SX;
    } else if (k == 9) {           // weight scales: lane (group l / (2 CT), columns 8 (l % 2 CT) ..)
      const int l = lane & (32 * CT - 1);
      d.base = wscales + (int64_t)min(16 * c0 + 8 * (l % (2 * CT)), geo.n_pad - 8) * 2;
      d.gs = (uint32_t)geo.n_pad * 2;
      d.gl = l / (2 * CT);
      d.lds = C::R_SW;
    } else {                       // L1 scales, region s: lane (group, ranks 8 (.) ..)
      const int s = k - 10;
      const int per = C::RPAD > 0 ? C::RPAD / 8 : 1;   // 16-byte pieces per group
      const int piece = (s * 64 + lane) % (DCG * per);
      d.base = l1scales + (int64_t)min(8 * (piece % per), geo.r_pad32 - 8) * 2;
      d.gs = (uint32_t)geo.r_pad32 * 2;
      d.gl = piece / per;
      d.lds = C::R_SL + s * 1024;
    }
  }
  auto issue_chunk = [&](int c) {
    const uint32_t slot = lds0 + C::OFF_RAW + (c % DRAW) * C::RSLOT;
#pragma unroll
    for (int t = 0; t < C::NCI; t++)
      ddma(it[t].base + (uint64_t)min(DCG * c + it[t].gl, KG - 1) * it[t].gs, slot + it[t].lds);
  };

  // ---- this wavefront's fragments: H tile (wave < NH) and residual pairs ----
  const bool hw = wave < C::NH;
  const int rw = C::SHARED ? wave : wave - C::NH;           // residual index (< 0: none)
  const int nres = C::SHARED ? 1 : (rw >= 0 ? (DCP - rw + C::NR - 1) / C::NR : 0);   // pairs per chunk
  const int F = (hw ? DCP : 0) + nres * CT;                 // fragment loads per chunk
  const uint32_t ring = lds0 + C::OFF_RING + wave * C::RING;
  // fragment of a 16-column (or 16-rank) slice of a packed 32-wide block pair:
  // lane (q, c16) -> group 2 p + q / 2, code half q % 2, column c16
  auto frag_addr = [&](const uint8_t *blocks, int col16, int p) {
    const int g = min(2 * min(p, NP - 1) + (q >> 1), KG - 1);
    const int L = (q & 1) * 32 + (col16 & 1) * 16 + c16;
    return blocks + (((int64_t)(col16 >> 1) * KG + g) * 64 + L) * 16;
  };
  auto issue_frags = [&](int c) {   // fragments of chunk c, in the consumption order
    int s = 0;
    if (hw) {
#pragma unroll
      for (int pl = 0; pl < DCP; pl++, s++) ddma(frag_addr(l1codes, wave, DCP * c + pl), ring + s * 1024);
    }
    for (int i = 0; i < nres; i++) {
      const int pl = C::SHARED ? rw : rw + C::NR * i;
#pragma unroll
      for (int j = 0; j < CT; j++, s++)
        ddma(frag_addr(wcodes, min(c0 + j, ct16 - 1), DCP * c + pl), ring + s * 1024);
    }
  };
  // wait until at most n loads are in flight (n is wave-uniform, < 64)
  auto wait_n = [&](int n) {
    switch (n) {
#define TQ_W(N) case N: dwait_vm<N>(); break;
      TQ_W(0) TQ_W(1) TQ_W(2) TQ_W(3) TQ_W(4) TQ_W(5) TQ_W(6) TQ_W(7) TQ_W(8) TQ_W(9)
      TQ_W(10) TQ_W(11) TQ_W(12) TQ_W(13) TQ_W(14) TQ_W(15) TQ_W(16) TQ_W(17) TQ_W(18)
      TQ_W(19) TQ_W(20) TQ_W(21) TQ_W(22) TQ_W(23) TQ_W(24)
#undef TQ_W
      default: dwait_vm<0>(); break;
    }
  };

  // expand raw chunk c into fp8 operand bytes: thread = (group, half, token)
  auto expand = [&](int c) {
    const uint8_t *R = smem + C::OFF_RAW + (c % DRAW) * C::RSLOT + C::R_X;
    const int g = tid >> 5, h = (tid >> 4) & 1, t = tid & 15;
    // raw pair layout: [pair][lane (group in pair, half, token)] x 16 B
    const u32x4 raw = *reinterpret_cast<const u32x4 *>(R + ((g >> 1) * 64 + (g & 1) * 32 + h * 16 + t) * 16);
    const v8i u = unpack32(raw);
    uint8_t *E = smem + C::OFF_XE + (c & 1) * C::XE + ((g * 2 + h) * 16 + t) * 32;
    *reinterpret_cast<u32x4 *>(E) = u32x4{(uint32_t)u[0], (uint32_t)u[1], (uint32_t)u[2], (uint32_t)u[3]};
    *reinterpret_cast<u32x4 *>(E + 16) = u32x4{(uint32_t)u[4], (uint32_t)u[5], (uint32_t)u[6], (uint32_t)u[7]};
  };

  if (tid < 16) reinterpret_cast<uint32_t *>(smem + C::OFF_ZERO)[tid] = 0;

  // ---- prologue ----
  dwait_vm<0>();
  issue_chunk(0);
  issue_chunk(1);
  issue_frags(0);
  wait_n(C::NCI + F);   // chunk 0's items have landed
  __syncthreads();
  expand(0);

  v4f hacc = v4f{0, 0, 0, 0};
  v4f acc[CT];
#pragma unroll
  for (int j = 0; j < CT; j++) acc[j] = v4f{0, 0, 0, 0};

  // operand addresses of a group pair within an expanded chunk: lanes 0-31
  // read group 2 pl (token c16, half q), lanes 32-63 group 2 pl + 1; the
  // other single-group operand reads zeros
  const uint32_t xe_lane = ((q & 1) * 16 + c16) * 32 + (q >> 1) * 1024;
  const uint32_t zero_off = C::OFF_ZERO;

  // The K loop of one wavefront role, with its per-chunk load count NF as a
  // compile-time constant: NH wavefronts walk the 8 pairs of their H tile,
  // residual wavefronts their NRP pairs x CT tiles.  Operands of the next
  // fragment slot are read from LDS while the current one computes.
  struct Ops {
    u32x4 b;   // raw codes, expanded just before their products
    v8i a1, a2;
    uint32_t sx1, sx2, sy1, sy2;
  };
  auto chunk_loop = [&](auto HC, auto NRPC) {
    constexpr bool H = decltype(HC)::value;       // this wavefront walks an H tile
    constexpr int NRP = decltype(NRPC)::value;    // residual pairs per chunk
    constexpr int NF = (H ? DCP : 0) + NRP * CT;  // fragment slots per chunk
    constexpr int NCI = C::NCI;
    // slot k -> (pair within the chunk, is H, residual tile)
    auto slot_pair = [&](int k) { return (H && k < DCP) ? k : (C::SHARED ? rw : rw + C::NR * ((k - (H ? DCP : 0)) / CT)); };
    auto slot_is_h = [&](int k) { return H && k < DCP; };
    auto slot_tile = [&](int k) { return (k - (H ? DCP : 0)) % CT; };
    auto read_ops = [&](int c, int k, Ops &O) {
      const uint8_t *RS = smem + C::OFF_RAW + (c % DRAW) * C::RSLOT;
      const int pl = slot_pair(k);
      const uint32_t pa = C::OFF_XE + (c & 1) * C::XE + pl * 2048 + xe_lane;
      O.b = *reinterpret_cast<const u32x4 *>(smem + C::OFF_RING + wave * C::RING + k * 1024 + lane * 16);
      O.a1 = dlds_v8i(smem + (q < 2 ? pa : zero_off));
      O.a2 = dlds_v8i(smem + (q < 2 ? zero_off : pa));
      const uint32_t zs = C::OFF_ZERO;   // lanes 16-63 read zero scales
      O.sx1 = *reinterpret_cast<const uint16_t *>(smem + (lane < 16 ? (uint32_t)(RS - smem) + C::R_SX + ((2 * pl) * 16 + c16) * 2 : zs));
      O.sx2 = *reinterpret_cast<const uint16_t *>(smem + (lane < 16 ? (uint32_t)(RS - smem) + C::R_SX + ((2 * pl + 1) * 16 + c16) * 2 : zs));
      uint32_t o1, o2;
      if (slot_is_h(k)) {
        o1 = C::R_SL + ((2 * pl) * C::RPAD + 16 * wave + c16) * 2;
        o2 = C::R_SL + ((2 * pl + 1) * C::RPAD + 16 * wave + c16) * 2;
      } else {
        const int j = slot_tile(k);
        o1 = C::R_SW + ((2 * pl) * 16 * CT + 16 * j + c16) * 2;
        o2 = C::R_SW + ((2 * pl + 1) * 16 * CT + 16 * j + c16) * 2;
      }
      O.sy1 = *reinterpret_cast<const uint16_t *>(smem + (lane < 16 ? (uint32_t)(RS - smem) + o1 : zs));
      O.sy2 = *reinterpret_cast<const uint16_t *>(smem + (lane < 16 ? (uint32_t)(RS - smem) + o2 : zs));
    };
    auto compute = [&](int c, int k, const Ops &O) {
      const int g1 = DCG * c + 2 * slot_pair(k);
      const v8i b = unpack32(O.b);
      const v4f m1 = mfma_codes_16x16x128(O.a1, b);
      const v4f o1 = outer16(O.sx1, O.sy1);
      const v4f m2 = mfma_codes_16x16x128(O.a2, b);
      const v4f o2 = outer16(O.sx2, O.sy2);
      v4f &t = slot_is_h(k) ? hacc : acc[slot_tile(k)];
      if (g1 < KG) {
#pragma unroll
        for (int v = 0; v < 4; v++) t[v] = fmaf(m1[v], o1[v], t[v]);
      }
      if (g1 + 1 < KG) {
#pragma unroll
        for (int v = 0; v < 4; v++) t[v] = fmaf(m2[v], o2[v], t[v]);
      }
    };
    auto refill = [&](int c, int k) {
      const int pl = slot_pair(k);
      if (slot_is_h(k)) ddma(frag_addr(l1codes, wave, DCP * c + pl), ring + k * 1024);
      else ddma(frag_addr(wcodes, min(c0 + slot_tile(k), ct16 - 1), DCP * c + pl), ring + k * 1024);
    };
    for (int c = 0; c < NCH; c++) {
      dwait_vm<NF>();     // chunk c + 1's items have landed
      __syncthreads();    // chunk c's expansion is visible; chunk c - 1 is consumed everywhere
      if (c + 1 < NCH) expand(c + 1);
      issue_chunk(c + 2);
      if constexpr (NF > 0) {
        Ops O, On;
        dwait_vm<NF - 1 + NCI>();   // slot 0 has landed
        read_ops(c, 0, O);
#pragma unroll
        for (int k = 0; k < NF; k++) {
          if (k + 1 < NF) {
            dwait_vm<(NF >= 2 ? NF - 2 + NCI : 0)>();   // slot k + 1 has landed
            read_ops(c, k + 1, On);
          }
          __builtin_amdgcn_sched_barrier(0);
          compute(c, k, O);
          __builtin_amdgcn_sched_barrier(0);
          refill(c + 1, k);   // slot k's reads were consumed above
          O = On;
        }
      }
    }
  };
  if (hw) {
    if constexpr (C::NH > 0) {
      if constexpr (C::SHARED) chunk_loop(std::true_type{}, std::integral_constant<int, 1>{});
      else chunk_loop(std::true_type{}, std::integral_constant<int, 0>{});
    }
  } else if (nres == 2) {
    chunk_loop(std::false_type{}, std::integral_constant<int, 2>{});
  } else {
    chunk_loop(std::false_type{}, std::integral_constant<int, 1>{});
  }
  dwait_vm<0>();
  __syncthreads();   // every load has landed and every wavefront is done with the rings

  // ---- H tiles and residual partials -> LDS ----
  float *HS = reinterpret_cast<float *>(smem + C::E_HS);
  uint8_t *QS = smem + C::E_QS;
  float *SHS = reinterpret_cast<float *>(smem + C::E_SH);
  float *RES = reinterpret_cast<float *>(smem + C::E_RES);
  const int orow0 = 4 * q;   // output rows 4q .. 4q + 3 of this lane
  if (hw) {
#pragma unroll
    for (int v = 0; v < 4; v++) HS[(orow0 + v) * C::HSTR + 16 * wave + c16] = hacc[v];
  }
  if (rw >= 0) {
#pragma unroll
    for (int j = 0; j < CT; j++)
#pragma unroll
      for (int v = 0; v < 4; v++) RES[((rw * CT + j) * 4 + v) * 64 + lane] = acc[j][v];
  }
  if constexpr (RT16 > 0) {
    const int r = geo.r;
    if (r < C::RB * 64)
      for (int idx = tid; idx < 16 * C::RB * 64; idx += 64 * DW) {
        const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
        if (j >= r) QS[row * C::QSTR + j] = 0;
      }
  }
  __syncthreads();

  // ---- re-quantize H per token and rank group (s_H stays fp32) ----
  if constexpr (RT16 > 0) {
    const int r = geo.r, gr = geo.gr, rg = r / gr;
    const int subs = gr / 8;                // lanes per (token, rank group): 1, 2, 4 or 8
    const int work = 16 * rg * subs;        // <= 256
    const bool dbg = a.dbg_h != nullptr && blockIdx.x == 0;
    const bool valid = tid < work;
    const int pair = tid / subs, sub = tid % subs;
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
    const float sh = amax / 7.0f;   // IEEE division
    if (valid) {
      uint32_t w0 = 0, w1 = 0;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        int qv = 0;
        if (sh != 0.0f) {
          float tq = __builtin_rintf(hv[e] / sh);
          tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
          qv = (int)tq;
        }
        const uint32_t bq = code_to_fp8(qv);
        if (e < 4) w0 |= bq << (8 * e); else w1 |= bq << (8 * (e - 4));
        if (dbg && row < m) {
          a.dbg_h[(int64_t)row * r + j0 + e] = hv[e];
          a.dbg_qh[(int64_t)row * r + j0 + e] = (int8_t)qv;
        }
      }
      *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0) = w0;
      *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0 + 4) = w1;
      if (sub == 0) {
        SHS[hg * 16 + row] = sh;
        if (dbg && row < m) a.dbg_sh[(int64_t)row * rg + hg] = sh;
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
      if constexpr (RT16 > 0) {
        // rank blocks in pairs: lanes q < 2 carry block rb, lanes q >= 2 block rb + 1
        for (int rb = 0; rb < C::RB; rb += 2) {
          const int rbq = min(rb + (q >> 1), C::RB - 1);
          const v8i qa = dlds_v8i(QS + c16 * C::QSTR + rbq * 64 + (q & 1) * 32);
          const int L = (q & 1) * 32 + (ct & 1) * 16 + c16;
          const v8i lb = unpack32(*reinterpret_cast<const u32x4 *>(
              l2codes + (((int64_t)(ct >> 1) * C::RB + rbq) * 64 + L) * 16));
          const v8i zero = {0, 0, 0, 0, 0, 0, 0, 0};
          const v8i qa1 = q < 2 ? qa : zero;
          const v8i qa2 = q < 2 ? zero : qa;
          const int col = ct * 16 + c16;
          {
            const float s2 = half_bits_to_float(l2scales[(int64_t)rb * geo.n_pad + col]);
            const v4f cb = mfma_codes_16x16x128(qa1, lb);
#pragma unroll
            for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[rb * 16 + orow0 + v] * s2, ylr[v]);
          }
          if (rb + 1 < C::RB) {
            const float s2 = half_bits_to_float(l2scales[(int64_t)(rb + 1) * geo.n_pad + col]);
            const v4f cb = mfma_codes_16x16x128(qa2, lb);
#pragma unroll
            for (int v = 0; v < 4; v++) ylr[v] = fmaf(cb[v], SHS[(rb + 1) * 16 + orow0 + v] * s2, ylr[v]);
          }
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
            for (int w2 = 0; w2 < C::NR; w2++) yres += RES[((w2 * CT + j) * 4 + v) * 64 + lane];
            const float yv = yres + ylr[v];
            const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
            reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
          }
        }
      }
    }
  }
}

template <int RT16, int CT>
hipError_t launch_decode(const GemmArgs &a, hipStream_t s) {
  using C = DCfg<RT16, CT>;
  const int tiles16 = a.geo.n_pad / 16;
  auto kern = dual_gemm_decode_kernel<RT16, CT>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((tiles16 + CT - 1) / CT), dim3(64 * DW), C::LDS, s, a);
  return hipGetLastError();
}

template <int CT>
hipError_t launch_decode_ct(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.r_pad32 / 16) {
    case 0: return launch_decode<0, CT>(a, s);
    case 2: return launch_decode<2, CT>(a, s);
    case 4: return launch_decode<4, CT>(a, s);
    case 8: return launch_decode<8, 1>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_dual_gemm_decode(const GemmArgs &a, hipStream_t s) {
  // two 16-column tiles per workgroup once one tile per workgroup would take
  // more than about two rounds of the 256 CUs
  const int tiles16 = a.geo.n_pad / 16;
  int ct = tiles16 > 2 * 256 ? 2 : 1;
  if (const char *env = getenv("TQ_DECODE_CT")) ct = atoi(env) == 2 ? 2 : 1;
  return ct == 2 ? launch_decode_ct<2>(a, s) : launch_decode_ct<1>(a, s);
}

}  // namespace tq
