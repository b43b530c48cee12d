// Fused dual-component W4A4 layer (paper Sec. 4.3) for prefill-sized token
// counts: the residual 4-bit GEMM, the stage-1 product H = Q(X) Q(L1) kept on
// chip, its on-the-fly re-quantization, stage 2 Q_H Q(L2) and one epilogue,
// in one kernel.
//
// Work decomposition.  A workgroup of 8 wavefronts (two per SIMD) owns a block
// of 128 tokens and a run of 256-column blocks.  Wavefront w = 4 wr + wc
// computes tokens [64 wr, +64) x columns [64 wc, +64) of a block: four 32x32
// tiles.  During the first column block of its run the workgroup also forms H
// for its 128 tokens: 4 x (r / 32) tiles of 32 tokens x 32 ranks, one or two
// per wavefront, each accumulated in ascending K-group order (the oracle's
// order, so H is bit-identical).  After that block H is re-quantized into LDS;
// later blocks of the run reuse Q_H and s_H.
//
// K pipeline.  Everything a K-group needs -- the 128 activation rows (fp8
// operand bytes: at these token counts the quantizer writes the codes
// expanded, so no wavefront unpacks an activation operand), the 256 weight
// columns, the rank columns of L1 (first block only) and all their scales --
// arrives once per workgroup by direct global->LDS loads
// (global_load_lds_dwordx4) into a D-slot ring; the loads of a group are
// spread over the 8 wavefronts, and one workgroup barrier per group hands
// slots over.  A wavefront's group step has a matrix-core phase (the eight
// products of the group, with its share of the loads of a later group in
// their shadow) and a vector phase (the rescaling fmas of those products, the
// next group's LDS reads and operand expansion).  The two wavefronts of a
// SIMD run these phases out of step --
// their barrier sits after the matrix-core phase on one and after the vector
// phase on the other -- so one issues matrix-core work while the other issues
// vector work: on gfx950 a wavefront that interleaves both itself overlaps
// them poorly, two wavefronts that split them overlap well.
//
// Arithmetic per 32x32 tile and group (Eq. 2): the exact integer group sum of
// code products comes from v_mfma_scale_f32_32x32x64_f8f6f4 (codes as fp8
// subnormals; block scales 2^8 and 2^9 return half of the integer sum), the
// exact scale product from v_mfma_f32_32x32x8f16 with both scale operands
// placed in k = 0 and k = 4 (twice the product), and one fma adds their
// product -- exactly I * s_x * s_w -- to the fp32 accumulator in ascending
// group order, the oracle's order for H and for the residual, so Y is
// bit-identical to the oracle's rounded result.  128-wide groups (Sec. 5.1)
// keep the 64-wide operand blocks: a group's two blocks add their integer
// sums in the matrix core (its accumulator input) before the one rescale.

#include <type_traits>

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int PBM = 128;   // tokens per workgroup block (four 32-row tiles)
constexpr int PBN = 256;   // columns per block (eight 32-column tiles)
constexpr int PNW = 8;     // wavefronts per workgroup
// one ring slot (one K-group).  Main loop: activation tiles, weight tiles,
// weight and activation scales.  H pass: activation tiles, L1 rank tiles in
// place of the weight tiles, activation and L1 scales.  Every load is one
// 16-byte-per-lane wave load; the scale runs fill part of a 1 KiB region.
constexpr int P_A = 0;          // 4 x 2 KiB fp8 activation tiles (two 1 KiB halves each)
constexpr int P_B = 8192;       // 8 x 1 KiB weight blocks as stored (H pass: L1 blocks)
constexpr int P_SW = 16384;     // weight scales of the 256 columns (H pass: all scales)
constexpr int P_SX = 16896;     // activation scales of the 128 tokens (256 B)
constexpr int P_STAGE = 17408;

template <int RT, int D>
struct PCfg {
  static constexpr int STAGE = P_STAGE;
  static constexpr int RING = D * STAGE;
  static constexpr int RB = (RT + 1) / 2;            // 64-rank blocks (= rank groups)
  static constexpr int HSTR = RT * 32 + 1;           // fp32 H staging: row stride in floats
  static constexpr int QSTR = RB * 64 + 16;          // Q_H bytes per token row
  static constexpr int OFF_Q = RING;
  static constexpr int OFF_SH = OFF_Q + (RT > 0 ? PBM * QSTR : 0);
  // stage-2 operands of each column pair (the two wavefronts with the same
  // wc share them), loaded while the K loop starts: 2 x RB L2 blocks, then a
  // 1 KiB scale region
  static constexpr int L2W = 2 * RB * 1024 + 1024;
  static constexpr int OFF_L2 = OFF_SH + (RT > 0 ? RB * PBM * 4 : 0);
  static constexpr int LDS = OFF_L2 + (RT > 0 ? 4 * L2W : 0);
  static constexpr int HT = RT >= 2 ? RT / 2 : 1;    // H tiles of an H wavefront
  static_assert(PBM * HSTR * 4 <= RING, "H staging fits in the ring");
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

// the same added to c: the two 64-wide blocks of a 128-wide group (exact
// while the sums stay integers below 2^24)
__device__ __forceinline__ v16f codes_half_acc(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, kScale2p9 - 1, 0,
                                                         kScale2p9);
}

__device__ __forceinline__ void fma16(v16f &acc, const v16f &c, const v16f &p) {
#pragma unroll
  for (int v = 0; v < 16; v++) acc[v] = fmaf(c[v], p[v], acc[v]);
}

__device__ __forceinline__ v8i join(u32x4 lo, u32x4 hi) {
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// s_waitcnt vmcnt(n) (n < 64), leaving the other counters alone
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt has 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// direct global -> LDS load of 16 bytes per lane into lds + 16 * lane:
// scalar base + 32-bit lane offset
__device__ __forceinline__ void dma_s(uint32_t voff, const uint8_t *sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase),
               "s"(lds)
               : "memory");
}
__device__ __forceinline__ void dma_v(const uint8_t *addr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(addr), "s"(lds)
               : "memory");
}

// wave-uniform 64-bit pointer, kept in scalar registers
__device__ __forceinline__ const uint8_t *uniform_ptr(const uint8_t *p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t *>(((uint64_t)hi << 32) | lo);
}

// This wavefront's share of one 64-wide K block's loads: two
// 16-byte-per-lane wave loads (item t reads b[t] + g * inc[t] + v[t] (lane)),
// and for wavefront 0 a third one, the scales of the block's quantization
// group (GK blocks per group): lane l reads 16 bytes at s3[l] + (g / GK) * inc3[l].
struct PPlan {
  const uint8_t *b1, *b2;     // wave-uniform bases of group 0
  uint32_t inc1, inc2;        // bytes per K-group
  uint32_t v1, v2;            // lane offsets
  uint32_t l1, l2;            // LDS offsets within a slot
  const uint8_t *s3;          // lane address of group 0 (wavefront 0)
  uint32_t inc3;              // lane bytes per quantization group
};

template <int GK>
__device__ __forceinline__ void p_issue(const PPlan &P, bool three, int g, uint32_t slot_lds) {
  // the bases are wave-uniform (scalar registers): the block offset is added
  // with scalar instructions
  dma_s(P.v1, P.b1 + (uint32_t)g * P.inc1, slot_lds + P.l1);
  dma_s(P.v2, P.b2 + (uint32_t)g * P.inc2, slot_lds + P.l2);
  if (three) dma_v(P.s3 + (uint64_t)(g / GK) * P.inc3, slot_lds + P_SW);
}

// activation tile t of the block (clamped to the last tile): its group-0
// block; the tile of one group is 2 KiB of fp8 operand bytes, two 1 KiB
// halves in matrix-core lane order
__device__ __forceinline__ const uint8_t *act_tile(const GemmArgs &a, int m0, int t) {
  const int tt = min(m0 / 32 + t, (a.m - 1) / 32);
  return reinterpret_cast<const uint8_t *>(a.xc) + (int64_t)tt * (a.geo.k / kGroup) * 2048;
}

// Main loop: wavefront w loads weight tile w and, as its second item, half
// w % 2 of activation tile w / 2.  Wavefront 0 also loads the scales: the weight
// scales of the 256 columns (lanes 0-31, eight each, to P_SW) and the
// activation scales of the 128 tokens (lanes 32-47, to P_SX; lanes 48-63
// repeat lane 32's run into unused bytes), clamped to the padded sizes.
__device__ __forceinline__ void plan_main(const GemmArgs &a, int lane, int wave, int m0, int n0,
                                          PPlan &P) {
  const Geometry &geo = a.geo;
  const int KG = geo.k / kGroup;
  const int ct = min(n0 / 32 + wave, geo.n_pad / 32 - 1);   // past the last tile: never stored
  P.b1 = uniform_ptr(a.packed + geo.off_w + (int64_t)ct * KG * 1024);
  P.inc1 = 1024;
  P.v1 = lane * 16;
  P.l1 = P_B + wave * 1024;
  P.b2 = uniform_ptr(act_tile(a, m0, wave >> 1) + (wave & 1) * 1024);
  P.inc2 = 2048;
  P.v2 = lane * 16;
  P.l2 = P_A + wave * 1024;
  if (lane < 32) {
    P.s3 = a.packed + geo.off_ws + (int64_t)min(n0 + 8 * lane, geo.n_pad - 8) * 2;
    P.inc3 = (uint32_t)geo.n_pad * 2;
  } else {
    const int l = lane < 48 ? lane - 32 : 0;
    P.s3 = reinterpret_cast<const uint8_t *>(a.xs) + (int64_t)min(m0 + 8 * l, a.ms - 8) * 2;
    P.inc3 = (uint32_t)a.ms * 2;
  }
}

// H pass.  A step covers one 64-wide K block, laid out in a slot as: the
// activation tiles at P_A (as in the main loop), L1 rank tile t at
// P_B + 1024 t, and at H_S the activation scales of the 128 tokens (256 B)
// followed by the L1 scales (256 B) of the block's quantization group.  Every
// item is a wave load whose lane l reads 16 bytes at base[l] + (g >> shift)
// * stride[l].
constexpr int H_S = P_SW;

struct HPlan {
  const uint8_t *base[2];   // lane addresses for block 0
  uint32_t stride[2];       // lane bytes per block (codes) or per quantization group (scales)
  uint32_t lds[2];          // wave-uniform LDS offset within a slot
  int shift[2];             // block index >> shift: 0 for codes, log2(GK) for scales
};

__device__ __forceinline__ void h_issue(const HPlan &P, int g, uint32_t slot_lds) {
#pragma unroll
  for (int t = 0; t < 2; t++)
    dma_v(P.base[t] + (uint64_t)(g >> P.shift[t]) * P.stride[t], slot_lds + P.lds[t]);
}

// items, in order: the 8 activation halves, RT L1 tiles, one scale item, then
// repeats of earlier items (same bytes to the same place); wavefront w takes
// items w and w + 8
__device__ __forceinline__ void plan_h(const GemmArgs &a, int lane, int wave, int m0, int RT,
                                       HPlan &P) {
  const Geometry &geo = a.geo;
  const int KG = geo.k / kGroup;
  const int nitem = 8 + RT + 1;
#pragma unroll
  for (int t = 0; t < 2; t++) {
    int it = wave + 8 * t;
    if (it >= nitem) it -= 8;   // a repeat of item it - 8
    P.shift[t] = 0;
    if (it < 8) {               // half it % 2 of activation tile it / 2
      P.base[t] = act_tile(a, m0, it >> 1) + (it & 1) * 1024 + lane * 16;
      P.stride[t] = 2048;
      P.lds[t] = P_A + 1024 * it;
    } else if (it < 8 + RT) {   // L1 rank tile it - 8
      P.base[t] = a.packed + geo.off_l1 + (int64_t)(it - 8) * KG * 1024 + lane * 16;
      P.stride[t] = 1024;
      P.lds[t] = P_B + 1024 * (it - 8);
    } else {   // scales: lanes 0-15 activation runs, 16-31 L1 runs, then repeats
      const int q = lane >> 4, r = lane & 15;
      if ((q & 1) == 0) {
        P.base[t] = reinterpret_cast<const uint8_t *>(a.xs) +
                    (int64_t)min(m0 + 8 * r, a.ms - 8) * 2;
        P.stride[t] = (uint32_t)a.ms * 2;
      } else {
        P.base[t] = a.packed + geo.off_l1s + (int64_t)min(8 * r, geo.r_pad32 - 8) * 2;
        P.stride[t] = (uint32_t)geo.r_pad32 * 2;
      }
      P.shift[t] = geo.gk - 1;   // one scale row per quantization group
      P.lds[t] = H_S;
    }
  }
}

template <int RT, int D>
struct PKernel {
  using C = PCfg<RT, D>;

  struct Raw {
    v8i a[2];      // fp8 activation operands, ready for the matrix cores
    u32x4 b[2];    // TQ4 weight operands
    uint32_t sa[2], sb[2];
  };

  // This lane's byte offsets within a slot (loop-invariant): one address add
  // per operand kind and group, the rest are immediate offsets.
  struct RawOff {
    uint32_t a, b, sa, sb;
  };
  __device__ __forceinline__ static RawOff raw_off(int lane, int wr, int wc) {
    const int l32 = lane & 31;
    RawOff o;
    o.a = P_A + 2 * wr * 2048 + lane * 16;
    o.b = P_B + 2 * wc * 1024 + lane * 16;
    o.sa = P_SX + (64 * wr + l32) * 2;
    o.sb = P_SW + (64 * wc + l32) * 2;
    return o;
  }

  __device__ __forceinline__ static void read_raw(const uint8_t *S, const RawOff &o, Raw &R) {
    const uint8_t *pa = S + o.a, *pb = S + o.b, *psa = S + o.sa, *psb = S + o.sb;
#pragma unroll
    for (int i = 0; i < 2; i++) {
      R.a[i] = join(*reinterpret_cast<const u32x4 *>(pa + i * 2048),
                    *reinterpret_cast<const u32x4 *>(pa + i * 2048 + 1024));
      R.sa[i] = *reinterpret_cast<const uint16_t *>(psa + i * 64);
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      R.b[j] = *reinterpret_cast<const u32x4 *>(pb + j * 1024);
      R.sb[j] = *reinterpret_cast<const uint16_t *>(psb + j * 64);
    }
  }

  // The residual K loop as two phases per group that the two wavefronts of a
  // SIMD run out of step, so that one issues matrix-core work while the other
  // issues vector work:
  //   X(g): the eight matrix-core products of group g (code and scale products
  //         of tiles 00, 01, 10, 11), with this wavefront's loads of a later
  //         group interleaved between them (their scalar address arithmetic
  //         issues while the matrix core works);
  //   Y(g): the LDS reads of group g + 1, the 64 rescaling fmas of group g (on
  //         products that X(g) has finished) and the expansion of the weight
  //         operands of group g + 1.
  // Every wavefront runs X(0) Y(0) X(1) Y(1) ... with one workgroup barrier per
  // group, placed after X(g) on wavefronts 0-3 (GA) and after Y(g) on
  // wavefronts 4-7 (each SIMD holds one of each), so between barriers k - 1 and
  // k wavefront A runs Y(k - 1) X(k) while wavefront B runs X(k) Y(k).
  //
  // Ring hand-over.  In that interval A reads group k and B group k + 1, so
  // the barrier that opens it must publish groups <= k + 1; slot s is free
  // once both readers of its group have passed the barrier after their reads.
  // Each wavefront issues its loads of group k + D - 1 into slot (k - 1) % D
  // in X(k), which lies in interval k for A and B alike, and before barrier k
  // waits until only its loads of groups k + 3 .. k + D - 1 may be in flight
  // (D - 3 groups), so groups <= k + 2 are complete when barrier k opens.  The
  // prologue loads groups 0 .. D - 2; loads past the last group repeat the
  // last group into a free slot.
  // (THREE: this wavefront also loads the scales, three loads per group; a
  // template parameter, so that the loop body is one basic block)
  //
  // 128-wide quantization groups (GK = 2): the ring still moves one 64-wide
  // block per step, and the steps go in pairs.  X of a group's first block
  // issues its four code products and holds them; X of the second adds the
  // second block's code products to them in the matrix core (the exact
  // integer sum of the whole group) and issues the group's four scale
  // products; only the second block's Y applies fmas.  Every wait and barrier
  // is the same per block as for 64-wide groups.
  template <bool GA, bool THREE, int GK, typename Pre>
  __device__ __forceinline__ static void main_loop_pp(const PPlan &P, uint8_t *smem,
                                                      uint32_t ring_lds, int KG, int lane, int wr,
                                                      int wc, v16f (&acc)[2][2], Pre pre) {
    static_assert(D >= 4, "the hand-over keeps D - 3 groups of loads in flight");
    static_assert(GK == 1 || GK == 2, "64- or 128-wide quantization groups");
    constexpr int L = THREE ? 3 : 2;   // loads per block
    wait_vm<0>();
    pre();
#pragma unroll
    for (int s = 0; s < D - 1; s++) p_issue<GK>(P, THREE, min(s, KG - 1), ring_lds + s * C::STAGE);
    wait_vm<L * (D - 3)>();
    __syncthreads();
    const RawOff ro = raw_off(lane, wr, wc);
    Raw R;
    read_raw(smem, ro, R);
    wait_lgkm0();
    v8i b0 = unpack32(R.b[0]), b1 = unpack32(R.b[1]);
    auto hand_over = [&]() {
      wait_vm<L * (D - 3)>();
      wait_lgkm0();
      __syncthreads();
    };
    // The slots read in Y(g) and loaded in X(g) advance one slot per block
    // (wave-uniform; no division in the loop): the read slot holds block
    // min(g + 1, KG - 1), the load slot (an LDS address) receives block
    // g + D - 1.
    uint32_t ring0 = ring_lds;
    asm volatile("" : "+s"(ring0));   // a plain scalar from here on
    const uint32_t ring_end = ring0 + C::RING;
    uint32_t rd_off = (uint32_t)(min(1, KG - 1) * C::STAGE);
    uint32_t ld_lds = ring0 + (uint32_t)((D - 1) * C::STAGE);
    // Y(g)'s reads: block g + 1's operands into the registers X(g) read (past
    // the last block: the last block again, never used); X(g)'s loads: this
    // wavefront's share of block g + D - 1 into the slot that block g - 1 left
    auto y_reads = [&](int g) {
      read_raw(smem + rd_off, ro, R);
      const uint32_t nx = rd_off + C::STAGE == (uint32_t)C::RING ? 0u : rd_off + C::STAGE;
      rd_off = g + 2 < KG ? nx : rd_off;
      asm volatile("" ::: "memory");
    };
    auto x_loads = [&](int g) {
      p_issue<GK>(P, THREE, min(g + D - 1, KG - 1), ld_lds);
      ld_lds += C::STAGE;
      ld_lds = ld_lds == ring_end ? ring0 : ld_lds;
    };
    auto y_expand = [&]() {
      wait_lgkm0();
      b0 = unpack32(R.b[0]);
      b1 = unpack32(R.b[1]);
    };
    for (int g = 0; g < KG; g += GK) {
      v16f c00, c01, c10, c11;
      if constexpr (GK == 2) {
        // ---- X(g): the group's first block, held ----
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
        c00 = codes_half(R.a[0], b0);
        c01 = codes_half(R.a[0], b1);
        c10 = codes_half(R.a[1], b0);
        c11 = codes_half(R.a[1], b1);
        x_loads(g);
#pragma unroll
        for (int i = 0; i < 4; i++) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x004, 6, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (GA) hand_over();
        __builtin_amdgcn_sched_barrier(0);
        // ---- Y(g) ----
        y_reads(g);
        __builtin_amdgcn_sched_barrier(0);
        y_expand();
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (!GA) hand_over();
      }
      const int gb = g + GK - 1;   // the group's last block
      // ---- X(gb) ----
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
      if constexpr (GK == 2) {
        c00 = codes_half_acc(R.a[0], b0, c00);
      } else {
        c00 = codes_half(R.a[0], b0);
      }
      const v16f p00 = outer2(R.sa[0], R.sb[0]);
      if constexpr (GK == 2) {
        c01 = codes_half_acc(R.a[0], b1, c01);
      } else {
        c01 = codes_half(R.a[0], b1);
      }
      const v16f p01 = outer2(R.sa[0], R.sb[1]);
      if constexpr (GK == 2) {
        c10 = codes_half_acc(R.a[1], b0, c10);
      } else {
        c10 = codes_half(R.a[1], b0);
      }
      const v16f p10 = outer2(R.sa[1], R.sb[0]);
      if constexpr (GK == 2) {
        c11 = codes_half_acc(R.a[1], b1, c11);
      } else {
        c11 = codes_half(R.a[1], b1);
      }
      const v16f p11 = outer2(R.sa[1], R.sb[1]);
      x_loads(gb);
      // one product, then a few of the loads' scalar, memory and address
      // instructions, in the shadow of the product
#pragma unroll
      for (int i = 0; i < 8; i++) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x004, 3, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (GA) hand_over();
      __builtin_amdgcn_sched_barrier(0);
      // ---- Y(gb) ----
      y_reads(gb);
      __builtin_amdgcn_sched_barrier(0);
      fma16(acc[0][0], c00, p00);
      fma16(acc[0][1], c01, p01);
      __builtin_amdgcn_sched_barrier(0);
      fma16(acc[1][0], c10, p10);
      fma16(acc[1][1], c11, p11);
      __builtin_amdgcn_sched_barrier(0);
      y_expand();
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (!GA) hand_over();
    }
    wait_vm<0>();   // the refills past the end have landed before the ring is reused
  }

  // The stage-1 pass: H tiles of 32 tokens x 32 ranks, accumulated over all
  // K-groups in ascending order (token tile ti, rank tiles hrt[]), one 64-wide
  // block per ring slot and step; a 128-wide group (GK = 2) adds its second
  // block's code products to its first's in the matrix core before its one
  // scale product.
  template <int GK>
  __device__ __forceinline__ static void h_loop(const HPlan &P, uint8_t *smem, uint32_t ring_lds,
                                                int KG, int lane, bool hw, int ti,
                                                const int (&hrt)[C::HT], v16f (&hacc)[C::HT]) {
    wait_vm<0>();
#pragma unroll
    for (int s = 0; s < D; s++) h_issue(P, min(s, KG - 1), ring_lds + s * C::STAGE);
    wait_vm<2 * (D - 1)>();
    __syncthreads();
    const int l32 = lane & 31;
    for (int s0 = 0; s0 < KG; s0 += GK) {
      v16f hc[C::HT];
#pragma unroll
      for (int u = 0; u < GK; u++) {
        const int s = s0 + u;
        const uint8_t *S = smem + (s % D) * C::STAGE;
        v8i ra = v8i{0};
        u32x4 rl[C::HT];
        uint32_t sa = 0, sl[C::HT];
        if (hw) {
          ra = join(*reinterpret_cast<const u32x4 *>(S + P_A + ti * 2048 + lane * 16),
                    *reinterpret_cast<const u32x4 *>(S + P_A + ti * 2048 + 1024 + lane * 16));
          sa = *reinterpret_cast<const uint16_t *>(S + H_S + (32 * ti + l32) * 2);
#pragma unroll
          for (int h = 0; h < C::HT; h++) {
            rl[h] = *reinterpret_cast<const u32x4 *>(S + P_B + 1024 * hrt[h] + lane * 16);
            sl[h] = *reinterpret_cast<const uint16_t *>(S + H_S + 256 + (32 * hrt[h] + l32) * 2);
          }
        }
        // block s + 1 has landed and every wavefront is done with slot s
        wait_vm<2 * (D - 2)>();
        wait_lgkm0();
        __syncthreads();
        h_issue(P, min(s + D, KG - 1), ring_lds + (s % D) * C::STAGE);
        if (hw) {
#pragma unroll
          for (int h = 0; h < C::HT; h++) {
            const v8i lb = unpack32(rl[h]);
            if (u == 0) {
              hc[h] = codes_half(ra, lb);
            } else {
              hc[h] = codes_half_acc(ra, lb, hc[h]);
            }
            if (u == GK - 1) fma16(hacc[h], hc[h], outer2(sa, sl[h]));
          }
        }
      }
    }
    wait_vm<0>();
  }
};

template <int RT, int D, int GK>
__global__ __launch_bounds__(64 * PNW, 1) void dual_gemm_prefill_kernel(GemmArgs a, int m_tiles,
                                                                        int n_tiles, int n_chunks,
                                                                        int cpw, int band) {
  using K = PKernel<RT, D>;
  using C = PCfg<RT, D>;
  // 64-rank blocks per rank group (a 128-rank group in 128-wide groups: 2)
  // and rank groups
  constexpr int BPG = GK == 2 && C::RB == 2 ? 2 : 1;
  constexpr int RG = C::RB / BPG;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wr = wave >> 2, wc = wave & 3;
  const int KG = geo.k / kGroup;
  const int m = a.m;
  const int ctiles = geo.n_pad / 32;
  const uint32_t ring_lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);

  // Workgroups are dealt round-robin to the 8 XCDs: give each XCD a
  // contiguous run of logical ids, ordered in bands of `band` token blocks,
  // column chunk by column chunk, so the workgroups of an XCD share their
  // activation rows and weight columns in its L2.
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
  const int m0 = m_tile * PBM;
  const int cb_begin = chunk * cpw;
  const int cb_end = min(cb_begin + cpw, n_tiles);

  // H tiles of this wavefront in the stage-1 pass: token tile hti, rank
  // tiles hrt[] (RT = 1: wavefronts 0-3, one per SIMD)
  const int hti = wave & 3;
  const bool hw = RT >= 2 || (RT == 1 && wave < 4);
  int hrt[C::HT];
#pragma unroll
  for (int h = 0; h < C::HT; h++) hrt[h] = RT >= 2 ? (wave >> 2) + 2 * h : 0;

  const uint8_t *l2codes = a.packed + geo.off_l2;
  const uint16_t *l2scales = reinterpret_cast<const uint16_t *>(a.packed + geo.off_l2s);

  for (int cb = cb_begin; cb < cb_end; cb++) {
    const int n0 = cb * PBN;
    if constexpr (RT > 0) {
      if (cb == cb_begin) {
        // ---- stage 1: H for the block's 128 tokens, then Q_H and s_H in LDS ----
        HPlan HP;
        plan_h(a, lane, wave, m0, RT, HP);
        v16f hacc[C::HT];
#pragma unroll
        for (int h = 0; h < C::HT; h++) hacc[h] = v16f{0};
        K::template h_loop<GK>(HP, smem, ring_lds, KG, lane, hw, hti, hrt, hacc);
        __syncthreads();   // every wavefront is done with the ring
        float *HS = reinterpret_cast<float *>(smem);
        uint8_t *QS = smem + C::OFF_Q;
        float *SHS = reinterpret_cast<float *>(smem + C::OFF_SH);
        const int r = geo.r, gr = geo.gr, rg = r / gr;
        if (hw) {
#pragma unroll
          for (int h = 0; h < C::HT; h++) {
#pragma unroll
            for (int v = 0; v < 16; v++) {
              const int row = 32 * hti + row_of_32x32(lane, v);
              HS[row * C::HSTR + hrt[h] * 32 + l32] = hacc[h][v];
            }
          }
        }
        if (r < C::RB * 64) {   // zero the fp8 padding ranks [r, 64 RB) of Q_H
          for (int idx = tid; idx < PBM * C::RB * 64; idx += 64 * PNW) {
            const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
            if (j >= r) QS[row * C::QSTR + j] = 0;
          }
        }
        __syncthreads();
        // per-token, per-rank-group re-quantization (s_H in fp32)
        const int subs = gr / 8;   // lanes per (token, rank group): 1, 2, 4 or 8
        const int work = PBM * rg * subs;
        const bool dbg = a.dbg_h != nullptr && chunk == 0;
        for (int base = 0; base < work; base += 64 * PNW) {
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
          const float s = amax / 7.0f;   // IEEE division; s_H stays fp32
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
              SHS[hg * PBM + row] = s;
              if (dbg && m0 + row < m) a.dbg_sh[(int64_t)(m0 + row) * rg + hg] = s;
            }
          }
        }
        __syncthreads();   // Q_H and s_H are published; the ring is free
      }
    }

    // ---- residual 4-bit GEMM of the block ----
    PPlan P;
    plan_main(a, lane, wave, m0, n0, P);
    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
      for (int j = 0; j < 2; j++) acc[i][j] = v16f{0};
    // the stage-2 operands of this column pair's two column tiles (L2 blocks
    // and scales) travel with the first groups of the K loop, loaded by the
    // wavefront with wr = 0 (published by the K loop's first barrier)
    const uint32_t l2_lds = ring_lds + C::OFF_L2 + wc * C::L2W;
    auto pre = [&]() {
      if (RT > 0 && wr == 0) {
#pragma unroll
        for (int j = 0; j < 2; j++) {
          const int ct = min(n0 / 32 + 2 * wc + j, ctiles - 1);
#pragma unroll
          for (int rbk = 0; rbk < C::RB; rbk++)
            dma_s(lane * 16, uniform_ptr(l2codes + ((int64_t)ct * C::RB + rbk) * 1024),
                  l2_lds + (j * C::RB + rbk) * 1024);
        }
        // lane q < 8 RG: 8 scales of column tile j = q / (4 RG), rank group
        // (q / 4) % RG, columns 8 (q % 4) .. + 8
        const int q = lane & (8 * RG - 1);
        const int jj = q / (4 * RG), hg = (q / 4) % RG;
        const int ct = min(n0 / 32 + 2 * wc + jj, ctiles - 1);
        dma_v(reinterpret_cast<const uint8_t *>(l2scales + (int64_t)hg * geo.n_pad + ct * 32 +
                                                8 * (q & 3)),
              l2_lds + 2 * C::RB * 1024);
      }
    };
    if (wave == 0) K::template main_loop_pp<true, true, GK>(P, smem, ring_lds, KG, lane, wr, wc, acc, pre);
    else if (wr == 0) K::template main_loop_pp<true, false, GK>(P, smem, ring_lds, KG, lane, wr, wc, acc, pre);
    else K::template main_loop_pp<false, false, GK>(P, smem, ring_lds, KG, lane, wr, wc, acc, pre);

    // ---- stage 2 (Q_H Q(L2)) and the single epilogue ----
    // (the index values are re-derived here, behind an opaque copy, so the
    // compiler does not keep per-row addresses alive across the K loop)
    int lane_e = lane, m0_e = m0;
    asm volatile("" : "+v"(lane_e), "+s"(m0_e));
    const int l32e = lane_e & 31;
#pragma unroll
    for (int i = 0; i < 2; i++) {
      const int ti = 2 * wr + i;   // token tile within the block
#pragma unroll
      for (int j = 0; j < 2; j++) {
        const int ct = n0 / 32 + 2 * wc + j;
        const bool cvalid = ct < ctiles;
        v16f ylr = v16f{0};
        if constexpr (RT > 0) {
          const uint8_t *QS = smem + C::OFF_Q;
          const float *SHS = reinterpret_cast<const float *>(smem + C::OFF_SH);
          const uint8_t *L2S = smem + C::OFF_L2 + wc * C::L2W;
          // one rescale per rank group: a 128-rank group first adds its two
          // 64-rank blocks' exact integer sums in the matrix core
#pragma unroll
          for (int hg = 0; hg < RG; hg++) {
            v16f cbv;
#pragma unroll
            for (int bb = 0; bb < BPG; bb++) {
              const int rbk = hg * BPG + bb;
              const uint8_t *qrow = QS + (32 * ti + l32e) * C::QSTR + rbk * 64 + (lane_e >> 5) * 32;
              const v8i qa = join(*reinterpret_cast<const u32x4 *>(qrow),
                                  *reinterpret_cast<const u32x4 *>(qrow + 16));
              const v8i lb = unpack32(*reinterpret_cast<const u32x4 *>(
                  L2S + (j * C::RB + rbk) * 1024 + lane_e * 16));
              if (bb == 0) {
                cbv = mfma_codes_32x32x64(qa, lb);
              } else {
                cbv = mfma_codes_32x32x64_acc(qa, lb, cbv);
              }
            }
            const float sl2 = half_bits_to_float(*reinterpret_cast<const uint16_t *>(
                L2S + 2 * C::RB * 1024 + ((j * RG + hg) * 32 + l32e) * 2));
            const float *shrow = SHS + hg * PBM + 32 * ti + 4 * (lane_e >> 5);
#pragma unroll
            for (int q = 0; q < 4; q++) {
              const v4f sh4 = *reinterpret_cast<const v4f *>(shrow + 8 * q);
#pragma unroll
              for (int e = 0; e < 4; e++) {
                const int v = 4 * q + e;
                ylr[v] = fmaf(cbv[v], sh4[e] * sl2, ylr[v]);
              }
            }
          }
        }
        // the matrix-core products above read operands from every lane: keep
        // them out of the per-lane store branch below
        asm volatile("" : "+v"(ylr));
        const int col = ct * 32 + l32e;
        if (cvalid && col < geo.n) {
#pragma unroll
          for (int v = 0; v < 16; v++) {
            const int row = m0_e + 32 * ti + row_of_32x32(lane_e, v);
            if (row < m) {
              const float yv = acc[i][j][v] + ylr[v];
              const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
              reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
            }
          }
        }
      }
    }
    wait_vm<0>();      // stores drained before the next block's loads are counted
    __syncthreads();   // the next block refills the ring
  }
}

template <int RT, int D, int GK>
hipError_t launch_prefill(const GemmArgs &a, hipStream_t s) {
  using C = PCfg<RT, D>;
  const int m_tiles = (a.m + PBM - 1) / PBM;
  const int n_tiles = (a.geo.n_pad + PBN - 1) / PBN;
  // column blocks per work-group: the fewest that fit the grid in one round
  // over the 256 CUs (one work-group per CU), so no second round runs a few
  // leftover work-groups alone (m_tiles > 256: one run of all column blocks)
  const int runs = m_tiles >= 256 ? 1 : 256 / m_tiles;
  int cpw = (n_tiles + runs - 1) / runs;
  if (cpw > n_tiles) cpw = n_tiles;
  const int n_chunks = (n_tiles + cpw - 1) / cpw;
  const int band = m_tiles < 8 ? m_tiles : 8;   // token blocks per band of the XCD order
  auto kern = dual_gemm_prefill_kernel<RT, D, GK>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(m_tiles * n_chunks), dim3(64 * PNW), C::LDS, s, a, m_tiles,
                     n_tiles, n_chunks, cpw, band);
  return hipGetLastError();
}

template <int D, int GK>
hipError_t launch_prefill_rt(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.r_pad32 / 32) {
    case 0: return launch_prefill<0, D, GK>(a, s);
    case 1: return launch_prefill<1, D, GK>(a, s);
    case 2: return launch_prefill<2, D, GK>(a, s);
    case 4: return launch_prefill<4, D - 1, GK>(a, s);   // the larger Q_H and stage-2 region leave D - 1 slots
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_dual_gemm_prefill(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.gk) {
    case 1: return launch_prefill_rt<8, 1>(a, s);
    case 2: return launch_prefill_rt<8, 2>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tq
