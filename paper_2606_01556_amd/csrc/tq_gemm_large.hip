// Fused dual-component W4A4 layer (paper Sec. 4.3) for large token counts:
// the residual 4-bit GEMM, the stage-1 product H = Q(X) Q(L1) kept on chip,
// its on-the-fly re-quantization, stage 2 Q_H Q(L2) and one epilogue, in one
// kernel.
//
// Work decomposition.  A work-group of 16 wavefronts (four per SIMD) owns a
// block of 128 tokens x 256 columns.  Wavefront w = 8 tp + cc computes the
// two 32 x 32 output tiles of token tiles 2 tp and 2 tp + 1 and column tile
// cc, so it expands one weight operand per group and reads its two activation
// operands ready-made: at these token counts the activation codes arrive as
// fp8 operand bytes, and the kernel is bound by vector-ALU work (4-bit
// expansion and the per-group rescaling fmas).  The 4 x RT tiles of H
// (RT = r / 32 rounded up) are spread over the wavefronts so that every SIMD
// forms the same number, in the same K loop.  Each tile walks the K-groups in
// ascending order with one fma per group, the oracle's order, so H, Q_H and Y
// are bit-identical to it.  Four wavefronts per SIMD with one tile in flight
// each hide the latency of the matrix-core results better than fewer
// wavefronts with more tiles.
//
// Per tile and group (Eq. 2): v_mfma_scale_f32_32x32x64_f8f6f4 returns half
// of the exact integer group sum (codes as fp8 subnormals), v_mfma_f32_32x32x8
// f16 twice the exact scale product, and one fma per element applies their
// product, exactly I * s_x * s_w.
//
// Data movement: everything a K-group needs -- 4 activation tiles (2 KiB
// each), 8 weight tiles, RT L1 tiles and all their scales -- arrives by direct
// global -> LDS loads (global_load_lds_dwordx4) into a D-slot ring, one 1 KiB
// wave load per wavefront and group (two for the first 2 + RT wavefronts), so
// every wait is one constant s_waitcnt.  A step consumes two K-groups behind
// one work-group barrier and refills their slots D groups ahead.  The stage-2
// operands (L2 blocks and scales of the 8 column tiles) are loaded at the
// start into a region of their own.

#include <type_traits>

#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {
namespace {

typedef _Float16 v4h __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int LW = 16;       // wavefronts per work-group
constexpr int LBM = 128;     // tokens per block (4 tiles)
constexpr int LBN = 256;     // columns per block (8 tiles)
constexpr int L_LDS = 160 * 1024;

template <int RT>
struct LCfg {
  static constexpr int RB = (RT + 1) / 2;              // 64-rank blocks (= rank groups)
  // one ring slot (one K-group)
  static constexpr int S_A = 0;                        // 4 activation tiles x 2 halves
  static constexpr int S_B = 8192;                     // 8 weight tiles
  static constexpr int S_L = 16384;                    // RT L1 tiles
  static constexpr int S_SX = S_L + RT * 1024;         // activation scales (256 B used)
  static constexpr int S_SW = S_SX + 1024;             // weight scales 512 B, then L1 64 RT B
  static constexpr int SLOT = S_SW + 1024;
  static constexpr int NI = 18 + RT;                   // wave loads per group
  // stage-2 operands: 8 x RB L2 blocks, then their scales
  static constexpr int L2B = RT > 0 ? 8 * RB * 1024 + 1024 : 0;
  static constexpr int DFIT = (L_LDS - L2B) / SLOT;
  static constexpr int D = DFIT > 8 ? 8 : DFIT;        // ring slots
  static constexpr int OFF_L2 = D * SLOT;
  static constexpr int LDS = OFF_L2 + L2B;
  // epilogue (aliases the ring)
  static constexpr int HSTR = RT * 32 + 1;
  static constexpr int QSTR = (RB > 0 ? RB : 1) * 64 + 16;
  static constexpr int E_HS = 0;                                   // [128][HSTR] fp32
  static constexpr int E_QS = E_HS + LBM * HSTR * 4;               // [128][QSTR] fp8 codes
  static constexpr int E_SH = E_QS + LBM * QSTR;                   // [RB][128] fp32
  static constexpr int E_END = E_SH + (RB > 0 ? RB : 1) * LBM * 4;
  static_assert(LDS <= L_LDS, "fits the 160 KiB LDS of a CU");
  static_assert(E_END <= D * SLOT, "the epilogue fits in the ring");
  static_assert(NI <= 2 * LW, "at most two wave loads per wavefront and group");
  static_assert(D >= 4, "two groups consumed per step, two more in flight");
};

template <int N>
__device__ __forceinline__ void lwait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt has 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xf) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// 16 bytes per lane from addr into LDS at lds + 16 * lane
__device__ __forceinline__ void ldma(const uint8_t *addr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(addr), "s"(lds)
               : "memory");
}

// the same with a wave-uniform base and a 32-bit lane offset
__device__ __forceinline__ void ldma_s(uint32_t voff, const uint8_t *sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory");
}

// a wave-uniform pointer, kept in scalar registers
__device__ __forceinline__ const uint8_t *l_uniform(const uint8_t *p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t *>(((uint64_t)hi << 32) | lo);
}

// one fp8 activation operand: the lane's two 16-byte halves, 1 KiB apart
__device__ __forceinline__ v8i l_v8h(const uint8_t *p) {
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(p);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(p + 1024);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

__device__ __forceinline__ v8i l_v8i(const uint8_t *p) {
  const u32x4 lo = *reinterpret_cast<const u32x4 *>(p);
  const u32x4 hi = *reinterpret_cast<const u32x4 *>(p + 16);
  return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// 2 * s_row * s_col of a 32x32 tile (both scales in k = 0 and k = 4)
__device__ __forceinline__ v16f l_outer2(uint32_t sa, uint32_t sb) {
  const v16f z = {0};
  const u32x2 a2 = {sa, 0u}, b2 = {sb, 0u};
  return __builtin_amdgcn_mfma_f32_32x32x8f16(__builtin_bit_cast(v4h, a2),
                                              __builtin_bit_cast(v4h, b2), z, 0, 0, 0);
}

// half of the exact integer group sum of a 32x32 tile of code products
__device__ __forceinline__ v16f l_codes_half(v8i a, v8i b) {
  const v16f z = {0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, z, 0, 0, 0, kScale2p9 - 1, 0,
                                                         kScale2p9);
}
// the same added to c (the second block of a 128-wide group: exact)
__device__ __forceinline__ v16f l_codes_half_acc(v8i a, v8i b, v16f c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, kScale2p9 - 1, 0,
                                                         kScale2p9);
}

// A wave load of one 64-wide K block g: lane reads 16 bytes at base + off +
// (g >> shift) * stride (base wave-uniform, off and stride per lane) into LDS
// at slot + dst + 16 * lane.  Scale rows are per quantization group, so scale
// items shift by log2(group / 64); each slot holds its block's group scales.
struct LItem {
  const uint8_t *base;
  uint32_t off, stride;
  uint32_t dst;          // offset within a slot
  int shift;
};

template <int RT>
__device__ __forceinline__ LItem l_item(const GemmArgs &a, int it, int lane, int m0, int n0) {
  using C = LCfg<RT>;
  const Geometry &geo = a.geo;
  const int KG = geo.k / kGroup;
  LItem d;
  d.shift = it < 16 + RT ? 0 : geo.gk - 1;
  if (it < 8) {                       // activation tile it / 2, half it % 2 (fp8 bytes)
    const int t = min(m0 / 32 + it / 2, a.ms / 32 - 1);
    d.base = reinterpret_cast<const uint8_t *>(a.xc) + (int64_t)t * KG * 2048 + (it & 1) * 1024;
    d.off = lane * 16;
    d.stride = 2048;
    d.dst = C::S_A + it * 1024;
  } else if (it < 16) {               // weight tile it - 8
    const int ct = min(n0 / 32 + it - 8, geo.n_pad / 32 - 1);
    d.base = a.packed + geo.off_w + (int64_t)ct * KG * 1024;
    d.off = lane * 16;
    d.stride = 1024;
    d.dst = C::S_B + (it - 8) * 1024;
  } else if (it < 16 + RT) {          // L1 rank tile it - 16
    d.base = a.packed + geo.off_l1 + (int64_t)(it - 16) * KG * 1024;
    d.off = lane * 16;
    d.stride = 1024;
    d.dst = C::S_L + (it - 16) * 1024;
  } else if (it == 16 + RT) {         // activation scales of the 128 tokens: lanes 0-15
    const int l = lane < 16 ? lane : 0;   // other lanes repeat lane 0's piece into their own place
    d.base = reinterpret_cast<const uint8_t *>(a.xs);
    d.off = (uint32_t)min(m0 + 8 * l, a.ms - 8) * 2;
    d.stride = (uint32_t)a.ms * 2;
    d.dst = C::S_SX;
  } else {                            // weight scales (lanes 0-31), L1 scales (32 ..)
    int l = lane;
    if (l >= 32 + 4 * RT) l = 0;      // spare lanes repeat lane 0's piece into their own place
    d.base = a.packed;
    if (l < 32) {
      d.off = (uint32_t)(geo.off_ws + (uint64_t)min(n0 + 8 * l, geo.n_pad - 8) * 2);
      d.stride = (uint32_t)geo.n_pad * 2;
    } else {
      d.off = (uint32_t)(geo.off_l1s + (uint64_t)(8 * (l - 32)) * 2);
      d.stride = (uint32_t)geo.r_pad32 * 2;
    }
    d.dst = C::S_SW;
  }
  return d;
}

// GK: 64-wide K blocks per quantization group (1 or 2, the descriptor's
// group / 64), a template parameter so that each variant keeps its registers
template <int RT, int GK>
__global__ __launch_bounds__(64 * LW, 1) void dual_gemm_large_kernel(GemmArgs a, int m_tiles,
                                                                     int n_tiles, int band) {
  using C = LCfg<RT>;
  constexpr int D = C::D;
  extern __shared__ __attribute__((aligned(1024))) uint8_t smem[];
  const Geometry &geo = a.geo;
  const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int tp = wave >> 3, cc = wave & 7;   // token tile pair, column tile
  const int KG = geo.k / kGroup;
  const int m = a.m;
  const int ct32 = geo.n_pad / 32;
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)smem);

  // Work-groups are dealt round-robin to the 8 XCDs: give each XCD a
  // contiguous run of logical ids, ordered in bands of `band` token blocks,
  // column block by column block, so the work-groups of an XCD share their
  // activation rows and weight columns in its L2.
  int logical;
  {
    const int nwg = gridDim.x, per = nwg / 8, rem = nwg % 8;
    const int x = blockIdx.x % 8, s = blockIdx.x / 8;
    logical = (x < rem ? x * (per + 1) : rem * (per + 1) + (x - rem) * per) + s;
  }
  const int bsz = band * n_tiles;
  const int bidx = logical / bsz, brem = logical % bsz;
  const int rows_in_band = min(band, m_tiles - bidx * band);
  const int nb = brem / rows_in_band;
  const int mb = bidx * band + brem % rows_in_band;
  const int m0 = mb * LBM, n0 = nb * LBN;

  // ---- this wavefront's loads: item `wave`, and for wavefronts below
  // NI - 16 also item wave + 16 ----
  const LItem it0 = l_item<RT>(a, wave, lane, m0, n0);
  const bool two = wave + LW < C::NI;

  // stage-2 operands: wavefront j < 8 the L2 blocks of column tile j,
  // wavefront 8 the L2 scales of the 8 tiles
  auto stage2_loads = [&]() {
    if constexpr (RT > 0) {
      if (wave < 8) {
        const int ct = min(n0 / 32 + wave, ct32 - 1);
#pragma unroll
        for (int rb = 0; rb < C::RB; rb++)
          ldma(a.packed + geo.off_l2 + (((int64_t)ct * C::RB + rb) * 64 + lane) * 16,
               lds0 + C::OFF_L2 + (wave * C::RB + rb) * 1024);
      } else if (wave == 8) {
        const int q = lane < 8 * C::RB * 4 ? lane : 0;   // 4 pieces per (rank group, tile)
        const int h = q / 32, j = (q / 4) % 8, part = q % 4;
        const int col = min(n0 + 32 * j + 8 * part, geo.n_pad - 8);
        const int hg = h * 64 / geo.gr;   // rank group of 64-rank block h (gr >= 64 here)
        ldma(a.packed + geo.off_l2s + ((int64_t)hg * geo.n_pad + col) * 2,
             lds0 + C::OFF_L2 + 8 * C::RB * 1024);
      }
    }
  };

  // H tiles: wavefront w runs on SIMD w mod 4 = cc mod 4.  RT = 1: the four
  // tiles (ti, 0) go to wavefronts (tp, cc) = (ti / 2, ti); RT = 2: tile
  // (2 tp + cc / 2, cc % 2) to wavefront (tp, cc < 4); RT = 4: tile
  // (2 tp + cc % 2, cc / 2) to every wavefront -- the same number per SIMD.
  // The token tile of this wavefront's H tile is its first tile tA, the other
  // one tB.
  int hsel = 0, hrt = 0;
  bool hw = false;
  if constexpr (RT == 1) { hw = cc < 4 && tp == (cc >> 1); hsel = cc & 1; }
  if constexpr (RT == 2) { hw = cc < 4; hsel = (cc >> 1) & 1; hrt = cc & 1; }
  if constexpr (RT == 4) { hw = true; hsel = cc & 1; hrt = cc >> 1; }
  const int tA = 2 * tp + hsel, tB = 2 * tp + 1 - hsel;
  v16f acc0 = v16f{0}, acc1 = v16f{0}, hacc = v16f{0};

  auto k_loop = [&](auto PC, auto HC) {
    constexpr int PER = decltype(PC)::value;   // wave loads per group
    constexpr bool HW = decltype(HC)::value;   // this wavefront forms an H tile
    auto issue = [&](int g) {
      const uint32_t slot = lds0 + (g % D) * C::SLOT;
      ldma_s(it0.off + (uint32_t)(GK == 1 ? g : g >> it0.shift) * it0.stride, l_uniform(it0.base), slot + it0.dst);
      if constexpr (PER == 2) {
        const LItem it1 = l_item<RT>(a, wave + LW, lane, m0, n0);
        ldma_s(it1.off + (uint32_t)(GK == 1 ? g : g >> it1.shift) * it1.stride, l_uniform(it1.base), slot + it1.dst);
      }
    };
    auto group = [&](int g) {
      const uint8_t *S = smem + (g % D) * C::SLOT;
      const v8i a0 = l_v8h(S + C::S_A + tA * 2048 + lane * 16);
      const v8i a1 = l_v8h(S + C::S_A + tB * 2048 + lane * 16);
      const uint32_t sa0 = *reinterpret_cast<const uint16_t *>(S + C::S_SX + (32 * tA + l32) * 2);
      const uint32_t sa1 = *reinterpret_cast<const uint16_t *>(S + C::S_SX + (32 * tB + l32) * 2);
      const v8i b = unpack32(*reinterpret_cast<const u32x4 *>(S + C::S_B + cc * 1024 + lane * 16));
      const uint32_t sb = *reinterpret_cast<const uint16_t *>(S + C::S_SW + (32 * cc + l32) * 2);
      {
        const v16f c = l_codes_half(a0, b);
        const v16f p = l_outer2(sa0, sb);
#pragma unroll
        for (int v = 0; v < 16; v++) acc0[v] = fmaf(c[v], p[v], acc0[v]);
      }
      {
        const v16f c = l_codes_half(a1, b);
        const v16f p = l_outer2(sa1, sb);
#pragma unroll
        for (int v = 0; v < 16; v++) acc1[v] = fmaf(c[v], p[v], acc1[v]);
      }
      if constexpr (HW) {
        const v8i bl = unpack32(*reinterpret_cast<const u32x4 *>(S + C::S_L + hrt * 1024 + lane * 16));
        const uint32_t sl = *reinterpret_cast<const uint16_t *>(S + C::S_SW + 512 + (32 * hrt + l32) * 2);
        const v16f c = l_codes_half(a0, bl);
        const v16f p = l_outer2(sa0, sl);
#pragma unroll
        for (int v = 0; v < 16; v++) hacc[v] = fmaf(c[v], p[v], hacc[v]);
      }
    };
    // a 128-wide group (blocks g and g + 1): each tile's two half sums add
    // exactly in the matrix core, then one fma per element (the oracle's step)
    auto group2 = [&](int g) {
      const uint8_t *S0 = smem + (g % D) * C::SLOT;
      const uint8_t *S1 = smem + ((g + 1) % D) * C::SLOT;
      const uint32_t sb = *reinterpret_cast<const uint16_t *>(S0 + C::S_SW + (32 * cc + l32) * 2);
      const v8i b0 = unpack32(*reinterpret_cast<const u32x4 *>(S0 + C::S_B + cc * 1024 + lane * 16));
      const v8i b1 = unpack32(*reinterpret_cast<const u32x4 *>(S1 + C::S_B + cc * 1024 + lane * 16));
      // one tile at a time, each finished before the next starts (registers)
      auto tile = [&](int t, const v8i &w0, const v8i &w1, uint32_t sw, v16f &acc) {
        const uint32_t sx = *reinterpret_cast<const uint16_t *>(S0 + C::S_SX + (32 * t + l32) * 2);
        const v16f c = l_codes_half_acc(l_v8h(S1 + C::S_A + t * 2048 + lane * 16), w1,
                                        l_codes_half(l_v8h(S0 + C::S_A + t * 2048 + lane * 16), w0));
        const v16f p = l_outer2(sx, sw);
#pragma unroll
        for (int v = 0; v < 16; v++) acc[v] = fmaf(c[v], p[v], acc[v]);
      };
      tile(tA, b0, b1, sb, acc0);
      tile(tB, b0, b1, sb, acc1);
      if constexpr (HW) {
        const v8i l0 = unpack32(*reinterpret_cast<const u32x4 *>(S0 + C::S_L + hrt * 1024 + lane * 16));
        const v8i l1 = unpack32(*reinterpret_cast<const u32x4 *>(S1 + C::S_L + hrt * 1024 + lane * 16));
        const uint32_t sl = *reinterpret_cast<const uint16_t *>(S0 + C::S_SW + 512 + (32 * hrt + l32) * 2);
        tile(tA, l0, l1, sl, hacc);
      }
    };
    lwait_vm<0>();
    stage2_loads();
    for (int s = 0; s < D - 2; s++)
      if (s < KG) issue(s);
    for (int g2 = 0; g2 < KG; g2 += 2) {
      // groups g2 and g2 + 1 have landed (loads complete in issue order; near
      // the end of K fewer groups are in flight, so everything is waited for)
      if (g2 + D - 3 < KG) lwait_vm<(D - 4) * PER>();
      else lwait_vm<0>();
      __syncthreads();   // groups g2, g2 + 1 are visible; g2 - 2, g2 - 1 are consumed everywhere
      if (g2 + D - 2 < KG) issue(g2 + D - 2);   // into group g2 - 2's slot
      if (g2 + D - 1 < KG) issue(g2 + D - 1);   // into group g2 - 1's slot
      if constexpr (GK == 2) {
        group2(g2);   // K is a multiple of 128 here
      } else {
        group(g2);
        if (g2 + 1 < KG) group(g2 + 1);
      }
    }
  };
  if constexpr (RT == 0) {
    if (two) k_loop(std::integral_constant<int, 2>{}, std::false_type{});
    else k_loop(std::integral_constant<int, 1>{}, std::false_type{});
  } else {
    if (two && hw) k_loop(std::integral_constant<int, 2>{}, std::true_type{});
    else if (two) k_loop(std::integral_constant<int, 2>{}, std::false_type{});
    else if (hw) k_loop(std::integral_constant<int, 1>{}, std::true_type{});
    else k_loop(std::integral_constant<int, 1>{}, std::false_type{});
  }
  __syncthreads();   // every wavefront is done with the ring

  // ---- H -> LDS, re-quantization per token and rank group (s_H in fp32) ----
  float *HS = reinterpret_cast<float *>(smem + C::E_HS);
  uint8_t *QS = smem + C::E_QS;
  float *SHS = reinterpret_cast<float *>(smem + C::E_SH);
  if constexpr (RT > 0) {
    if (hw) {
#pragma unroll
      for (int v = 0; v < 16; v++) HS[(32 * tA + row_of_32x32(lane, v)) * C::HSTR + 32 * hrt + l32] = hacc[v];
    }
    const int r = geo.r, gr = geo.gr, rg = r / gr;
    if (r < C::RB * 64)
      for (int idx = tid; idx < LBM * C::RB * 64; idx += 64 * LW) {
        const int row = idx / (C::RB * 64), j = idx % (C::RB * 64);
        if (j >= r) QS[row * C::QSTR + j] = 0;
      }
    __syncthreads();
    const int subs = gr / 8;                // lanes per (token, rank group): 1, 2, 4 or 8
    const int work = LBM * rg * subs;       // <= 2048
    const bool dbg = a.dbg_h != nullptr && nb == 0;
    for (int base = 0; base < work; base += 64 * LW) {
      const int idx = base + tid;
      const bool valid = idx < work;
      const int pair = idx / subs, sub = idx % subs;
      const int row = pair / rg, hg = pair % rg;
      const int j0 = hg * gr + sub * 8;
      const int grow = m0 + row;
      float hv[8];
      float amax = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        hv[e] = valid ? HS[row * C::HSTR + j0 + e] : 0.0f;
        amax = fmaxf(amax, fabsf(hv[e]));
      }
      for (int msk = 1; msk < subs; msk <<= 1) amax = fmaxf(amax, __shfl_xor(amax, msk));
      const float shv = amax / 7.0f;   // IEEE division
      if (valid) {
        uint32_t w0 = 0, w1 = 0;
#pragma unroll
        for (int e = 0; e < 8; e++) {
          int qv = 0;
          if (shv != 0.0f) {
            float tq = __builtin_rintf(hv[e] / shv);
            tq = tq > 7.0f ? 7.0f : (tq < -7.0f ? -7.0f : tq);
            qv = (int)tq;
          }
          const uint32_t bq = code_to_fp8(qv);
          if (e < 4) w0 |= bq << (8 * e); else w1 |= bq << (8 * (e - 4));
          if (dbg && grow < m) {
            a.dbg_h[(int64_t)grow * r + j0 + e] = hv[e];
            a.dbg_qh[(int64_t)grow * r + j0 + e] = (int8_t)qv;
          }
        }
        *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0) = w0;
        *reinterpret_cast<uint32_t *>(QS + row * C::QSTR + j0 + 4) = w1;
        if (sub == 0) {
          SHS[hg * LBM + row] = shv;
          if (dbg && grow < m) a.dbg_sh[(int64_t)grow * rg + hg] = shv;
        }
      }
    }
    __syncthreads();
  }

  // ---- stage 2 and the single epilogue: this wavefront's two tiles ----
#pragma unroll
  for (int j = 0; j < 2; j++) {
    const int ti = j == 0 ? tA : tB;    // token tile within the block
    const int jt = cc;                  // column tile within the block
    const int ct = n0 / 32 + jt;
    v16f ylr = v16f{0};
    if constexpr (RT > 0) {
      const uint8_t *L2S = smem + C::OFF_L2;
      // one fma per rank group (the oracle's step): a 128-rank group (r = 128
      // in 128-wide groups) first adds its two 64-rank blocks' exact integer
      // sums in the matrix core
      constexpr int bpg = RT == 4 && GK == 2 ? 2 : 1;   // 64-rank blocks per rank group
#pragma unroll
      for (int hg = 0; hg < C::RB / bpg; hg++) {
        v16f cbv = v16f{0};
#pragma unroll
        for (int q = 0; q < bpg; q++) {
          const int rb = hg * bpg + q;
          const v8i qa = l_v8i(QS + (32 * ti + l32) * C::QSTR + rb * 64 + (lane >> 5) * 32);
          const v8i lb = unpack32(*reinterpret_cast<const u32x4 *>(L2S + (jt * C::RB + rb) * 1024 + lane * 16));
          cbv = q == 0 ? mfma_codes_32x32x64(qa, lb) : mfma_codes_32x32x64_acc(qa, lb, cbv);
        }
        const float sl2 = half_bits_to_float(*reinterpret_cast<const uint16_t *>(
            L2S + 8 * C::RB * 1024 + ((hg * bpg * 8 + jt) * 32 + l32) * 2));
#pragma unroll
        for (int v = 0; v < 16; v++)
          ylr[v] = fmaf(cbv[v], SHS[hg * LBM + 32 * ti + row_of_32x32(lane, v)] * sl2, ylr[v]);
      }
    }
    // the matrix-core products above read operands from every lane: keep
    // them out of the per-lane store branch below
    asm volatile("" : "+v"(ylr));
    const v16f &acc = j == 0 ? acc0 : acc1;
    const int col = ct * 32 + l32;
    if (ct < ct32 && col < geo.n) {
#pragma unroll
      for (int v = 0; v < 16; v++) {
        const int row = m0 + 32 * ti + row_of_32x32(lane, v);
        if (row < m) {
          const float yv = acc[v] + ylr[v];
          const uint16_t bits = a.bf16_out ? float_to_bf16_bits(yv) : float_to_half_bits(yv);
          reinterpret_cast<uint16_t *>(a.y)[(int64_t)row * geo.n + col] = bits;
        }
      }
    }
  }
}

template <int RT, int GK>
hipError_t launch_large(const GemmArgs &a, hipStream_t s) {
  using C = LCfg<RT>;
  const int m_tiles = (a.m + LBM - 1) / LBM;
  const int n_tiles = (a.geo.n_pad + LBN - 1) / LBN;
  const int band = m_tiles < 8 ? m_tiles : 8;   // token blocks per band of the XCD order
  auto kern = dual_gemm_large_kernel<RT, GK>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(m_tiles * n_tiles), dim3(64 * LW), C::LDS, s, a, m_tiles, n_tiles,
                     band);
  return hipGetLastError();
}

template <int GK>
hipError_t launch_large_rt(const GemmArgs &a, hipStream_t s) {
  switch (a.geo.r_pad32 / 32) {
    case 0: return launch_large<0, GK>(a, s);
    case 1: return launch_large<1, GK>(a, s);
    case 2: return launch_large<2, GK>(a, s);
    case 4: return launch_large<4, GK>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_dual_gemm_large(const GemmArgs &a, hipStream_t s) {
  return a.geo.gk == 2 ? launch_large_rt<2>(a, s) : launch_large_rt<1>(a, s);
}

}  // namespace tq
