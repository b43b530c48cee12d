// Activation quantizer, weight packing and weight export kernels.
//
// Quantizer: paper Sec. 2 Eq. (1) with q_max = 7, one fp16 scale per group of
// 64 or 128 consecutive values along the reduction axis (Sec. 5.1), round half
// to even, codes clamped to [-7, 7], an all-zero group gets scale 0.  Codes
// are stored in 64-wide K blocks whatever the group; a 128-wide group spans two
// blocks and has one scale.
#include "tq_device.hpp"
#include "tq_kernels.hpp"

namespace tq {

// ---------------------------------------------------------------------------
// Activations: one work-group of 4 wavefronts per quantization group (GK
// consecutive 1 KiB matrix-core blocks) of one token tile, or per QPW
// consecutive groups (the fp8 output of 64-wide groups).  Wavefront
// w takes tokens 8 w .. 8 w + 7 of the tile; for each of the GK blocks, lane
// 8 j + 4 h + l quantizes codes 32 h + 8 l .. + 7 of the group for token
// 8 w + j (16 bytes of the row) into one TQ4 word, and the 8 lanes of a token
// share the group max through three DPP lane swizzles.  All GK loads of a
// lane are issued before any is used.  TQ4 output (m <= kMidMaxTokens): token
// 32 t + i, codes 32 h .. 32 h + 31 of group g land at byte
// ((t * KG + g) * 64 + 32 h + i) * 16 (the lane order of one matrix-core
// operand), so each wavefront stores two contiguous 128-byte runs per block.
// fp8 output (larger m): the same operand as 32 fp8 bytes per lane, split into
// two 1 KiB halves -- bytes 16 p .. 16 p + 15 of lane slot 32 h + i at byte
// ((t * KG + g) * 2 + p) * 1024 + (32 h + i) * 16 -- so each half is one
// 16-byte-per-lane wave load and one conflict-free LDS read.  The padding
// tokens [m, m32) of the last tile get zero codes.  Scales are stored
// group-major with the token count padded to m32 (padding entries are zero).
// ---------------------------------------------------------------------------
// (max8_dpp and quant8_fp8, the per-lane quantizer step, are in tq_device.hpp:
// the decode kernel quantizes fp16 activations with the same code.)

template <bool FP8, int GK, int QPW = 1>
__global__ __launch_bounds__(256) void quant_act_kernel(const uint16_t *__restrict__ x, int m,
                                                        int k, uint32_t *__restrict__ codes,
                                                        uint16_t *__restrict__ scales) {
  // QPW consecutive quantization groups of GK 64-wide blocks each: a group's
  // max spans its blocks
  const int KG = k / kGroup;
  const int t = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int j = lane >> 3, h = (lane >> 2) & 1, l = lane & 3;
  const int i = 8 * w + j;          // token within the tile
  const int row = 32 * t + i;
  const int m32 = (int)gridDim.y * 32;
  u32x4 raw[QPW][GK];
  // padding tokens read the last real row (m >= 1) and quantize zeros; every
  // load is issued before the first is used
  const bool live = row < m;
  const uint16_t *src = x + (int64_t)(live ? row : m - 1) * k + blockIdx.x * QPW * GK * kGroup + 32 * h + 8 * l;
#pragma unroll
  for (int u = 0; u < QPW; u++)
#pragma unroll
    for (int q = 0; q < GK; q++) raw[u][q] = *reinterpret_cast<const u32x4 *>(src + (u * GK + q) * kGroup);
#pragma unroll
  for (int u = 0; u < QPW; u++) {
    const int q0 = blockIdx.x * QPW + u, g0 = q0 * GK;
#pragma unroll
    for (int q = 0; q < GK; q++)
      if (!live) raw[u][q] = u32x4{0, 0, 0, 0};
    float v[GK][8];
    float amax = 0.0f;
#pragma unroll
    for (int q = 0; q < GK; q++) {
#pragma unroll
      for (int e = 0; e < 4; e++) {
        v[q][2 * e] = half_bits_to_float((uint16_t)(raw[u][q][e] & 0xffffu));
        v[q][2 * e + 1] = half_bits_to_float((uint16_t)(raw[u][q][e] >> 16));
      }
#pragma unroll
      for (int e = 0; e < 8; e++) amax = fmaxf(amax, fabsf(v[q][e]));
    }
    amax = max8_dpp(amax);
    uint16_t s16;
    const float s = q4_scale(amax, s16);
    const float y = s == 0.0f ? 0.0f : __builtin_amdgcn_rcpf(s);
#pragma unroll
    for (int q = 0; q < GK; q++) {
      const int g = g0 + q;   // the launch covers the K blocks exactly
      uint32_t b0, b1;
      quant8_fp8(v[q], s, y, b0, b1);
      if constexpr (FP8) {
        const int64_t off = (((int64_t)t * KG + g) * 2 + (l >> 1)) * 256 + (32 * h + i) * 4 + 2 * (l & 1);
        *reinterpret_cast<uint2 *>(codes + off) = make_uint2(b0, b1);
      } else {
        // TQ4 word: the inverse of tq4_to_fp8 (codes 4..7 rotated into the
        // bits 0x78787878 that codes 0..3 leave free)
        codes[(((int64_t)t * KG + g) * 64 + 32 * h + i) * 4 + l] = b0 | __builtin_amdgcn_alignbit(b1, b1, 28);
      }
    }
    if ((lane & 7) == 0) scales[(int64_t)q0 * m32 + row] = row < m ? s16 : (uint16_t)0;
  }
}

// Rows of x quantized into TQ4 words in the layout of the packed weight
// blocks: block (t, g) holds rows 32 t .. 32 t + 31 of K block g, and the
// scales are group-major with the row count padded to 32 -- the same layout as
// the packed W_res codes and scales, so the weight packing uses this launch.
static void launch_quant_rows_tq4(const uint16_t *x, int m, int k, int gk, uint32_t *codes,
                                  uint16_t *scales, hipStream_t s) {
  const int m32 = (m + 31) / 32 * 32;
  const dim3 grid((unsigned)(k / kGroup / gk), (unsigned)(m32 / 32));
  if (gk == 2) hipLaunchKernelGGL((quant_act_kernel<false, 2>), grid, dim3(256), 0, s, x, m, k, codes, scales);
  else hipLaunchKernelGGL((quant_act_kernel<false, 1>), grid, dim3(256), 0, s, x, m, k, codes, scales);
}

hipError_t launch_quant_act(const uint16_t *x, int m, int k, int gk, uint32_t *codes,
                            uint16_t *scales, hipStream_t s) {
  // TQ4 output (up to kMidMaxTokens tokens): one quantization group per
  // work-group (more groups per work-group measured slower there)
  if (!act_codes_fp8(m)) {
    launch_quant_rows_tq4(x, m, k, gk, codes, scales, s);
    return hipGetLastError();
  }
  const int m32 = (m + 31) / 32 * 32;
  const int kq = k / kGroup / gk;   // quantization groups per row
  // 64-wide groups: four groups per work-group with all loads of a lane
  // issued first (more bytes in flight per work-group: the 70B down layer's
  // 8192 x 28672 activations quantize in 140-143 us instead of 149-154 us;
  // no change at the smaller sizes, 2 % slower for 128-wide groups)
  if (gk == 1 && kq % 4 == 0) {
    const dim3 grid((unsigned)(kq / 4), (unsigned)(m32 / 32));
    hipLaunchKernelGGL((quant_act_kernel<true, 1, 4>), grid, dim3(256), 0, s, x, m, k, codes, scales);
    return hipGetLastError();
  }
  const dim3 grid((unsigned)kq, (unsigned)(m32 / 32));
  if (gk == 2) hipLaunchKernelGGL((quant_act_kernel<true, 2>), grid, dim3(256), 0, s, x, m, k, codes, scales);
  else hipLaunchKernelGGL((quant_act_kernel<true, 1>), grid, dim3(256), 0, s, x, m, k, codes, scales);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight packing.  W_res rows go through the activation quantizer's TQ4 path
// (launch_quant_rows_tq4), whose output is the packed block layout.  The
// strided vectors -- columns of L1 and of L2 -- take one thread per (vector,
// group): it quantizes its group and writes the codes into the two 16-byte
// lane slots of its block plus the scale.  Vectors past the real sizes
// (padding to 32 columns / 64 ranks) get zero codes and zero scales, so every
// byte of the packed buffer is written.
// ---------------------------------------------------------------------------
// The fp16 scale of `len` values at src with the given element stride (0 if
// !present), and the TQ4 words of the 64 of them starting at element e0
// (codes past len are zero).
__device__ __forceinline__ float group_scale_strided(const uint16_t *src, int64_t stride, int len,
                                                     bool present, uint16_t &s16) {
  float amax = 0.0f;
  if (present)
    for (int i = 0; i < len; i++) amax = fmaxf(amax, fabsf(half_bits_to_float(src[i * stride])));
  return q4_scale(amax, s16);
}
__device__ __forceinline__ void codes_strided(const uint16_t *src, int64_t stride, int len, int e0,
                                              bool present, float s, uint32_t out[8]) {
  for (int wd = 0; wd < 8; wd++) {
    int c[8];
    for (int i = 0; i < 8; i++) {
      const int e = e0 + wd * 8 + i;
      c[i] = (present && e < len) ? q4_code(half_bits_to_float(src[e * stride]), s) : 0;
    }
    out[wd] = tq4_pack8(c);
  }
}

// W_res [n][k] rows and L1 [k][r] columns share the block format: one thread
// per (vector, quantization group of gk 64-wide blocks).
__global__ __launch_bounds__(256) void pack_kgroups_kernel(const uint16_t *__restrict__ src,
                                                           int64_t vec_stride, int64_t elem_stride,
                                                           int nvec, int nvec_pad, int kblocks, int gk,
                                                           uint8_t *__restrict__ codes,
                                                           uint16_t *__restrict__ scales) {
  const int kq = kblocks / gk;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)nvec_pad * kq) return;
  const int g = (int)(t % kq);
  const int v = (int)(t / kq);
  const bool present = v < nvec;
  const int len = gk * kGroup;
  const uint16_t *p = present ? src + (int64_t)v * vec_stride + (int64_t)g * len * elem_stride : src;
  uint16_t s16;
  const float s = group_scale_strided(p, elem_stride, len, present, s16);
  for (int b = 0; b < gk; b++) {
    uint32_t w[8];
    codes_strided(p, elem_stride, len, b * kGroup, present, s, w);
    uint8_t *blk = codes + ((int64_t)(v >> 5) * kblocks + g * gk + b) * 1024;
    const int c = v & 31;
    *reinterpret_cast<u32x4 *>(blk + c * 16) = u32x4{w[0], w[1], w[2], w[3]};
    *reinterpret_cast<u32x4 *>(blk + (32 + c) * 16) = u32x4{w[4], w[5], w[6], w[7]};
  }
  scales[(int64_t)g * nvec_pad + v] = s16;
}

// L2 [r][n]: column n along the rank axis, one 64-rank block per thread.  A
// rank group is gr <= 64 ranks inside the block, or (gr = 128) two blocks,
// whose threads each compute the group's scale and code their own half.
__global__ __launch_bounds__(256) void pack_l2_kernel(const uint16_t *__restrict__ l2, int n,
                                                      int n_pad, int r, int gr, int rblocks,
                                                      uint8_t *__restrict__ codes,
                                                      uint16_t *__restrict__ scales) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)n_pad * rblocks) return;
  const int rb = (int)(t % rblocks);
  const int col = (int)(t / rblocks);
  const bool present = col < n;
  uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  const int j0 = rb * 64;
  if (gr > 64) {
    const int jg = j0 / gr * gr;
    const uint16_t *p = present ? l2 + (int64_t)jg * n + col : l2;
    uint16_t s16;
    const float s = group_scale_strided(p, n, gr, present, s16);
    codes_strided(p, n, gr, j0 - jg, present, s, w);
    if (j0 == jg) scales[(int64_t)(jg / gr) * n_pad + col] = s16;
  } else {
    const int jend = r < j0 + 64 ? r : j0 + 64;
    for (int jg = j0; jg < jend; jg += gr) {
      uint32_t part[8];
      uint16_t s16;
      const uint16_t *p = present ? l2 + (int64_t)jg * n + col : l2;
      const float s = group_scale_strided(p, n, gr, present, s16);
      codes_strided(p, n, gr, 0, present, s, part);
      const int w0 = (jg - j0) / 8;
      for (int i = 0; i < gr / 8; i++) w[w0 + i] = part[i];
      scales[(int64_t)(jg / gr) * n_pad + col] = s16;
    }
  }
  uint8_t *blk = codes + ((int64_t)(col >> 5) * rblocks + rb) * 1024;
  const int c = col & 31;
  *reinterpret_cast<u32x4 *>(blk + c * 16) = u32x4{w[0], w[1], w[2], w[3]};
  *reinterpret_cast<u32x4 *>(blk + (32 + c) * 16) = u32x4{w[4], w[5], w[6], w[7]};
}

static unsigned nblocks(int64_t threads) { return (unsigned)((threads + 255) / 256); }

// Zero n16 16-byte words (the slack after a section).
__global__ __launch_bounds__(256) void zero16_kernel(uint8_t *__restrict__ p, int64_t n16) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t < n16) *reinterpret_cast<u32x4 *>(p + 16 * t) = u32x4{0u, 0u, 0u, 0u};
}

hipError_t launch_pack(const Geometry &g, const uint16_t *w, const uint16_t *l1,
                       const uint16_t *l2, uint8_t *packed, hipStream_t s) {
  const int kg = g.k / kGroup, kq = kg / g.gk;   // 64-wide blocks, quantization groups
  // W_res rows: the quantizer of activation rows writes exactly this block
  // layout (n_pad = n rounded up to 32; padding rows get zero codes and scales)
  launch_quant_rows_tq4(w, g.n, g.k, g.gk, reinterpret_cast<uint32_t *>(packed + g.off_w),
                        reinterpret_cast<uint16_t *>(packed + g.off_ws), s);
  // the slack read past the last K block: 1 KiB of codes, one scale row
  hipLaunchKernelGGL(zero16_kernel, dim3(1), dim3(256), 0, s,
                     packed + g.off_w + (uint64_t)g.n_pad / 32 * kg * 1024, (int64_t)64);
  hipLaunchKernelGGL(zero16_kernel, dim3(nblocks(g.n_pad / 8)), dim3(256), 0, s,
                     packed + g.off_ws + (uint64_t)kq * g.n_pad * 2, (int64_t)g.n_pad / 8);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.r == 0) return e;
  hipLaunchKernelGGL(zero16_kernel, dim3(1), dim3(256), 0, s,
                     packed + g.off_l1 + (uint64_t)g.r_pad32 / 32 * kg * 1024, (int64_t)64);
  hipLaunchKernelGGL(zero16_kernel, dim3(1), dim3(256), 0, s,
                     packed + g.off_l1s + (uint64_t)kq * g.r_pad32 * 2, (int64_t)g.r_pad32 / 8);
  hipLaunchKernelGGL(pack_kgroups_kernel, dim3(nblocks((int64_t)g.r_pad32 * kq)), dim3(256), 0,
                     s, l1, (int64_t)1, (int64_t)g.r, g.r, g.r_pad32, kg, g.gk, packed + g.off_l1,
                     reinterpret_cast<uint16_t *>(packed + g.off_l1s));
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rblocks = g.r_pad64 / 64;
  hipLaunchKernelGGL(pack_l2_kernel, dim3(nblocks((int64_t)g.n_pad * rblocks)), dim3(256), 0, s,
                     l2, g.n, g.n_pad, g.r, g.gr, rblocks, packed + g.off_l2,
                     reinterpret_cast<uint16_t *>(packed + g.off_l2s));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Export to the canonical layout (tests / debugging).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void export_kgroups_kernel(const uint8_t *__restrict__ codes,
                                                             const uint16_t *__restrict__ scales,
                                                             int nvec, int nvec_pad, int kblocks,
                                                             int gk, uint32_t *__restrict__ out_c,
                                                             uint16_t *__restrict__ out_s) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)nvec * kblocks) return;
  const int g = (int)(t % kblocks);
  const int v = (int)(t / kblocks);
  const uint8_t *blk = codes + ((int64_t)(v >> 5) * kblocks + g) * 1024;
  const int c = v & 31;
  const u32x4 a = *reinterpret_cast<const u32x4 *>(blk + c * 16);
  const u32x4 b = *reinterpret_cast<const u32x4 *>(blk + (32 + c) * 16);
  uint32_t *o = out_c + (int64_t)v * kblocks * 8 + g * 8;
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  const int kq = kblocks / gk;
  if (g % gk == 0) out_s[(int64_t)v * kq + g / gk] = scales[(int64_t)(g / gk) * nvec_pad + v];
}

__global__ __launch_bounds__(256) void export_l2_kernel(const uint8_t *__restrict__ codes,
                                                        const uint16_t *__restrict__ scales, int n,
                                                        int n_pad, int r, int gr, int rblocks,
                                                        uint32_t *__restrict__ out_c,
                                                        uint16_t *__restrict__ out_s) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)n * rblocks) return;
  const int rb = (int)(t % rblocks);
  const int col = (int)(t / rblocks);
  const uint8_t *blk = codes + ((int64_t)(col >> 5) * rblocks + rb) * 1024;
  const int c = col & 31;
  const u32x4 a = *reinterpret_cast<const u32x4 *>(blk + c * 16);
  const u32x4 b = *reinterpret_cast<const u32x4 *>(blk + (32 + c) * 16);
  const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  const int j0 = rb * 64;
  const int words = ((r < j0 + 64 ? r : j0 + 64) - j0) / 8;
  uint32_t *o = out_c + (int64_t)col * (r / 8) + j0 / 8;
  for (int i = 0; i < words; i++) o[i] = w[i];
  const int ng = r / gr;
  for (int jg = j0; jg < j0 + words * 8; jg += gr)
    out_s[(int64_t)col * ng + jg / gr] = scales[(int64_t)(jg / gr) * n_pad + col];
}

// ---------------------------------------------------------------------------
// Canonical layout: two's-complement nibbles, element 2 i in the low nibble
// and 2 i + 1 in the high nibble of byte i, contiguous along the reduction
// axis; scales as IEEE fp16 bit patterns.
// ---------------------------------------------------------------------------
// fp8 code byte (sign << 7 | |q|) -> the code's two's-complement nibble
__device__ __forceinline__ uint32_t fp8_code_to_nibble(uint32_t b) {
  const int m = (int)(b & 7u);
  return (uint32_t)((b & 0x80u) ? -m : m) & 0xfu;
}
// 8 codes (one TQ4 word) -> 4 canonical bytes
__device__ __forceinline__ uint32_t tq4_to_canonical(uint32_t w) {
  uint32_t lo, hi;
  tq4_to_fp8(w, lo, hi);   // bytes of codes 0..3, 4..7
  const uint32_t c[8] = {lo & 0xffu, (lo >> 8) & 0xffu, (lo >> 16) & 0xffu, lo >> 24,
                         hi & 0xffu, (hi >> 8) & 0xffu, (hi >> 16) & 0xffu, hi >> 24};
  uint32_t out = 0;
#pragma unroll
  for (int i = 0; i < 4; i++)
    out |= (fp8_code_to_nibble(c[2 * i]) | (fp8_code_to_nibble(c[2 * i + 1]) << 4)) << (8 * i);
  return out;
}

// W_res rows / L1 columns: one thread per (vector, 64-wide block).  Scales go
// to [vector][k / group] (vec_major) or [k / group][vector].
__global__ __launch_bounds__(256) void export_canonical_kgroups_kernel(
    const uint8_t *__restrict__ codes, const uint16_t *__restrict__ scales, int nvec, int nvec_pad,
    int kblocks, int gk, bool vec_major, uint8_t *__restrict__ out_q, uint16_t *__restrict__ out_s) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)nvec * kblocks) return;
  const int g = (int)(t % kblocks);
  const int v = (int)(t / kblocks);
  const uint8_t *blk = codes + ((int64_t)(v >> 5) * kblocks + g) * 1024;
  const int c = v & 31;
  const u32x4 a = *reinterpret_cast<const u32x4 *>(blk + c * 16);
  const u32x4 b = *reinterpret_cast<const u32x4 *>(blk + (32 + c) * 16);
  uint8_t *o = out_q + (int64_t)v * kblocks * 32 + g * 32;
  *reinterpret_cast<u32x4 *>(o) = u32x4{tq4_to_canonical(a.x), tq4_to_canonical(a.y),
                                        tq4_to_canonical(a.z), tq4_to_canonical(a.w)};
  *reinterpret_cast<u32x4 *>(o + 16) = u32x4{tq4_to_canonical(b.x), tq4_to_canonical(b.y),
                                             tq4_to_canonical(b.z), tq4_to_canonical(b.w)};
  const int kq = kblocks / gk;
  if (g % gk == 0) {
    const uint16_t sv = scales[(int64_t)(g / gk) * nvec_pad + v];
    if (vec_major) out_s[(int64_t)v * kq + g / gk] = sv;
    else out_s[(int64_t)(g / gk) * nvec + v] = sv;
  }
}

// L2 columns along the rank axis: one thread per (column, 64-rank block);
// codes [n][r / 2], scales [r / group_r][n].
__global__ __launch_bounds__(256) void export_canonical_l2_kernel(
    const uint8_t *__restrict__ codes, const uint16_t *__restrict__ scales, int n, int n_pad, int r,
    int gr, int rblocks, uint8_t *__restrict__ out_q, uint16_t *__restrict__ out_s) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)n * rblocks) return;
  const int rb = (int)(t % rblocks);
  const int col = (int)(t / rblocks);
  const uint8_t *blk = codes + ((int64_t)(col >> 5) * rblocks + rb) * 1024;
  const int c = col & 31;
  const u32x4 a = *reinterpret_cast<const u32x4 *>(blk + c * 16);
  const u32x4 b = *reinterpret_cast<const u32x4 *>(blk + (32 + c) * 16);
  const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  const int j0 = rb * 64;
  const int words = ((r < j0 + 64 ? r : j0 + 64) - j0) / 8;   // 8 ranks per word
  uint32_t *o = reinterpret_cast<uint32_t *>(out_q + (int64_t)col * (r / 2) + j0 / 2);
  for (int i = 0; i < words; i++) o[i] = tq4_to_canonical(w[i]);
  for (int jg = j0 / gr * gr; jg < j0 + words * 8; jg += gr)
    if (jg >= j0) out_s[(int64_t)(jg / gr) * n + col] = scales[(int64_t)(jg / gr) * n_pad + col];
}

// Activation codes (either tiled format) -> canonical [m][k / 2], scales
// [m][k / group]: one thread per (token, 64-wide block).
__global__ __launch_bounds__(256) void act_canonical_kernel(const uint8_t *__restrict__ x_codes,
                                                            const uint16_t *__restrict__ x_scales,
                                                            int m, int k, int gk, bool fp8,
                                                            uint8_t *__restrict__ out_q,
                                                            uint16_t *__restrict__ out_s) {
  const int KG = k / kGroup, m32 = (m + 31) / 32 * 32;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)m * KG) return;
  const int g = (int)(t % KG), row = (int)(t / KG);
  const int tile = row / 32, i = row % 32;
  uint32_t outw[8];
  if (fp8) {
    // block of 2 KiB: half p, lane slot 32 h + i holds bytes 16 p .. 16 p + 15
    // of codes 32 h .. 32 h + 31
    const uint8_t *blk = x_codes + ((int64_t)tile * KG + g) * 2048;
    for (int h = 0; h < 2; h++)
      for (int pp = 0; pp < 2; pp++) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(blk + pp * 1024 + (32 * h + i) * 16);
        const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
        for (int q = 0; q < 4; q++) {   // 4 codes -> 2 canonical bytes
          const uint32_t x = wv[q];
          const uint32_t b0 = fp8_code_to_nibble(x & 0xffu) | (fp8_code_to_nibble((x >> 8) & 0xffu) << 4);
          const uint32_t b1 = fp8_code_to_nibble((x >> 16) & 0xffu) | (fp8_code_to_nibble(x >> 24) << 4);
          const int e = 32 * h + 16 * pp + 4 * q;   // first code of the four
          const int wi = e / 8, sh = (e % 8) * 4;
          if (sh == 0) outw[wi] = b0 | (b1 << 8);
          else outw[wi] |= (b0 | (b1 << 8)) << 16;
        }
      }
  } else {
    const uint8_t *blk = x_codes + ((int64_t)tile * KG + g) * 1024;
    for (int h = 0; h < 2; h++) {
      const u32x4 v = *reinterpret_cast<const u32x4 *>(blk + (32 * h + i) * 16);
      outw[4 * h + 0] = tq4_to_canonical(v.x);
      outw[4 * h + 1] = tq4_to_canonical(v.y);
      outw[4 * h + 2] = tq4_to_canonical(v.z);
      outw[4 * h + 3] = tq4_to_canonical(v.w);
    }
  }
  uint8_t *o = out_q + (int64_t)row * (k / 2) + g * 32;
  *reinterpret_cast<u32x4 *>(o) = u32x4{outw[0], outw[1], outw[2], outw[3]};
  *reinterpret_cast<u32x4 *>(o + 16) = u32x4{outw[4], outw[5], outw[6], outw[7]};
  if (g % gk == 0) out_s[(int64_t)row * (KG / gk) + g / gk] = x_scales[(int64_t)(g / gk) * m32 + row];
}

hipError_t launch_export_canonical(const Geometry &g, const uint8_t *packed, uint8_t *wq, uint16_t *ws,
                                   uint8_t *l1q, uint16_t *l1s, uint8_t *l2q, uint16_t *l2s,
                                   hipStream_t s) {
  const int kg = g.k / kGroup;
  hipLaunchKernelGGL(export_canonical_kgroups_kernel, dim3(nblocks((int64_t)g.n * kg)), dim3(256), 0, s,
                     packed + g.off_w, reinterpret_cast<const uint16_t *>(packed + g.off_ws), g.n,
                     g.n_pad, kg, g.gk, true, wq, ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.r == 0) return e;
  hipLaunchKernelGGL(export_canonical_kgroups_kernel, dim3(nblocks((int64_t)g.r * kg)), dim3(256), 0, s,
                     packed + g.off_l1, reinterpret_cast<const uint16_t *>(packed + g.off_l1s), g.r,
                     g.r_pad32, kg, g.gk, false, l1q, l1s);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rblocks = g.r_pad64 / 64;
  hipLaunchKernelGGL(export_canonical_l2_kernel, dim3(nblocks((int64_t)g.n * rblocks)), dim3(256), 0, s,
                     packed + g.off_l2, reinterpret_cast<const uint16_t *>(packed + g.off_l2s), g.n,
                     g.n_pad, g.r, g.gr, rblocks, l2q, l2s);
  return hipGetLastError();
}

hipError_t launch_act_canonical(const uint8_t *x_codes, const uint16_t *x_scales, int m, int k, int gk,
                                uint8_t *out_q, uint16_t *out_s, hipStream_t s) {
  hipLaunchKernelGGL(act_canonical_kernel, dim3(nblocks((int64_t)m * (k / kGroup))), dim3(256), 0, s,
                     x_codes, x_scales, m, k, gk, act_codes_fp8(m), out_q, out_s);
  return hipGetLastError();
}

hipError_t launch_export(const Geometry &g, const uint8_t *packed, uint32_t *wc, uint16_t *ws,
                         uint32_t *l1c, uint16_t *l1s, uint32_t *l2c, uint16_t *l2s,
                         hipStream_t s) {
  const int kg = g.k / kGroup;
  hipLaunchKernelGGL(export_kgroups_kernel, dim3(nblocks((int64_t)g.n * kg)), dim3(256), 0, s,
                     packed + g.off_w, reinterpret_cast<const uint16_t *>(packed + g.off_ws), g.n,
                     g.n_pad, kg, g.gk, wc, ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || g.r == 0) return e;
  hipLaunchKernelGGL(export_kgroups_kernel, dim3(nblocks((int64_t)g.r * kg)), dim3(256), 0, s,
                     packed + g.off_l1, reinterpret_cast<const uint16_t *>(packed + g.off_l1s),
                     g.r, g.r_pad32, kg, g.gk, l1c, l1s);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rblocks = g.r_pad64 / 64;
  hipLaunchKernelGGL(export_l2_kernel, dim3(nblocks((int64_t)g.n * rblocks)), dim3(256), 0, s,
                     packed + g.off_l2, reinterpret_cast<const uint16_t *>(packed + g.off_l2s),
                     g.n, g.n_pad, g.r, g.gr, rblocks, l2c, l2s);
  return hipGetLastError();
}

}  // namespace tq
