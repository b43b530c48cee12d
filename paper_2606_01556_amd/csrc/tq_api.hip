// C ABI of libtq: argument validation on the host, then one or more kernel
// launches on the caller's stream.  No allocation and no synchronization.
// The only global state is the static scratch array of
// tq_dual_gemm_unfused_noalloc and its per-device address, looked up once.
#include <stdint.h>

#include <mutex>

#include "tq.h"
#include "tq_kernels.hpp"

namespace {

constexpr int32_t kMagic = 0x54513402;  // "TQ4" + layout version 2

inline bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

bool desc_ok(const tq_weight_desc *d) {
  return d != nullptr && d->magic == kMagic && (d->group == 64 || d->group == 128) &&
         d->k % d->group == 0 && d->n >= 1 &&
         d->n_pad == (int32_t)round_up((uint64_t)d->n, 32) &&
         d->r_pad32 == (int32_t)round_up((uint64_t)d->rank, 32) &&
         d->r_pad64 == (int32_t)round_up((uint64_t)d->rank, 64);
}

tq::Geometry geometry(const tq_weight_desc *d) {
  tq::Geometry g;
  g.n = d->n; g.k = d->k; g.r = d->rank; g.gr = d->group_r;
  g.gk = d->group / 64;
  g.n_pad = d->n_pad; g.r_pad32 = d->r_pad32; g.r_pad64 = d->r_pad64;
  g.off_w = d->off_w; g.off_ws = d->off_ws; g.off_l1 = d->off_l1;
  g.off_l1s = d->off_l1s; g.off_l2 = d->off_l2; g.off_l2s = d->off_l2s;
  return g;
}

tq_status hip_status(hipError_t e) { return e == hipSuccess ? TQ_OK : TQ_ERR_HIP; }

}  // namespace

extern "C" {

tq_status tq_weight_desc_init(int n, int k, int rank, int group, tq_weight_desc *out) {
  if (out == nullptr) return TQ_ERR_NULL;
  if (group != 64 && group != 128) return TQ_ERR_GROUP;
  if (n < 1 || k < 1 || n > (1 << 24) || k > (1 << 24)) return TQ_ERR_SHAPE;
  if (k % group != 0) return TQ_ERR_GROUP;
  if (!(rank == 0 || rank == 8 || rank == 16 || rank == 32 || rank == 64 || rank == 128))
    return TQ_ERR_RANK;
  tq_weight_desc d = {};
  d.n = n; d.k = k; d.rank = rank; d.group = group;
  d.group_r = rank == 0 ? 0 : (rank < group ? rank : group);
  d.n_pad = (int32_t)round_up((uint64_t)n, 32);
  d.r_pad32 = (int32_t)round_up((uint64_t)rank, 32);
  d.r_pad64 = (int32_t)round_up((uint64_t)rank, 64);
  d.magic = kMagic;
  const uint64_t kg = (uint64_t)k / 64;         // 64-wide code blocks along K
  const uint64_t kgs = (uint64_t)k / group;     // quantization groups along K
  uint64_t off = 0;
  // The code sections end in 1 KiB of zeros and the scale sections in one
  // row of zero scales: a kernel may read one K-group past the last, where
  // the activation codes are zero, and its products then add exactly zero.
  d.off_w = off;   off = round_up(off + (uint64_t)d.n_pad / 32 * kg * 1024 + 1024, 256);
  d.off_ws = off;  off = round_up(off + (kgs + 1) * (uint64_t)d.n_pad * 2, 256);
  d.off_l1 = off;  off = round_up(off + (uint64_t)d.r_pad32 / 32 * kg * 1024 + (rank ? 1024 : 0), 256);
  d.off_l1s = off; off = round_up(off + (rank ? kgs + 1 : 0) * (uint64_t)d.r_pad32 * 2, 256);
  d.off_l2 = off;  off = round_up(off + (uint64_t)d.n_pad / 32 * ((uint64_t)d.r_pad64 / 64) * 1024, 256);
  d.off_l2s = off;
  const uint64_t rgroups = rank == 0 ? 0 : (uint64_t)rank / (uint64_t)d.group_r;
  off = round_up(off + rgroups * (uint64_t)d.n_pad * 2, 256);
  d.packed_bytes = off;
  // the kernels form offsets inside one packed buffer in 32 bits
  if (off >= ((uint64_t)1 << 32)) return TQ_ERR_SHAPE;
  *out = d;
  return TQ_OK;
}

tq_status tq_pack_weights(const tq_weight_desc *d, const void *w_res, const void *l1,
                          const void *l2, void *packed, void *stream) {
  if (d == nullptr || w_res == nullptr || packed == nullptr) return TQ_ERR_NULL;
  if (!desc_ok(d)) return TQ_ERR_BUFFER;
  if (d->rank > 0 && (l1 == nullptr || l2 == nullptr)) return TQ_ERR_NULL;
  if (!aligned16(w_res) || !aligned16(packed) || (d->rank > 0 && (!aligned16(l1) || !aligned16(l2))))
    return TQ_ERR_ALIGN;
  return hip_status(tq::launch_pack(geometry(d), static_cast<const uint16_t *>(w_res),
                                    static_cast<const uint16_t *>(l1),
                                    static_cast<const uint16_t *>(l2),
                                    static_cast<uint8_t *>(packed),
                                    static_cast<hipStream_t>(stream)));
}

tq_status tq_quant_act(const void *x, int m, int k, int group, void *x_codes, void *x_scales,
                       void *stream) {
  if (x == nullptr || x_codes == nullptr || x_scales == nullptr) return TQ_ERR_NULL;
  if (group != 64 && group != 128) return TQ_ERR_GROUP;
  if (m < 0 || m > 65535 * 32 || k < 1 || k > (1 << 24)) return TQ_ERR_SHAPE;
  if (k % group != 0) return TQ_ERR_GROUP;
  if (!aligned16(x) || !aligned16(x_codes) || !aligned16(x_scales)) return TQ_ERR_ALIGN;
  if ((int64_t)m * k >= ((int64_t)1 << 40)) return TQ_ERR_SHAPE;
  if (m == 0) return TQ_OK;
  return hip_status(tq::launch_quant_act(static_cast<const uint16_t *>(x), m, k, group / 64,
                                         static_cast<uint32_t *>(x_codes),
                                         static_cast<uint16_t *>(x_scales),
                                         static_cast<hipStream_t>(stream)));
}

}  // extern "C"

namespace tq {
// Scratch memory of tq_dual_gemm_unfused_noalloc, for callers that cannot
// allocate: every device the library runs on holds one copy for the life of
// the process.  Host code uses it only through the device address that
// hipGetSymbolAddress returns for the device (static_scratch below).
__device__ __align__(256) uint8_t scratch[TQ_NOALLOC_SCRATCH_BYTES];
}  // namespace tq

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of the static scratch array on the device of `stream` (the
// current device for the NULL stream), looked up on the first call for that
// device with the device current, then cached.
hipError_t static_scratch(hipStream_t stream, void **out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr) {
    hipDevice_t sd = 0;
    e = hipStreamGetDevice(stream, &sd);
    if (e != hipSuccess) return e;
    dev = sd;
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(tq::scratch));
    if (dev != cur) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

enum class Path { Fused, Unfused, UnfusedStatic };

// What one layer call runs, beyond the common arguments.
struct Call {
  Path path = Path::Fused;
  void *scratch = nullptr;                     // Path::Unfused: the caller's scratch
  void *h = nullptr, *sh = nullptr, *qh = nullptr;   // optional copies of H, s_H, Q_H
  int kernel = -1, mid_ct = 0;                 // forced kernel / mid tile count (tests)
  const void *x16 = nullptr;                   // fp16 activations quantized in the kernel
};

}  // namespace

extern "C" {

static tq_status dual_gemm_impl(const tq_weight_desc *d, const void *packed, const void *x_codes,
                                const void *x_scales, int m, void *y, tq_dtype y_dtype,
                                void *stream, const Call &c) {
  const bool fq = c.x16 != nullptr;
  if (d == nullptr || packed == nullptr || y == nullptr) return TQ_ERR_NULL;
  if (!fq && (x_codes == nullptr || x_scales == nullptr)) return TQ_ERR_NULL;
  if (c.path == Path::Unfused && c.scratch == nullptr) return TQ_ERR_NULL;
  const int ndbg = (c.h != nullptr) + (c.sh != nullptr) + (c.qh != nullptr);
  if (ndbg != 0 && ndbg != 3) return TQ_ERR_NULL;
  if (!desc_ok(d)) return TQ_ERR_BUFFER;
  if (m < 0 || m > (1 << 24)) return TQ_ERR_SHAPE;
  if (y_dtype != TQ_F16 && y_dtype != TQ_BF16) return TQ_ERR_DTYPE;
  if (ndbg == 3 && d->rank == 0) return TQ_ERR_RANK;
  if (!aligned16(packed) || !aligned16(x_codes) || !aligned16(x_scales) || !aligned16(y) ||
      !aligned16(c.scratch) || !aligned16(c.x16))
    return TQ_ERR_ALIGN;
  if (ndbg == 3 && (!aligned16(c.h) || !aligned16(c.sh) || !aligned16(c.qh))) return TQ_ERR_ALIGN;
  if (fq && m > 0 && (m > tq::kDecodeMaxTokens || !tq::decode_fits(m, d->k))) return TQ_ERR_SHAPE;
  if (c.kernel < -1 || c.kernel > tq::kKernelPrefill) return TQ_ERR_SHAPE;
  if (c.mid_ct != 0 && c.mid_ct != 1 && c.mid_ct != 2 && c.mid_ct != 4) return TQ_ERR_SHAPE;
  if (m > 0) {
    // a forced kernel must be one that serves m tokens
    if (c.kernel == tq::kKernelDecode && (m > tq::kDecodeMaxTokens || !tq::decode_fits(m, d->k)))
      return TQ_ERR_SHAPE;
    if ((c.kernel == tq::kKernelLarge || c.kernel == tq::kKernelPrefill) && !tq::act_codes_fp8(m))
      return TQ_ERR_SHAPE;
  }
  if (c.path == Path::UnfusedStatic &&
      tq::unfused_scratch_bytes(m, geometry(d)) > (size_t)TQ_NOALLOC_SCRATCH_BYTES)
    return TQ_ERR_TOO_LARGE;
  if (m == 0) return TQ_OK;
  tq::GemmArgs a{};
  a.packed = static_cast<const uint8_t *>(packed);
  a.geo = geometry(d);
  a.xc = static_cast<const uint32_t *>(x_codes);
  a.xs = static_cast<const uint16_t *>(x_scales);
  a.y = y;
  a.m = m;
  a.ms = (m + 31) / 32 * 32;
  a.bf16_out = y_dtype == TQ_BF16;
  a.dbg_h = static_cast<float *>(c.h);
  a.dbg_sh = static_cast<float *>(c.sh);
  a.dbg_qh = static_cast<int8_t *>(c.qh);
  a.force_kernel = c.kernel;
  a.mid_ct = c.mid_ct;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (fq) return hip_status(tq::launch_dual_gemm_decode(a, static_cast<const uint16_t *>(c.x16), s));
  if (c.path == Path::Unfused) return hip_status(tq::launch_dual_gemm_unfused(a, c.scratch, s));
  if (c.path == Path::UnfusedStatic) {
    void *scr = nullptr;
    if (static_scratch(s, &scr) != hipSuccess) return TQ_ERR_HIP;
    return hip_status(tq::launch_dual_gemm_unfused(a, scr, s));
  }
  return hip_status(tq::launch_dual_gemm(a, s));
}

int tq_dual_gemm_kernel(const tq_weight_desc *d, int m) {
  if (d == nullptr || !desc_ok(d) || m < 1 || m > (1 << 24)) return -1;
  tq::GemmArgs a{};
  a.geo = geometry(d);
  a.m = m;
  a.ms = (m + 31) / 32 * 32;
  a.force_kernel = -1;
  return tq::choose_kernel(a);
}

size_t tq_act_codes_bytes(int m, int k) {
  if (m < 0 || m > 65535 * 32 || k < 1 || k > (1 << 24) || k % 64 != 0) return 0;
  return tq::act_codes_bytes(m, k);
}

tq_status tq_dual_gemm(const tq_weight_desc *d, const void *packed, const void *x_codes,
                       const void *x_scales, int m, void *y, tq_dtype y_dtype, void *stream) {
  return dual_gemm_impl(d, packed, x_codes, x_scales, m, y, y_dtype, stream, Call{});
}

tq_status tq_dual_gemm_fused_quant(const tq_weight_desc *d, const void *packed, const void *x,
                                   int m, void *y, tq_dtype y_dtype, void *stream) {
  if (x == nullptr) return TQ_ERR_NULL;
  Call c;
  c.x16 = x;
  return dual_gemm_impl(d, packed, nullptr, nullptr, m, y, y_dtype, stream, c);
}

tq_status tq_dual_gemm_debug(const tq_weight_desc *d, const void *packed, const void *x_codes,
                             const void *x_scales, const void *x, int m, void *y, tq_dtype y_dtype,
                             int kernel, int mid_tiles, void *h, void *sh, void *qh, void *stream) {
  Call c;
  if (x != nullptr) {
    // the fused-quantization path: no codes, and only the decode kernel
    if (x_codes != nullptr || x_scales != nullptr) return TQ_ERR_SHAPE;
    if (kernel != -1 && kernel != tq::kKernelDecode) return TQ_ERR_SHAPE;
    c.x16 = x;
  }
  c.kernel = kernel;
  c.mid_ct = mid_tiles;
  c.h = h;
  c.sh = sh;
  c.qh = qh;
  return dual_gemm_impl(d, packed, x_codes, x_scales, m, y, y_dtype, stream, c);
}

size_t tq_unfused_scratch_bytes(const tq_weight_desc *d, int m) {
  if (!desc_ok(d) || m < 0 || m > (1 << 24)) return 0;
  return tq::unfused_scratch_bytes(m, geometry(d));
}

tq_status tq_dual_gemm_unfused(const tq_weight_desc *d, const void *packed, const void *x_codes,
                               const void *x_scales, int m, void *y, tq_dtype y_dtype,
                               void *scratch, void *stream) {
  Call c;
  c.path = Path::Unfused;
  c.scratch = scratch;
  return dual_gemm_impl(d, packed, x_codes, x_scales, m, y, y_dtype, stream, c);
}

tq_status tq_dual_gemm_unfused_noalloc(const tq_weight_desc *d, const void *packed,
                                       const void *x_codes, const void *x_scales, int m, void *y,
                                       tq_dtype y_dtype, void *stream) {
  Call c;
  c.path = Path::UnfusedStatic;
  return dual_gemm_impl(d, packed, x_codes, x_scales, m, y, y_dtype, stream, c);
}

tq_status tq_export_weights(const tq_weight_desc *d, const void *packed, void *w_codes,
                            void *w_scales, void *l1_codes, void *l1_scales, void *l2_codes,
                            void *l2_scales, void *stream) {
  if (d == nullptr || packed == nullptr || w_codes == nullptr || w_scales == nullptr)
    return TQ_ERR_NULL;
  if (!desc_ok(d)) return TQ_ERR_BUFFER;
  if (d->rank > 0 && (!l1_codes || !l1_scales || !l2_codes || !l2_scales)) return TQ_ERR_NULL;
  if (!aligned16(packed) || !aligned16(w_codes) || !aligned16(w_scales)) return TQ_ERR_ALIGN;
  if (d->rank > 0 && (!aligned16(l1_codes) || !aligned16(l1_scales) || !aligned16(l2_codes) ||
                      !aligned16(l2_scales)))
    return TQ_ERR_ALIGN;
  return hip_status(tq::launch_export(
      geometry(d), static_cast<const uint8_t *>(packed), static_cast<uint32_t *>(w_codes),
      static_cast<uint16_t *>(w_scales), static_cast<uint32_t *>(l1_codes),
      static_cast<uint16_t *>(l1_scales), static_cast<uint32_t *>(l2_codes),
      static_cast<uint16_t *>(l2_scales), static_cast<hipStream_t>(stream)));
}

tq_status tq_export_weights_canonical(const tq_weight_desc *d, const void *packed, void *wq, void *ws,
                                      void *l1q, void *l1s, void *l2q, void *l2s, void *stream) {
  if (d == nullptr || packed == nullptr || wq == nullptr || ws == nullptr) return TQ_ERR_NULL;
  if (!desc_ok(d)) return TQ_ERR_BUFFER;
  if (d->rank > 0 && (!l1q || !l1s || !l2q || !l2s)) return TQ_ERR_NULL;
  if (!aligned16(packed) || !aligned16(wq) || !aligned16(ws)) return TQ_ERR_ALIGN;
  if (d->rank > 0 && (!aligned16(l1q) || !aligned16(l1s) || !aligned16(l2q) || !aligned16(l2s)))
    return TQ_ERR_ALIGN;
  return hip_status(tq::launch_export_canonical(
      geometry(d), static_cast<const uint8_t *>(packed), static_cast<uint8_t *>(wq),
      static_cast<uint16_t *>(ws), static_cast<uint8_t *>(l1q), static_cast<uint16_t *>(l1s),
      static_cast<uint8_t *>(l2q), static_cast<uint16_t *>(l2s), static_cast<hipStream_t>(stream)));
}

tq_status tq_act_codes_canonical(const void *x_codes, const void *x_scales, int m, int k, int group,
                                 void *codes_out, void *scales_out, void *stream) {
  if (x_codes == nullptr || x_scales == nullptr || codes_out == nullptr || scales_out == nullptr)
    return TQ_ERR_NULL;
  if (group != 64 && group != 128) return TQ_ERR_GROUP;
  if (m < 0 || m > 65535 * 32 || k < 1 || k > (1 << 24)) return TQ_ERR_SHAPE;
  if (k % group != 0) return TQ_ERR_GROUP;
  if (!aligned16(x_codes) || !aligned16(x_scales) || !aligned16(codes_out) || !aligned16(scales_out))
    return TQ_ERR_ALIGN;
  if (m == 0) return TQ_OK;
  return hip_status(tq::launch_act_canonical(static_cast<const uint8_t *>(x_codes),
                                             static_cast<const uint16_t *>(x_scales), m, k, group / 64,
                                             static_cast<uint8_t *>(codes_out),
                                             static_cast<uint16_t *>(scales_out),
                                             static_cast<hipStream_t>(stream)));
}

const char *tq_status_string(tq_status s) {
  switch (s) {
    case TQ_OK: return "ok";
    case TQ_ERR_NULL: return "a required pointer is NULL";
    case TQ_ERR_SHAPE: return "size out of range";
    case TQ_ERR_GROUP: return "unsupported group size or k not a multiple of it";
    case TQ_ERR_RANK: return "unsupported rank";
    case TQ_ERR_DTYPE: return "unknown output dtype";
    case TQ_ERR_ALIGN: return "device pointer not 16-byte aligned";
    case TQ_ERR_BUFFER: return "weight descriptor not initialised or inconsistent";
    case TQ_ERR_HIP: return "HIP runtime error on launch";
    case TQ_ERR_TOO_LARGE: return "the call needs more scratch memory than the static buffer holds";
  }
  return "unknown status";
}

}  // extern "C"
