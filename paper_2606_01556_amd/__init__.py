"""TwinQuant dual-component W4A4 linear layer on AMD MI355X (gfx950).

Thin Python binding of ``libtq.so`` (C ABI in ``include/tq.h``).  Every step of
the layer runs in the library's HIP kernels; this module only marshals
arguments (device pointers from torch tensors, the current HIP stream) and
turns non-zero status codes into exceptions.  It never computes the layer
itself and has no CPU fallback: if the library is missing it raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtq.so")
GROUP = 64

TQ_F16, TQ_BF16 = 0, 1
STATUS = {0: "TQ_OK", 1: "TQ_ERR_NULL", 2: "TQ_ERR_SHAPE", 3: "TQ_ERR_GROUP", 4: "TQ_ERR_RANK",
          5: "TQ_ERR_DTYPE", 6: "TQ_ERR_ALIGN", 7: "TQ_ERR_BUFFER", 8: "TQ_ERR_HIP",
          9: "TQ_ERR_TOO_LARGE"}
NOALLOC_SCRATCH_BYTES = 8 << 20   # TQ_NOALLOC_SCRATCH_BYTES


class TQError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {STATUS.get(code, code)} ({lib().tq_status_string(code).decode()})")


class WeightDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("group", ctypes.c_int32), ("group_r", ctypes.c_int32), ("n_pad", ctypes.c_int32),
                ("r_pad32", ctypes.c_int32), ("r_pad64", ctypes.c_int32), ("magic", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("packed_bytes", ctypes.c_uint64),
                ("off_w", ctypes.c_uint64), ("off_ws", ctypes.c_uint64), ("off_l1", ctypes.c_uint64),
                ("off_l1s", ctypes.c_uint64), ("off_l2", ctypes.c_uint64), ("off_l2s", ctypes.c_uint64)]


EXPORTS = ("tq_weight_desc_init", "tq_pack_weights", "tq_quant_act", "tq_dual_gemm",
           "tq_dual_gemm_fused_quant", "tq_dual_gemm_debug", "tq_export_weights",
           "tq_act_codes_bytes", "tq_unfused_scratch_bytes", "tq_dual_gemm_unfused",
           "tq_dual_gemm_unfused_noalloc", "tq_dual_gemm_kernel", "tq_status_string",
           "tq_export_weights_canonical", "tq_act_codes_canonical")

_lib = None


def lib() -> ctypes.CDLL:
    """Load libtq.so (built by ``paper_2606_01556_amd.build``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_01556_amd.build` (there is no fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P, I = ctypes.c_void_p, ctypes.c_int
        D = ctypes.POINTER(WeightDesc)
        L.tq_weight_desc_init.argtypes = [I, I, I, I, D]
        L.tq_pack_weights.argtypes = [D, P, P, P, P, P]
        L.tq_quant_act.argtypes = [P, I, I, I, P, P, P]
        L.tq_dual_gemm.argtypes = [D, P, P, P, I, P, I, P]
        L.tq_dual_gemm_fused_quant.argtypes = [D, P, P, I, P, I, P]
        L.tq_dual_gemm_debug.argtypes = [D, P, P, P, P, I, P, I, I, I, P, P, P, P]
        L.tq_act_codes_bytes.argtypes = [I, I]
        L.tq_act_codes_bytes.restype = ctypes.c_size_t
        L.tq_dual_gemm_kernel.argtypes = [D, I]
        L.tq_dual_gemm_kernel.restype = I
        L.tq_unfused_scratch_bytes.argtypes = [D, I]
        L.tq_unfused_scratch_bytes.restype = ctypes.c_size_t
        L.tq_dual_gemm_unfused.argtypes = [D, P, P, P, I, P, I, P, P]
        L.tq_dual_gemm_unfused_noalloc.argtypes = [D, P, P, P, I, P, I, P]
        L.tq_export_weights.argtypes = [D, P, P, P, P, P, P, P, P]
        L.tq_export_weights_canonical.argtypes = [D, P, P, P, P, P, P, P, P]
        L.tq_act_codes_canonical.argtypes = [P, P, I, I, I, P, P, P]
        L.tq_status_string.argtypes = [I]
        L.tq_status_string.restype = ctypes.c_char_p
        for name in EXPORTS:
            if name not in ("tq_act_codes_bytes", "tq_unfused_scratch_bytes",
                            "tq_dual_gemm_kernel", "tq_status_string"):
                getattr(L, name).restype = I
        _lib = L
    return _lib


def _check(code: int, where: str):
    if code != 0:
        raise TQError(code, where)


def _ptr(t):
    """Device pointer of a torch tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------ argument checks
# Every wrapper below checks its tensors before the C call: the library sees
# only raw pointers and would read or write out of bounds on a wrong shape.
def _tensor(t, name, dtype=None, shape=None, min_bytes=None):
    if t is None:
        raise ValueError(f"{name}: missing")
    if isinstance(t, int):
        return                          # a raw device address: the caller vouches for it
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if min_bytes is not None and t.numel() * t.element_size() < min_bytes:
        raise ValueError(f"{name}: {t.numel() * t.element_size()} bytes, needs {min_bytes}")


def _act_checks(desc, x_codes, x_scales, m):
    k = desc.k
    _tensor(x_codes, "x_codes", min_bytes=act_codes_bytes(m, k))
    _tensor(x_scales, "x_scales", min_bytes=(k // desc.group) * padded_tokens(m) * 2)


def _y_check(desc, y, m, bf16):
    import torch
    _tensor(y, "y", torch.bfloat16 if bf16 else torch.float16, (m, desc.n))


# ------------------------------------------------------------------ C ABI
def weight_desc_init(n: int, k: int, rank: int, group: int = GROUP) -> WeightDesc:
    d = WeightDesc()
    _check(lib().tq_weight_desc_init(n, k, rank, group, ctypes.byref(d)), "tq_weight_desc_init")
    return d


def pack_weights(desc: WeightDesc, w_res, l1, l2, packed, stream=None):
    import torch
    f16 = torch.float16
    _tensor(w_res, "w_res", f16, (desc.n, desc.k))
    if desc.rank:
        _tensor(l1, "l1", f16, (desc.k, desc.rank))
        _tensor(l2, "l2", f16, (desc.rank, desc.n))
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    _check(lib().tq_pack_weights(ctypes.byref(desc), _ptr(w_res), _ptr(l1), _ptr(l2), _ptr(packed),
                                 _stream(stream)), "tq_pack_weights")


def quant_act(x, x_codes, x_scales, group: int = GROUP, stream=None):
    import torch
    _tensor(x, "x", torch.float16)
    if x.dim() != 2:
        raise ValueError(f"x: expected [m, k], got shape {tuple(x.shape)}")
    m, k = x.shape
    _tensor(x_codes, "x_codes", min_bytes=act_codes_bytes(m, k))
    _tensor(x_scales, "x_scales", min_bytes=(k // group) * padded_tokens(m) * 2)
    _check(lib().tq_quant_act(_ptr(x), m, k, group, _ptr(x_codes), _ptr(x_scales), _stream(stream)),
           "tq_quant_act")


def dual_gemm(desc: WeightDesc, packed, x_codes, x_scales, m: int, y, bf16: bool = False,
              stream=None):
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    _act_checks(desc, x_codes, x_scales, m)
    _y_check(desc, y, m, bf16)
    _check(lib().tq_dual_gemm(ctypes.byref(desc), _ptr(packed), _ptr(x_codes), _ptr(x_scales), m,
                              _ptr(y), TQ_BF16 if bf16 else TQ_F16, _stream(stream)),
           "tq_dual_gemm")


def dual_gemm_fused_quant(desc: WeightDesc, packed, x, y, bf16: bool = False, stream=None):
    """The fused layer from fp16 activations x [m, k], quantized inside the
    kernel (decode-sized m; tq_dual_gemm_fused_quant)."""
    import torch
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    _tensor(x, "x", torch.float16)
    if x.dim() != 2 or x.shape[1] != desc.k:
        raise ValueError(f"x: expected [m, {desc.k}], got shape {tuple(x.shape)}")
    m = x.shape[0]
    _y_check(desc, y, m, bf16)
    _check(lib().tq_dual_gemm_fused_quant(ctypes.byref(desc), _ptr(packed), _ptr(x), m, _ptr(y),
                                          TQ_BF16 if bf16 else TQ_F16, _stream(stream)),
           "tq_dual_gemm_fused_quant")


def unfused_scratch_bytes(desc: WeightDesc, m: int) -> int:
    return int(lib().tq_unfused_scratch_bytes(ctypes.byref(desc), m))


def empty_unfused_scratch(desc: WeightDesc, m: int, device="cuda"):
    import torch
    return torch.empty(unfused_scratch_bytes(desc, m), dtype=torch.uint8, device=device)


def unfused_parts(desc: WeightDesc, m: int, scratch):
    """Views of (H [m32, r_pad32] fp32, Q_H codes [m32, r_pad64] uint8, s_H
    [r/group_r, m32] fp32) inside a tq_dual_gemm_unfused scratch buffer."""
    import torch
    m32 = padded_tokens(m)
    up = lambda v: (v + 255) // 256 * 256
    r, r32, r64, gr = desc.rank, desc.r_pad32, desc.r_pad64, desc.group_r
    o1 = up(m32 * r32 * 4)
    o2 = o1 + up(m32 * r64)
    h = scratch[:m32 * r32 * 4].view(torch.float32).view(m32, r32)
    qh = scratch[o1:o1 + m32 * r64].view(m32, r64)
    sh = scratch[o2:o2 + (r // gr) * m32 * 4].view(torch.float32).view(r // gr, m32)
    return h, qh, sh


def dual_gemm_unfused(desc: WeightDesc, packed, x_codes, x_scales, m: int, y, scratch,
                      bf16: bool = False, stream=None):
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    _act_checks(desc, x_codes, x_scales, m)
    _y_check(desc, y, m, bf16)
    _tensor(scratch, "scratch", min_bytes=unfused_scratch_bytes(desc, m))
    _check(lib().tq_dual_gemm_unfused(ctypes.byref(desc), _ptr(packed), _ptr(x_codes), _ptr(x_scales),
                                      m, _ptr(y), TQ_BF16 if bf16 else TQ_F16, _ptr(scratch),
                                      _stream(stream)), "tq_dual_gemm_unfused")


def dual_gemm_unfused_noalloc(desc: WeightDesc, packed, x_codes, x_scales, m: int, y,
                              bf16: bool = False, stream=None):
    """tq_dual_gemm_unfused with the library's static scratch (allocates nothing)."""
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    _act_checks(desc, x_codes, x_scales, m)
    _y_check(desc, y, m, bf16)
    _check(lib().tq_dual_gemm_unfused_noalloc(ctypes.byref(desc), _ptr(packed), _ptr(x_codes),
                                              _ptr(x_scales), m, _ptr(y), TQ_BF16 if bf16 else TQ_F16,
                                              _stream(stream)), "tq_dual_gemm_unfused_noalloc")


KERNEL_NAMES = ("decode", "mid", "large", "prefill")


def dual_gemm_debug(desc: WeightDesc, packed, x_codes, x_scales, m: int, y, h=None, sh=None, qh=None,
                    bf16: bool = False, kernel: str | None = None, mid_tiles: int = 0, x=None,
                    stream=None):
    """tq_dual_gemm_debug: the fused layer with an optional forced kernel
    (one of KERNEL_NAMES) and mid-kernel tile count, and optional copies of
    H [m, r] fp32, s_H [m, r/group_r] fp32 and Q_H [m, r] int8.  With x (fp16
    [m, k]) instead of x_codes / x_scales it runs the fused-quantization
    path of tq_dual_gemm_fused_quant."""
    import torch
    _tensor(packed, "packed", min_bytes=int(desc.packed_bytes))
    if x is None:
        _act_checks(desc, x_codes, x_scales, m)
    else:
        _tensor(x, "x", torch.float16, (m, desc.k))
    _y_check(desc, y, m, bf16)
    if h is not None or sh is not None or qh is not None:
        r = desc.rank
        _tensor(h, "h", torch.float32, (m, r))
        _tensor(sh, "sh", torch.float32, (m, r // max(desc.group_r, 1)))
        _tensor(qh, "qh", torch.int8, (m, r))
    kid = -1 if kernel is None else KERNEL_NAMES.index(kernel)
    _check(lib().tq_dual_gemm_debug(ctypes.byref(desc), _ptr(packed), _ptr(x_codes), _ptr(x_scales),
                                    _ptr(x), m, _ptr(y), TQ_BF16 if bf16 else TQ_F16, kid, mid_tiles,
                                    _ptr(h), _ptr(sh), _ptr(qh), _stream(stream)), "tq_dual_gemm_debug")


def export_weights(desc: WeightDesc, packed, w_codes, w_scales, l1_codes=None, l1_scales=None,
                   l2_codes=None, l2_scales=None, stream=None):
    _check(lib().tq_export_weights(ctypes.byref(desc), _ptr(packed), _ptr(w_codes), _ptr(w_scales),
                                   _ptr(l1_codes), _ptr(l1_scales), _ptr(l2_codes), _ptr(l2_scales),
                                   _stream(stream)), "tq_export_weights")


def export_weights_canonical(desc: WeightDesc, packed, stream=None):
    """The packed weights in the canonical layout (tq_export_weights_canonical):
    (wq [n, k/2] uint8, ws [n, k/group] fp16, l1q [r, k/2], l1s [k/group, r],
    l2q [n, r/2], l2s [r/group_r, n]); the low-rank ones are None for r = 0."""
    import torch
    n, k, r, g, gr = desc.n, desc.k, desc.rank, desc.group, desc.group_r
    dv = packed.device
    wq = torch.empty((n, k // 2), dtype=torch.uint8, device=dv)
    ws = torch.empty((n, k // g), dtype=torch.float16, device=dv)
    l1q = l1s = l2q = l2s = None
    if r:
        l1q = torch.empty((r, k // 2), dtype=torch.uint8, device=dv)
        l1s = torch.empty((k // g, r), dtype=torch.float16, device=dv)
        l2q = torch.empty((n, r // 2), dtype=torch.uint8, device=dv)
        l2s = torch.empty((r // gr, n), dtype=torch.float16, device=dv)
    _check(lib().tq_export_weights_canonical(ctypes.byref(desc), _ptr(packed), _ptr(wq), _ptr(ws), _ptr(l1q),
                                             _ptr(l1s), _ptr(l2q), _ptr(l2s), _stream(stream)),
           "tq_export_weights_canonical")
    return wq, ws, l1q, l1s, l2q, l2s


def act_codes_canonical(x_codes, x_scales, m: int, k: int, group: int = GROUP, stream=None):
    """Activation codes and scales of tq_quant_act in the canonical layout
    (tq_act_codes_canonical): (codes [m, k/2] uint8, scales [m, k/group] fp16)."""
    import torch
    _tensor(x_codes, "x_codes", min_bytes=act_codes_bytes(m, k))
    _tensor(x_scales, "x_scales", min_bytes=(k // group) * padded_tokens(m) * 2)
    q = torch.empty((m, k // 2), dtype=torch.uint8, device=x_codes.device)
    s = torch.empty((m, k // group), dtype=torch.float16, device=x_codes.device)
    _check(lib().tq_act_codes_canonical(_ptr(x_codes), _ptr(x_scales), m, k, group, _ptr(q), _ptr(s),
                                        _stream(stream)), "tq_act_codes_canonical")
    return q, s


def canonical_decode(b) -> np.ndarray:
    """Canonical nibble bytes [..., w] (uint8) -> int8 codes [..., 2w] (host side)."""
    b = np.ascontiguousarray(b).astype(np.uint8)
    lo = (b & 0xF).astype(np.int8)
    hi = (b >> 4).astype(np.int8)
    lo = np.where(lo >= 8, lo - 16, lo).astype(np.int8)
    hi = np.where(hi >= 8, hi - 16, hi).astype(np.int8)
    return np.stack([lo, hi], axis=-1).reshape(*b.shape[:-1], 2 * b.shape[-1])


# ------------------------------------------------------------------ buffers
def empty_packed(desc: WeightDesc, device="cuda"):
    import torch
    return torch.empty(int(desc.packed_bytes), dtype=torch.uint8, device=device)


def padded_tokens(m: int) -> int:
    """m32: the token count rounded up to the 32-token activation tile (at least 32)."""
    return max((m + 31) // 32 * 32, 32)


def dual_gemm_kernel(desc: WeightDesc, m: int) -> str:
    """Name of the kernel tq_dual_gemm launches for this layer and m tokens
    (tq_dual_gemm_kernel); raises ValueError for an invalid descriptor or m."""
    k = int(lib().tq_dual_gemm_kernel(ctypes.byref(desc), m))
    if k < 0:
        raise ValueError(f"tq_dual_gemm_kernel: invalid descriptor or m = {m}")
    return KERNEL_NAMES[k]


def act_codes_bytes(m: int, k: int) -> int:
    """Bytes of the x_codes buffer of m tokens (tq_act_codes_bytes)."""
    return int(lib().tq_act_codes_bytes(m, k))


def empty_act(m: int, k: int, device="cuda", group: int = GROUP):
    """(x_codes, x_scales) buffers for tq_quant_act / tq_dual_gemm:
    x_codes [m32/32, k/64, W] int32, one tile-major block per 32 tokens and
    64-wide K block (W = 256: 1 KiB of TQ4 nibbles for m <= 512; W = 512: 2 KiB
    of fp8 operand bytes for larger m), x_scales [k/group, m32] fp16, m32 =
    padded_tokens(m)."""
    import torch
    m32 = padded_tokens(m)
    nbytes = act_codes_bytes(max(m, 1), k)
    words = nbytes // (m32 // 32 * (k // GROUP) * 4)
    assert words in (256, 512), (m, k, nbytes)
    return (torch.empty((m32 // 32, k // GROUP, words), dtype=torch.int32, device=device),
            torch.empty((k // group, m32), dtype=torch.float16, device=device))


class Layer:
    """One packed layer: descriptor and packed device buffer (device memory from
    torch).  Calls may run concurrently on any streams: the layer keeps no
    per-call state."""

    def __init__(self, w_res, l1=None, l2=None, group: int = GROUP, stream=None):
        n, k = w_res.shape
        r = 0 if l1 is None else l1.shape[1]
        self.desc = weight_desc_init(n, k, r, group)
        self.packed = empty_packed(self.desc, w_res.device)
        pack_weights(self.desc, w_res.contiguous(), None if l1 is None else l1.contiguous(),
                     None if l2 is None else l2.contiguous(), self.packed, stream)
        self.n, self.k, self.rank = n, k, r

    def __call__(self, x, bf16: bool = False, stream=None):
        """Y = layer(x) for fp16 x [m, k]: tq_quant_act, then tq_dual_gemm."""
        import torch
        _tensor(x, "x", torch.float16)
        if x.dim() != 2 or x.shape[1] != self.k:
            raise ValueError(f"x: expected [m, {self.k}], got shape {tuple(x.shape)}")
        m = x.shape[0]
        xc, xs = empty_act(m, self.k, x.device, self.desc.group)
        y = torch.empty((m, self.n), dtype=torch.bfloat16 if bf16 else torch.float16, device=x.device)
        quant_act(x, xc, xs, self.desc.group, stream=stream)
        dual_gemm(self.desc, self.packed, xc, xs, m, y, bf16, stream)
        return y


# ------------------------------------------------------------------ format helpers
def tq4_decode(words) -> np.ndarray:
    """TQ4 words (uint32/int32 array [..., w]) -> int8 codes [..., 8w] (host side)."""
    w = np.ascontiguousarray(words).view(np.uint32)
    out = np.zeros(w.shape + (8,), np.int8)
    for i in range(4):
        mag = (w >> (8 * i)) & 7
        sgn = (w >> (8 * i + 7)) & 1
        out[..., i] = np.where(sgn == 1, -mag.astype(np.int16), mag).astype(np.int8)
        mag2 = (w >> (8 * i + 4)) & 7
        sgn2 = (w >> (8 * ((i + 1) % 4) + 3)) & 1
        out[..., 4 + i] = np.where(sgn2 == 1, -mag2.astype(np.int16), mag2).astype(np.int8)
    return out.reshape(w.shape[:-1] + (w.shape[-1] * 8,))


def tq4_encode(codes) -> np.ndarray:
    """int8 codes in [-7, 7], last axis a multiple of 8 -> TQ4 words (uint32)."""
    c = np.ascontiguousarray(codes).astype(np.int32)
    assert c.shape[-1] % 8 == 0 and np.all(np.abs(c) <= 7)
    c = c.reshape(c.shape[:-1] + (c.shape[-1] // 8, 8))
    mag = np.abs(c).astype(np.uint32)
    neg = (c < 0).astype(np.uint32)
    w = np.zeros(c.shape[:-1], np.uint32)
    for i in range(4):
        w |= mag[..., i] << (8 * i)
        w |= neg[..., i] << (8 * i + 7)
        w |= mag[..., 4 + i] << (8 * i + 4)
        w |= neg[..., 4 + i] << (8 * ((i + 1) % 4) + 3)
    return w


def fp8_code_decode(b) -> np.ndarray:
    """fp8 operand bytes sign << 7 | |q| (uint8 array) -> int8 codes (host side)."""
    b = np.ascontiguousarray(b).view(np.uint8)
    mag = (b & 0x7F).astype(np.int16)
    assert np.all(mag <= 7), "not a code byte"
    return np.where(b >> 7 == 1, -mag, mag).astype(np.int8)


def act_codes_rows(x_codes, m: int) -> np.ndarray:
    """Tile-major activation codes (host copy of x_codes [tiles, k/64, W]
    int32, TQ4 blocks for W = 256 and fp8 blocks for W = 512) -> int8 codes
    [m, k] (host side, for inspection and tests)."""
    w = np.ascontiguousarray(x_codes).view(np.uint32)
    tiles, kg, words = w.shape[0], w.shape[1], w.shape[2]
    if words == 256:
        w = w.reshape(tiles, kg, 2, 32, 4)            # tile, group, half, token, word
        w = w.transpose(0, 3, 1, 2, 4)                 # tile, token, group, half, word
        return tq4_decode(w.reshape(tiles * 32, kg * 8))[:m]
    assert words == 512, words
    b = w.view(np.uint8).reshape(tiles, kg, 2, 2, 32, 16)   # tile, group, part, half, token, byte
    b = b.transpose(0, 4, 1, 3, 2, 5)                        # tile, token, group, half, part, byte
    return fp8_code_decode(b.reshape(tiles * 32, kg * 64))[:m]
