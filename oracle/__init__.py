"""TEST INFRASTRUCTURE ONLY: ctypes front-end of the plain CPU oracle.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never does, and the two share no code.

The oracle (``tq_oracle.c``) computes the TwinQuant dual-component W4A4 layer
step by step (Sec. 2 Eq. 1-2, Sec. 4.1 Eq. 4/6, Sec. 4.3, Sec. 5.1 of the
paper); every parity test compares the HIP path against it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")


def build_cmd(src: str = _SRC, out: str = _LIB) -> list:
    # -ffp-contract=off: no implicit fma; every float op is IEEE single precision.
    return ["gcc", "-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
            "-fPIC", "-shared", "-Wall", "-Wno-unknown-pragmas", src, "-o", out, "-lm"]


BUILD_CMD = build_cmd()


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle library (in place by default) and return its path."""
    subprocess.run(build_cmd(src, out), check=True)
    return out


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = load(_LIB)
    return _lib


def load(path: str):
    """Load an oracle library file and declare its entry points."""
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    L.tqo_f16_to_f64.argtypes = [ctypes.c_uint16]
    L.tqo_f16_to_f64.restype = ctypes.c_double
    L.tqo_f64_to_f16.argtypes = [ctypes.c_double]
    L.tqo_f64_to_f16.restype = ctypes.c_uint16
    L.tqo_f32_to_bf16.argtypes = [ctypes.c_float]
    L.tqo_f32_to_bf16.restype = ctypes.c_uint16
    L.tqo_quantize.argtypes = [P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                               ctypes.c_int64, ctypes.c_int, P, P]
    L.tqo_quantize.restype = ctypes.c_int
    L.tqo_layer.argtypes = [ctypes.c_int] * 5 + [P] * 4 + [P, ctypes.c_int, P, ctypes.c_int] + [P] * 7
    L.tqo_layer.restype = ctypes.c_int
    return L


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _as_f16_bits(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    if a.dtype == np.uint16:
        return a
    raise TypeError(f"expected float16 (or its uint16 bit pattern), got {a.dtype}")


def f16_to_f64(h: int) -> float:
    return lib().tqo_f16_to_f64(h)


def f64_to_f16(x: float) -> int:
    return lib().tqo_f64_to_f16(x)


def f32_to_bf16(x: float) -> int:
    return lib().tqo_f32_to_bf16(x)


def quantize(v, group: int, axis: int = -1):
    """Group-wise symmetric 4-bit quantization along ``axis`` (Sec. 2, Eq. 1).

    ``v`` is a 2-D float16 array.  Returns ``(codes, scales)``: int8 codes in
    [-7, 7] with the shape of ``v``, and float16 scales with ``axis`` divided
    by ``group`` (groups are contiguous runs along ``axis``).
    """
    v = _as_f16_bits(v)
    assert v.ndim == 2
    axis = axis % 2
    rows, cols = v.shape
    q = np.zeros(v.shape, np.int8)
    if axis == 1:
        n_vec, length, vs, es = rows, cols, cols, 1
    else:
        n_vec, length, vs, es = cols, rows, 1, cols
    s = np.zeros((n_vec, length // group), np.uint16)
    rc = lib().tqo_quantize(_ptr(v), n_vec, length, vs, es, group, _ptr(q), _ptr(s))
    if rc != 0:
        raise ValueError("bad quantization arguments")
    s = s.view(np.float16)
    return q, (s if axis == 1 else s.T.copy())


def layer(X, W_res, L1, L2, group: int, rows=None, cols=None):
    """The full layer, steps O1-O7, for the selected tokens / output channels.

    Returns a dict with H [nr,r] fp32, sH [nr,r/Gr] fp32, qH [nr,r] int8,
    Y32 [nr,nc] fp32, Y64 [nr,nc] fp64, Y16 [nr,nc] fp16, Ybf [nr,nc] (bf16
    bit patterns as uint16).
    """
    X = _as_f16_bits(X)
    W_res = _as_f16_bits(W_res)
    M, K = X.shape
    N = W_res.shape[0]
    assert W_res.shape[1] == K
    r = 0 if L1 is None else L1.shape[1]
    if r:
        L1 = _as_f16_bits(L1)
        L2 = _as_f16_bits(L2)
        assert L1.shape == (K, r) and L2.shape == (r, N)
    Gr = min(group, r) if r else 1
    rows_a = None if rows is None else np.ascontiguousarray(rows, np.int32)
    cols_a = None if cols is None else np.ascontiguousarray(cols, np.int32)
    nr = M if rows_a is None else len(rows_a)
    nc = N if cols_a is None else len(cols_a)
    out = {
        "H": np.zeros((nr, r), np.float32),
        "sH": np.zeros((nr, r // Gr if r else 0), np.float32),
        "qH": np.zeros((nr, r), np.int8),
        "Y32": np.zeros((nr, nc), np.float32),
        "Y64": np.zeros((nr, nc), np.float64),
        "Y16": np.zeros((nr, nc), np.uint16),
        "Ybf": np.zeros((nr, nc), np.uint16),
    }
    rc = lib().tqo_layer(M, N, K, r, group, _ptr(X), _ptr(W_res),
                         _ptr(L1) if r else None, _ptr(L2) if r else None,
                         _ptr(rows_a), nr, _ptr(cols_a), nc,
                         _ptr(out["H"]), _ptr(out["sH"]), _ptr(out["qH"]),
                         _ptr(out["Y32"]), _ptr(out["Y64"]), _ptr(out["Y16"]), _ptr(out["Ybf"]))
    if rc != 0:
        raise ValueError(f"oracle layer failed ({rc})")
    out["Y16"] = out["Y16"].view(np.float16)
    return out
