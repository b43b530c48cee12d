"""Seeded synthetic inputs for the TwinQuant dual-component linear layer.

This module is the only code shared by the HIP path's tests/benchmark and the
CPU oracle's tests.  It holds none of the method's arithmetic (no quantizer,
no GEMM of the layer): it only draws activations and weights with the shapes
and value distributions of the paper's workloads (LLaMA3 / Qwen3 projection
layers, Sec. 5.1 and the kernel-profile appendix), and splits each weight into
a rank-r part and a residual the way an offline SVD decomposition would
(Sec. 2, Eq. 3: W = U V + R), so that the layer sees realistic L1 = U',
L2 = V' and W_res = R'^T.  The learned transforms Q and G of Sec. 4.1 are not
available (no checkpoints here); they are taken as the identity, which the
paper's layer definition allows (they are folded into the weights offline).

Recipe (numpy PCG64, every stream seeded from the workload id and sizes):
  * weights: Student-t (nu = 4) scaled to standard deviation 0.02; the tiny
    workload uses N(0, 0.02^2) with 1 % of the input channels scaled x20.
  * activations: N(0, 1) with a seeded 0.5 % of the input channels scaled
    x30 (x50 for the 70B-shaped layers; the tiny workload uses 1 % x30, on
    the same channels as its weight outliers).
  * split: rank-r truncated SVD of W^T (exact for the tiny workload,
    randomized range finder with 16 extra columns and 4 power iterations
    otherwise), L1 = U_r diag(sqrt(s)), L2 = diag(sqrt(s)) V_r^T, both stored
    as fp16; W_res = fp16(W - (L1 L2)^T) with the fp16-rounded factors.
"""
from __future__ import annotations

import dataclasses

import numpy as np

GROUP = 64


@dataclasses.dataclass(frozen=True)
class Layer:
    name: str
    K: int
    N: int
    r: int


@dataclasses.dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    layers: tuple
    Ms: tuple
    w_dist: str            # "normal" or "t4"
    w_outlier_scale: float  # 1.0 = none
    x_outlier_frac: float
    x_outlier_scale: float


WORKLOADS = {
    "tiny": Workload(1, "tiny", (Layer("tiny", 512, 512, 16),), (16,), "normal", 20.0, 0.01, 30.0),
    "llama3-8b-qo": Workload(2, "llama3-8b-qo", (Layer("q_proj", 4096, 4096, 64),),
                             (1, 16, 128, 2048), "t4", 1.0, 0.005, 30.0),
    "llama3-8b-mlp": Workload(3, "llama3-8b-mlp", (Layer("gate_up", 4096, 14336, 64),
                                                   Layer("down", 14336, 4096, 64)),
                              (1, 16, 4096), "t4", 1.0, 0.005, 30.0),
    "qwen3-8b": Workload(4, "qwen3-8b", tuple(
        Layer(f"{nm}_r{r}", K, N, r) for r in (32, 64, 128)
        for nm, K, N in (("qo", 4096, 4096), ("gate_up", 4096, 12288), ("down", 12288, 4096))),
        (1, 256, 4096), "t4", 1.0, 0.005, 30.0),
    "llama3-70b": Workload(5, "llama3-70b", (Layer("gate_up", 8192, 28672, 128),
                                             Layer("down", 28672, 8192, 128)),
                           (1, 32, 8192), "t4", 1.0, 0.005, 50.0),
}


def _rng(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([int(k) for k in key]))


def outlier_channels(wl: Workload, K: int) -> np.ndarray:
    n = max(1, int(round(wl.x_outlier_frac * K)))
    return np.sort(_rng(wl.wid, K, 7).choice(K, size=n, replace=False))


def activations(wl: Workload, M: int, K: int, seed: int = 0) -> np.ndarray:
    """X [M, K] float16."""
    x = _rng(wl.wid, M, K, 1, seed).standard_normal((M, K), dtype=np.float32)
    ch = outlier_channels(wl, K)
    x[:, ch] *= wl.x_outlier_scale
    return x.astype(np.float16)


def dense_weight(wl: Workload, K: int, N: int, seed: int = 0) -> np.ndarray:
    """W [N, K] float32 (PyTorch Linear layout: Y = X W^T)."""
    g = _rng(wl.wid, K, N, 2, seed)
    if wl.w_dist == "normal":
        w = g.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)
    else:
        w = g.standard_t(4.0, size=(N, K)).astype(np.float32) * np.float32(0.02 / np.sqrt(2.0))
    if wl.w_outlier_scale != 1.0:
        w[:, outlier_channels(wl, K)] *= np.float32(wl.w_outlier_scale)
    return w


def _truncated_svd(A: np.ndarray, r: int, exact: bool, key) -> tuple:
    """Rank-r SVD of A [K, N] (fp32): returns U [K,r], s [r], Vt [r,N]."""
    if exact:
        U, s, Vt = np.linalg.svd(A.astype(np.float64), full_matrices=False)
        return U[:, :r], s[:r], Vt[:r]
    K, N = A.shape
    p = min(16, min(K, N) - r)
    omega = _rng(*key).standard_normal((N, r + p), dtype=np.float32)
    Y = A @ omega
    Qm, _ = np.linalg.qr(Y)
    for _ in range(4):
        Z, _ = np.linalg.qr(A.T @ Qm)
        Qm, _ = np.linalg.qr(A @ Z)
    B = Qm.T @ A
    Ub, s, Vt = np.linalg.svd(B.astype(np.float64), full_matrices=False)
    U = Qm.astype(np.float64) @ Ub
    return U[:, :r], s[:r], Vt[:r]


def weights(wl: Workload, layer: Layer, seed: int = 0, rank: int | None = None) -> dict:
    """W_res [N,K], L1 [K,r], L2 [r,N] (float16) for one layer.

    ``rank`` overrides the layer's rank (0 gives W_res = W and no factors).
    """
    K, N = layer.K, layer.N
    r = layer.r if rank is None else rank
    w = dense_weight(wl, K, N, seed)
    if r == 0:
        return {"W_res": w.astype(np.float16), "L1": None, "L2": None}
    U, s, Vt = _truncated_svd(w.T, r, exact=(K * N <= 512 * 512),
                              key=(wl.wid, K, N, r, 3, seed))
    root = np.sqrt(s)
    L1 = (U * root[None, :]).astype(np.float16)
    L2 = (root[:, None] * Vt).astype(np.float16)
    low = L1.astype(np.float32) @ L2.astype(np.float32)          # [K, N]
    W_res = (w - low.T).astype(np.float16)
    return {"W_res": W_res, "L1": L1, "L2": L2}


def layer_inputs(wl_name: str, layer_idx: int, M: int, seed: int = 0, rank: int | None = None) -> dict:
    wl = WORKLOADS[wl_name]
    layer = wl.layers[layer_idx]
    d = weights(wl, layer, seed, rank)
    d["X"] = activations(wl, M, layer.K, seed)
    d["layer"] = layer
    d["workload"] = wl
    return d


def random_codes_layer(M: int, K: int, N: int, r: int, seed: int) -> dict:
    """Small fp16 inputs with no structure (uniform and normal mixtures),
    used for edge-case parity tests (ragged shapes, zero groups)."""
    g = _rng(99, M, K, N, r, seed)
    X = (g.standard_normal((M, K), dtype=np.float32) * 2.0).astype(np.float16)
    W = (g.standard_normal((N, K), dtype=np.float32) * 0.05).astype(np.float16)
    L1 = (g.standard_normal((K, r), dtype=np.float32) * 0.1).astype(np.float16) if r else None
    L2 = (g.standard_normal((r, N), dtype=np.float32) * 0.1).astype(np.float16) if r else None
    return {"X": X, "W_res": W, "L1": L1, "L2": L2}
