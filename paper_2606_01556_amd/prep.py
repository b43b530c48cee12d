"""Offline weight preparation for the fused W4A4 layer: the step before
tq_pack_weights.

A linear layer Y = X W (W of shape [K, N], input channels as rows; PyTorch
stores the transpose, ``weight`` [N, K]) is turned into the three fp16
operands that tq_pack_weights quantizes:

1. per-channel smoothing (Sec. 2, "Per-channel Scaling"; smoothing factor of
   the implementation details, Appendix "Implement Detail"):
   X^ = X diag(lam)^-1 and W^ = diag(lam) W with
   lam_i = max|X[:, i]|^alpha / max|W[i, :]|^(1 - alpha);
2. the low-rank / residual split of W^ (Sec. 2, "Low-Rank Decomposition"):
   W^ = U V + R, U [K, r] and V [r, N] from a rank-r truncated SVD;
3. the transforms of the re-parameterization (Sec. 4.1): a global orthogonal
   Q [K, K] applied to the activation (X^ Q) and a layer-specific invertible
   G [r, r], folded into the weights as U' = Q^-1 U G, V' = G^-1 V and
   R' = Q^-1 R.  In full precision (X^ Q)(U' V' + R') = X W exactly.

The kernel then computes Q(X^ Q) [Q(U') Q(V') + Q(R')]: L1 = U', L2 = V' and
W_res = R'^T.  Learning Q and G (Sec. 4.2) is outside this module; it takes
them as given, e.g. from ``hadamard`` (the fixed-rotation variant of the
ablation study, Sec. 5.5) or ``g_from_polar`` (the polar form G = P S,
S = e^gamma L L^T, of Sec. 4.2).

Everything here runs on the host in float64 except ``search_alpha``, which
measures each candidate through the library's fused layer on the GPU.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

__all__ = ["smooth_factors", "hadamard", "g_from_polar", "svd_split", "fold_transforms",
           "PreparedLayer", "prepare_layer", "transform_activations", "search_alpha"]


def smooth_factors(x_absmax, w, alpha: float, eps: float = 1e-5) -> np.ndarray:
    """Per-input-channel smoothing factors lam [K] (Appendix, Implement Detail):
    lam_i = max|X[:, i]|^alpha / max|W[i, :]|^(1 - alpha).

    x_absmax  [K] per-channel max |X| over the calibration tokens
    w         [K, N] weight, input channels as rows
    alpha     migration strength in [0, 1]
    Channel maxima are floored at eps so that dead channels give finite
    factors."""
    a = np.maximum(np.asarray(x_absmax, np.float64), eps)
    w = np.asarray(w, np.float64)
    if a.ndim != 1 or w.ndim != 2 or w.shape[0] != a.shape[0]:
        raise ValueError(f"x_absmax [{a.shape}] and w [{w.shape}] do not match as [K] and [K, N]")
    if not 0.0 <= alpha <= 1.0:
        raise ValueError("alpha must lie in [0, 1]")
    wmax = np.maximum(np.abs(w).max(axis=1), eps)
    return a ** alpha / wmax ** (1.0 - alpha)


def hadamard(n: int) -> np.ndarray:
    """Orthonormal Hadamard matrix of order n (a power of two), Sylvester's
    construction scaled by 1/sqrt(n): a fixed orthogonal Q."""
    if n < 1 or n & (n - 1):
        raise ValueError("the Sylvester construction needs a power of two")
    h = np.ones((1, 1))
    while h.shape[0] < n:
        h = np.block([[h, h], [h, -h]])
    return h / np.sqrt(n)


def g_from_polar(P, L, gamma: float) -> np.ndarray:
    """G = P S with S = e^gamma L L^T (Sec. 4.2, Eq. polar): P orthogonal, L
    lower triangular with a non-zero diagonal, so G is invertible."""
    P = np.asarray(P, np.float64)
    L = np.tril(np.asarray(L, np.float64))
    if P.shape != L.shape or P.shape[0] != P.shape[1]:
        raise ValueError("P and L must be square and of the same size")
    return P @ (np.exp(gamma) * (L @ L.T))


def svd_split(w_hat, rank: int):
    """W^ = U V + R with U = U_r Sigma_r^(1/2) [K, r], V = Sigma_r^(1/2) V_r^T
    [r, N] from the rank-r truncated SVD (Sec. 2, Eq. for the low-rank
    branch), and the residual R = W^ - U V [K, N].  The singular values are
    split evenly between the two factors, so U^T U = V V^T = Sigma_r."""
    w_hat = np.asarray(w_hat, np.float64)
    K, N = w_hat.shape
    if not 0 <= rank <= min(K, N):
        raise ValueError(f"rank {rank} outside [0, {min(K, N)}]")
    if rank == 0:
        return np.zeros((K, 0)), np.zeros((0, N)), w_hat.copy()
    u, s, vt = np.linalg.svd(w_hat, full_matrices=False)
    root = np.sqrt(s[:rank])
    U = u[:, :rank] * root
    V = root[:, None] * vt[:rank]
    return U, V, w_hat - U @ V


def fold_transforms(U, V, R, Q=None, G=None, tol: float = 1e-8):
    """Fold the transforms into the weights (Sec. 4.1): U' = Q^-1 U G,
    V' = G^-1 V, R' = Q^-1 R, with Q^-1 = Q^T for the orthogonal Q.  None
    stands for the identity.  Raises ValueError for a Q that is not
    orthogonal to within tol (relative) or a G that is singular or
    ill-conditioned beyond 1 / tol."""
    U = np.asarray(U, np.float64)
    V = np.asarray(V, np.float64)
    R = np.asarray(R, np.float64)
    K, r = U.shape
    if V.shape[0] != r or R.shape != (K, V.shape[1]):
        raise ValueError("U [K, r], V [r, N] and R [K, N] do not match")
    if Q is not None:
        Q = np.asarray(Q, np.float64)
        if Q.shape != (K, K):
            raise ValueError(f"Q must be [{K}, {K}]")
        if np.abs(Q.T @ Q - np.eye(K)).max() > tol * max(1.0, K ** 0.5):
            raise ValueError("Q is not orthogonal")
        U = Q.T @ U
        R = Q.T @ R
    if G is not None and r > 0:
        G = np.asarray(G, np.float64)
        if G.shape != (r, r):
            raise ValueError(f"G must be [{r}, {r}]")
        if not np.all(np.isfinite(G)) or np.linalg.cond(G) > 1.0 / tol:
            raise ValueError("G is singular or too ill-conditioned to invert")
        U = U @ G
        V = np.linalg.solve(G, V)
    return U, V, R


@dataclass
class PreparedLayer:
    """fp16 operands of tq_pack_weights and the activation-side transforms.
    w_res [N, K], l1 [K, r], l2 [r, N] (None for rank 0); lam [K] or None;
    Q [K, K] or None.  The layer's input must be transform_activations(x,
    lam, Q) (in a model, folded into the previous layer)."""
    w_res: np.ndarray
    l1: np.ndarray | None
    l2: np.ndarray | None
    lam: np.ndarray | None
    Q: np.ndarray | None


def prepare_layer(weight, rank: int, x_absmax=None, alpha: float = 0.5, Q=None, G=None) -> PreparedLayer:
    """The three steps above for one layer.  weight [N, K] as nn.Linear
    stores it.  x_absmax [K] enables smoothing with strength alpha.  The fp16
    residual is formed after rounding the low-rank factors to fp16, in the
    transformed basis: w_res = fp16((Q^T W^ - fp16(U') fp16(V'))^T), so it
    also absorbs the rounding of U' and V'."""
    W = np.asarray(weight, np.float64).T          # [K, N]
    lam = None
    if x_absmax is not None:
        lam = smooth_factors(x_absmax, W, alpha)
        W = lam[:, None] * W
    U, V, R = svd_split(W, rank)
    U, V, R = fold_transforms(U, V, R, Q, G)
    Wt = W if Q is None else np.asarray(Q, np.float64).T @ W
    if rank == 0:
        return PreparedLayer(Wt.T.astype(np.float16), None, None, lam, Q)
    l1 = U.astype(np.float16)
    l2 = V.astype(np.float16)
    w_res = (Wt - l1.astype(np.float64) @ l2.astype(np.float64)).T.astype(np.float16)
    return PreparedLayer(w_res, l1, l2, lam, Q)


def transform_activations(x, lam=None, Q=None) -> np.ndarray:
    """X^ Q = X diag(lam)^-1 Q in float64, returned as fp16 [M, K]: the input
    the prepared layer expects."""
    x = np.asarray(x, np.float64)
    if lam is not None:
        x = x / np.asarray(lam, np.float64)[None, :]
    if Q is not None:
        x = x @ np.asarray(Q, np.float64)
    return x.astype(np.float16)


def search_alpha(x_calib, weight, rank: int, alphas=(0.3, 0.4, 0.5, 0.6, 0.7), Q=None, G=None,
                 device="cuda"):
    """Choose the migration strength per layer as the candidate whose
    quantized layer (run through tq_quant_act and tq_dual_gemm on `device`)
    has the smallest output mean squared error against the float64 product
    X W on the calibration tokens (Appendix, Implement Detail).  Returns
    (best alpha, {alpha: mse})."""
    import torch
    from . import Layer

    x = np.asarray(x_calib, np.float64)
    ref = x @ np.asarray(weight, np.float64).T
    x_absmax = np.abs(x).max(axis=0)
    errs = {}
    for a in alphas:
        p = prepare_layer(weight, rank, x_absmax, a, Q, G)
        dev = torch.device(device)
        lay = Layer(torch.from_numpy(p.w_res).to(dev),
                    None if p.l1 is None else torch.from_numpy(p.l1).to(dev),
                    None if p.l2 is None else torch.from_numpy(p.l2).to(dev))
        xt = torch.from_numpy(transform_activations(x, p.lam, p.Q)).to(dev)
        y = lay(xt).float().cpu().numpy().astype(np.float64)
        errs[a] = float(np.mean((y - ref) ** 2))
    best = min(errs, key=errs.get)
    return best, errs
