"""Offline weight preparation (smoothing, SVD split, transform folding),
pinned in float64 against closed forms and the exact equivalence the
re-parameterization preserves (Sec. 2 and Sec. 4.1)."""
import numpy as np
import pytest

from paper_2606_01556_amd import prep


def rand_orthogonal(n, rng):
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def test_smooth_factors_closed_forms():
    """alpha = 0.5 equalizes the per-channel maxima of X^ and W^ (both become
    sqrt(max|X_i| max|W_i|)); alpha = 1 makes every X^ channel max 1; alpha = 0
    makes every W^ row max 1."""
    rng = np.random.default_rng(0)
    X = rng.standard_normal((64, 48)) * rng.uniform(0.1, 30, 48)
    W = rng.standard_normal((48, 40)) * rng.uniform(0.01, 1, 48)[:, None]
    a = np.abs(X).max(0)
    for alpha, check in ((0.5, None), (1.0, "x"), (0.0, "w")):
        lam = prep.smooth_factors(a, W, alpha)
        xm = np.abs(X / lam).max(0)
        wm = np.abs(lam[:, None] * W).max(1)
        if check is None:
            np.testing.assert_allclose(xm, wm, rtol=1e-12)
            np.testing.assert_allclose(xm, np.sqrt(a * np.abs(W).max(1)), rtol=1e-12)
        elif check == "x":
            np.testing.assert_allclose(xm, 1.0, rtol=1e-12)
        else:
            np.testing.assert_allclose(wm, 1.0, rtol=1e-12)
    with pytest.raises(ValueError):
        prep.smooth_factors(a, W, 1.5)
    with pytest.raises(ValueError):
        prep.smooth_factors(a[:-1], W, 0.5)


def test_svd_split_known_spectrum():
    """A matrix with known singular values: the rank-r split leaves exactly the
    tail energy sum_{i>r} sigma_i^2 in R (Eckart-Young), and the factors carry
    sigma evenly: U^T U = V V^T = diag(sigma_1..r)."""
    rng = np.random.default_rng(1)
    K, N, r = 40, 30, 6
    sig = np.sort(rng.uniform(0.1, 5.0, N))[::-1]
    A = rand_orthogonal(K, rng)[:, :N]
    B = rand_orthogonal(N, rng)
    W = A @ np.diag(sig) @ B.T
    U, V, R = prep.svd_split(W, r)
    assert U.shape == (K, r) and V.shape == (r, N) and R.shape == (K, N)
    np.testing.assert_allclose(np.sum(R ** 2), np.sum(sig[r:] ** 2), rtol=1e-10)
    np.testing.assert_allclose(U.T @ U, np.diag(sig[:r]), atol=1e-10)
    np.testing.assert_allclose(V @ V.T, np.diag(sig[:r]), atol=1e-10)
    np.testing.assert_allclose(U @ V + R, W, atol=1e-12)
    U0, V0, R0 = prep.svd_split(W, 0)
    assert U0.shape == (K, 0) and V0.shape == (0, N)
    np.testing.assert_array_equal(R0, W)


def test_fold_transforms_preserve_the_layer():
    """(X diag(lam)^-1 Q)(U'V' + R') = X W in float64 for a random orthogonal
    Q, a Hadamard Q and a polar-form G."""
    rng = np.random.default_rng(2)
    M, K, N, r = 20, 64, 48, 8
    X = rng.standard_normal((M, K)) * rng.uniform(0.5, 20, K)
    W = rng.standard_normal((K, N)) * 0.05
    lam = prep.smooth_factors(np.abs(X).max(0), W, 0.5)
    U, V, R = prep.svd_split(lam[:, None] * W, r)
    P = rand_orthogonal(r, rng)
    L = np.tril(rng.standard_normal((r, r)) * 0.2) + np.eye(r)
    G = prep.g_from_polar(P, L, 0.3)
    for Q in (rand_orthogonal(K, rng), prep.hadamard(K), None):
        U2, V2, R2 = prep.fold_transforms(U, V, R, Q, G)
        Xt = X / lam
        if Q is not None:
            Xt = Xt @ Q
        np.testing.assert_allclose(Xt @ (U2 @ V2 + R2), X @ W, rtol=1e-9, atol=1e-9)
        if Q is not None:   # the residual is the rotated residual, U'V' the rotated low-rank part
            np.testing.assert_allclose(R2, Q.T @ R, atol=1e-12)
            np.testing.assert_allclose(U2 @ V2, Q.T @ U @ V, atol=1e-10)


def test_fold_transforms_rejects_invalid():
    rng = np.random.default_rng(3)
    U, V, R = prep.svd_split(rng.standard_normal((16, 12)), 4)
    with pytest.raises(ValueError):
        prep.fold_transforms(U, V, R, Q=rng.standard_normal((16, 16)))     # not orthogonal
    G = np.eye(4)
    G[3, 3] = 0.0
    with pytest.raises(ValueError):
        prep.fold_transforms(U, V, R, G=G)                                  # singular
    with pytest.raises(ValueError):
        prep.fold_transforms(U, V, R, Q=np.eye(8))                          # wrong size
    with pytest.raises(ValueError):
        prep.fold_transforms(U, V[:3], R)                                   # shapes do not match


def test_hadamard_and_polar():
    for n in (1, 2, 8, 64):
        H = prep.hadamard(n)
        np.testing.assert_allclose(H @ H.T, np.eye(n), atol=1e-13)
        np.testing.assert_allclose(np.abs(H), 1.0 / np.sqrt(n))
    with pytest.raises(ValueError):
        prep.hadamard(12)
    rng = np.random.default_rng(4)
    np.testing.assert_array_equal(prep.g_from_polar(np.eye(5), np.eye(5), 0.0), np.eye(5))
    P = rand_orthogonal(6, rng)
    L = np.tril(rng.standard_normal((6, 6))) + 3 * np.eye(6)
    G = prep.g_from_polar(P, L, -0.7)
    # G^T G = S^2 with S = e^gamma L L^T symmetric positive definite
    S = np.exp(-0.7) * L @ L.T
    np.testing.assert_allclose(G.T @ G, S @ S, rtol=1e-10)
    assert np.all(np.linalg.eigvalsh(S) > 0)


def test_prepare_layer_fp16_operands():
    """The fp16 operands rebuild the transformed weight to fp16 precision; the
    residual absorbs the rounding of the low-rank factors; rank 0 and
    identity transforms reduce to the plain layer."""
    rng = np.random.default_rng(5)
    M, K, N, r = 24, 128, 96, 16
    weight = (rng.standard_normal((N, K)) * 0.02).astype(np.float16)   # nn.Linear layout [N, K]
    X = rng.standard_normal((M, K)) * 2
    X[:, 5] *= 30
    Q = prep.hadamard(K)
    P = rand_orthogonal(r, rng)
    G = prep.g_from_polar(P, np.eye(r) + np.tril(rng.standard_normal((r, r)) * 0.1, -1), 0.1)
    p = prep.prepare_layer(weight, r, np.abs(X).max(0), 0.5, Q, G)
    assert p.w_res.dtype == np.float16 and p.w_res.shape == (N, K)
    assert p.l1.shape == (K, r) and p.l2.shape == (r, N)
    Wt = Q.T @ (p.lam[:, None] * weight.astype(np.float64).T)
    rebuilt = p.l1.astype(np.float64) @ p.l2.astype(np.float64) + p.w_res.astype(np.float64).T
    # only the final fp16 rounding of the residual remains
    assert np.abs(rebuilt - Wt).max() <= np.abs(Wt - p.l1.astype(np.float64) @ p.l2.astype(np.float64)).max() * 2.0 ** -11
    xt = prep.transform_activations(X, p.lam, p.Q).astype(np.float64)
    ref = X @ weight.astype(np.float64).T
    rel = np.linalg.norm(xt @ rebuilt - ref) / np.linalg.norm(ref)
    assert rel < 2e-3, rel                    # fp16 rounding of the activations and the residual
    p0 = prep.prepare_layer(weight, 0)
    assert p0.l1 is None and p0.l2 is None and p0.lam is None
    np.testing.assert_array_equal(p0.w_res, weight)
    p1 = prep.prepare_layer(weight, r)
    U, V, _ = prep.svd_split(weight.astype(np.float64).T, r)
    np.testing.assert_array_equal(p1.l1, U.astype(np.float16))
    np.testing.assert_array_equal(p1.l2, V.astype(np.float16))


def test_prepared_layers_through_the_oracle(oracle_mod):
    """Smoothing on a layer whose activations carry a few x40 outlier
    channels, through the oracle's W4A4 layer: migrating the outliers into the
    weights lowers the output error against the exact float64 product; the
    prepared operands (any rank, any transform) stay valid layer inputs.
    (Whether the 4-bit low-rank branch helps depends on the weight's spectrum:
    on this structureless random weight it does not, so that is not asserted.)"""
    rng = np.random.default_rng(6)
    M, K, N, r = 64, 256, 128, 32
    weight = (rng.standard_t(4, size=(N, K)) * 0.02 / np.sqrt(2)).astype(np.float16)
    X = rng.standard_normal((M, K))
    X[:, rng.choice(K, 3, replace=False)] *= 40
    ref = X @ weight.astype(np.float64).T

    def err(p):
        xt = prep.transform_activations(X, p.lam, p.Q)
        y = oracle_mod.layer(xt, p.w_res, p.l1, p.l2, 64)["Y64"]
        assert np.all(np.isfinite(y))
        return np.linalg.norm(y - ref) / np.linalg.norm(ref)

    amax = np.abs(X).max(0)
    e_plain = err(prep.prepare_layer(weight, 0))
    e_smooth = err(prep.prepare_layer(weight, 0, amax, 0.5))
    assert e_smooth < 0.5 * e_plain, (e_plain, e_smooth)
    for Q in (None, prep.hadamard(K)):
        assert err(prep.prepare_layer(weight, r, amax, 0.5, Q)) < e_plain
