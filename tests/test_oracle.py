"""Pins of the CPU oracle against facts the paper and the mathematics fix.

Nothing here compares the oracle with a retyped copy of itself.  The pins are:
hand-derived quantizer cases (Sec. 2, Eq. 1), exact rational arithmetic,
library conversions (numpy float16, torch bfloat16), integer-exact designed
layers checked against numpy integer matmul, dyadic-scale layers checked
against fp64 matmul, a brute-force fp64 layer on tiny inputs, and the
invariants the layer definition implies (rank-0, zero residual,
power-of-two scaling, permutation equivariance, locality).
"""
import os
from fractions import Fraction as Fr

import numpy as np
import pytest
import torch

from tq_synth import GROUP, random_codes_layer

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------- helpers
def fp16_rne_exact(x: Fr) -> Fr:
    """Nearest binary16 value of an exact rational (ties to even), no overflow."""
    if x == 0:
        return Fr(0)
    sgn = -1 if x < 0 else 1
    x = abs(x)
    e = 0
    while x >= 2:
        x /= 2
        e += 1
    while x < 1:
        x *= 2
        e -= 1
    ulp = Fr(2) ** max(e - 10, -24)
    q = x * Fr(2) ** e / ulp
    fl = q.numerator // q.denominator
    rem = q - fl
    if rem > Fr(1, 2) or (rem == Fr(1, 2) and fl % 2 == 1):
        fl += 1
    return sgn * fl * ulp


def rne_int(x: Fr) -> int:
    fl = x.numerator // x.denominator
    rem = x - fl
    if rem > Fr(1, 2) or (rem == Fr(1, 2) and fl % 2 == 1):
        fl += 1
    return fl


def q4_exact(vals):
    """Eq. (1) in exact rational arithmetic: codes and the fp16 scale."""
    vs = [Fr(float(v)) for v in vals]
    a = max(abs(v) for v in vs)
    s = fp16_rne_exact(a / 7)
    if s == 0:
        return [0] * len(vs), Fr(0)
    return [max(-7, min(7, rne_int(v / s))) for v in vs], s


def load_hand_cases():
    cases, cur = [], None
    with open(os.path.join(HERE, "golden", "q4_hand_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, rest = line.partition(" ")
            if key == "case":
                cur = {"name": rest}
                cases.append(cur)
            elif key == "in":
                cur["in"] = [float(t) for t in rest.split()]
            elif key == "scale":
                cur["scale"] = float(rest)
            elif key == "codes":
                cur["codes"] = [int(t) for t in rest.split()]
    return cases


def dequant(codes, scales, group, axis):
    s = np.repeat(scales.astype(np.float64), group, axis=axis)
    return codes.astype(np.float64) * s


# ---------------------------------------------------------------- fp16 / bf16
def test_f16_roundtrip_all_patterns(oracle_mod):
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = bits[np.isfinite(bits.view(np.float16))]
    ref = finite.view(np.float16).astype(np.float64)
    L = oracle_mod.lib()
    got = np.array([L.tqo_f16_to_f64(int(b)) for b in finite[::7]])
    np.testing.assert_array_equal(got, ref[::7])
    back = np.array([L.tqo_f64_to_f16(float(v)) for v in ref[::7]], np.uint16)
    # +0/-0 both encode; compare values
    np.testing.assert_array_equal(back.view(np.float16).astype(np.float64), ref[::7])


def test_f16_rounding_matches_numpy(oracle_mod):
    g = np.random.default_rng(5)
    L = oracle_mod.lib()
    xs = np.concatenate([
        g.standard_normal(4000) * 10.0 ** g.integers(-8, 5, 4000),
        (np.arange(-3000, 3000) + 0.5) * 2.0 ** -24,       # subnormal ties
        (np.arange(1024, 2048) + 0.5) * 2.0 ** -5,          # normal ties
        [65504.0, 65519.0, 65520.0, 1e6, -65520.0, 2.0 ** -25, 3 * 2.0 ** -26],
    ])
    with np.errstate(over="ignore"):
        ref = xs.astype(np.float16)
    got = np.array([L.tqo_f64_to_f16(float(x)) for x in xs], np.uint16).view(np.float16)
    np.testing.assert_array_equal(got.astype(np.float64), ref.astype(np.float64))


def test_bf16_rounding_matches_torch(oracle_mod):
    g = np.random.default_rng(6)
    L = oracle_mod.lib()
    xs = (g.standard_normal(5000) * 10.0 ** g.integers(-30, 30, 5000)).astype(np.float32)
    ties = ((np.arange(128, 256) * 2 + 1).astype(np.float32) * np.float32(2.0 ** -8))  # exact bf16 midpoints
    xs = np.concatenate([xs, ties, -ties]).astype(np.float32)
    got = np.array([L.tqo_f32_to_bf16(float(x)) for x in xs], np.uint16)
    ref = torch.from_numpy(xs).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, ref)


# ---------------------------------------------------------------- quantizer
@pytest.mark.parametrize("case", load_hand_cases(), ids=lambda c: c["name"])
def test_quantizer_hand_cases(oracle_mod, case):
    vals = np.zeros(GROUP, np.float16)
    vals[: len(case["in"])] = case["in"]
    q, s = oracle_mod.quantize(vals[None, :], GROUP)
    assert float(s[0, 0]) == case["scale"]
    assert q[0, : len(case["codes"])].tolist() == case["codes"]
    assert np.all(q[0, len(case["codes"]):] == 0)


def test_quantizer_matches_exact_rational(oracle_mod):
    """Codes and scales equal Eq. (1) evaluated in exact rational arithmetic
    (fp32 division inside the oracle never changes a decision)."""
    g = np.random.default_rng(11)
    rows = []
    for i in range(120):
        if i % 5 == 0:
            # dyadic scale 2^e with planted exact ties (k + 1/2) * 2^e
            e = int(g.integers(-10, 6))
            half = g.integers(-14, 15, size=GROUP)
            half[0] = 14
            v = (half * 2.0 ** (e - 1)).astype(np.float16)
        else:
            scale = 10.0 ** g.uniform(-6, 3)
            v = (g.standard_normal(GROUP) * scale).astype(np.float16)
        rows.append(v)
    V = np.stack(rows)
    q, s = oracle_mod.quantize(V, GROUP)
    for i in range(V.shape[0]):
        codes, sc = q4_exact(V[i])
        assert Fr(float(s[i, 0])) == sc, i
        assert q[i].tolist() == codes, i


@pytest.mark.parametrize("e", [-24, -20, -14, -3, 0, 5, 10, 13])
def test_quantizer_round_trip_dyadic(oracle_mod, e):
    g = np.random.default_rng(e + 100)
    q0 = g.integers(-7, 8, size=(6, GROUP))
    q0[:, 3] = 7 * np.where(g.integers(0, 2, 6) > 0, 1, -1)   # |q| = 7 in every group
    v = (q0 * 2.0 ** e).astype(np.float16)
    assert np.all(v.astype(np.float64) == q0 * 2.0 ** e)
    q, s = oracle_mod.quantize(v, GROUP)
    np.testing.assert_array_equal(q, q0)
    assert np.all(s.astype(np.float64) == 2.0 ** e)


def test_quantizer_sign_symmetry_and_locality(oracle_mod):
    g = np.random.default_rng(3)
    v = (g.standard_normal((4, 4 * GROUP)) * 3).astype(np.float16)
    q, s = oracle_mod.quantize(v, GROUP)
    qn, sn = oracle_mod.quantize(-v, GROUP)
    np.testing.assert_array_equal(qn, -q)
    np.testing.assert_array_equal(sn, s)
    v2 = v.copy()
    v2[1, GROUP:2 * GROUP] *= np.float16(5)
    q2, s2 = oracle_mod.quantize(v2, GROUP)
    changed = np.ones_like(q, bool)
    changed[1, GROUP:2 * GROUP] = False
    np.testing.assert_array_equal(q2[changed], q[changed])
    sm = np.ones_like(s, bool)
    sm[1, 1] = False
    np.testing.assert_array_equal(s2[sm], s[sm])
    assert s2[1, 1] != s[1, 1]


def test_quantizer_axis0_groups(oracle_mod):
    """Groups along axis 0 equal groups along axis 1 of the transpose."""
    g = np.random.default_rng(4)
    v = (g.standard_normal((2 * GROUP, 24))).astype(np.float16)
    q0, s0 = oracle_mod.quantize(v, GROUP, axis=0)
    q1, s1 = oracle_mod.quantize(np.ascontiguousarray(v.T), GROUP, axis=1)
    np.testing.assert_array_equal(q0, q1.T)
    np.testing.assert_array_equal(s0, s1.T)


# ---------------------------------------------------------------- designed layers
def _designed_integer_layer(M, K, N, r, seed, G=GROUP):
    """fp16 inputs whose every group has max |value| = 7, so all stored scales
    are exactly 1 and the codes are the values themselves.  The low-rank part
    is built so that H = X L1 is integer with max |H| = 7 per r-group, so
    s_H = 1 and q_H = H (no rounding anywhere)."""
    g = np.random.default_rng(seed)
    X = g.integers(-6, 7, size=(M, K)).astype(np.float64)
    W = g.integers(-7, 8, size=(N, K)).astype(np.float64)
    for kg in range(K // G):
        X[:, kg * G + 5] = 7 * np.sign(g.standard_normal(M) + 0.01)
        W[:, kg * G + 9] = -7
    L1 = np.zeros((K, r))
    L2 = g.integers(-7, 8, size=(r, N)).astype(np.float64)
    Gr = max(1, min(G, r))
    for hg in range(r // Gr):
        L2[hg * Gr, :] = 7
    if r:
        # X column k1 = +-1 carries H; column k7 = 7 (already in X), zero L1 there.
        k1 = 2
        X[:, k1] = np.sign(g.standard_normal(M) + 0.01)
        k0 = 3
        X[:, k0] = 0
        v = g.integers(-7, 8, size=r).astype(np.float64)
        for hg in range(r // Gr):
            v[hg * Gr] = 7
        L1[k1, :] = v
        L1[k0, :] = 7                # sets every L1 column group's max to 7 (X is 0 there)
        for kg in range(1, K // G):  # later groups: max 7 where X is 0
            X[:, kg * G + 11] = 0
            L1[kg * G + 11, :] = -7
    return {k: a.astype(np.float16) for k, a in
            dict(X=X, W_res=W, L1=L1 if r else None, L2=L2 if r else None).items() if a is not None}, X, W, L1, L2


@pytest.mark.parametrize("M,K,N,r,G", [(5, 128, 48, 16, 64), (3, 192, 64, 64, 64), (4, 128, 32, 128, 64),
                                       (2, 64, 16, 0, 64), (3, 256, 40, 128, 128), (4, 384, 24, 32, 128)])
def test_integer_designed_layer(oracle_mod, M, K, N, r, G):
    d, X, W, L1, L2 = _designed_integer_layer(M, K, N, r, seed=M * 7 + r, G=G)
    out = oracle_mod.layer(d["X"], d["W_res"], d.get("L1"), d.get("L2"), G)
    Xi, Wi = X.astype(np.int64), W.astype(np.int64)
    Y = Xi @ Wi.T
    if r:
        H = Xi @ L1.astype(np.int64)
        np.testing.assert_array_equal(out["H"], H.astype(np.float32))
        np.testing.assert_array_equal(out["qH"], H)
        assert np.all(out["sH"] == 1.0)
        Y = Y + H @ L2.astype(np.int64)
    np.testing.assert_array_equal(out["Y32"], Y.astype(np.float32))
    np.testing.assert_array_equal(out["Y64"], Y.astype(np.float64))
    np.testing.assert_array_equal(out["Y16"], Y.astype(np.float16))


def test_dyadic_scale_layer(oracle_mod):
    """Per-group power-of-two scales: the layer equals the fp64 matmul of the
    dequantized operands exactly (every product and sum is exact)."""
    g = np.random.default_rng(21)
    M, K, N, G = 6, 256, 40, GROUP
    qx = g.integers(-7, 8, size=(M, K))
    qw = g.integers(-7, 8, size=(N, K))
    qx[:, ::G] = 7
    qw[:, 1::G] = -7
    ex = g.integers(-6, 4, size=(M, K // G))
    ew = g.integers(-9, -3, size=(N, K // G))
    X = qx * np.repeat(2.0 ** ex, G, axis=1)
    W = qw * np.repeat(2.0 ** ew, G, axis=1)
    out = oracle_mod.layer(X.astype(np.float16), W.astype(np.float16), None, None, G)
    np.testing.assert_array_equal(out["Y64"], X @ W.T)
    np.testing.assert_array_equal(out["Y32"], (X @ W.T).astype(np.float32))


# ---------------------------------------------------------------- brute force
def _brute_force(X, W, L1, L2, G):
    """quantize (exact rationals) -> dequantize -> fp64 matmul, H requantized in fp64."""
    def quant_rows(A, group):
        Q = np.zeros(A.shape, np.int64)
        S = np.zeros((A.shape[0], A.shape[1] // group))
        for i in range(A.shape[0]):
            for gi in range(A.shape[1] // group):
                c, s = q4_exact(A[i, gi * group:(gi + 1) * group])
                Q[i, gi * group:(gi + 1) * group] = c
                S[i, gi] = float(s)
        return Q, S
    qx, sx = quant_rows(X, G)
    qw, sw = quant_rows(W, G)
    Xd = dequant(qx, sx, G, 1)
    Y = Xd @ dequant(qw, sw, G, 1).T
    res = {"Yres": Y.copy()}
    if L1 is not None:
        r = L1.shape[1]
        Gr = min(G, r)
        ql1, sl1 = quant_rows(np.ascontiguousarray(L1.T), G)
        ql2, sl2 = quant_rows(np.ascontiguousarray(L2.T), Gr)
        H = Xd @ dequant(ql1, sl1, G, 1).T                     # [M, r]
        Hg = H.reshape(H.shape[0], r // Gr, Gr)
        sH = np.abs(Hg).max(axis=2) / 7.0
        with np.errstate(invalid="ignore", divide="ignore"):
            t = np.where(sH[..., None] > 0, Hg / sH[..., None], 0.0)
        qH = np.clip(np.rint(t), -7, 7).reshape(H.shape)
        Y = Y + dequant(qH, sH, Gr, 1) @ dequant(ql2, sl2, Gr, 1).T
        res.update(H=H, t=t.reshape(H.shape), qH=qH)
    res["Y"] = Y
    return res


@pytest.mark.parametrize("M,K,N,r,G", [(4, 128, 24, 16, 64), (3, 192, 16, 64, 64), (2, 128, 8, 128, 64),
                                       (3, 128, 16, 0, 64), (4, 256, 24, 128, 128), (3, 384, 16, 64, 128),
                                       (2, 128, 8, 16, 128), (3, 256, 16, 0, 128)])
def test_brute_force_fp64(oracle_mod, M, K, N, r, G):
    d = random_codes_layer(M, K, N, r, seed=r + 1 + G)
    if G == 128:
        # halves of very different size: a 128-wide group codes the smaller
        # half with the larger half's scale, which 64-wide groups would not
        d["X"][:, 64:128] = (d["X"][:, 64:128].astype(np.float32) * 40).astype(np.float16)
    bf = _brute_force(d["X"].astype(np.float64), d["W_res"].astype(np.float64),
                      None if d["L1"] is None else d["L1"].astype(np.float64),
                      None if d["L2"] is None else d["L2"].astype(np.float64), G)
    out = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], G)
    if G == 128:
        o64 = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], 64)
        assert not np.array_equal(o64["Y32"], out["Y32"]), "the group width must matter here"
    if r:
        np.testing.assert_allclose(out["H"], bf["H"], rtol=1e-6, atol=1e-6 * np.abs(bf["H"]).max())
        near_tie = np.abs(np.abs(bf["t"] - np.floor(bf["t"])) - 0.5) < 1e-4
        assert not near_tie.any(), "seed lands on a q_H tie; pick another"
        np.testing.assert_array_equal(out["qH"], bf["qH"])
    rel = np.linalg.norm(out["Y64"] - bf["Y"]) / np.linalg.norm(bf["Y"])
    assert rel <= 1e-6
    rel32 = np.linalg.norm(out["Y32"] - bf["Y"]) / np.linalg.norm(bf["Y"])
    assert rel32 <= 1e-5


# ---------------------------------------------------------------- invariants
def test_rank0_is_plain_w4a4(oracle_mod):
    d = random_codes_layer(5, 256, 32, 16, seed=3)
    full = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    r0 = oracle_mod.layer(d["X"], d["W_res"], None, None, GROUP)
    bf = _brute_force(d["X"].astype(np.float64), d["W_res"].astype(np.float64), None, None, GROUP)
    assert np.linalg.norm(r0["Y64"] - bf["Yres"]) <= 1e-12 * np.linalg.norm(bf["Yres"])
    assert not np.array_equal(full["Y32"], r0["Y32"])


def test_zero_residual_is_pure_low_rank(oracle_mod):
    d = random_codes_layer(4, 128, 24, 32, seed=8)
    Wz = np.zeros_like(d["W_res"])
    out = oracle_mod.layer(d["X"], Wz, d["L1"], d["L2"], GROUP)
    full = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    r0 = oracle_mod.layer(d["X"], d["W_res"], None, None, GROUP)
    np.testing.assert_array_equal(out["H"], full["H"])
    # with W_res = 0 every residual scale is 0: Y is the low-rank branch alone
    np.testing.assert_allclose(out["Y64"] + r0["Y64"], full["Y64"], rtol=1e-12, atol=1e-12)


def test_power_of_two_scaling(oracle_mod):
    d = random_codes_layer(4, 192, 16, 64, seed=9)
    a = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    b = oracle_mod.layer((d["X"].astype(np.float32) * 4).astype(np.float16), d["W_res"], d["L1"], d["L2"], GROUP)
    np.testing.assert_array_equal(b["qH"], a["qH"])
    np.testing.assert_array_equal(b["H"], a["H"] * 4)
    np.testing.assert_array_equal(b["sH"], a["sH"] * 4)
    np.testing.assert_array_equal(b["Y32"], a["Y32"] * 4)


def test_permutation_equivariance(oracle_mod):
    d = random_codes_layer(6, 128, 20, 64, seed=10)
    base = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    g = np.random.default_rng(0)
    pm = g.permutation(6)
    t = oracle_mod.layer(d["X"][pm], d["W_res"], d["L1"], d["L2"], GROUP)
    np.testing.assert_array_equal(t["Y32"], base["Y32"][pm])
    pn = g.permutation(20)
    o = oracle_mod.layer(d["X"], d["W_res"][pn], d["L1"], np.ascontiguousarray(d["L2"][:, pn]), GROUP)
    np.testing.assert_array_equal(o["Y32"], base["Y32"][:, pn])
    pr = g.permutation(64)       # one r-group (r = G): any rank permutation
    rr = oracle_mod.layer(d["X"], d["W_res"], np.ascontiguousarray(d["L1"][:, pr]),
                          np.ascontiguousarray(d["L2"][pr]), GROUP)
    np.testing.assert_array_equal(rr["Y32"], base["Y32"])
    np.testing.assert_array_equal(rr["H"], base["H"][:, pr])


def test_row_col_selection_matches_full(oracle_mod):
    d = random_codes_layer(7, 128, 33, 32, seed=12)
    full = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    rows, cols = [6, 0, 3], [32, 1, 5, 5]
    sub = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP, rows=rows, cols=cols)
    np.testing.assert_array_equal(sub["Y32"], full["Y32"][np.ix_(rows, cols)])
    np.testing.assert_array_equal(sub["qH"], full["qH"][rows])
    np.testing.assert_array_equal(sub["Y16"], full["Y16"][np.ix_(rows, cols)])


# ---------------------------------------------------------------- H order and Q_H ties
def f32_rne_exact(x: Fr) -> Fr:
    """Nearest binary32 value of an exact rational, ties to even (normal range)."""
    if x == 0:
        return Fr(0)
    sgn = -1 if x < 0 else 1
    x = abs(x)
    e = 0
    while x >= 2:
        x /= 2
        e += 1
    while x < 1:
        x *= 2
        e -= 1
    ulp = Fr(2) ** (e - 23)
    return sgn * rne_int(x * Fr(2) ** e / ulp) * ulp


def check_h_chain_order(oracle_mod):
    """O4 (Sec. 4.3, stage 1; reading R11): H is summed over K-groups in
    ascending order, one fused multiply-add (a single rounding) per group, with
    the exact fp32 scale product s_x s_L1.  The designed layer fixes the codes
    and scales, so the integer group sums A_g and the scale products c_g are
    known exactly; the expected H is the ascending chain
    h <- rn32(A_g c_g + h) evaluated in exact rationals.  The design also
    checks that it tells this chain apart from a descending chain, from an
    unfused chain (the product rounded before the add) and from the correctly
    rounded sum."""
    from designed import chain_order_layer
    d = chain_order_layer(M=8, r=32, seed=1)
    out = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    M, r = out["H"].shape
    KG = d["sx"].shape[1]
    qx = d["qx"].reshape(M, KG, GROUP)
    ql1 = d["ql1"].reshape(KG, GROUP, r)
    A = np.einsum("mgk,gkj->mjg", qx, ql1)                      # exact int64 sums
    diffs = {"descending": 0, "unfused": 0, "exact_sum": 0}
    for m in range(M):
        for j in range(r):
            terms = [int(A[m, j, g]) * Fr(float(d["sx"][m, g])) * Fr(float(d["sl1"][g, j]))
                     for g in range(KG)]
            asc = Fr(0)
            for t in terms:
                asc = f32_rne_exact(t + asc)
            desc = Fr(0)
            for t in reversed(terms):
                desc = f32_rne_exact(t + desc)
            unf = Fr(0)
            for t in terms:
                unf = f32_rne_exact(f32_rne_exact(t) + unf)
            exact = f32_rne_exact(sum(terms))
            assert Fr(float(out["H"][m, j])) == asc, (m, j)
            diffs["descending"] += desc != asc
            diffs["unfused"] += unf != asc
            diffs["exact_sum"] += exact != asc
    assert all(v > 0 for v in diffs.values()), diffs


def check_qh_ties(oracle_mod):
    """O5 (Sec. 4.3, on-the-fly scaling; readings R1, R10): on the designed
    layer of tests/golden/qh_ties.txt, H / s_H lands exactly on k + 1/2 and
    the codes are the fixture's hand-derived round-half-to-even values."""
    from designed import qh_tie_layer
    fx_u = [1.0, 3.0, 0.125]
    d = qh_tie_layer(M=3, N=16)
    out = oracle_mod.layer(d["X"], d["W_res"], d["L1"], d["L2"], GROUP)
    np.testing.assert_array_equal(out["sH"][:, 0], np.array(fx_u, np.float32))
    np.testing.assert_array_equal(out["H"], (d["t"] * np.array(fx_u)[:, None]).astype(np.float32))
    np.testing.assert_array_equal(out["qH"], d["qh"])


def test_h_chain_order_exact(oracle_mod):
    check_h_chain_order(oracle_mod)


def test_qh_ties_golden(oracle_mod):
    check_qh_ties(oracle_mod)


# Each pin above must fail on an oracle with the corresponding plausible
# mistake; the mutants are built from the oracle's source on the CPU.
MUTANTS = {
    "h_descending": ("for (int g = 0; g < KG; g++) {\n                    int32_t a = 0;",
                     "for (int g = KG - 1; g >= 0; g--) {\n                    int32_t a = 0;",
                     check_h_chain_order),
    "h_unfused": ("acc = fmaf((float)a, sxf * slf, acc);",
                  "acc = (float)a * (sxf * slf) + acc;", check_h_chain_order),
    "qh_half_away": ("double rr = nearbyint((double)t);", "double rr = round((double)t);",
                     check_qh_ties),
    "qh_truncate": ("double rr = nearbyint((double)t);", "double rr = trunc((double)t);",
                    check_qh_ties),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant_oracle(oracle_mod, tmp_path, monkeypatch, name):
    old, new, check = MUTANTS[name]
    with open(oracle_mod._SRC) as f:
        src = f.read()
    assert src.count(old) == 1, "mutation site not found once in the oracle source"
    mut = tmp_path / "mutant.c"
    mut.write_text(src.replace(old, new))
    lib = oracle_mod.load(oracle_mod.build(str(mut), str(tmp_path / "libmutant.so")))
    monkeypatch.setattr(oracle_mod, "_lib", lib)
    with pytest.raises(AssertionError):
        check(oracle_mod)
