"""Designed fp16 inputs whose quantized codes and scales are known in advance.

Input generators only: nothing here quantizes or multiplies anything of the
layer.  Each generator places values so that the group quantizer of Sec. 2,
Eq. (1) returns chosen codes and scales exactly (a group holding q * s with
max |q| = 7 and an fp16 scale s of at most 8 significant bits quantizes to
exactly (q, s)), so the tests can derive what the layer must produce with
exact arithmetic of their own.
"""
from __future__ import annotations

import os

import numpy as np

from tq_synth import GROUP

HERE = os.path.dirname(os.path.abspath(__file__))


def _rng(*key):
    return np.random.Generator(np.random.PCG64([int(k) for k in key]))


def _codes_with_max7(g, shape, axis_len):
    """Random codes in [-7, 7] whose every run of `axis_len` along the last
    axis holds a +-7 (so each group's max |code| is 7)."""
    q = g.integers(-7, 8, size=shape)
    flat = q.reshape(-1, shape[-1] // axis_len, axis_len)
    pos = g.integers(0, axis_len, size=flat.shape[:2])
    sign = np.where(g.integers(0, 2, size=flat.shape[:2]) > 0, 7, -7)
    np.put_along_axis(flat, pos[..., None], sign[..., None], axis=2)
    return flat.reshape(shape)


def _scales8(g, shape, e_lo, e_hi):
    """fp16-exact scales m * 2^(e - 7) with an 8-bit significand m in
    [128, 255] and e in [e_lo, e_hi] (elementwise)."""
    m = g.integers(128, 256, size=shape).astype(np.float64)
    e = g.integers(e_lo, e_hi + 1, size=shape)
    return m * np.exp2(e - 7.0)


def chain_order_layer(M: int, r: int, seed: int):
    """A layer of three K-groups built so that the fp32 sum of the stage-1
    group terms A_g * (s_x s_L1) depends on the order and on whether each
    term is rounded before it is added:
      * group 1 holds the negated activation codes of group 0 with the same
        scale, and the same L1 codes with a different scale of the same
        binade, so the first two terms nearly cancel and the low bits of the
        second product survive in the sum;
      * group 2's activation scale is about 2^-9 of the others, so adding it
        first or last rounds differently.
    Returns the fp16 inputs and the exact codes and scales: qx [M, K],
    sx [M, 3], ql1 [K, r], sl1 [3, r]."""
    g = _rng(31, M, r, seed)
    K = 3 * GROUP
    # group 0: codes of magnitude 4..7 with one sign pattern along K shared by
    # the activations and L1, so every integer sum is 1024..3136 (11-12
    # significant bits) and a product with two 8-bit scales needs more than
    # fp32's 24
    sign = np.where(g.integers(0, 2, size=GROUP) > 0, 1, -1)
    q0 = sign * g.integers(4, 8, size=(M, GROUP))
    q0[:, 0] = 7 * sign[0]
    q2 = _codes_with_max7(g, (M, GROUP), GROUP)
    qx = np.concatenate([q0, -q0, q2], axis=1)
    s0 = _scales8(g, (M, 1), -1, 1)
    sx = np.concatenate([s0, s0, _scales8(g, (M, 1), -10, -8)], axis=1)
    l0 = sign[:, None] * g.integers(4, 8, size=(GROUP, r))
    l0[1, :] = 7 * sign[1]
    l2 = _codes_with_max7(g, (r, GROUP), GROUP).T
    ql1 = np.concatenate([l0, l0, l2], axis=0)
    e01 = g.integers(-5, -2, size=(1, r))
    sl1 = np.concatenate([g.integers(128, 256, size=(2, r)) * np.exp2(e01 - 7.0),
                          _scales8(g, (1, r), -5, -3)], axis=0)
    X = qx * np.repeat(sx, GROUP, axis=1)
    L1 = ql1 * np.repeat(sl1, GROUP, axis=0)
    N = 16
    W = (g.standard_normal((N, K)) * 0.05).astype(np.float16)
    L2 = (g.standard_normal((r, N)) * 0.1).astype(np.float16)
    X16, L116 = X.astype(np.float16), L1.astype(np.float16)
    assert np.array_equal(X16.astype(np.float64), X) and np.array_equal(L116.astype(np.float64), L1)
    return {"X": X16, "W_res": W, "L1": L116, "L2": L2,
            "qx": qx, "sx": sx, "ql1": ql1, "sl1": sl1}


def load_qh_ties():
    """The fixture tests/golden/qh_ties.txt as a dict of lists."""
    out = {}
    with open(os.path.join(HERE, "golden", "qh_ties.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, rest = line.partition(" ")
            out[key] = [float(t) for t in rest.split()]
    return out


def qh_tie_layer(M: int, N: int, r: int = 8, K: int = GROUP, gpos: int = 0, seed: int = 0):
    """The designed layer of tests/golden/qh_ties.txt, widened to r ranks and
    K input channels.  Rank column j takes the fixture's column j % 8, so every
    rank group (8 columns or more, starting at a multiple of 8) holds the
    column with a + b = 14 and keeps s_H = u_t.  The design sits in K-group
    `gpos`; the activations are zero in every other K-group (scale 0, codes 0:
    those groups add nothing), and the weights there are random.  Token t takes
    the fixture's token scale u[t % len(u)].  Returns the fp16 inputs and the
    expected H / s_H and Q_H per token [M, r]."""
    fx = load_qh_ties()
    a, b, u = np.array(fx["a"]), np.array(fx["b"]), np.array(fx["u"])
    t8, q8 = np.array(fx["t"]), np.array(fx["qh"]).astype(np.int64)
    g = _rng(41, M, N, r, K, gpos, seed)
    k0 = gpos * GROUP
    X = np.zeros((M, K))
    ut = u[np.arange(M) % len(u)]
    X[:, k0 + 0] = ut
    X[:, k0 + 2] = ut
    X[:, k0 + 63] = 7 * ut
    L1 = (g.standard_normal((K, r)) * 0.1)
    L1[k0:k0 + GROUP, :] = 0.0
    cols = np.arange(r) % 8
    L1[k0 + 0, :] = a[cols] / 2
    L1[k0 + 2, :] = b[cols] / 2
    L1[k0 + 1, :] = 3.5
    W = g.standard_normal((N, K)) * 0.05
    L2 = g.standard_normal((r, N)) * 0.1
    d = {"X": X.astype(np.float16), "W_res": W.astype(np.float16),
         "L1": L1.astype(np.float16), "L2": L2.astype(np.float16)}
    assert np.array_equal(d["X"].astype(np.float64), X)
    assert np.array_equal(d["L1"][k0:k0 + GROUP].astype(np.float64), L1[k0:k0 + GROUP])
    d["t"] = np.tile(t8[cols], (M, 1))
    d["qh"] = np.tile(q8[cols], (M, 1))
    return d
