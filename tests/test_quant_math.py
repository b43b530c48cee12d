"""CPU check of the activation quantizer's division-free rounding.

The kernel forms the code of an fp16 value v in a group with fp16 scale s as
rint(v * y), y an approximate reciprocal of s, and resolves exact half-integer
quotients with the exact remainder v - q s (round half to even).  That equals
rint of the IEEE fp32 quotient v / s -- the definition, Eq. (1) -- for every
fp16 v, s because a non-tie quotient of two fp16 values is never within 2.4e-4
of a half-integer.  This test evaluates the same arithmetic in numpy (float32
products and rounding, the fma remainder in float64, where it is exact) with
reciprocals up to 2 ulp off, over all fp16 values v with |v| <= 7.5 s, for
several hundred scales (normal and subnormal fp16), against numpy's IEEE
float32 division.
"""
import numpy as np


def _codes_reference(v32, s32):
    q = np.rint(v32 / s32)
    return np.clip(q, -7, 7)


def _codes_fast(v32, s32, y32):
    q = np.rint((v32 * y32).astype(np.float32))
    r = (v32.astype(np.float64) - q.astype(np.float64) * np.float64(s32)).astype(np.float32)
    tie = (np.abs(r) == np.float32(0.5) * s32) & (np.mod(q, 2) != 0)
    q = np.where(tie, q + np.sign(r), q)
    return np.clip(q, -7, 7)


def test_fast_rounding_matches_ieee_division():
    rng = np.random.default_rng(5)
    all16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16).view(np.float16)
    finite = all16[np.isfinite(all16)].astype(np.float32)
    # scales: random normal fp16 significands at several exponents, subnormals,
    # and scales with few significant bits (where exact ties are common)
    sig = rng.integers(1024, 2048, 240)
    exps = rng.integers(-14, 12, 240)
    scales = [np.float32(np.float16(s * 2.0 ** (e - 10))) for s, e in zip(sig, exps)]
    scales += [np.float32(np.float16(k * 2.0 ** -24)) for k in (1, 3, 5, 7, 100, 1023)]
    scales += [np.float32(np.float16(v)) for v in (3.0, 5.0, 0.375, 1.25, 1.75, 6.0, 11 / 4, 13 / 32)]
    checked = ties = 0
    for s in scales:
        assert np.isfinite(s) and s > 0
        v = finite[np.abs(finite) <= 7.5 * s]
        ref = _codes_reference(v, s)
        y0 = np.float32(1.0) / s
        for d in (-2, -1, 0, 1, 2):
            y = y0
            for _ in range(abs(d)):
                y = np.nextafter(y, np.float32(np.inf if d > 0 else -np.inf))
            np.testing.assert_array_equal(_codes_fast(v, s, np.float32(y)), ref)
        checked += v.size
        ties += int(np.count_nonzero(np.abs(v / s - np.trunc(v / s)) == 0.5))
    assert checked > 1_000_000 and ties > 1000
