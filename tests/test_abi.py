"""CPU tests of the C ABI: the library loads, exports every declared entry
point, and validates arguments on the host without touching a GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_01556_amd as tq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "tq.h")).read()
    return sorted(set(re.findall(r"\b(tq_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(tq.LIB_PATH):
        from paper_2606_01556_amd import build
        build.build()
    return tq.lib()


def test_exports_every_declared_symbol(L):
    syms = declared_symbols()
    assert set(syms) == set(tq.EXPORTS)
    for s in syms:
        assert hasattr(L, s), s


def test_status_strings(L):
    for code in range(0, 10):
        assert L.tq_status_string(code) != b"unknown status"
    assert L.tq_status_string(1234) == b"unknown status"


@pytest.mark.parametrize("n,k,r,g,code", [
    (512, 512, 16, 64, 0), (4096, 4096, 64, 64, 0), (100, 64, 0, 64, 0), (1, 64, 128, 64, 0),
    (512, 512, 16, 128, 0), (512, 576, 16, 128, 3), (512, 512, 16, 32, 3), (512, 512, 16, 256, 3),
    (512, 500, 16, 64, 3), (0, 512, 16, 64, 2), (512, 0, 16, 64, 2),
    (512, 512, 24, 64, 4), (512, 512, 256, 64, 4), (512, 512, -8, 64, 4),
])
def test_desc_init_validation(L, n, k, r, g, code):
    d = tq.WeightDesc()
    assert L.tq_weight_desc_init(n, k, r, g, ctypes.byref(d)) == code


def test_desc_init_null(L):
    assert L.tq_weight_desc_init(64, 64, 0, 64, None) == 1


def test_desc_sizes(L):
    d = tq.weight_desc_init(4096, 4096, 64)
    assert d.n_pad == 4096 and d.r_pad32 == 64 and d.r_pad64 == 64 and d.group_r == 64
    # codes: n*k/2 + scales 2*n*k/64 + L1 codes k*r/2 + scales + L2 codes + scales
    # + 1 KiB of zeros after each code section and a zero row after each
    # K-group scale section; sections start at multiples of 256 bytes
    up = lambda b: (b + 255) // 256 * 256
    expect = (up(4096 * 4096 // 2 + 1024) + up(2 * 4096 * 65) + up(4096 * 64 // 2 + 1024) + up(2 * 64 * 65)
              + up(4096 * 64 // 2) + up(2 * 4096))
    assert d.packed_bytes == expect
    offs = [d.off_w, d.off_ws, d.off_l1, d.off_l1s, d.off_l2, d.off_l2s, d.packed_bytes]
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
    d2 = tq.weight_desc_init(100, 128, 16)
    assert d2.n_pad == 128 and d2.r_pad32 == 32 and d2.r_pad64 == 64 and d2.group_r == 16
    # 128-wide groups: codes in the same 64-wide blocks, one scale row per 128
    d3 = tq.weight_desc_init(4096, 4096, 128, 128)
    assert d3.group == 128 and d3.group_r == 128
    expect3 = (up(4096 * 4096 // 2 + 1024) + up(2 * 4096 * 33) + up(4096 * 128 // 2 + 1024) + up(2 * 128 * 33)
               + up(4096 * 128 // 2) + up(2 * 4096))
    assert d3.packed_bytes == expect3


FAKE = 1 << 20     # 16-byte aligned fake device address; never dereferenced


def test_quant_act_validation(L):
    assert L.tq_quant_act(None, 4, 64, 64, FAKE, FAKE, None) == 1
    assert L.tq_quant_act(FAKE, 4, 64, 32, FAKE, FAKE, None) == 3
    assert L.tq_quant_act(FAKE, 4, 100, 64, FAKE, FAKE, None) == 3
    assert L.tq_quant_act(FAKE, -1, 64, 64, FAKE, FAKE, None) == 2
    assert L.tq_quant_act(FAKE, 65535 * 32 + 1, 64, 64, FAKE, FAKE, None) == 2   # more token tiles than the grid holds
    assert L.tq_quant_act(FAKE + 8, 4, 64, 64, FAKE, FAKE, None) == 6
    assert L.tq_quant_act(FAKE, 0, 64, 64, FAKE, FAKE, None) == 0      # empty: no launch


def test_dual_gemm_validation(L):
    d = tq.weight_desc_init(128, 128, 16)
    bad = tq.WeightDesc()
    D = ctypes.byref
    assert L.tq_dual_gemm(D(d), None, FAKE, FAKE, 4, FAKE, 0, None) == 1
    assert L.tq_dual_gemm(D(bad), FAKE, FAKE, FAKE, 4, FAKE, 0, None) == 7
    assert L.tq_dual_gemm(D(d), FAKE, FAKE, FAKE, 4, FAKE, 7, None) == 5
    assert L.tq_dual_gemm(D(d), FAKE, FAKE, FAKE, -2, FAKE, 0, None) == 2
    assert L.tq_dual_gemm(D(d), FAKE, FAKE + 4, FAKE, 4, FAKE, 0, None) == 6
    assert L.tq_dual_gemm(D(d), FAKE, FAKE, FAKE, 0, FAKE, 0, None) == 0
    # a descriptor edited after init is rejected
    d3 = tq.weight_desc_init(128, 128, 16)
    d3.n_pad = 64
    assert L.tq_dual_gemm(D(d3), FAKE, FAKE, FAKE, 4, FAKE, 0, None) == 7


def test_debug_entry_validation(L):
    """The test entry: H / s_H / Q_H copies all or none (and only with r > 0),
    forced kernels only where they serve m, mid tile counts 1, 2, 4."""
    d = tq.weight_desc_init(128, 128, 16)
    d0 = tq.weight_desc_init(128, 128, 0)
    D = ctypes.byref
    dbg = lambda dd, m, kern, ct, h, sh, qh, x=None, xc=FAKE: L.tq_dual_gemm_debug(
        D(dd), FAKE, xc, xc, x, m, FAKE, 0, kern, ct, h, sh, qh, None)
    assert dbg(d0, 4, -1, 0, FAKE, FAKE, FAKE) == 4
    assert dbg(d, 4, -1, 0, None, FAKE, FAKE) == 1
    assert dbg(d, 4, 4, 0, None, None, None) == 2            # no such kernel
    assert dbg(d, 4, -2, 0, None, None, None) == 2
    assert dbg(d, 4, 2, 0, None, None, None) == 2            # large kernel needs m > 512
    assert dbg(d, 100, 3, 0, None, None, None) == 2          # prefill kernel needs m > 512
    assert dbg(d, 17, 0, 0, None, None, None) == 2           # decode kernel needs m <= 16
    assert dbg(d, 4, 1, 3, None, None, None) == 2            # mid tiles 1, 2 or 4
    # the fused-quantization path: no codes, decode kernel only
    assert dbg(d, 4, -1, 0, None, None, None, x=FAKE) == 2
    assert dbg(d, 4, 1, 0, None, None, None, x=FAKE, xc=None) == 2
    assert dbg(d, 17, -1, 0, None, None, None, x=FAKE, xc=None) == 2


def test_fused_quant_validation(L):
    D = ctypes.byref
    d = tq.weight_desc_init(128, 4096, 64)
    assert L.tq_dual_gemm_fused_quant(D(d), FAKE, None, 4, FAKE, 0, None) == 1
    assert L.tq_dual_gemm_fused_quant(D(d), FAKE, FAKE + 2, 4, FAKE, 0, None) == 6
    assert L.tq_dual_gemm_fused_quant(D(d), FAKE, FAKE, 17, FAKE, 0, None) == 2
    assert L.tq_dual_gemm_fused_quant(D(d), FAKE, FAKE, 0, FAKE, 0, None) == 0
    # the activation codes of m tokens must fit the decode kernel's LDS
    big = tq.weight_desc_init(128, 14400, 64)
    assert L.tq_dual_gemm_fused_quant(D(big), FAKE, FAKE, 16, FAKE, 0, None) == 2


def test_desc_rejects_4gib_packed_buffer(L):
    d = tq.WeightDesc()
    assert L.tq_weight_desc_init(1 << 17, 1 << 16, 0, 64, ctypes.byref(d)) == 2
    assert L.tq_weight_desc_init(1 << 16, 1 << 16, 0, 64, ctypes.byref(d)) == 0
    assert d.packed_bytes < (1 << 32)


def test_noalloc_validation(L):
    """The allocation-free entry point validates on the host and rejects a call
    whose scratch exceeds the static buffer before touching any device."""
    d = tq.weight_desc_init(128, 1024, 128)
    D = ctypes.byref
    assert L.tq_dual_gemm_unfused_noalloc(D(d), None, FAKE, FAKE, 4, FAKE, 0, None) == 1
    assert L.tq_dual_gemm_unfused_noalloc(D(d), FAKE, FAKE, FAKE, 4, FAKE, 9, None) == 5
    assert tq.unfused_scratch_bytes(d, 12928) <= tq.NOALLOC_SCRATCH_BYTES
    assert tq.unfused_scratch_bytes(d, 12929) > tq.NOALLOC_SCRATCH_BYTES
    assert L.tq_dual_gemm_unfused_noalloc(D(d), FAKE, FAKE, FAKE, 12929, FAKE, 0, None) == 9
    assert L.tq_dual_gemm_unfused_noalloc(D(d), FAKE, FAKE, FAKE, 0, FAKE, 0, None) == 0


def test_pack_export_validation(L):
    d = tq.weight_desc_init(128, 128, 16)
    D = ctypes.byref
    assert L.tq_pack_weights(D(d), FAKE, None, FAKE, FAKE, None) == 1
    assert L.tq_pack_weights(D(d), FAKE + 2, FAKE, FAKE, FAKE, None) == 6
    assert L.tq_export_weights(D(d), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, None) == 1
    d0 = tq.weight_desc_init(128, 128, 0)
    assert L.tq_export_weights(D(d0), FAKE, FAKE, FAKE + 1, None, None, None, None, None) == 6


def test_canonical_export_validation(L):
    d = tq.weight_desc_init(256, 256, 16)
    assert L.tq_export_weights_canonical(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 1
    assert L.tq_export_weights_canonical(ctypes.byref(d), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, None) == 1
    assert L.tq_export_weights_canonical(ctypes.byref(d), FAKE + 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 6
    bad = tq.WeightDesc()
    assert L.tq_export_weights_canonical(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 7
    assert L.tq_act_codes_canonical(None, FAKE, 4, 64, 64, FAKE, FAKE, None) == 1
    assert L.tq_act_codes_canonical(FAKE, FAKE, 4, 64, 32, FAKE, FAKE, None) == 3
    assert L.tq_act_codes_canonical(FAKE, FAKE, 4, 192, 128, FAKE, FAKE, None) == 3
    assert L.tq_act_codes_canonical(FAKE, FAKE, -1, 64, 64, FAKE, FAKE, None) == 2
    assert L.tq_act_codes_canonical(FAKE, FAKE, 4, 64, 64, FAKE + 2, FAKE, None) == 6
    assert L.tq_act_codes_canonical(FAKE, FAKE, 0, 64, 64, FAKE, FAKE, None) == 0


def test_canonical_decode_helper():
    """Two's-complement nibbles, element 2i low: the binding's host decoder."""
    codes = np.array([[0, 1, -1, 7, -7, 3, -4, 2]], dtype=np.int8)
    b = (codes[:, 0::2].astype(np.uint8) & 0xF) | ((codes[:, 1::2].astype(np.uint8) & 0xF) << 4)
    assert b.tolist() == [[0x10, 0x7F, 0x39, 0x2C]]
    np.testing.assert_array_equal(tq.canonical_decode(b), codes)


def test_tq4_roundtrip():
    g = np.random.default_rng(0)
    c = g.integers(-7, 8, size=(5, 64)).astype(np.int8)
    w = tq.tq4_encode(c)
    assert w.shape == (5, 8)
    np.testing.assert_array_equal(tq.tq4_decode(w), c)
    # the documented bit positions, spelled out for one word
    one = np.array([[1, -2, 3, -4, 5, -6, 7, 0]], np.int8)
    word = int(tq.tq4_encode(one)[0, 0])
    assert word & 0x87 == 0x01
    assert (word >> 8) & 0x87 == 0x82
    assert (word >> 4) & 7 == 5 and (word >> 11) & 1 == 0      # c4 = +5, sign in bit 11
    assert (word >> 12) & 7 == 6 and (word >> 19) & 1 == 1     # c5 = -6, sign in bit 19
    assert (word >> 28) & 7 == 0 and (word >> 3) & 1 == 0      # c7 = 0, sign in bit 3


def test_act_codes_tile_layout_roundtrip():
    """act_codes_rows inverts the tile-major activation layout of tq_quant_act:
    token 32 t + i, codes 32 h .. 32 h + 31 of group g sit in 16-byte lane slot
    32 h + i of the 1 KiB block (t, g)."""
    rng = np.random.default_rng(5)
    m, k = 45, 192
    m32 = tq.padded_tokens(m)
    codes = np.zeros((m32, k), np.int8)
    codes[:m] = rng.integers(-7, 8, size=(m, k))
    kg = k // 64
    blocks = np.zeros((m32 // 32, kg, 64, 4), np.uint32)   # tile, group, lane slot, word
    for t in range(m32 // 32):
        for g in range(kg):
            for h in range(2):
                for i in range(32):
                    seg = codes[32 * t + i, 64 * g + 32 * h: 64 * g + 32 * h + 32]
                    blocks[t, g, 32 * h + i] = tq.tq4_encode(seg)
    back = tq.act_codes_rows(blocks.reshape(m32 // 32, kg, 256), m)
    np.testing.assert_array_equal(back, codes[:m])
    assert tq.padded_tokens(1) == 32 and tq.padded_tokens(32) == 32 and tq.padded_tokens(33) == 64


def test_act_codes_fp8_layout_roundtrip():
    """act_codes_rows inverts the fp8 activation layout used above 512 tokens:
    token 32 t + i, codes 32 h + 16 p .. + 15 of group g are the bytes
    sign << 7 | |q| of lane slot 32 h + i in half p of the 2 KiB block (t, g)."""
    rng = np.random.default_rng(6)
    m, k = 520, 128
    m32 = tq.padded_tokens(m)
    codes = np.zeros((m32, k), np.int8)
    codes[:m] = rng.integers(-7, 8, size=(m, k))
    kg = k // 64
    blocks = np.zeros((m32 // 32, kg, 2, 64, 16), np.uint8)   # tile, group, half p, slot, byte
    for t in range(m32 // 32):
        for g in range(kg):
            for p in range(2):
                for h in range(2):
                    for i in range(32):
                        q = codes[32 * t + i, 64 * g + 32 * h + 16 * p: 64 * g + 32 * h + 16 * p + 16]
                        blocks[t, g, p, 32 * h + i] = np.where(q < 0, 0x80 | -q.astype(np.int16), q)
    back = tq.act_codes_rows(blocks.view(np.uint32).reshape(m32 // 32, kg, 512), m)
    np.testing.assert_array_equal(back, codes[:m])
    assert tq.fp8_code_decode(np.array([0x87, 0x07, 0x00, 0x81], np.uint8)).tolist() == [-7, 7, 0, -1]


def test_act_codes_bytes(L):
    """x_codes sizes: 4 bits per code up to 512 tokens, 8 bits beyond; 0 for bad shapes."""
    assert L.tq_act_codes_bytes(1, 4096) == 32 * 4096 // 2
    assert L.tq_act_codes_bytes(512, 4096) == 512 * 4096 // 2
    assert L.tq_act_codes_bytes(513, 4096) == 544 * 4096
    assert L.tq_act_codes_bytes(2048, 64) == 2048 * 64
    assert L.tq_act_codes_bytes(0, 4096) == 0
    assert L.tq_act_codes_bytes(16, 100) == 0 and L.tq_act_codes_bytes(-1, 64) == 0


def test_unfused_sizes_and_validation(L):
    """Scratch of the unfused layer: H fp32 [m32][r_pad32], Q_H [m32][r_pad64],
    s_H [r/group_r][m32], each at a 256-byte-aligned offset; 0 for a bad
    descriptor; argument errors as tq_dual_gemm."""
    D = tq.WeightDesc
    d = tq.weight_desc_init(4096, 4096, 64, 64)
    up = lambda v: (v + 255) // 256 * 256
    assert L.tq_unfused_scratch_bytes(ctypes.byref(d), 1) == up(32 * 64 * 4) + up(32 * 64) + up(32 * 4)
    d8 = tq.weight_desc_init(512, 256, 8, 64)
    assert L.tq_unfused_scratch_bytes(ctypes.byref(d8), 40) == up(64 * 32 * 4) + up(64 * 64) + up(64 * 4)
    bad = D()
    assert L.tq_unfused_scratch_bytes(ctypes.byref(bad), 16) == 0
    assert L.tq_dual_gemm_unfused(ctypes.byref(d), FAKE, FAKE, FAKE, 1, FAKE, 0, None, None) == 1
    assert L.tq_dual_gemm_unfused(ctypes.byref(d), FAKE, FAKE, FAKE, 1, FAKE, 0, FAKE + 4, None) == 6
    assert L.tq_dual_gemm_unfused(ctypes.byref(d), FAKE, FAKE, FAKE, 0, FAKE, 0, FAKE, None) == 0


def test_kernel_choice(L):
    """tq_dual_gemm_kernel: the decode kernel up to 16 tokens (while their
    activation codes fit its LDS), the mid kernel up to 512, past that the
    large kernel where its 128 x 256 blocks fill the CUs, the mid kernel where
    they would leave most CUs idle, the prefill kernel beyond one round of
    blocks (for r <= 64 in 64-wide groups only where a work-group's run of
    column blocks spans at least 256 K-groups; in 128-wide groups at every
    rank but 0); -1 for a bad descriptor or m."""
    d = tq.weight_desc_init(4096, 4096, 64)           # n, k, r
    assert [tq.dual_gemm_kernel(d, m) for m in (1, 16, 17, 512, 2048)] == \
        ["decode", "decode", "mid", "mid", "large"]
    assert tq.dual_gemm_kernel(tq.weight_desc_init(96, 4096, 64), 600) == "mid"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(14336, 4096, 128), 4096) == "prefill"
    # r = 64 beyond one round: runs of 7 blocks x 64 groups take the prefill
    # kernel, runs of 2 x 64 stay on the large kernel
    assert tq.dual_gemm_kernel(tq.weight_desc_init(14336, 4096, 64), 4096) == "prefill"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 64), 4096) == "large"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 14336, 64), 4096) == "prefill"
    # 128-wide groups: past one round of blocks the prefill kernel unless r = 0
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 64, 128), 4096) == "prefill"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 16, 128), 4096) == "prefill"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 0, 128), 4096) == "large"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 128, 128), 2048) == "large"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(28672, 8192, 128, 128), 8192) == "prefill"
    # the mid kernel's threshold over the large kernel is lower for 128-wide
    # groups (28 against 34 of its cost units per round of large blocks)
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 0), 1024) == "mid"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 4096, 0, 128), 1024) == "large"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 14336, 128), 576) == "mid"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 14336, 128, 128), 576) == "large"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(8192, 28672, 128), 1) == "decode"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(8192, 28672, 128), 8) == "decode"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(8192, 28672, 128), 9) == "mid"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 14336, 64), 16) == "decode"
    assert tq.dual_gemm_kernel(tq.weight_desc_init(4096, 14400, 64), 16) == "mid"
    assert L.tq_dual_gemm_kernel(ctypes.byref(d), 0) == -1
    assert L.tq_dual_gemm_kernel(ctypes.byref(tq.WeightDesc()), 100) == -1
    assert L.tq_dual_gemm_kernel(None, 100) == -1
    with pytest.raises(ValueError):
        tq.dual_gemm_kernel(d, 0)
