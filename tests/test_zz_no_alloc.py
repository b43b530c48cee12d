"""GPU test of tq_dual_gemm_unfused_noalloc, the entry point for callers that
cannot allocate: through the C ABI, its output must equal tq_dual_gemm_unfused's
(same kernels, caller scratch) bit for bit, on two calls in a row, the second
with a smaller input, and it must reject a call whose scratch exceeds the
static buffer before launching anything."""
import ctypes

import numpy as np
import pytest

import paper_2606_01556_amd as tq
from tq_synth import random_codes_layer

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tq.lib()
    yield
    torch.cuda.synchronize()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _call_both(lay, X, bf16):
    M, K = X.shape
    xc, xs = tq.empty_act(M, K)
    tq.quant_act(dev(X), xc, xs)
    dt = torch.bfloat16 if bf16 else torch.float16
    y_ref = torch.empty((M, lay.n), dtype=dt, device="cuda")
    scratch = tq.empty_unfused_scratch(lay.desc, M)
    tq.dual_gemm_unfused(lay.desc, lay.packed, xc, xs, M, y_ref, scratch, bf16)
    y_na = torch.full((M, lay.n), float("nan"), dtype=dt, device="cuda")
    tq.dual_gemm_unfused_noalloc(lay.desc, lay.packed, xc, xs, M, y_na, bf16)
    torch.cuda.synchronize()
    return (y_ref.view(torch.int16).cpu().numpy(), y_na.view(torch.int16).cpu().numpy())


@pytest.mark.parametrize("K,N,r,bf16", [(1024, 512, 64, False), (4096, 4096, 128, True)])
def test_noalloc_matches_caller_scratch(K, N, r, bf16):
    d = random_codes_layer(640, K, N, r, seed=5)
    lay = tq.Layer(dev(d["W_res"]), dev(d["L1"]), dev(d["L2"]))
    # two calls in a row on the same static array, the second smaller; the
    # first (640 tokens) runs the 8-bit activation format, the second the
    # 4-bit one, so the second reads scratch rows the first also wrote
    for M in (640, 37, 1):
        say("noalloc", K, N, r, "bf16" if bf16 else "f16", "M =", M)
        ref, got = _call_both(lay, d["X"][:M], bf16)
        np.testing.assert_array_equal(got, ref)


def test_noalloc_rejects_oversized_call():
    K, N, r = 1024, 256, 128
    d = random_codes_layer(8, K, N, r, seed=6)
    lay = tq.Layer(dev(d["W_res"]), dev(d["L1"]), dev(d["L2"]))
    M = 13000   # needs more scratch than the static buffer (8 MiB at r = 128)
    assert tq.unfused_scratch_bytes(lay.desc, M) > tq.NOALLOC_SCRATCH_BYTES
    xc, xs = tq.empty_act(M, K)
    y = torch.zeros((M, N), dtype=torch.float16, device="cuda")
    say("noalloc oversized M =", M)
    rc = tq.lib().tq_dual_gemm_unfused_noalloc(ctypes.byref(lay.desc), xc.data_ptr(), xc.data_ptr(),
                                               xs.data_ptr(), M, y.data_ptr(), 0, None)
    assert rc == 9, tq.STATUS.get(rc, rc)
    torch.cuda.synchronize()
    assert int(y.view(torch.int16).abs().sum()) == 0   # nothing written
