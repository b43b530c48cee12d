"""GPU parity at every point of the five workload configurations (the tiny
layer, LLaMA3-8B q/o and MLP, the Qwen3-8B rank sweep and the LLaMA3-70B
layers, each at its token counts): 44 points; and the LLaMA3-70B points again
with the paper's default 128-wide quantization groups (Sec. 5.1).

At each point the activation codes and scales are compared bit-exactly over
all tokens, H, s_H and Q_H bit-exactly and Y at the tolerance (bit-exactly
where the kernel sums in the oracle's order) over the checked tokens: every
token where M*N*K <= 2e11, else 64 seeded tokens including the first and the
last, across all N.  Weight codes and scales are compared once per layer.
Each layer's weights are drawn and packed once per module.
"""
import functools

import numpy as np
import pytest

import paper_2606_01556_amd as tq
from tq_synth import GROUP, WORKLOADS, activations, weights
from test_gpu_parity import check_output, dev, say

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]

FULL_LIMIT = 2e11
SAMPLE_ROWS = 64


def config_points():
    pts = []
    for name, wl in WORKLOADS.items():
        for li, layer in enumerate(wl.layers):
            for M in wl.Ms:
                pts.append(pytest.param(name, li, M, id=f"{name}-{layer.name}-M{M}"))
    return pts


POINTS = config_points()
assert len(POINTS) == 44


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tq.lib()
    yield
    _layer.cache_clear()
    torch.cuda.synchronize()


@functools.lru_cache(maxsize=2)
def _layer(name, li, group=GROUP):
    wl = WORKLOADS[name]
    w = weights(wl, wl.layers[li])
    lay = tq.Layer(dev(w["W_res"]), dev(w["L1"]), dev(w["L2"]), group=group)
    return w, lay, {"weights_checked": False}


def _check_weights(oracle_mod, w, lay):
    d = lay.desc
    N, K, r, G = d.n, d.k, d.rank, d.group
    wc = torch.empty((N, K // 8), dtype=torch.int32, device="cuda")
    ws = torch.empty((N, K // G), dtype=torch.float16, device="cuda")
    l1c = torch.empty((r, K // 8), dtype=torch.int32, device="cuda")
    l1s = torch.empty((r, K // G), dtype=torch.float16, device="cuda")
    l2c = torch.empty((N, r // 8), dtype=torch.int32, device="cuda")
    l2s = torch.empty((N, r // d.group_r), dtype=torch.float16, device="cuda")
    tq.export_weights(d, lay.packed, wc, ws, l1c, l1s, l2c, l2s)
    torch.cuda.synchronize()
    qw, sw = oracle_mod.quantize(w["W_res"], G)
    np.testing.assert_array_equal(tq.tq4_decode(wc.cpu().numpy()), qw)
    np.testing.assert_array_equal(ws.cpu().numpy().view(np.uint16), sw.view(np.uint16))
    q1, s1 = oracle_mod.quantize(w["L1"], G, axis=0)
    np.testing.assert_array_equal(tq.tq4_decode(l1c.cpu().numpy()).T, q1)
    np.testing.assert_array_equal(l1s.cpu().numpy().T.view(np.uint16), s1.view(np.uint16))
    q2, s2 = oracle_mod.quantize(w["L2"], min(G, r), axis=0)
    np.testing.assert_array_equal(tq.tq4_decode(l2c.cpu().numpy()).T, q2)
    np.testing.assert_array_equal(l2s.cpu().numpy().T.view(np.uint16), s2.view(np.uint16))


@pytest.mark.parametrize("name,li,M", POINTS)
def test_config_point(oracle_mod, name, li, M):
    check_point(oracle_mod, name, li, M, GROUP)


# The LLaMA3-70B layers with the paper's default group width of 128 (every
# kernel takes it; past 512 tokens the prefill kernel runs it)
G128_POINTS = [pytest.param("llama3-70b", li, M, id=f"llama3-70b-{l.name}-M{M}-g128")
               for li, l in enumerate(WORKLOADS["llama3-70b"].layers) for M in WORKLOADS["llama3-70b"].Ms]


@pytest.mark.parametrize("name,li,M", G128_POINTS)
def test_config_point_group128(oracle_mod, name, li, M):
    check_point(oracle_mod, name, li, M, 128)


def check_point(oracle_mod, name, li, M, group):
    wl = WORKLOADS[name]
    layer = wl.layers[li]
    K, N, r = layer.K, layer.N, layer.r
    say(f"{name} {layer.name} M={M} K={K} N={N} r={r} group={group}")
    w, lay, state = _layer(name, li, group)
    if not state["weights_checked"]:
        _check_weights(oracle_mod, w, lay)
        state["weights_checked"] = True
    X = activations(wl, M, K)
    xd = dev(X)
    xc, xs = tq.empty_act(M, K, group=group)
    tq.quant_act(xd, xc, xs, group)
    y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    h = torch.empty((M, r), dtype=torch.float32, device="cuda")
    sh = torch.empty((M, r // lay.desc.group_r), dtype=torch.float32, device="cuda")
    qh = torch.empty((M, r), dtype=torch.int8, device="cuda")
    tq.dual_gemm_debug(lay.desc, lay.packed, xc, xs, M, y, h, sh, qh)
    torch.cuda.synchronize()
    kernel = tq.dual_gemm_kernel(lay.desc, M)
    # activation codes and scales, every token
    qx, sx = oracle_mod.quantize(X, group)
    np.testing.assert_array_equal(tq.act_codes_rows(xc.cpu().numpy(), M), qx)
    np.testing.assert_array_equal(xs.cpu().numpy()[:, :M].T.view(np.uint16), sx.view(np.uint16))
    del qx, sx
    if M * N * K <= FULL_LIMIT:
        rows = np.arange(M)
    else:
        rng = np.random.default_rng(M + N + K + r)
        rows = np.unique(np.concatenate([[0, M - 1], rng.choice(M, SAMPLE_ROWS - 2, replace=False)]))
        while len(rows) < SAMPLE_ROWS:
            rows = np.unique(np.concatenate([rows, rng.integers(0, M, SAMPLE_ROWS - len(rows))]))
    o = oracle_mod.layer(X, w["W_res"], w["L1"], w["L2"], group, rows=rows)
    np.testing.assert_array_equal(h.cpu().numpy()[rows].view(np.uint32), o["H"].view(np.uint32))
    np.testing.assert_array_equal(sh.cpu().numpy()[rows].view(np.uint32), o["sH"].view(np.uint32))
    np.testing.assert_array_equal(qh.cpu().numpy()[rows], o["qH"])
    g = {"kernel": kernel, "Y": y.float().cpu().numpy(),
         "Ybits": y.view(torch.int16).cpu().numpy().view(np.uint16)}
    check_output(g, o, False, rows=rows, cols=np.arange(N))
    assert np.all(np.isfinite(g["Y"]))
