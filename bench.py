#!/usr/bin/env python3
"""Benchmark of the TwinQuant dual-component W4A4 linear layer on one MI355X.

One step = one forward of each LLaMA3-70B-shaped layer on one GPU (gate_up
K = 8192 -> N = 28672 and down K = 28672 -> N = 8192, rank 128, group 64) at
each token count M in {8192, 1, 32}: six layer calls.  A layer call is the
whole layer from fp16 activations: for a single token the one fused launch
that quantizes the activation in its prologue (tq_dual_gemm_fused_quant),
otherwise the quantizer (tq_quant_act) followed by the fused layer
(tq_dual_gemm).  (Quantizing inside the kernel repeats the work in every
work-group: it wins at one token and loses at sixteen, where per_m shows both.)
Inputs are seeded synthetic tensors of the workload's distributions, resident
in HBM before timing starts.  The packed weights are replicated over >= 1 GiB
of distinct copies and the activations and outputs over several copies, and
every call takes the next copy, so decode-sized calls read their operands from
HBM rather than from the 256 MB last-level cache.

Prints one JSON line: nominal TFLOPS (2 M N K summed over the step / step
time), per-call microseconds next to an fp16 GEMM of the same shape
(torch.matmul -> hipBLASLt) and next to the same layer without kernel fusion
(tq_dual_gemm_unfused), the roofline position of the dominant kernel (the
M = 8192 calls, fp8 matrix-core bound) and of the single-token kernel (HBM
bound), each timed with HIP events on its launch stream inside the timed
region, and the CPU oracle timed on the host as a reported baseline.

Other modes print markdown tables (--configs, --ranks, --kernel-choice), run
one layer call repeatedly for a profiler (--kernel-only), or turn rocprofv3
output into the summaries kept under profiles/ (--trace-summary,
--traffic-summary).
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "dual-component W4A4 linear: µs/layer & TFLOPS (M=1..4096) vs fp16 GEMM"
HEADLINE = "llama3-70b"
HEAD_MS = (8192, 1, 32)    # step order: the long calls first, so the queue never drains
DETAIL_EXTRA = "llama3-8b-qo"
GROUP = 64
FP8_MFMA_PEAK_TFLOPS = 5000.0   # MI355X dense fp8 matrix peak (5.0 PFLOP/s)
HBM_PEAK_GBS = 8000.0
ROTATE_BYTES = 1 << 30
CALIB_COPY_BYTES = 256 << 20
CPU_SLICE_ROWS = 64
FUSED_QUANT_MAX_M = 1      # layer calls up to this many tokens quantize inside the kernel
CSRC = os.path.join(ROOT, "paper_2606_01556_amd", "csrc")
KERNEL_SOURCES = {"decode": "tq_gemm_decode.hip", "mid": "tq_gemm_mid.hip",
                  "large": "tq_gemm_large.hip", "prefill": "tq_gemm_prefill.hip"}


# ---------------------------------------------------------------------------
# algorithmic work
# ---------------------------------------------------------------------------
def alg_ops(m, n, k, r):
    """Multiply-adds x 2 of the layer: residual GEMM, stage 1 and stage 2."""
    return 2.0 * m * (n * k + k * r + r * n)


def weight_bytes(n, k, r, g=GROUP):
    gr = min(g, r) if r else 1
    return (n * k / 2 + 2 * n * k / g + k * r / 2 + 2 * r * k / g + r * n / 2
            + (2 * n * r / gr if r else 0))


def alg_bytes(m, n, k, r, fused_quant):
    """Bytes a launch must move at least: packed weights once, the
    activations (fp16 for the fused-quantization entry, else 4-bit codes and
    fp16 scales) and the fp16 output."""
    act = 2 * m * k if fused_quant else m * k / 2 + 2 * m * k / GROUP
    return weight_bytes(n, k, r) + act + 2 * m * n


# ---------------------------------------------------------------------------
# committed profiler summaries
# ---------------------------------------------------------------------------
def kernel_sha(kname):
    h = hashlib.sha256()
    for f in (KERNEL_SOURCES[kname], "tq_device.hpp", "tq_kernels.hpp"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def traffic_file(kname, tag):
    return os.path.join(ROOT, "profiles", f"traffic_{kname}_kernel_{tag}.json")


def measured_traffic(kname, tag):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE runs,
    scaled by the copy-kernel calibration; None when no such summary exists
    or it was taken on another version of the kernel's source."""
    try:
        with open(traffic_file(kname, tag)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_sha(kname):
        return None
    return t.get("hbm_bytes_per_launch")


def _csv_rows(d, suffix):
    import csv
    rows = []
    for f in glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    return rows


def traffic_summary(fetch_dir, write_dir, layer_name, m, cmds):
    """Write profiles/traffic_<kernel>_kernel_<tag>.json from two rocprofv3
    --pmc runs of --kernel-only (FETCH_SIZE, then WRITE_SIZE): the kernel's
    per-dispatch KiB and the calibration by the 256 MiB copy that run does."""
    import paper_2606_01556_amd as tq
    from tq_synth import WORKLOADS
    wl = WORKLOADS[HEADLINE]
    layer = [l for l in wl.layers if l.name == layer_name][0]
    kname = tq.dual_gemm_kernel(tq.weight_desc_init(layer.N, layer.K, layer.r), m)
    sym = f"dual_gemm_{kname}_kernel"
    out = {"kernel": f"{sym}, {HEADLINE} {layer_name} (K={layer.K}, N={layer.N}, r={layer.r}) at M={m}",
           "kernel_source_sha256": kernel_sha(kname)}
    for ctr, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        per = {}
        names = {}
        for r in _csv_rows(d, "counter_collection.csv"):
            if r["Counter_Name"] != ctr:
                continue
            key = r["Dispatch_Id"]
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
            names[key] = r["Kernel_Name"]
        mine = [v for k, v in per.items() if sym in names[k]]
        others = [v for k, v in per.items() if "tq::" not in names[k]]
        if not mine or not others:
            raise SystemExit(f"{ctr}: no {sym} dispatch or no calibration copy in {d}")
        cal = max(others)   # the 256 MiB copy (or fill): the largest other dispatch
        factor = (CALIB_COPY_BYTES / 1024.0) / cal
        key = "fetch" if ctr == "FETCH_SIZE" else "write"
        out[f"{key}_size_kib_raw_per_launch"] = float(np.mean(mine))
        out[f"{key}_dispatches"] = len(mine)
        out[f"{key}_calibration_kib_raw"] = cal
        out[f"{key}_factor"] = factor
    out["hbm_bytes_per_launch"] = int(round(1024.0 * (out["fetch_size_kib_raw_per_launch"] * out["fetch_factor"]
                                                      + out["write_size_kib_raw_per_launch"] * out["write_factor"])))
    out["algorithmic_bytes_per_launch"] = int(alg_bytes(m, layer.N, layer.K, layer.r, m <= FUSED_QUANT_MAX_M))
    out["commands"] = cmds
    path = traffic_file(kname, f"{HEADLINE.replace('-', '_')}_{layer_name}_m{m}")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(path)
    print(json.dumps(out, indent=1))


def trace_summary(trace_dir, title, cmd):
    """Markdown summary of a rocprofv3 --kernel-trace --stats run: calls and
    average / total duration per kernel symbol."""
    rows = _csv_rows(trace_dir, "kernel_stats.csv")
    if not rows:
        raise SystemExit(f"no kernel_stats.csv under {trace_dir}")
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    print(f"# {title}\n")
    print("Command (from the repository root on the GPU box):\n")
    print("```\n" + cmd + "\n```\n")
    print("| kernel | calls | avg µs | min µs | max µs | share of GPU time |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        name = r["Name"]
        if len(name) > 110:
            name = name[:107] + "..."
        print(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
              f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['TotalDurationNs']) / total * 100:.1f} % |")


SIMDS = 1024          # MI355X: 256 CUs x 4 SIMDs
XCCS = 8


def counter_summary(dirs, layer_name, m, cmd):
    """Markdown summary of rocprofv3 --pmc passes of --kernel-only: the SQ
    counters of the layer's fused kernel, summed over the chip and averaged
    over its dispatches, and the unit-busy fractions derived from them."""
    import paper_2606_01556_amd as tq
    from tq_synth import WORKLOADS
    wl = WORKLOADS[HEADLINE]
    layer = [l for l in wl.layers if l.name == layer_name][0]
    kname = tq.dual_gemm_kernel(tq.weight_desc_init(layer.N, layer.K, layer.r), m)
    sym = f"dual_gemm_{kname}_kernel"
    per = {}
    for d in dirs:
        disp = {}
        for r in _csv_rows(d, "counter_collection.csv"):
            if sym not in r["Kernel_Name"]:
                continue
            key = (r["Dispatch_Id"], r["Counter_Name"])
            disp[key] = disp.get(key, 0.0) + float(r["Counter_Value"])
        by_ctr = {}
        for (_, c), v in disp.items():
            by_ctr.setdefault(c, []).append(v)
        for c, vs in by_ctr.items():
            per[c] = float(np.mean(vs))
    if not per:
        raise SystemExit(f"no {sym} dispatch in {dirs}")
    cyc = per["GRBM_GUI_ACTIVE"] / XCCS          # GPU cycles of one dispatch
    wave_cyc = per.get("SQ_WAVE_CYCLES", 0.0)    # quad-cycles, summed over waves
    print(f"# SQ counters: {sym}, {HEADLINE} {layer_name} (K={layer.K}, N={layer.N}, r={layer.r}) at M={m}\n")
    print("Commands (from the repository root on the GPU box; one rocprofv3 --pmc pass per line):\n")
    print("```\n" + cmd + "\n```\n")
    print(f"Kernel source sha256: `{kernel_sha(kname)}`. Values: per dispatch, summed over the chip,")
    print("averaged over the dispatches of the kernel.\n")
    print("| counter | value |")
    print("|---|---|")
    for c in sorted(per):
        print(f"| `{c}` | {per[c]:.4g} |")
    print("\n| derived | value |")
    print("|---|---|")
    print(f"| GPU cycles per dispatch (GRBM_GUI_ACTIVE / {XCCS} XCCs) | {cyc:.4g} |")
    if "SQ_VALU_MFMA_BUSY_CYCLES" in per:
        print(f"| matrix cores busy, share of SIMD cycles (MFMA_BUSY / (cycles x {SIMDS})) | "
              f"{per['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * SIMDS) * 100:.1f} % |")
    if wave_cyc:
        for c, label in (("SQ_ACTIVE_INST_VALU", "vector instructions active"),
                         ("SQ_ACTIVE_INST_SCA", "scalar instructions active"),
                         ("SQ_ACTIVE_INST_LDS", "LDS instructions active"),
                         ("SQ_ACTIVE_INST_ANY", "any instruction active"),
                         ("SQ_WAIT_INST_ANY", "waiting to issue"),
                         ("SQ_WAIT_ANY", "waiting on counters / barriers")):
            if c in per:
                print(f"| {label}, share of wave cycles | {per[c] / wave_cyc * 100:.1f} % |")
    if "SQ_WAVES" in per:
        w = per["SQ_WAVES"]
        for c in ("SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_INSTS_SALU"):
            if c in per:
                print(f"| `{c}` per wavefront | {per[c] / w:.0f} |")
    if "SQ_INSTS_VALU" in per and "SQ_WAVES" in per:
        print(f"| `SQ_INSTS_VALU` per wavefront | {per['SQ_INSTS_VALU'] / per['SQ_WAVES']:.0f} |")
    if "SQ_LDS_BANK_CONFLICT" in per and per.get("SQ_LDS_IDX_ACTIVE"):
        print(f"| LDS bank-conflict cycles per LDS-active cycle | "
              f"{per['SQ_LDS_BANK_CONFLICT'] / per['SQ_LDS_IDX_ACTIVE']:.3f} |")


# ---------------------------------------------------------------------------
# the CPU baseline: the oracle on the host cores
# ---------------------------------------------------------------------------
def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_oracle_child(threads):
    """Runs in a child process that imports no GPU library.  For each headline
    layer (weights drawn once), times oracle.layer on a 1-row and a 64-row
    call with `threads` OpenMP threads, then on a 1-row and a 4-row call with
    one thread (omp_set_num_threads on the oracle's own runtime), and returns
    the fixed (weight quantization) and per-row seconds of each."""
    import ctypes
    import oracle
    from tq_synth import WORKLOADS, weights, activations
    oracle.lib()
    gomp = ctypes.CDLL("libgomp.so.1")
    wl = WORKLOADS[HEADLINE]
    res = {}
    for layer in wl.layers:
        w = weights(wl, layer)
        X = activations(wl, CPU_SLICE_ROWS, layer.K)
        for th, big in ((threads, CPU_SLICE_ROWS), (1, 4)):
            gomp.omp_set_num_threads(th)
            t = {}
            for nrow in (1, big):
                t0 = time.perf_counter()
                oracle.layer(X, w["W_res"], w["L1"], w["L2"], GROUP, rows=np.arange(nrow))
                t[nrow] = time.perf_counter() - t0
            per_row = max((t[big] - t[1]) / (big - 1), 0.0)
            res.setdefault(str(th), {})[layer.name] = {
                "fixed_s": max(t[1] - per_row, 0.0), "per_row_s": per_row,
                "rows_timed": [1, big], "seconds": t[1] + t[big]}
        del w, X
    return res


def cpu_baseline(step_flops):
    """The oracle as it stands on the host: all cores, then one thread.  A
    headline layer call costs a fixed part (the weight quantization the
    oracle redoes per call) plus a part linear in M; both are measured (1-row
    and 64-row calls with all cores, 1-row and 4-row calls with one thread)
    and the step's six calls are extrapolated from them."""
    from tq_synth import WORKLOADS
    wl = WORKLOADS[HEADLINE]
    threads = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
    env = dict(os.environ, OMP_NUM_THREADS=str(threads))
    p = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-oracle-child", str(threads)],
                       env=env, capture_output=True, text=True, check=True)
    out = json.loads(p.stdout.strip().splitlines()[-1])

    def step_seconds(r):
        return sum(r[l.name]["fixed_s"] + m * r[l.name]["per_row_s"] for l in wl.layers for m in HEAD_MS)
    t_all, t_one = step_seconds(out[str(threads)]), step_seconds(out["1"])
    sampled = sum(v["seconds"] for th in out for v in out[th].values())
    return {"value": round(step_flops / t_all / 1e12, 6), "unit": "TFLOPS", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(), "nproc": len(os.sched_getaffinity(0)),
            "value_1thread": round(step_flops / t_one / 1e12, 7),
            "seconds_per_step": round(t_all, 3), "seconds_per_step_1thread": round(t_one, 3),
            "sample": (f"per headline layer, oracle calls on 1 and {CPU_SLICE_ROWS} token rows with {threads} "
                       f"threads and on 1 and 4 rows with one thread; the step's six calls "
                       f"(M = {', '.join(map(str, HEAD_MS))}) are extrapolated as fixed + M x per-row (the "
                       f"work is linear in M); {sampled:.1f} s of oracle time sampled"),
            "extrapolated": True}


# ---------------------------------------------------------------------------
# device-side setup
# ---------------------------------------------------------------------------
class LayerBench:
    """One layer's packed weights (rotated copies), and per token count the
    fp16 activations, activation codes and outputs (rotated copies)."""

    def __init__(self, wl, layer, ms, stream, with_fp16=True, group=GROUP, rank=None):
        import torch
        import paper_2606_01556_amd as tq
        from tq_synth import weights, activations
        dev = torch.device("cuda")
        self.layer = layer
        self.group = group
        self.K, self.N = layer.K, layer.N
        self.r = layer.r if rank is None else rank
        w = weights(wl, layer, rank=self.r)
        with torch.cuda.stream(stream):
            W = torch.from_numpy(w["W_res"]).to(dev)
            lay = tq.Layer(W, torch.from_numpy(w["L1"]).to(dev), torch.from_numpy(w["L2"]).to(dev),
                           group=group, stream=stream)
            self.desc = lay.desc
            self.ncopy = max(2, int(np.ceil(ROTATE_BYTES / self.desc.packed_bytes)))
            self.packed = [lay.packed] + [lay.packed.clone() for _ in range(self.ncopy - 1)]
            self.WT = []
            if with_fp16:
                WT = W.t().contiguous()
                nwt = max(2, int(np.ceil(ROTATE_BYTES / (WT.numel() * 2))))
                self.WT = [WT] + [WT.clone() for _ in range(nwt - 1)]
            del W, lay
            self.X, self.act, self.Y = {}, {}, {}
            for m in ms:
                x = torch.from_numpy(activations(wl, m, self.K)).to(dev)
                per = 2 * m * (self.K + self.N) + tq.act_codes_bytes(m, self.K)
                nx = max(2, min(self.ncopy, int(np.ceil(ROTATE_BYTES / per))))
                self.X[m] = [x] + [x.clone() for _ in range(nx - 1)]
                self.act[m] = [tq.empty_act(m, self.K, group=group) for _ in range(nx)]
                self.Y[m] = [torch.empty((m, self.N), dtype=torch.float16, device=dev) for _ in range(nx)]
        self.i = 0

    def kernel(self, m):
        import paper_2606_01556_amd as tq
        return tq.dual_gemm_kernel(self.desc, m)

    def call(self, m, s, ev=None, fused_quant=True, force=False):
        """One layer call on the next copies; ev = (start, end) events around
        the fused layer's launch (recorded on the current stream, which the
        caller makes the launch stream)."""
        import paper_2606_01556_amd as tq
        i = self.i
        self.i += 1
        p = self.packed[i % self.ncopy]
        j = i % len(self.X[m])
        x, (xc, xs), y = self.X[m][j], self.act[m][j], self.Y[m][j]
        if fused_quant and (m <= FUSED_QUANT_MAX_M or (force and m <= 16)):
            if ev is not None:
                ev[0].record()
            tq.dual_gemm_fused_quant(self.desc, p, x, y, stream=s)
        else:
            tq.quant_act(x, xc, xs, self.group, stream=s)
            if ev is not None:
                ev[0].record()
            tq.dual_gemm(self.desc, p, xc, xs, m, y, stream=s)
        if ev is not None:
            ev[1].record()


def timed(stream, fn, reps):
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        for _ in range(2):
            fn()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
    torch.cuda.synchronize()
    return 1e3 * e0.elapsed_time(e1) / reps


def detail_rows(L, ms, stream, wl_name):
    """Per token count (outside the timed region): the layer call, its parts,
    the fp16 hipBLASLt GEMM of the same shape and the layer without fusion."""
    import torch
    import paper_2606_01556_amd as tq
    s = stream.cuda_stream
    rows = []
    for m in ms:
        reps = 20 if m <= 256 else 5
        j = [0]

        def nxt():
            j[0] += 1
            return j[0]

        def gemm():
            i = nxt()
            xc, xs = L.act[m][i % len(L.act[m])]
            tq.dual_gemm(L.desc, L.packed[i % L.ncopy], xc, xs, m, L.Y[m][i % len(L.Y[m])], stream=s)

        def quant():
            i = nxt()
            xc, xs = L.act[m][i % len(L.act[m])]
            tq.quant_act(L.X[m][i % len(L.X[m])], xc, xs, L.group, stream=s)

        def f16():
            i = nxt()
            torch.matmul(L.X[m][i % len(L.X[m])], L.WT[i % len(L.WT)])

        scratch = tq.empty_unfused_scratch(L.desc, m)

        def unf():
            i = nxt()
            xc, xs = L.act[m][i % len(L.act[m])]
            tq.quant_act(L.X[m][i % len(L.X[m])], xc, xs, L.group, stream=s)
            tq.dual_gemm_unfused(L.desc, L.packed[i % L.ncopy], xc, xs, m, L.Y[m][i % len(L.Y[m])],
                                 scratch, stream=s)

        timed(stream, lambda: L.call(m, s), reps)   # warm-up: the clocks after the host-side set-up
        us_layer = timed(stream, lambda: L.call(m, s), reps)
        us_two = timed(stream, lambda: L.call(m, s, fused_quant=False), reps)
        us_gemm = timed(stream, gemm, reps)
        us_quant = timed(stream, quant, reps)
        us_fp16 = timed(stream, f16, reps)
        us_unf = timed(stream, unf, reps)
        del scratch
        row = {"workload": wl_name, "layer": L.layer.name, "K": L.K, "N": L.N, "r": L.r, "group": L.group, "M": m,
               "kernel": L.kernel(m), "us_layer": round(us_layer, 3),
               "layer_launches": 1 if m <= FUSED_QUANT_MAX_M else 2,
               "us_quant_act_plus_dual_gemm": round(us_two, 3),
               "us_dual_gemm": round(us_gemm, 3), "us_quant_act": round(us_quant, 3),
               "tflops_nominal": round(2.0 * m * L.N * L.K / us_layer / 1e6, 3),
               "fp16_gemm_us": round(us_fp16, 3), "speedup_vs_fp16": round(us_fp16 / us_layer, 3),
               "us_layer_unfused": round(us_unf, 3), "fusion_speedup": round(us_unf / us_layer, 3)}
        if m <= 16:
            b = alg_bytes(m, L.N, L.K, L.r, m <= FUSED_QUANT_MAX_M)
            row["hbm_frac_layer"] = round(b / us_layer / 1e3 / HBM_PEAK_GBS, 4)
            if m > FUSED_QUANT_MAX_M:
                row["us_fused_quant"] = round(timed(stream, lambda: L.call(m, s, fused_quant=True, force=True), reps), 3)
        else:
            row["fp8_frac_dual_gemm"] = round(alg_ops(m, L.N, L.K, L.r) / us_gemm / 1e6 / FP8_MFMA_PEAK_TFLOPS, 4)
        rows.append(row)
        print(json.dumps(row), file=sys.stderr, flush=True)
    return rows


# ---------------------------------------------------------------------------
# the benchmark line
# ---------------------------------------------------------------------------
def main_bench(args):
    import torch
    from tq_synth import WORKLOADS
    wl = WORKLOADS[HEADLINE]
    stream = torch.cuda.Stream()
    s = stream.cuda_stream
    t_setup = time.perf_counter()
    layers = [LayerBench(wl, layer, HEAD_MS, stream, with_fp16=not args.no_detail) for layer in wl.layers]
    torch.cuda.synchronize()
    t_setup = time.perf_counter() - t_setup
    print(f"setup {t_setup:.1f} s", file=sys.stderr, flush=True)
    if args.calib_copy:
        src = torch.empty(CALIB_COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step(evs=None):
        for m in HEAD_MS:
            for li, L in enumerate(layers):
                L.call(m, s, None if evs is None else evs[(li, m)])

    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step()
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` steps ----
    keys = [(li, m) for m in HEAD_MS for li in range(len(layers))]
    evs = [{k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for k in keys}
           for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        t_start.record()
        for i in range(args.steps):
            step(evs[i])
        t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    kern_us = {k: 1e3 * float(np.mean([e[k][0].elapsed_time(e[k][1]) for e in evs])) for k in keys}
    print(f"timed {args.steps} steps: {ms_step:.3f} ms/step", file=sys.stderr, flush=True)

    step_flops = sum(2.0 * m * L.N * L.K for m in HEAD_MS for L in layers)
    tag = HEADLINE.replace("-", "_")

    def roof(k, bound):
        li, m = k
        L = layers[li]
        kname = L.kernel(m)
        us = kern_us[k]
        if bound == "mfma":
            ops = alg_ops(m, L.N, L.K, L.r)
            ach = ops / us / 1e6
            d = {"bound": "mfma", "achieved": round(ach, 1), "peak": FP8_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(ach / FP8_MFMA_PEAK_TFLOPS, 4), "ops_per_launch": ops}
        else:
            b = alg_bytes(m, L.N, L.K, L.r, m <= FUSED_QUANT_MAX_M)
            ach = b / us / 1e3
            d = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                 "frac": round(ach / HBM_PEAK_GBS, 4), "bytes_per_launch": int(b)}
        d["traffic"] = measured_traffic(kname, f"{tag}_{L.layer.name}_m{m}")
        d.update({"kernel": f"dual_gemm_{kname}_kernel", "call": f"{HEADLINE} {L.layer.name} M={m}",
                  "avg_launch_us": round(us, 3), "timing": "HIP events on the launch stream, timed region"})
        return d

    dom = max((k for k in keys if k[1] == max(HEAD_MS)), key=lambda k: kern_us[k])
    dec = max((k for k in keys if k[1] == 1), key=lambda k: kern_us[k])

    per_call = []
    for k in keys:
        li, m = k
        L = layers[li]
        r = {"layer": L.layer.name, "M": m, "kernel": L.kernel(m), "avg_launch_us": round(kern_us[k], 3)}
        if m <= 16:
            b = alg_bytes(m, L.N, L.K, L.r, m <= FUSED_QUANT_MAX_M)
            r["hbm_frac"] = round(b / kern_us[k] / 1e3 / HBM_PEAK_GBS, 4)
        else:
            r["fp8_frac"] = round(alg_ops(m, L.N, L.K, L.r) / kern_us[k] / 1e6 / FP8_MFMA_PEAK_TFLOPS, 4)
        per_call.append(r)

    out = {
        "metric": METRIC,
        "value": round(step_flops / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOPS",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int4",
        "data": "synthetic (seeded Student-t weights split by a rank-128 SVD, activations with 0.5 % "
                "outlier channels x50; random-init, no checkpoint)",
        "config": {"workload": "LLaMA3-70B-shaped layers on one GPU: gate_up K=8192->N=28672 and down "
                               "K=28672->N=8192, rank 128, group 64; one step = one layer call of each "
                               "at each M in (8192, 1, 32)",
                   "layers": [{"name": L.layer.name, "K": L.K, "N": L.N, "rank": L.r} for L in layers],
                   "M": list(HEAD_MS), "group": GROUP,
                   "layer_call": "M=1: tq_dual_gemm_fused_quant (one launch); else tq_quant_act + tq_dual_gemm",
                   "weight_copies_rotated": [L.ncopy for L in layers],
                   "activation_output_copies_rotated": {str(m): len(layers[0].X[m]) for m in HEAD_MS},
                   "compute": "int4 codes as exact fp8-e4m3 matrix-core operands, fp32 accumulate"},
        "per_call": per_call,
        "roofline": roof(dom, "mfma"),
        "roofline_decode": roof(dec, "hbm"),
        "setup_s": round(t_setup, 1),
    }
    if not args.no_detail:
        rows = []
        for L in layers:
            rows += detail_rows(L, HEAD_MS, stream, HEADLINE)
        del layers
        torch.cuda.empty_cache()
        wl2 = WORKLOADS[DETAIL_EXTRA]
        L2 = LayerBench(wl2, wl2.layers[0], wl2.Ms, stream)
        rows += detail_rows(L2, wl2.Ms, stream, DETAIL_EXTRA)
        del L2
        torch.cuda.empty_cache()
        # the paper's default configuration (group 128, rank 128) on the same shape
        L3 = LayerBench(wl2, wl2.layers[0], wl2.Ms, stream, group=128, rank=128)
        rows += detail_rows(L3, wl2.Ms, stream, DETAIL_EXTRA + "-g128-r128")
        del L3
        torch.cuda.empty_cache()
        # and at the headline's prefill point (gate_up, r = 128, the largest M)
        gate_up = [l for l in wl.layers if l.name == "gate_up"][0]
        L4 = LayerBench(wl, gate_up, (max(HEAD_MS),), stream, group=128)
        rows += detail_rows(L4, (max(HEAD_MS),), stream, HEADLINE + "-g128")
        del L4
        torch.cuda.empty_cache()
        out["per_m"] = rows
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(step_flops)
    print(json.dumps(out), flush=True)


def kernel_only(args):
    """--kernel-only LAYER M: one headline layer call, repeated, after a
    256 MiB calibration copy (for rocprofv3 counter runs)."""
    import torch
    from tq_synth import WORKLOADS
    wl = WORKLOADS[HEADLINE]
    layer = [l for l in wl.layers if l.name == args.kernel_only[0]][0]
    m = int(args.kernel_only[1])
    stream = torch.cuda.Stream()
    L = LayerBench(wl, layer, (m,), stream, with_fp16=False)
    src = torch.empty(CALIB_COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    with torch.cuda.stream(stream):
        for _ in range(args.reps):
            L.call(m, stream.cuda_stream)
    torch.cuda.synchronize()
    print(f"done: {args.reps} calls of {HEADLINE} {layer.name} M={m} ({L.kernel(m)} kernel)", flush=True)


# ---------------------------------------------------------------------------
# table modes
# ---------------------------------------------------------------------------
def config_sweep():
    """Every layer and token count of the four GPU-sized workload configs
    (LLaMA3-8B q/o and MLP, Qwen3-8B with its rank sweep, LLaMA3-70B on one
    GPU): per call, the layer, the fused kernel alone and an fp16 hipBLASLt
    GEMM of the same shape, each with HIP events on the launch stream over
    rotated copies, and the kernel's roofline fraction (HBM bytes for
    M <= 16, fp8 matrix-core ops otherwise).  Prints a markdown table."""
    import torch
    from tq_synth import WORKLOADS
    stream = torch.cuda.Stream()
    print("| config | layer K→N | r | M | kernel | layer µs | tq_dual_gemm µs | roofline | fp16 GEMM µs | "
          "speedup vs fp16 |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for name in ("llama3-8b-qo", "llama3-8b-mlp", "qwen3-8b", "llama3-70b"):
        wl = WORKLOADS[name]
        for layer in wl.layers:
            L = LayerBench(wl, layer, wl.Ms, stream)
            torch.cuda.synchronize()
            for r in detail_rows(L, wl.Ms, stream, name):
                m = r["M"]
                roof = (f"{r['hbm_frac_layer'] * 100:.1f} % HBM" if m <= 16
                        else f"{r['fp8_frac_dual_gemm'] * 100:.1f} % fp8")
                print(f"| {name} | {layer.name} {L.K}→{L.N} | {L.r} | {m} | {r['kernel']} | {r['us_layer']:.1f} | "
                      f"{r['us_dual_gemm']:.1f} | {roof} | {r['fp16_gemm_us']:.1f} | {r['speedup_vs_fp16']:.2f} |",
                      flush=True)
            del L
            torch.cuda.empty_cache()


def rank_overhead():
    """tq_dual_gemm at ranks 0, 32, 64 and 128 on the LLaMA3-8B q_proj and
    gate_up shapes: the latency the low-rank branch adds to the plain 4-bit
    layer (r = 0) at the same shape.  HIP events, rotated weight copies,
    random-init weights.  Prints a markdown table."""
    import torch
    import paper_2606_01556_amd as tq
    dev = torch.device("cuda")
    stream = torch.cuda.Stream()
    s = stream.cuda_stream
    torch.manual_seed(0)
    print("| layer K→N | M | r = 0 µs | r = 32 | r = 64 | r = 128 |")
    print("|---|---|---|---|---|---|")
    for name, Kl, Nl in (("q_proj", 4096, 4096), ("gate_up", 4096, 14336)):
        with torch.cuda.stream(stream):
            W = (torch.randn(Nl, Kl, device=dev) * 0.02).half()
        res = {}
        for rl in (0, 32, 64, 128):
            with torch.cuda.stream(stream):
                L1 = (torch.randn(Kl, rl, device=dev) * 0.05).half() if rl else None
                L2 = (torch.randn(rl, Nl, device=dev) * 0.05).half() if rl else None
                lay = tq.Layer(W, L1, L2, stream=stream)
                ncopy = max(2, int(np.ceil(ROTATE_BYTES / lay.desc.packed_bytes)))
                copies = [lay.packed] + [lay.packed.clone() for _ in range(ncopy - 1)]
            torch.cuda.synchronize()
            call = [0]
            for m in (1, 16, 128, 2048):
                with torch.cuda.stream(stream):
                    X = torch.randn(m, Kl, device=dev).half()
                    xc, xs = tq.empty_act(m, Kl, dev)
                    Y = torch.empty((m, Nl), dtype=torch.float16, device=dev)
                    tq.quant_act(X, xc, xs, stream=s)

                def gemm():
                    p = copies[call[0] % ncopy]
                    call[0] += 1
                    tq.dual_gemm(lay.desc, p, xc, xs, m, Y, stream=s)
                res[(rl, m)] = timed(stream, gemm, 30)
            del lay, copies
            torch.cuda.empty_cache()
        for m in (1, 16, 128, 2048):
            base = res[(0, m)]
            cells = " | ".join(f"{res[(r, m)]:.1f} (+{(res[(r, m)] / base - 1) * 100:.0f} %)"
                               for r in (32, 64, 128))
            print(f"| {name} {Kl}→{Nl} | {m} | {base:.1f} | {cells} |", flush=True)


def kernel_choice(group):
    """Past 512 tokens tq_dual_gemm picks the large kernel (128 x 256 blocks),
    the prefill kernel (beyond one round of blocks) or the mid kernel
    (32-token blocks, where the large blocks would leave most CUs idle).  Times
    each of them, forced through tq_dual_gemm_debug, beside the one it picks,
    on LLaMA3 layer shapes in quantization groups of `group` (HIP events,
    rotated weight copies, random-init weights).  Prints a markdown table."""
    import torch
    import paper_2606_01556_amd as tq
    dev = torch.device("cuda")
    stream = torch.cuda.Stream()
    s = stream.cuda_stream
    torch.manual_seed(0)
    print("| layer K→N | r | M | picked | large µs | prefill µs | mid µs | picked / fastest |")
    print("|---|---|---|---|---|---|---|---|")
    shapes = (("k/v_proj 8B", 4096, 1024), ("q/o_proj 8B", 4096, 4096), ("gate_up 8B", 4096, 14336),
              ("down 8B", 14336, 4096), ("k/v_proj 70B", 8192, 1024))
    for name, Kl, Nl in shapes:
        with torch.cuda.stream(stream):
            W = (torch.randn(Nl, Kl, device=dev) * 0.02).half()
        for rl in ((0, 64, 128) if group == 128 else (64, 128)):
            with torch.cuda.stream(stream):
                L1 = (torch.randn(Kl, rl, device=dev) * 0.05).half() if rl else None
                L2 = (torch.randn(rl, Nl, device=dev) * 0.05).half() if rl else None
                lay = tq.Layer(W, L1, L2, group=group, stream=stream)
                ncopy = max(2, int(np.ceil(ROTATE_BYTES / lay.desc.packed_bytes)))
                copies = [lay.packed] + [lay.packed.clone() for _ in range(ncopy - 1)]
            torch.cuda.synchronize()
            call = [0]
            for m in (576, 1024, 2048, 4096):
                with torch.cuda.stream(stream):
                    X = torch.randn(m, Kl, device=dev).half()
                    xc, xs = tq.empty_act(m, Kl, dev, group=group)
                    Y = torch.empty((m, Nl), dtype=torch.float16, device=dev)
                    tq.quant_act(X, xc, xs, group, stream=s)
                picked = tq.dual_gemm_kernel(lay.desc, m)
                res = {}
                for kname in ("large", "prefill", "mid"):

                    def gemm():
                        p = copies[call[0] % ncopy]
                        call[0] += 1
                        tq.dual_gemm_debug(lay.desc, p, xc, xs, m, Y, kernel=kname, stream=s)
                    res[kname] = timed(stream, gemm, 20)
                cell = lambda k: f"{res[k]:.1f}" if k in res else "–"
                print(f"| {name} {Kl}→{Nl} | {rl} | {m} | {picked} | {cell('large')} | {cell('prefill')} | "
                      f"{cell('mid')} | {res[picked] / min(res.values()):.2f} |", flush=True)
            del lay, copies
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-detail", action="store_true", help="skip the per-M detail")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 256 MiB device copy first (calibrates the HBM byte counters of "
                         "a profiler run)")
    ap.add_argument("--configs", action="store_true",
                    help="time every layer and token count of the workload configs (markdown table)")
    ap.add_argument("--ranks", action="store_true",
                    help="the low-rank branch's overhead at ranks 0/32/64/128 (markdown table)")
    ap.add_argument("--kernel-choice", action="store_true",
                    help="the large, prefill and mid kernels past 512 tokens beside the picked one")
    ap.add_argument("--group", type=int, default=64, choices=(64, 128),
                    help="quantization group of --kernel-choice")
    ap.add_argument("--kernel-only", nargs=2, metavar=("LAYER", "M"),
                    help="repeat one headline layer call (gate_up or down) after a calibration copy")
    ap.add_argument("--reps", type=int, default=5)
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "LAYER", "M"),
                    help="write the traffic summary of a --kernel-only counter pair under profiles/")
    ap.add_argument("--counter-summary", nargs="+", metavar="ARG",
                    help="PASS_DIR... LAYER M: print the SQ counter summary of --kernel-only --pmc passes")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "TITLE"),
                    help="print a markdown summary of a rocprofv3 --kernel-trace --stats run")
    ap.add_argument("--cmd", action="append", default=[],
                    help="the profiler commands a summary came from (recorded in it)")
    ap.add_argument("--cpu-oracle-child", type=int, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.cpu_oracle_child is not None:
        print(json.dumps(cpu_oracle_child(args.cpu_oracle_child)), flush=True)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary[0], args.trace_summary[1], "\n".join(args.cmd))
        return
    if args.traffic_summary:
        f, w, layer, m = args.traffic_summary
        traffic_summary(f, w, layer, int(m), args.cmd)
        return
    if args.counter_summary:
        *dirs, layer, m = args.counter_summary
        counter_summary(dirs, layer, int(m), "\n".join(args.cmd))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the layer runs on a single MI355X "
              "(multi-GPU sharding is a design note, not built)", file=sys.stderr)
        sys.exit(2)
    if args.configs:
        config_sweep()
    elif args.ranks:
        rank_overhead()
    elif args.kernel_choice:
        kernel_choice(args.group)
    elif args.kernel_only:
        kernel_only(args)
    else:
        main_bench(args)


if __name__ == "__main__":
    main()
