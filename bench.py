#!/usr/bin/env python3
"""Triangle-attention benchmark on one MI355X.

One step = the whole hot path on one batch of synthetic input: forward and
backward of triangle attention around the starting node and around the
ending node, N = 768 tokens, H = 4 heads, d = 32, bf16 inputs with fp32
accumulation, no padding (bias ~ N(0, 2)).  The metric is nominal fwd+bwd
TFLOP/s (14 N^3 H d per node variant: 4 forward, 10 backward) and its
fraction of the MI355X dense bf16 MFMA peak; peak HBM bytes are reported
beside it.

Prints ONE JSON line.  Inputs, outputs and workspaces are resident in HBM
before the timed region; the timed region runs exactly --steps steps between
two device synchronisations.  Per-kernel durations come from HIP events the
library records on its launch stream during the same timed steps.

The "cpu_baseline" leg times the fp64 oracle on the host cores on a bounded
sample of the same workload (it is a reference point, not a target).

--workload lnl_bf16_n768 instead measures the fused layer-norm + linear
projection that produces the attention inputs (m = 768^2 rows of 128
features -> Q, K, V, G [m][128] and the bias logits [m][4]): one step is its
forward and backward, the metric is algorithmic HBM GB/s (every input read
once, every output written once, per step time), and the roofline is HBM
bandwidth.

--workload tri_rows_bf16_n768_r96 measures one GPU's share of the row-sharded
starting node (Section IV-B): rows 288..383 of the N = 768 map through the
row-range entry points, forward and backward, nominal 14 R N^2 H d flop.

--workload trn_bf16_n768 measures the fused transition layer (layer norm,
W1 [128][1024], SwiGLU, W2 [512][128]) on the N = 768 pair representation
(m = 768^2 rows): forward and backward, algorithmic 18 m c F flop per step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 flop/clk/CU
MFMA_FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0

# Algorithmic MFMA flop per logit (per (row, query, key, head)) of each main
# kernel: d-long dot products, 2 d flop each.  fwd: S, P V.  dq: S, dP, dQ.
# dkdv: S, dP, dV, dK.  db: S, dP (it only reduces dS over rows).
KERNEL_FLOP_PER_LOGIT_D = {"fwd": 4, "dq": 6, "dkdv": 8, "db": 4}
PROFILE_DIR = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="workload name (default: the N=768 attention one; lnl_bf16_n768 runs "
                         "the fused layer-norm + linear projection; tri_rows_bf16_n768_r96 "
                         "one GPU's 96-row shard of the starting node; trn_bf16_n768 the fused "
                         "transition layer)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample (0 disables it)")
    ap.add_argument("--configs", type=int, default=1,
                    help="with the default workload: also time every workload configuration "
                         "(N = 32 fp32 ... N = 1536, each node variant) and report its fwd and "
                         "bwd time, TFLOP/s and peak HBM bytes in the same JSON line "
                         "(0 skips it, as the profiling runs do)")
    ap.add_argument("--mfma-probe", type=int, default=0,
                    help="only run the library's MFMA-only calibration kernel this many times "
                         "(1024 workgroups of 4 waves, 2000 rounds of 8 bf16 32x32x16 MFMAs per "
                         "wave): the reference kernel for the MFMA-activity counters")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run a plain device-to-device copy of this many bytes 5 times "
                         "(reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def copy_calibration(nbytes):
    """A plain copy of known size: under rocprofv3 --pmc its FETCH_SIZE and WRITE_SIZE per
    dispatch, divided by nbytes, are the scale factors of those counters."""
    import torch
    dev = torch.device("cuda:0")
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize(dev)
    print(json.dumps({"copy_bytes": src.numel() * 4, "launches": 5}), flush=True)


def mfma_calibration(launches, blocks=1024, iters=2000):
    """The library's MFMA-only kernel (one workgroup of 4 waves per SIMD quad,
    `iters` rounds of 8 bf16 32x32x16 MFMAs per wave): under rocprofv3 --pmc the
    MFMA-busy counter of a dispatch, divided by the cycles its MFMAs need at
    the dense rate (32 per MFMA on each SIMD), calibrates that counter."""
    import torch

    from paper_2506_20686_amd import binding as B
    dev = torch.device("cuda:0")
    out = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for i in range(launches + 1):
        if i == 1:
            ev[0].record()
        st = B.tri_attn_mfma_probe(blocks, iters, out.data_ptr(), stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_attn_mfma_probe")
    ev[1].record()
    torch.cuda.synchronize(dev)
    ms = ev[0].elapsed_time(ev[1]) / max(1, launches)
    mfmas = blocks * 4 * iters * 8
    print(json.dumps({"mfma_probe_launches": launches, "blocks": blocks, "iters": iters,
                      "mfma_per_launch": mfmas, "ms_per_launch": round(ms, 5),
                      "tflops": round(mfmas * 32768 / (ms * 1e-3) / 1e12, 2)}), flush=True)


# Sources whose change can change a kernel family's memory traffic (its
# kernels, the shared device headers, the host code that picks launch shapes).
SOURCE_FAMILIES = {
    "tri": ("fwd.hip", "bwd.hip", "dkdv.hip", "dkdv_end.hip", "dkdv_dma.h", "bwd.h", "api.hip",
            "common.h", "dma.h", "stage.h", "kernels.h"),
    "lnl": ("lnl.hip", "api.hip", "common.h", "dma.h", "kernels.h"),
    "trn": ("trn.hip", "api.hip", "common.h", "dma.h", "kernels.h"),
}


def _code_only(text):
    """C++ source without its comments and with runs of whitespace collapsed, so that
    editing a comment leaves the hash of the code unchanged (the sources hold no string
    literal with comment markers)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(family="tri"):
    """Hash of the code (comments aside) of a kernel family's sources; a traffic figure
    measured on other code is stale."""
    from paper_2506_20686_amd import build as hip_build
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2506_20686_amd", "csrc")
    for name in sorted(SOURCE_FAMILIES[family]):
        with open(os.path.join(csrc, name), encoding="utf-8") as f:
            h.update(name.encode() + b"\0" + _code_only(f.read()).encode())
    # the compile options shape the code as much as the sources do
    h.update(repr((hip_build.FLAGS, hip_build.MAX_ILP, hip_build.ILP_FLAGS)).encode())
    return h.hexdigest()[:16]


def time_steps(step, dev, steps, candidates):
    """Time `steps` calls of `step`.  A first pass of min(steps, 10) steps with
    every kernel timed gives the per-kernel breakdown and the dominant kernel
    (the largest total among `candidates`); the timed region then records HIP
    events around the dominant kernel's launches only, since events around
    every launch cost the step about 1.5%.  Returns (ms per step, breakdown
    {name: (total ms, launches)}, dominant name, (its total ms, launches) over
    the timed region)."""
    import torch
    from paper_2506_20686_amd import binding as B
    B.tri_attn_timing_select(None)
    B.tri_attn_timing_reset()
    B.tri_attn_timing_enable(True)
    for _ in range(min(steps, 10)):
        step()
    torch.cuda.synchronize(dev)
    B.tri_attn_timing_enable(False)
    breakdown = {k: v for k, v in B.kernel_times().items() if v[1] > 0}
    dom = max((k for k in breakdown if k in candidates), key=lambda k: breakdown[k][0])
    B.tri_attn_timing_select([dom])
    B.tri_attn_timing_reset()
    B.tri_attn_timing_enable(True)
    torch.cuda.synchronize(dev)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize(dev)
    t1 = time.perf_counter()
    B.tri_attn_timing_enable(False)
    live = B.kernel_times()[dom]
    B.tri_attn_timing_select(None)
    return (t1 - t0) * 1e3 / steps, breakdown, dom, live


def recorded_traffic(kernel, workload, family="tri"):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 --pmc summary, or
    None if there is none or it was taken on different kernel sources."""
    path = os.path.join(PROFILE_DIR, f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"bytes_per_launch:\s*([0-9.eE+]+)", text)
    s = re.search(r"source_hash:\s*([0-9a-f]+)", text)
    if not m or not s or s.group(1) != kernel_source_hash(family):
        return None
    return float(m.group(1))


def host_cpu():
    """CPU model and logical core count of the host running the benchmark."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count()}


class native_oracle:
    """The oracle's sources built for this host (-O3 -march=native, OpenMP) and
    swapped in for the duration of a `with` block; the tests use the generic build."""

    def __enter__(self):
        import oracle
        from oracle import build as ob
        self.flags = " ".join(ob.NATIVE_FLAGS)
        self.prev = oracle.use_library(oracle.load(ob.build_native()))
        return self

    def __exit__(self, *exc):
        import oracle
        oracle.use_library(self.prev)


def cpu_baseline(w, t, target_s, row_range=None, whole=()):
    """Time the fp64 oracle (as it stands, built -O3 -march=native for this
    host) on a sample of the workload.  A whole fwd+bwd is the forward of every
    row, the per-row gradients (dQ, dK, dV, dG) of every row and the bias
    gradient of every query (a sum over all rows); the sample takes R evenly
    spaced rows and R evenly spaced bias-gradient queries, R / N of that work,
    nominal 14 N^2 H d flop per row.  R is sized from a trial of one row and
    one query per oracle thread to about target_s seconds.  row_range = (r0,
    rows) draws the rows from that range and leaves the bias gradient out (the
    oracle sums it over every row of the map, not over a range's).  `whole`
    lists small workloads timed in full as well."""
    import numpy as np

    import oracle
    from paper_2506_20686_amd import workloads as W

    def arrays(tt):
        arr = {k: np.ascontiguousarray(tt[k].double().numpy())
               for k in ("q", "k", "v", "g", "bias", "dout")}
        m = tt.get("mask")
        return arr, (None if m is None else m.numpy())

    def run(ww, tt, node, rows, qs):
        arr, mask = arrays(tt)
        t0 = time.perf_counter()
        oracle.fwd(node, arr["q"], arr["k"], arr["v"], arr["g"], arr["bias"], mask, rows=rows)
        oracle.bwd(node, arr["q"], arr["k"], arr["v"], arr["g"], arr["bias"], arr["dout"], mask,
                   rows=rows, db_queries=qs)
        return time.perf_counter() - t0

    with native_oracle() as nat:
        node = w.nodes[0]
        r0, span = (0, w.n) if row_range is None else row_range
        nt = max(1, min(span, oracle.max_threads()))
        with_db = row_range is None

        def sample(count):
            rows = [r0 + int(i * span / count) for i in range(count)]
            qs = [int(i * w.n / count) for i in range(count)] if with_db else []
            return run(w, t, node, rows, qs)

        trial = sample(nt)
        rows = max(nt, min(span, int(nt * target_s / max(trial, 1e-3)) // nt * nt))
        dt = sample(rows)
        flop = 14.0 * w.n ** 2 * w.h * w.d * rows
        where = f"{w.n} rows" if row_range is None else f"rows {r0}..{r0 + span - 1} of {w.n}"
        res = {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.max_threads(),
               "kind": "oracle", "seconds": round(dt, 3), "build": f"gcc {nat.flags}",
               **host_cpu(),
               "sample": (f"{W.NODE_NAMES[node]} node of {w.name}: forward and per-row gradients "
                          f"(dQ, dK, dV, dG) of {rows} of {where}" +
                          (f", and the bias gradient of {rows} of {w.n} query indices (each a "
                           f"sum over all {w.n} rows): {rows}/{w.n} of one node's fwd+bwd"
                           if with_db else "; the range's bias-gradient term not included") +
                          ", fp64, nominal 14*N^2*H*d flop per row")}
        timed = {}
        for wname in whole:
            ww = W.WORKLOADS[wname]
            tt = W.workload_inputs(ww)
            sec = run(ww, tt, tt["node"], None, None)
            timed[wname] = {"seconds": round(sec, 3),
                            "tflops": round(ww.flops_fwd_bwd / sec / 1e12, 6)}
        if timed:
            res["whole"] = timed
    return res


def lnl_kernel_bytes(m, cols, k=128):
    """Algorithmic HBM bytes per launch of the fused projection's main kernels."""
    n = int(sum(cols))
    return {"lnl_fwd": m * k * 2 + m * n * 2 + m * 8,
            "lnl_bwd_dx": 2 * m * k * 2 + m * n * 2 + m * 8,
            "lnl_bwd_g": m * k * 2 + m * n * 2 + m * 8}


def lnl_cpu_baseline(t, target_s):
    """Time the fp64 oracle on a sample of R rows: forward, then the backward
    of those rows (dx and their sums over rows).  Unit: algorithmic GB/s."""
    import numpy as np
    import torch

    import oracle
    from paper_2506_20686_amd import workloads as W

    m = t["x"].shape[0]
    arr = {k: np.ascontiguousarray(t[k].double().numpy()) for k in ("gamma", "beta", "w")}

    def run(rows):
        sel = torch.as_tensor(rows)
        xs = np.ascontiguousarray(t["x"][sel].double().numpy())
        ds = np.ascontiguousarray(t["do2"][sel].double().numpy())
        t0 = time.perf_counter()
        oracle.lnl_fwd(xs, arr["gamma"], arr["beta"], arr["w"])
        oracle.lnl_bwd(xs, arr["gamma"], arr["beta"], arr["w"], ds)
        return time.perf_counter() - t0

    trial_rows = 512
    trial = run([int(i * m / trial_rows) for i in range(trial_rows)])
    rows = max(trial_rows, min(m, int(trial_rows * target_s / max(trial, 1e-3))))
    dt = run([int(i * m / rows) for i in range(rows)])
    b = W.lnl_step_bytes(rows, t["cols"])
    return {"value": (b["fwd"] + b["bwd"]) / dt / 1e9, "unit": "GB/s",
            "cores": oracle.max_threads(), "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"{rows} of {m} rows (evenly spaced): forward and backward of those rows, "
                      f"fp64, their sums over rows only; algorithmic bytes of {rows} rows"}


def bench_lnl(args, name):
    """Forward + backward of the fused layer-norm + linear projection."""
    import torch

    from paper_2506_20686_amd import binding as B
    from paper_2506_20686_amd import workloads as W

    spec = W.LNL_WORKLOADS[name]
    m, cols = spec["m"], tuple(spec["cols"])
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch.zeros(1, device=dev)
    torch.cuda.reset_peak_memory_stats(dev)
    t = W.lnl_inputs(m, cols, seed=0)
    x, gamma, beta, w = (t[k].to(dev) for k in ("x", "gamma", "beta", "w"))
    douts = [p.contiguous().to(dev) for p in torch.split(t["do2"], list(cols), dim=1)]
    ncols = sum(cols)
    outs = [torch.empty((m, c), dtype=torch.bfloat16, device=dev) for c in cols]
    mean = torch.empty(m, dtype=torch.float32, device=dev)
    rstd = torch.empty(m, dtype=torch.float32, device=dev)
    dx = torch.empty_like(x)
    dw = torch.empty((128, ncols), dtype=torch.float32, device=dev)
    dg = torch.empty(128, dtype=torch.float32, device=dev)
    db = torch.empty(128, dtype=torch.float32, device=dev)
    ws_bytes = B.tri_ln_linear_bwd_workspace_bytes(B.BF16, m, 128, cols)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda a: a.data_ptr()  # noqa: E731

    def step():
        st = B.tri_ln_linear_fwd(B.BF16, m, 128, cols, 1e-5, P(x), P(gamma), P(beta), P(w),
                                 [P(o) for o in outs], P(mean), P(rstd), stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_ln_linear_fwd")
        st = B.tri_ln_linear_bwd(B.BF16, m, 128, cols, P(x), P(gamma), P(beta), P(w), P(mean),
                                 P(rstd), [P(d) for d in douts], P(dx), P(dw), P(dg), P(db),
                                 P(ws), ws_bytes, stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_ln_linear_bwd")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    kb = lnl_kernel_bytes(m, cols)
    ms, ktimes, dom, dom_t = time_steps(step, dev, args.steps, kb)
    peak_bytes = torch.cuda.max_memory_allocated(dev)

    sb = W.lnl_step_bytes(m, cols)
    step_bytes = sb["fwd"] + sb["bwd"]
    gbs = step_bytes / (ms * 1e-3) / 1e9
    per_kernel = {k: {"avg_ms": round(v[0] / v[1], 5), "launches": v[1],
                      "share": round(v[0] / max(1e-9, sum(x[0] for x in ktimes.values())), 4)}
                  for k, v in ktimes.items() if v[1] > 0}
    avg_s = dom_t[0] / dom_t[1] * 1e-3
    achieved = kb[dom] / avg_s / 1e9
    out = {
        "metric": "fused layer-norm + linear projection fwd+bwd, algorithmic HBM GB/s at m=768^2",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals; the paper's pair representations are not available)",
        "config": {"workload": name, "m": m, "k": 128, "cols": list(cols),
                   "parallelism": "none (1 GPU)"},
        "step_bytes": int(step_bytes),
        "peak_hbm_bytes": int(peak_bytes),
        "workspace_bytes": int(ws_bytes),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 5),
                     "traffic": recorded_traffic(dom, name, "lnl")},
        "per_kernel": per_kernel,
    }
    out["cpu_baseline"] = lnl_cpu_baseline(t, args.cpu_seconds) if args.cpu_seconds > 0 else None
    print(json.dumps(out), flush=True)


def trn_kernel_flops(m, c=128, f=512):
    """MFMA flop per launch of the transition layer's main kernels: the
    products each performs (the backward kernels recompute [a | b] = o1 W1
    and du = dout W2^T, which counts here but not in the step's 18 m c f)."""
    return {"trn_fwd": 6.0 * m * c * f,           # o1 W1 (2 m c 2f), u W2 (2 m f c)
            "trn_bwd_dx": 10.0 * m * c * f,       # du, o1 W1, dh W1^T
            "trn_bwd_w": 12.0 * m * c * f}        # o1 W1, du, xhat^T dh, u^T dout


def trn_cpu_baseline(t, target_s):
    """Time the fp64 oracle on a sample of R rows: forward, then the backward
    of those rows with their sums over rows.  Unit: algorithmic TFLOP/s (18 c
    f flop per row)."""
    import numpy as np

    from oracle import transition as OT
    from paper_2506_20686_amd import workloads as W

    m = t["x"].shape[0]
    w = {k: np.ascontiguousarray(t[k].double().numpy()) for k in ("gamma", "beta", "w1", "w2")}

    def run(rows):
        sel = np.asarray(rows)
        xs = np.ascontiguousarray(t["x"].double().numpy()[sel])
        ds = np.ascontiguousarray(t["dout"].double().numpy()[sel])
        t0 = time.perf_counter()
        OT.trn_fwd(xs, w["gamma"], w["beta"], w["w1"], w["w2"])
        OT.trn_bwd(xs, w["gamma"], w["beta"], w["w1"], w["w2"], ds)
        return time.perf_counter() - t0

    trial_rows = 4096
    trial = run([int(i * m / trial_rows) for i in range(trial_rows)])
    rows = max(trial_rows, min(m, int(trial_rows * target_s / max(trial, 1e-3))))
    dt = run([int(i * m / rows) for i in range(rows)])
    flop = W.trn_step_flops(rows)
    threads = os.environ.get("OMP_NUM_THREADS") or str(os.cpu_count())
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "seconds": round(dt, 3),
            "sample": f"{rows} of {m} rows (evenly spaced): forward and backward of those rows "
                      f"with their sums over rows, fp64 numpy (BLAS threads: {threads}); "
                      f"algorithmic 18*c*f flop per row"}


def bench_trn(args, name):
    """Forward + backward of the fused transition layer."""
    import torch

    from paper_2506_20686_amd import binding as B
    from paper_2506_20686_amd import workloads as W

    m, c, f = W.TRN_WORKLOADS[name], W.TRN_C, W.TRN_F
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    torch.zeros(1, device=dev)
    torch.cuda.reset_peak_memory_stats(dev)
    t = W.trn_inputs(m, seed=0)
    x, gamma, beta, w1, w2, dout = (t[k].to(dev) for k in ("x", "gamma", "beta", "w1", "w2",
                                                             "dout"))
    out = torch.empty_like(x)
    mean = torch.empty(m, dtype=torch.float32, device=dev)
    rstd = torch.empty(m, dtype=torch.float32, device=dev)
    dx = torch.empty_like(x)
    dw1 = torch.empty((c, 2 * f), dtype=torch.float32, device=dev)
    dw2 = torch.empty((f, c), dtype=torch.float32, device=dev)
    dg = torch.empty(c, dtype=torch.float32, device=dev)
    db = torch.empty(c, dtype=torch.float32, device=dev)
    ws_bytes = max(B.tri_transition_fwd_workspace_bytes(B.BF16, m, c, f),
                   B.tri_transition_bwd_workspace_bytes(B.BF16, m, c, f))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda a: a.data_ptr()  # noqa: E731

    def step():
        st = B.tri_transition_fwd(B.BF16, m, c, f, 1e-5, P(x), P(gamma), P(beta), P(w1), P(w2),
                                  P(out), P(mean), P(rstd), P(ws), ws_bytes, stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_transition_fwd")
        st = B.tri_transition_bwd(B.BF16, m, c, f, P(x), P(gamma), P(beta), P(w1), P(w2),
                                  P(mean), P(rstd), P(dout), P(dx), P(dw1), P(dw2), P(dg), P(db),
                                  P(ws), ws_bytes, stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_transition_bwd")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    kf = trn_kernel_flops(m, c, f)
    ms, ktimes, dom, dom_t = time_steps(step, dev, args.steps, kf)
    peak_bytes = torch.cuda.max_memory_allocated(dev)

    tflops = W.trn_step_flops(m) / (ms * 1e-3) / 1e12
    per_kernel = {k: {"avg_ms": round(v[0] / v[1], 5), "launches": v[1],
                      "share": round(v[0] / max(1e-9, sum(y[0] for y in ktimes.values())), 4)}
                  for k, v in ktimes.items() if v[1] > 0}
    avg_s = dom_t[0] / dom_t[1] * 1e-3
    achieved = kf[dom] / avg_s / 1e12
    peak = MFMA_BF16_PEAK_TFLOPS
    out_line = {
        "metric": "fused transition layer (layer norm, W1, SwiGLU, W2) fwd+bwd TFLOP/s at "
                  "m=768^2, c=128, F=512",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals; the paper's pair representations are not available)",
        "config": {"workload": name, "m": m, "c": c, "f": f, "parallelism": "none (1 GPU)"},
        "pct_of_peak": round(100.0 * tflops / peak, 3),
        "peak_hbm_bytes": int(peak_bytes),
        "workspace_bytes": int(ws_bytes),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 3),
                     "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 5),
                     "traffic": recorded_traffic(dom, name, "trn")},
        "per_kernel": per_kernel,
    }
    out_line["cpu_baseline"] = (trn_cpu_baseline(t, args.cpu_seconds) if args.cpu_seconds > 0
                                else None)
    print(json.dumps(out_line), flush=True)


def bench_rows(args, name):
    """One GPU's share of the row-sharded starting node: forward + backward of
    `rows` rows of the whole map through tri_attn_rows_{fwd,bwd}, shard-local
    tensors, the whole bias, an fp32 bias-gradient term.  Nominal 14 R N^2 H d
    flop per step; MFMA roofline of the dominant kernel."""
    import torch

    from paper_2506_20686_amd import binding as B
    from paper_2506_20686_amd import workloads as W

    rw = W.ROWS_WORKLOADS[name]
    w = W.WORKLOADS[rw.base]
    dev = torch.device("cuda:0")
    dt = B.BF16
    n, h, d, R = w.n, w.h, w.d, rw.rows
    scale = 1.0 / math.sqrt(d)
    torch.cuda.set_device(dev)
    torch.zeros(1, device=dev)
    torch.cuda.reset_peak_memory_stats(dev)
    s = W.rows_inputs(rw)
    x = {k: s[k].to(dev) for k in ("q", "k", "v", "g", "bias", "dout", "mask")}
    x["out"] = torch.empty_like(x["q"])
    x["lse"] = torch.empty((R, n, h), dtype=torch.float32, device=dev)
    for gname in ("dq", "dk", "dv", "dg"):
        x[gname] = torch.empty_like(x["q"])
    x["dbp"] = torch.empty((n, n, h), dtype=torch.float32, device=dev)
    ws_bytes = max(B.tri_attn_rows_fwd_workspace_bytes(dt, n, R, h, d),
                   B.tri_attn_rows_bwd_workspace_bytes(dt, n, R, h, d))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda a: a.data_ptr()  # noqa: E731

    def step():
        st = B.tri_attn_rows_fwd(dt, n, R, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]),
                                 P(x["g"]), P(x["bias"]), P(x["mask"]), P(x["out"]), P(x["lse"]),
                                 P(ws), ws_bytes, stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_attn_rows_fwd")
        st = B.tri_attn_rows_bwd(dt, n, R, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]),
                                 P(x["g"]), P(x["bias"]), P(x["mask"]), P(x["out"]), P(x["lse"]),
                                 P(x["dout"]), P(x["dq"]), P(x["dk"]), P(x["dv"]), P(x["dg"]),
                                 P(x["dbp"]), P(ws), ws_bytes, stream)
        if st != B.OK:
            raise B.TriAttnError(st, "tri_attn_rows_bwd")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    ms, ktimes, dom, dom_t = time_steps(step, dev, args.steps, KERNEL_FLOP_PER_LOGIT_D)
    peak_bytes = torch.cuda.max_memory_allocated(dev)

    tflops = rw.flops_fwd_bwd / (ms * 1e-3) / 1e12
    peak = MFMA_BF16_PEAK_TFLOPS
    per_kernel = {k: {"avg_ms": round(v[0] / v[1], 5), "launches": v[1],
                      "share": round(v[0] / max(1e-9, sum(y[0] for y in ktimes.values())), 4)}
                  for k, v in ktimes.items() if v[1] > 0}
    avg_s = dom_t[0] / dom_t[1] * 1e-3
    achieved = KERNEL_FLOP_PER_LOGIT_D[dom] * d * R * n * n * h / avg_s / 1e12
    out = {
        "metric": f"triangle-attn fwd+bwd TFLOP/s on one GPU's {R}-row shard of the N={n} "
                  "starting node",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded normals, rows of the N=768 attention workload's inputs)",
        "config": {"workload": name, "n": n, "rows": R, "first_row": rw.r0, "heads": h,
                   "head_dim": d, "nodes": ["starting"], "mask": "all keys valid",
                   "parallelism": f"one of {n // R} row shards (1 GPU)"},
        "pct_of_peak": round(100.0 * tflops / peak, 3),
        "peak_hbm_bytes": int(peak_bytes),
        "workspace_bytes": int(ws_bytes),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 3),
                     "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 5),
                     "traffic": recorded_traffic(dom, name)},
        "per_kernel": per_kernel,
    }
    out["cpu_baseline"] = (cpu_baseline(w, s["whole"], args.cpu_seconds, (rw.r0, R))
                           if args.cpu_seconds > 0 else None)
    print(json.dumps(out), flush=True)


# The workload configurations reported beside the headline (one entry per
# node variant): the small fp32 case, the padded N = 256 and N = 384 cases,
# N = 768 and the N = 1536 memory stress.
CONFIG_SWEEP = ("tri_start_fp32_n32", "tri_start_bf16_n256_pad10", "tri_end_bf16_n384_randpad15",
                "tri_bf16_n768", "tri_start_bf16_n1536_pad5")


def sweep_configs(steps):
    """Forward and backward time, nominal and valid-key TFLOP/s and peak HBM
    bytes of one fwd+bwd for every workload configuration and node variant.
    Peak bytes are torch's max_memory_allocated over one fwd+bwd: `peak_hbm_bytes`
    with the inputs and outputs resident, `extra_hbm_bytes` above them (the
    workspace, i.e. what the method itself needs besides its operands)."""
    import torch

    from paper_2506_20686_amd import binding as B
    from paper_2506_20686_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda a: a.data_ptr()  # noqa: E731
    res = []
    for name in CONFIG_SWEEP:
        w = W.WORKLOADS[name]
        dt = B.BF16 if w.dtype == torch.bfloat16 else B.F32
        n, h, d = w.n, w.h, w.d
        scale = 1.0 / math.sqrt(d)
        for node in w.nodes:
            t = W.workload_inputs(w, node)
            valid_keys = int(t["mask"].to(torch.int64).sum().item())  # over all rows
            x = {k: t[k].to(dev) for k in ("q", "k", "v", "g", "bias", "dout", "mask")}
            del t
            x["out"] = torch.empty_like(x["q"])
            x["lse"] = torch.empty(x["bias"].shape, dtype=torch.float32, device=dev)
            for gname in ("dq", "dk", "dv", "dg"):
                x[gname] = torch.empty_like(x["q"])
            x["dbias"] = torch.empty_like(x["bias"])
            torch.cuda.synchronize(dev)
            resident = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            ws_bytes = max(B.tri_attn_fwd_workspace_bytes(node, dt, n, h, d),
                           B.tri_attn_bwd_workspace_bytes(node, dt, n, h, d))
            ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)

            def fwd():
                st = B.tri_attn_fwd(node, dt, n, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]),
                                    P(x["g"]), P(x["bias"]), P(x["mask"]), P(x["out"]),
                                    P(x["lse"]), P(ws), ws_bytes, stream)
                if st != B.OK:
                    raise B.TriAttnError(st, "tri_attn_fwd")

            def bwd():
                st = B.tri_attn_bwd(node, dt, n, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]),
                                    P(x["g"]), P(x["bias"]), P(x["mask"]), P(x["out"]),
                                    P(x["lse"]), P(x["dout"]), P(x["dq"]), P(x["dk"]),
                                    P(x["dv"]), P(x["dg"]), P(x["dbias"]), P(ws), ws_bytes,
                                    stream)
                if st != B.OK:
                    raise B.TriAttnError(st, "tri_attn_bwd")

            fwd()
            bwd()
            torch.cuda.synchronize(dev)
            peak = torch.cuda.max_memory_allocated(dev)
            k = max(1, steps if n <= 768 else steps // 4)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            tf = tb = 0.0
            for _ in range(k):
                ev[0].record()
                fwd()
                ev[1].record()
                bwd()
                ev[2].record()
                ev[2].synchronize()
                tf += ev[0].elapsed_time(ev[1])
                tb += ev[1].elapsed_time(ev[2])
            tf, tb = tf / k, tb / k
            nominal = w.flops_fwd_bwd
            effective = 14.0 * n * valid_keys * h * d  # logits of valid keys only
            pk = MFMA_BF16_PEAK_TFLOPS if dt == B.BF16 else MFMA_FP32_PEAK_TFLOPS
            res.append({
                "workload": name, "node": W.NODE_NAMES[node], "n": n, "heads": h, "head_dim": d,
                "dtype": "bf16" if dt == B.BF16 else "f32", "steps": k,
                "fwd_ms": round(tf, 4), "bwd_ms": round(tb, 4),
                "tflops": round(nominal / ((tf + tb) * 1e-3) / 1e12, 3),
                "tflops_valid_keys": round(effective / ((tf + tb) * 1e-3) / 1e12, 3),
                "pct_of_peak": round(100.0 * nominal / ((tf + tb) * 1e-3) / 1e12 / pk, 3),
                "peak_hbm_bytes": int(peak), "extra_hbm_bytes": int(peak - resident),
                "naive_logits_bytes": int(n ** 3 * h * (2 if dt == B.BF16 else 4)),
            })
            del x, ws
            torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (one GPU's share "
              "of a row-sharded run is --workload tri_rows_bf16_n768_r96); run it with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.copy_bytes > 0:
        copy_calibration(args.copy_bytes)
        return
    if args.mfma_probe > 0:
        mfma_calibration(args.mfma_probe)
        return

    import torch

    from paper_2506_20686_amd import binding as B
    from paper_2506_20686_amd import workloads as W

    if not os.path.exists(B.LIB_PATH):
        from paper_2506_20686_amd import build
        build.build()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    name = args.workload or W.HEADLINE
    if name in W.LNL_WORKLOADS:
        bench_lnl(args, name)
        return
    if name in W.ROWS_WORKLOADS:
        bench_rows(args, name)
        return
    if name in W.TRN_WORKLOADS:
        bench_trn(args, name)
        return
    w = W.WORKLOADS[name]
    dev = torch.device("cuda:0")
    dt = B.BF16 if w.dtype == torch.bfloat16 else B.F32
    scale = 1.0 / math.sqrt(w.d)
    n, h, d = w.n, w.h, w.d

    torch.cuda.set_device(dev)
    torch.zeros(1, device=dev)  # initialise the context before the memory counters
    torch.cuda.reset_peak_memory_stats(dev)
    host = {}
    per_node = []
    for node in w.nodes:
        t = W.workload_inputs(w, node)
        host[node] = t
        x = {k: t[k].to(dev) for k in ("q", "k", "v", "g", "bias", "dout", "mask")}
        x["out"] = torch.empty_like(x["q"])
        x["lse"] = torch.empty(x["bias"].shape, dtype=torch.float32, device=dev)
        for gname in ("dq", "dk", "dv", "dg"):
            x[gname] = torch.empty_like(x["q"])
        x["dbias"] = torch.empty_like(x["bias"])
        per_node.append((node, x))
    if w.batch > 1:  # one copy per sample: one launch per kernel for the whole batch
        ws_bytes = max(max(B.tri_attn_fwd_batched_workspace_bytes(nd, dt, w.batch, n, h, d),
                           B.tri_attn_bwd_batched_workspace_bytes(nd, dt, w.batch, n, h, d))
                       for nd in w.nodes)
    else:
        ws_bytes = max(max(B.tri_attn_fwd_workspace_bytes(nd, dt, n, h, d),
                           B.tri_attn_bwd_workspace_bytes(nd, dt, n, h, d)) for nd in w.nodes)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    P = lambda a: a.data_ptr()  # noqa: E731

    if w.batch > 1:
        fwd_call = lambda node, *a: B.tri_attn_fwd_batched(node, dt, w.batch, *a)  # noqa: E731
        bwd_call = lambda node, *a: B.tri_attn_bwd_batched(node, dt, w.batch, *a)  # noqa: E731
    else:
        fwd_call = lambda node, *a: B.tri_attn_fwd(node, dt, *a)  # noqa: E731
        bwd_call = lambda node, *a: B.tri_attn_bwd(node, dt, *a)  # noqa: E731

    def step():
        for node, x in per_node:
            st = fwd_call(node, n, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]), P(x["g"]),
                          P(x["bias"]), P(x["mask"]), P(x["out"]), P(x["lse"]), P(ws), ws_bytes,
                          stream)
            if st != B.OK:
                raise B.TriAttnError(st, "tri_attn_fwd")
            st = bwd_call(node, n, h, d, scale, P(x["q"]), P(x["k"]), P(x["v"]), P(x["g"]),
                          P(x["bias"]), P(x["mask"]), P(x["out"]), P(x["lse"]), P(x["dout"]),
                          P(x["dq"]), P(x["dk"]), P(x["dv"]), P(x["dg"]), P(x["dbias"]), P(ws),
                          ws_bytes, stream)
            if st != B.OK:
                raise B.TriAttnError(st, "tri_attn_bwd")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize(dev)
    ms, ktimes, dom, dom_t = time_steps(step, dev, args.steps, KERNEL_FLOP_PER_LOGIT_D)
    peak_bytes = torch.cuda.max_memory_allocated(dev)

    flop_step = w.flops_fwd_bwd * len(w.nodes)
    tflops = flop_step / (ms * 1e-3) / 1e12
    peak = MFMA_BF16_PEAK_TFLOPS if dt == B.BF16 else MFMA_FP32_PEAK_TFLOPS

    per_kernel = {k: {"avg_ms": round(v[0] / v[1], 5), "launches": v[1],
                      "share": round(v[0] / max(1e-9, sum(x[0] for x in ktimes.values())), 4)}
                  for k, v in ktimes.items() if v[1] > 0}
    avg_s = dom_t[0] / dom_t[1] * 1e-3
    flop_launch = KERNEL_FLOP_PER_LOGIT_D[dom] * d * n ** 3 * h
    achieved = flop_launch / avg_s / 1e12
    traffic = recorded_traffic(dom, name)

    out = {
        "metric": ("triangle-attn fwd+bwd TFLOP/s (% of bf16 MFMA peak) at N=768; peak HBM bytes"
                   if name == W.HEADLINE else
                   f"triangle-attn fwd+bwd TFLOP/s (nominal 14 N^3 H d per sample) on {name}"),
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if dt == B.BF16 else "f32",
        "data": "synthetic (seeded normals; the paper's PDB-derived pair representations are "
                "not available)",
        "config": {"workload": name, "batch": w.batch, "n": n, "heads": h, "head_dim": d,
                   "nodes": [W.NODE_NAMES[x] for x in w.nodes], "mask": "all keys valid"
                   if w.pad_frac == 0 and w.rand_pad_frac == 0 else "key padding",
                   "bias_std": round(w.bias_std, 4), "parallelism": "none (1 GPU)"},
        "pct_of_peak": round(100.0 * tflops / peak, 3),
        "peak_hbm_bytes": int(peak_bytes),
        "workspace_bytes": int(ws_bytes),
        "naive_logits_bytes": int(n ** 3 * h * 2),
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 3),
                     "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 5),
                     "traffic": traffic},
        "per_kernel": per_kernel,
    }
    if name == W.HEADLINE and args.configs:
        del per_node, ws, x
        torch.cuda.empty_cache()
        out["configs"] = sweep_configs(args.steps)
    if args.cpu_seconds > 0:
        h0 = host[w.nodes[0]]
        if w.batch > 1:  # sample 0
            h0 = {k: (v[0] if hasattr(v, "dim") else v) for k, v in h0.items()}
        out["cpu_baseline"] = cpu_baseline(
            w, h0, args.cpu_seconds,
            whole=("tri_start_fp32_n32", "tri_start_bf16_n256_pad10") if name == W.HEADLINE
            else ())
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
