"""Benchmark of one MoE layer step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5]

A step is one pass of the whole layer over one batch of synthetic inputs:
gate + top-k (or cached ids) -> per-expert load count -> capacity update ->
dispatch -> expert FFN -> combine, and for training workloads the backward
(combine, FFN, gate, dispatch).  Inputs are resident in HBM before timing.
Prints ONE JSON line.  Per-kernel times come from HIP events that libmoe
records around each of its launches during the timed steps.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE layer tokens/sec fwd(+bwd) on 1 MI355X; % MFMA peak (GEMM), % HBM BW (dispatch)"
PEAK_BF16_TFLOPS = 2516.6    # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 flop/clk)
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0

DESCR = {
    "c1": "T=256 d=64 E=4 top-1 d_ff=128 ReLU fp32, static capacity 1.25, forward",
    "c2": "T=8192 d=512 E=16 top-2 d_ff=2048 GELU-tanh bf16, dynamic capacity 1.1, forward",
    "c3": "T=16384 d=1024 E=64 top-1 d_ff=4096 ReLU bf16 Zipf gate bias, dynamic capacity 1.1, forward+backward",
    "c4": "T=32768 d=2048 E=32 top-2 d_ff=8192 ReLU bf16 cached Zipf(1.2) assignments, exact capacity, forward+backward",
    "c5": "T=65536 d=4096 E=8 top-2 d_ff=14336 SwiGLU bf16, dynamic capacity 1.05, forward+backward",
}
VARIANTS = {
    "balance": "with the Eq. 3 balance term and its gate gradient",
    "spec": "with AggregateSpec and the Eq. 2 specification loss (squared error) driving "
            "the backward",
    "cached": "sample assignment caching on: dispatch and FFN from cached picks (4% of "
              "samples reassigned) while the gate runs on a second stream",
    "policy": "capacities from the host launch-frontier policy (pinned counts ring)",
}
# bounded oracle sample (tokens) per workload, about 10-30 s of CPU work
CPU_SAMPLE = {"c1": 256, "c2": 8192, "c3": 16384, "c4": 2048, "c5": 4096}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c5", choices=sorted(DESCR))
    ap.add_argument("--capacity", default=None,
                    help="override: static:num/den or dynamic:num/den")
    ap.add_argument("--rows", default="fill", choices=["fill", "capacity"],
                    help="capacity = padded static-shape baseline")
    ap.add_argument("--variant", default="base", choices=["base", "balance", "spec", "cached",
                                                          "policy"],
                    help="base: the layer step; balance: + Eq. 3 balance term and its gate "
                         "gradient; spec: + AggregateSpec, backward driven by the Eq. 2 "
                         "specification loss; cached: caching on, gate on a second stream; "
                         "policy: capacities from the host launch-frontier policy")
    ap.add_argument("--lam", type=float, default=0.01, help="balance term weight")
    ap.add_argument("--delta", type=int, default=1, help="policy: delta_launch")
    ap.add_argument("--policy-sweep", action="store_true",
                    help="instead of the layer: routing-only run of a drifting trajectory "
                         "of mini-batches, drops vs average capacity factor for static "
                         "capacities and for launch-frontier policies")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--configs", action="store_true",
                    help="also time every other workload into detail.configs (the default "
                         "c5 run does this unless --no-configs)")
    ap.add_argument("--no-configs", action="store_true")
    ap.add_argument("--reps", type=int, default=50,
                    help="repetitions per run of detail.configs (median reported)")
    ap.add_argument("--row-align", type=int, default=None,
                    help="rows each expert region of the grouped buffers is aligned to "
                         "(default: the layer's, one GEMM tile of 256 rows; 1 packs them)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time its replays (per-kernel "
                         "times then come from as many instrumented eager steps)")
    ap.add_argument("--blas-gemm", default=None, metavar="M,N,K",
                    help="instead of the layer: time hipBLASLt (torch.matmul) on one bf16 "
                         "product C[M,N] = A[M,K] B[N,K]^T with N(0,1) operands (context: "
                         "an achievable GEMM rate on this GPU; not part of the path)")
    ap.add_argument("--iso-gemm", default=None, metavar="M,D,F",
                    help="instead of the layer: the library's two forward products of one "
                         "ReLU expert (H = X W1^T: M x F x D, Y = A W2^T: M x D x F; no saved "
                         "planes) and hipBLASLt (torch.matmul) on the same tensors, each "
                         "sustained for a second after a half-second warm-up")
    ap.add_argument("--gate-alone", action="store_true",
                    help="instead of the layer: the gate forward on the workload's shapes, "
                         "sustained for a second, alone and after writing (or reading) as many "
                         "bytes as x elsewhere in memory (shows what the previous kernel's "
                         "dirty cache lines cost the next one)")
    ap.add_argument("--tiles", type=int, default=0, choices=[0, 1, 2],
                    help="GEMM tiles: 0 the library's choice per product, 1 256x256 "
                         "only (also fp32), 2 128x128 only (bf16; two workgroups per CU)")
    ap.add_argument("--dx-weight-copy", type=int, default=0, choices=[0, 1, 2],
                    help="bf16 dX operand: 0 the library's choice, 1 W1/W3 read K-major, "
                         "2 from a transposed copy made in the backward")
    ap.add_argument("--copy-gib", type=float, default=0.0,
                    help="instead of the layer: time a plain device-to-device copy of this "
                         "many GiB (achievable HBM bandwidth; byte-counter calibration)")
    return ap.parse_args()


def copy_calibration(gib, steps):
    """Plain device copy of a known size: achieved HBM GB/s (read + write)."""
    import torch
    n = int(gib * (1 << 30))
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(json.dumps({"copy_bytes_each_way": n, "ms_per_copy": round(ms, 4),
                      "hbm_GBps_read_plus_write": round(2 * n / (ms / 1e3) / 1e9, 1)}))


def blas_gemm(shape, steps, warmup):
    """hipBLASLt through torch.matmul on A [M,K] times B [N,K]^T (both operands
    K-contiguous, as every forward product of the layer reads them)."""
    import torch
    M, N, K = (int(v) for v in shape.split(","))
    g = torch.Generator(device="cuda:0").manual_seed(1)
    a = torch.randn(M, K, device="cuda:0", dtype=torch.bfloat16, generator=g)
    b = torch.randn(N, K, device="cuda:0", dtype=torch.bfloat16, generator=g)
    c = torch.empty(M, N, device="cuda:0", dtype=torch.bfloat16)
    # the clock ramps up over the first few hundred milliseconds of load: warm
    # up for at least 0.5 s (and `warmup` products), then time at least
    # `steps` products and 1 s
    t0 = time.perf_counter()
    n = 0
    while n < warmup or time.perf_counter() - t0 < 0.5:
        torch.matmul(a, b.t(), out=c)
        n += 1
        if n % 20 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    n = 0
    e0.record()
    while n < steps or time.perf_counter() - t0 < 1.0:
        torch.matmul(a, b.t(), out=c)
        n += 1
        if n % 20 == 0:
            torch.cuda.synchronize()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n
    print(json.dumps({"blas_gemm": [M, N, K], "ms": round(ms, 4),
                      "tflops": round(2.0 * M * N * K / (ms / 1e3) / 1e12, 1),
                      "frac_bf16_peak": round(2.0 * M * N * K / (ms / 1e3) / 1e12 /
                                              PEAK_BF16_TFLOPS, 4)}))


def iso_gemm(shape):
    """The library's forward products of one ReLU expert against hipBLASLt on
    the same tensors (X ~ N(0,1), W ~ N(0,0.02), bf16)."""
    import torch

    from paper_2205_01848_amd import binding as B
    M, d, f = (int(v) for v in shape.split(","))
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(1)
    x = torch.randn(M, d, device=dev, generator=g).to(torch.bfloat16)
    w1 = (torch.randn(1, f, d, device=dev, generator=g) * 0.02).to(torch.bfloat16)
    w2 = (torch.randn(1, d, f, device=dev, generator=g) * 0.02).to(torch.bfloat16)
    off = torch.tensor([0, M], device=dev, dtype=torch.int32)
    rows = torch.tensor([M], device=dev, dtype=torch.int32)
    y = torch.empty(M, d, device=dev, dtype=torch.bfloat16)
    ws = torch.empty(B.moe_ffn_fwd_workspace_bytes(B.MOE_BF16, B.MOE_RELU, 1, d, f, M),
                     device=dev, dtype=torch.uint8)
    h = torch.empty(M, f, device=dev, dtype=torch.bfloat16)
    yb = torch.empty(M, d, device=dev, dtype=torch.bfloat16)

    def ours():
        B.moe_expert_ffn_fwd(B.MOE_RELU, off, rows, x, w1, None, w2, None, y, ws)

    def blas():
        torch.matmul(x, w1[0].t(), out=h)
        torch.matmul(h, w2[0].t(), out=yb)

    def sustain(fn, timing):
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.5:
            fn()
            torch.cuda.synchronize()
        if timing:
            B.moe_timing_report()
            B.moe_timing_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        n = 0
        t0 = time.perf_counter()
        e0.record()
        while time.perf_counter() - t0 < 1.0:
            fn()
            n += 1
            if n % 4 == 0:
                torch.cuda.synchronize()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / n
        rep = None
        if timing:
            B.moe_timing_enable(False)
            rep = B.moe_timing_report()
        return ms, rep

    fl = 2.0 * M * d * f
    out = {"iso_gemm": [M, d, f]}
    ms, _ = sustain(blas, False)
    out["hipblaslt_ms"] = round(ms, 4)
    out["hipblaslt_tflops"] = round(2 * fl / (ms / 1e3) / 1e12, 1)
    ms, rep = sustain(ours, True)
    out["ours_ms"] = round(ms, 4)
    out["ours_tflops"] = round(2 * fl / (ms / 1e3) / 1e12, 1)
    for k in ("gemm_fwd_h", "gemm_fwd_y"):
        c, t = rep[k]
        out[k + "_tflops"] = round(fl / (t / c / 1e3) / 1e12, 1)
    print(json.dumps(out))


def gate_alone(name):
    """Gate forward time on the workload's shapes (x ~ N(0,1), w_g ~ N(0,0.02)),
    alone and after another kernel writes or reads as many bytes as x."""
    import torch

    import workloads as W
    from paper_2205_01848_amd import binding as B
    wl = W.config(name)
    assert wl.gate == "linear", "the workload has no gate"
    T, d, E, k = wl.T, wl.d, wl.E, wl.k
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(1)
    x = torch.randn(T, d, device=dev, generator=g).to(torch.bfloat16)
    wg = (torch.randn(E, d, device=dev, generator=g) * 0.02).to(torch.bfloat16)
    bias = torch.zeros(E, device=dev, dtype=torch.float32)
    logits = torch.empty(T, E, device=dev, dtype=torch.float32)
    ids = torch.empty(T, k, device=dev, dtype=torch.int32)
    wts = torch.empty(T, k, device=dev, dtype=torch.float32)
    other = torch.empty(T, d, device=dev, dtype=torch.bfloat16)
    before = {"alone": lambda: None,
              "after_write_of_x_bytes": lambda: other.fill_(1.0),
              "after_read_of_x_bytes": lambda: torch.sum(other, dtype=torch.float32)}
    nbytes = T * d * 2 + E * d * 2 + T * E * 4 + T * k * 8
    out = {"gate_alone": name, "T": T, "d": d, "E": E, "algorithmic_bytes": nbytes}
    for label, pre in before.items():
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 0.3:
            pre()
            B.moe_gate_topk(x, wg, bias, k, wl.renorm, logits, ids, wts)
            torch.cuda.synchronize()
        B.moe_timing_report()
        B.moe_timing_enable(True)
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 1.0:
            for _ in range(10):
                pre()
                B.moe_gate_topk(x, wg, bias, k, wl.renorm, logits, ids, wts)
            torch.cuda.synchronize()
        B.moe_timing_enable(False)
        n, ms = B.moe_timing_report()["gate_fwd"]
        us = ms / n * 1e3
        out[label] = {"us": round(us, 2), "GBps": round(nbytes / us / 1e3, 1),
                      "frac_hbm": round(nbytes / us / 1e3 / PEAK_HBM_GBS, 4), "launches": n}
    print(json.dumps(out))


def gemm_flops(wl, kept):
    """Algorithmic MFMA flops per GEMM pass over `kept` rows: 2 flops per multiply-add
    of each rows x d x f product the pass computes (gated FFN: two for H1 and H3)."""
    unit = 2 * kept * wl.d * wl.f
    g = 2 if wl.act == "swiglu" else 1
    fl = {"gemm_fwd_h": g * unit, "gemm_fwd_y": unit}
    if wl.backward:
        fl.update({"gemm_bwd_da": unit, "gemm_bwd_dx": g * unit, "gemm_bwd_dw2": unit,
                   "gemm_bwd_dw13": g * unit})
    return fl


def hbm_bytes(wl, kept, active, padded=0):
    """Algorithmic HBM bytes per launch of the row-moving kernels (`padded`:
    rows the padded static baseline zeroes beyond the kept ones)."""
    s, T, d, E, k = wl.esize, wl.T, wl.d, wl.E, wl.k
    b = {
        "gate_fwd": T * d * s + E * d * s + T * E * 4 + T * k * 8,
        "dispatch_gather": active * d * s + kept * d * s + T * k * 4,
        "combine": kept * d * s + T * d * s + T * k * 8,
    }
    if wl.backward:
        b["combine_bwd"] = T * d * s + 2 * kept * d * s + T * k * 12
        b["dispatch_bwd"] = kept * d * s + T * d * s + T * k * 4 + \
            (T * E * 4 + E * d * s if wl.gate == "linear" else 0)
        if wl.dtype == "bf16":
            # the transposed copy of [W1; W3] read by dX (large experts only):
            # the weights read once and written once
            g = 2 if wl.act == "swiglu" else 1
            b["transpose_w"] = 2 * E * g * wl.f * d * s
    if wl.gate != "linear":
        del b["gate_fwd"]
    # operators of the variants
    b["balance_fwd"] = T * E * 4 + E * 4
    b["aggregate_spec"] = kept * d * s + T * k * d * s + T * k * 4
    b["spec_loss"] = 2 * kept * d * s + T * d * s + T * k * 12
    b["cache_update"] = 3 * T * k * 4
    b["cached_weights"] = T * E * 4 + 2 * T * k * 4
    if padded:
        b["zero_pad_rows"] = padded * d * s
    return b


def profiled_traffic(workload, kernel):
    """Calibrated HBM bytes per launch of `kernel` from profiles/traffic_<workload>.json,
    or None when the summary is missing or the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    from paper_2205_01848_amd.rocprof_summary import source_hash
    with open(path) as f:
        t = json.load(f)
    if t.get("source_hash") != source_hash() or kernel not in t.get("kernels", {}):
        return None
    k = t["kernels"][kernel]
    return int(k["read_bytes"] + k["write_bytes"])


def cpu_baseline(wl, I, cap_rule, ntok):
    """The oracle as it stands, on the first `ntok` tokens of the batch (the
    same per-token work: gate, capacity on the sample's own counts,
    dispatch, FFN, combine, backward)."""
    import numpy as np
    import threadpoolctl

    import oracle as O
    f64 = O.bf16_to_f64 if wl.dtype == "bf16" else (lambda a: np.asarray(a, np.float64))
    X = f64(I.x[:ntok])
    W1, W2 = f64(I.w1), f64(I.w2)
    W3 = f64(I.w3) if I.w3 is not None else None
    WG = f64(I.w_g) if I.w_g is not None else None
    dY = f64(I.dy[:ntok]) if I.dy is not None else None
    kind, num, den = cap_rule
    t0 = time.perf_counter()
    if wl.gate == "linear":
        r = O.route(X, WG, I.bias, wl.k, wl.renorm)
        ids, wts, logits = r["ids"], r["weights"], r["logits"]
    else:
        ids, wts, logits = I.ids[:ntok], I.cw[:ntok].astype(np.float64), None
    counts = O.count_assignments(ids, wl.E)
    if kind == "static":
        cap = O.capacity_static(ntok, wl.k, wl.E, num, den)
    else:
        cap = O.capacity_dynamic(counts, ntok, num, den)
    R = int(cap.sum())
    fw = O.layer_forward(X, W1, W3, W2, wl.act, wl.dtype, ids, wts, cap, R, wl.E)
    if wl.backward:
        O.layer_backward(fw, X, dY, W1, W3, W2, wl.act, wl.dtype, ids, wts, wl.E,
                         logits=logits, renorm=wl.renorm, w_g=WG)
    el = time.perf_counter() - t0
    threads = max([p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()] + [1])
    return {"value": ntok / el, "unit": "tokens/s", "cores": int(threads),
            "host_cpus": os.cpu_count(), "kind": "oracle",
            "sample": f"first {ntok} of {wl.T} tokens of the workload, "
                      f"{'forward+backward' if wl.backward else 'forward'}, float64 numpy "
                      f"({el:.1f} s)"}


def policy_sweep(args):
    """Drops vs average capacity factor over a drifting trajectory of
    mini-batches (routing only: count -> capacity -> dispatch of narrow
    rows), for static capacities (Eq. 4) and launch-frontier policies
    (Section 4.1 with the recompile appendix).  The demand per mini-batch is
    the library's own count; the capacity trajectories of these settings are
    checked against the oracle in the GPU tests, not here."""
    import numpy as np
    import torch

    import workloads as W
    from paper_2205_01848_amd import binding as B

    wl = W.config(args.workload)
    T, E, k, N, dw = wl.T, wl.E, wl.k, args.steps, 8
    log(f"policy sweep on {args.workload} shapes: {N} drifting mini-batches")
    traj = W.drifting_assignments(wl.seed, T, E, k, N)
    dev = torch.device("cuda:0")
    ids_dev = [torch.from_numpy(a).to(dev) for a in traj]
    R = E * T
    x = torch.zeros(T, dw, dtype=torch.bfloat16, device=dev)
    cap = torch.empty(E, dtype=torch.int32, device=dev)
    off = torch.empty(E + 1, dtype=torch.int32, device=dev)
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    fill = torch.empty(E, dtype=torch.int32, device=dev)
    dest = torch.empty(T, k, dtype=torch.int32, device=dev)
    src = torch.empty(R, dtype=torch.int32, device=dev)
    xd = torch.empty(R, dw, dtype=torch.bfloat16, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = B.workspace(B.moe_dispatch_workspace_bytes(T, E, k), dev)
    fills = torch.empty(N, E, dtype=torch.int32, device=dev)
    caps = torch.empty(N, E, dtype=torch.int32, device=dev)
    demands = torch.empty(N, E, dtype=torch.int32, device=dev)
    for i in range(N):                     # per-expert demand of every mini-batch
        B.moe_count(ids_dev[i], E, counts, status)
        demands[i].copy_(counts)
    torch.cuda.synchronize()
    seq = demands.cpu().numpy().astype(np.int64)
    demand = float(T * k)

    def summarise(name, extra):
        torch.cuda.synchronize()
        f = fills.cpu().numpy().astype(np.int64)
        c = caps.cpu().numpy().astype(np.int64)
        drops = (seq - f).sum()
        row = {"setting": name, "dropped_pct": round(100.0 * drops / (N * demand), 3),
               "avg_capacity_factor": round(float(c.sum(axis=1).mean()) / demand, 4)}
        row.update(extra)
        return row, c

    rows = []
    for a in [(1, 1), (5, 4), (3, 2), (2, 1), (3, 1)]:
        for i in range(N):
            B.moe_update_capacity(T, k, E, None, a[0], a[1], 0, cap, off)
            B.moe_dispatch(x, ids_dev[i], E, cap, off, R, counts, fill, dest, src, xd, status, ws)
            fills[i].copy_(fill)
            caps[i].copy_(cap)
        rows.append(summarise(f"static alpha {a[0]}/{a[1]}", {})[0])
    for margin in [(21, 20), (11, 10)]:
        for i in range(N):
            B.moe_count(ids_dev[i], E, counts, status)
            B.moe_update_capacity(T, k, E, counts, margin[0], margin[1], 0, cap, off)
            B.moe_dispatch(x, ids_dev[i], E, cap, off, R, counts, fill, dest, src, xd, status, ws)
            fills[i].copy_(fill)
            caps[i].copy_(cap)
        rows.append(summarise(f"device dynamic {margin[0]}/{margin[1]} (this batch's counts)",
                              {})[0])
    B.moe_update_capacity(T, k, E, None, 1, 1, 0, cap, off)   # static alpha = 1
    init = cap.cpu().numpy().astype(np.int64)
    for grow, shrink in [((21, 20), (5, 4)), ((11, 10), (13, 10)), ((6, 5), (3, 2)),
                         ((5, 4), (2, 1))]:
        for delta in (0, 1, 2):
            pol = B.CapacityPolicy(T, k, E, delta, grow, shrink, init)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(N):
                pol.begin(cap, off)
                B.moe_dispatch(x, ids_dev[i], E, cap, off, R, counts, fill, dest, src, xd,
                               status, ws)
                pol.end(counts)
                fills[i].copy_(fill)
                caps[i].copy_(cap)
            torch.cuda.synchronize()
            wall = (time.perf_counter() - t0) * 1e3 / N
            st = pol.state()
            pol.close()
            row, c = summarise(f"policy grow {grow[0]}/{grow[1]} shrink {shrink[0]}/{shrink[1]} "
                               f"delta {delta}",
                               {"recompiles": st["recompiles"], "ms_per_iteration": round(wall, 3)})
            rows.append(row)
    out = {"metric": "capacity policy: dropped assignments vs average capacity factor",
           "workload": f"{args.workload} shapes T={T} E={E} k={k}, {N} mini-batches with "
                       "drifting Zipf loads (exponent 1.2 -> 0.6, adjacent experts swap "
                       "every 5)",
           "status": int(status.item()), "rows": rows}
    print(json.dumps(out))


def upload(wl, dev):
    """Seeded inputs of a workload, resident in device memory."""
    import numpy as np
    import torch

    import workloads as W
    t0 = time.perf_counter()
    I = W.make_inputs(wl)
    t_gen = time.perf_counter() - t0

    def up(a):
        if a is None:
            return None
        if wl.dtype == "bf16" and a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    return I, up, t_gen


def build_step(wl, I, up, cap_rule, rows, variant, args, dev):
    """The layer, its device inputs and one step (closure) for this run."""
    import torch

    import workloads as W
    from paper_2205_01848_amd import MoELayer, binding as B, rows_alloc_for
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x, w1, w3, w2, dy = (up(a) for a in (I.x, I.w1, I.w3, I.w2, I.dy))
    from paper_2205_01848_amd.layer import ROW_ALIGN
    align = ROW_ALIGN if getattr(args, "row_align", None) is None else args.row_align
    kind, num, den = cap_rule
    R = rows_alloc_for(kind, wl.T, wl.k, wl.E, num, den, align)
    L = MoELayer(wl.T, wl.d, wl.E, wl.k, wl.f, wl.act, td, R, backward=wl.backward,
                 gate=wl.gate == "linear", row_align=align)
    if wl.gate == "linear":
        fkw = dict(w_g=up(I.w_g), bias=None if I.bias is None else up(I.bias), renorm=wl.renorm)
        bkw = dict(w_g=fkw["w_g"], renorm=wl.renorm)
    else:
        fkw = dict(ids=up(I.ids), weights=up(I.cw))
        bkw = dict(weights=fkw["weights"])

    if variant in ("balance", "cached") and wl.gate != "linear":
        raise SystemExit(f"--variant {variant} needs a workload with a gate")
    if variant in ("balance", "spec", "cached") and not wl.backward:
        raise SystemExit(f"--variant {variant} needs a training workload")
    extra = {}
    if variant == "spec":
        extra["target"] = up(W.make_target(wl))
        extra["spec_rows"] = torch.empty(wl.T * wl.k, wl.d, dtype=td, device=dev)
    if variant == "cached":
        # last epoch's picks: the gate's own, with 4% of the samples reassigned
        L.gate(x, fkw["w_g"], fkw["bias"], wl.renorm)
        fresh = L.ids.cpu().numpy()
        extra["cached"] = torch.from_numpy(W.reassign_some(wl.seed, fresh, wl.E, 0.04)).to(dev)
        extra["cache_out"] = torch.empty_like(extra["cached"])
        extra["unchanged"] = torch.zeros(1, dtype=torch.int32, device=dev)
        extra["gate_stream"] = torch.cuda.Stream()
    if variant == "policy":
        T_, k_, E_ = wl.T, wl.k, wl.E
        init = [-(-T_ * k_ // E_)] * E_                 # Eq. 4 with alpha = 1
        grow = (cap_rule[1], cap_rule[2]) if cap_rule[0] == "dynamic" else (21, 20)
        extra["policy"] = B.CapacityPolicy(T_, k_, E_, args.delta, grow, (5, 4), init,
                                           row_align=L.row_align)

    def step():
        if variant == "cached":
            L.forward_cached(x, w1, w3, w2, cached=extra["cached"], cache_out=extra["cache_out"],
                             unchanged=extra["unchanged"], w_g=fkw["w_g"], bias=fkw["bias"],
                             renorm=wl.renorm, capacity=cap_rule, gate_stream=extra["gate_stream"],
                             rows=rows)
            L.backward(x, dy, w1, w3, w2, rows=rows, ids=extra["cached"],
                       weights=L.cached_weights, **bkw)
            return
        if variant == "policy":
            rows_needed, _ = extra["policy"].begin(L.capacity, L.offsets)
            if rows_needed > L.rows_alloc:
                raise SystemExit(f"policy asks for {rows_needed} rows > {L.rows_alloc}")
            L.forward(x, w1, w3, w2, capacity=("policy", 1, 1), rows=rows, **fkw)
            extra["policy"].end(L.counts)
        else:
            L.forward(x, w1, w3, w2, capacity=cap_rule, rows=rows,
                      balance=args.lam if variant == "balance" else None, **fkw)
        if variant == "spec":
            L.aggregate_spec(extra["spec_rows"])
        if wl.backward:
            L.backward(x, dy, w1, w3, w2, rows=rows, target=extra.get("target"), **bkw)

    return L, step, extra


def kernel_table(wl, kern, kern_ms, kept, executed, active):
    """Per-kernel rates from the library's timing report, the dominant kernel
    and the GEMM totals."""
    fl_alg = gemm_flops(wl, kept)
    by = hbm_bytes(wl, kept, active, executed - kept)
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    detail = {}
    for name, (n, ms) in kern.items():
        avg = ms / max(n, 1)
        row = {"launches": n, "avg_ms": round(avg, 4), "share": round(ms / kern_ms, 4)}
        if name in fl_alg:
            row["tflops"] = round(fl_alg[name] / avg / 1e9, 1)
            row["frac_mfma_peak"] = round(fl_alg[name] / avg / 1e9 / peak, 4)
        if name in by:
            row["gbs"] = round(by[name] / avg / 1e6, 1)
            row["frac_hbm"] = round(by[name] / avg / 1e6 / PEAK_HBM_GBS, 4)
        detail[name] = row
    dom = max(kern.items(), key=lambda kv: kv[1][1])[0] if kern else None
    gemm_ms = sum(kern[k][1] for k in kern if k in fl_alg)
    gemm_fl = sum(fl_alg[k] * kern[k][0] for k in kern if k in fl_alg)
    gemm = round(gemm_fl / (gemm_ms / 1e3) / 1e12, 1) if gemm_ms else None
    return detail, dom, gemm, round(gemm_ms / kern_ms, 4), fl_alg, by, peak


# extra runs reported in detail.configs of the default run: every workload,
# with the static-capacity runs both on kept rows and padded to capacity
EXTRA_RUNS = [("c1", 0, "fill"), ("c2", 1, "fill"), ("c2", 0, "fill"), ("c2", 0, "capacity"),
              ("c3", 1, "fill"), ("c3", 0, "fill"), ("c3", 0, "capacity"), ("c4", 0, "fill")]
FLUSH_BYTES = 512 << 20       # scratch written between repetitions (> the 256 MB MALL)


def median_runs(args, dev):
    """detail.configs: each run's median step over args.reps repetitions
    (uninstrumented, a FLUSH_BYTES scratch write before each, so no
    repetition finds the last one's data in the L2 or the MALL), then the
    same number of instrumented repetitions (flushed the same way) for the
    per-kernel rates."""
    import statistics

    import torch

    import workloads as W
    from paper_2205_01848_amd import binding as B
    scratch = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    out = []
    cache = {}
    for name, run, rows in EXTRA_RUNS:
        wl = W.config(name)
        cap_rule = wl.capacity[run]
        if name not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            cache[name] = upload(wl, dev)
        I, up, _ = cache[name]
        log(f"config {name} capacity {cap_rule} rows={rows}: {args.reps} reps")
        L, step, _ = build_step(wl, I, up, cap_rule, rows, "base", args, dev)
        for _ in range(max(args.warmup, 2)):
            step()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.reps)]
        for i in range(args.reps):
            scratch.fill_(i & 0xFF)
            ev[i][0].record()
            step()
            ev[i][1].record()
        torch.cuda.synchronize()
        times = [a.elapsed_time(b) for a, b in ev]
        med = statistics.median(times)
        B.moe_timing_report()
        B.moe_timing_enable(True)
        for i in range(args.reps):
            scratch.fill_((i + 128) & 0xFF)
            step()
        torch.cuda.synchronize()
        B.moe_timing_enable(False)
        kern = B.moe_timing_report()
        kern_ms = sum(ms for _, ms in kern.values())
        kept = int(L.fill.sum().item())
        executed = int((L.fill if rows == "fill" else L.capacity).sum().item())
        active = int((L.dest_row >= 0).any(dim=1).sum().item())
        detail, dom, gemm, gshare, _, _, _ = kernel_table(wl, kern, kern_ms, kept, executed, active)
        out.append({"workload": f"{name}: {DESCR[name]}".split(",")[0],
                    "capacity": f"{cap_rule[0]} {cap_rule[1]}/{cap_rule[2]}", "rows": rows,
                    "pass": "fwd+bwd" if wl.backward else "fwd",
                    "ms_per_step_median": round(med, 4),
                    "ms_per_step_min": round(min(times), 4),
                    "tokens_per_s": round(wl.T / (med / 1e3), 1), "reps": args.reps,
                    "flush_bytes": FLUSH_BYTES, "kept_rows": kept, "executed_rows": executed,
                    "status": int(L.status.item()), "gemm_tflops": gemm, "gemm_share": gshare,
                    "dominant": dom, "kernels": detail})
        del L, step
    del scratch
    cache.clear()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the layer is not "
              "sharded across GPUs.", file=sys.stderr)
        sys.exit(2)
    if args.copy_gib > 0:
        copy_calibration(args.copy_gib, args.steps)
        return
    if args.blas_gemm:
        blas_gemm(args.blas_gemm, args.steps, args.warmup)
        return
    if args.iso_gemm:
        iso_gemm(args.iso_gemm)
        return
    if args.gate_alone:
        gate_alone(args.workload)
        return
    if args.policy_sweep:
        policy_sweep(args)
        return
    import torch

    import workloads as W
    from paper_2205_01848_amd import binding as B

    B.moe_set_gemm_tiles(args.tiles)
    B.moe_set_dx_weight_copy(args.dx_weight_copy)
    wl = W.config(args.workload)
    cap_rule = wl.capacity[-1]
    if args.capacity:
        kind, frac = args.capacity.split(":")
        num, den = (int(v) for v in frac.split("/"))
        cap_rule = (kind, num, den)
    dev = torch.device("cuda:0")
    log(f"workload {args.workload}: generating inputs")
    I, up, t_gen = upload(wl, dev)
    log(f"inputs ready in {t_gen:.1f} s")
    variant = args.variant
    L, step, extra = build_step(wl, I, up, cap_rule, args.rows, variant, args, dev)

    warmup = args.warmup
    if variant == "policy":
        warmup = max(warmup, args.delta + 2)    # the first recompile has taken effect
    log("warmup")
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    log("timed steps")
    kept = int(L.fill.sum().item())
    executed = int((L.fill if args.rows == "fill" else L.capacity).sum().item())
    active = int((L.dest_row >= 0).any(dim=1).sum().item())
    status = int(L.status.item())

    graph = None
    if args.graph:
        if variant in ("cached", "policy"):
            raise SystemExit(f"--graph does not apply to --variant {variant} (host work per step)")
        log("capturing one step")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()                   # a step on the capture stream before capturing
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()

    def timed(run, instrument):
        B.moe_timing_enable(instrument)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            run()
        e1.record()
        torch.cuda.synchronize()
        B.moe_timing_enable(False)
        return e0.elapsed_time(e1)

    B.moe_timing_report()            # drop warmup records
    if graph is None:
        total_ms = timed(step, True)
        kern_ms = total_ms
    else:
        total_ms = timed(graph.replay, False)
        kern_ms = timed(step, True)  # per-kernel times: instrumented eager steps
    kern = B.moe_timing_report()
    ms_step = total_ms / args.steps

    detail, dom, gemm, gshare, fl_alg, by, peak = kernel_table(wl, kern, kern_ms, kept, executed,
                                                              active)
    roof = None
    if dom in fl_alg:
        n, ms = kern[dom]
        ach = fl_alg[dom] / (ms / n / 1e3) / 1e12
        roof = {"bound": "mfma", "kernel": dom, "achieved": round(ach, 1), "peak": peak,
                "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                "traffic": profiled_traffic(args.workload, dom)}
    elif dom in by:
        n, ms = kern[dom]
        ach = by[dom] / (ms / n / 1e3) / 1e9
        roof = {"bound": "hbm", "kernel": dom, "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                "traffic": profiled_traffic(args.workload, dom)}

    out = {
        "metric": METRIC,
        "value": round(wl.T / (ms_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": f"{args.workload}: {DESCR[args.workload]}"
                   + ("" if variant == "base" else f" [{VARIANTS[variant]}]"),
                   "T": wl.T, "d": wl.d,
                   "E": wl.E, "k": wl.k, "d_ff": wl.f, "act": wl.act,
                   "capacity": f"{cap_rule[0]} {cap_rule[1]}/{cap_rule[2]}",
                   "rows": args.rows, "pass": "fwd+bwd" if wl.backward else "fwd",
                   "row_align": L.row_align, "parallelism": "single GPU",
                   "gemm_tiles": ["auto", "256x256", "128x128"][args.tiles],
                   "dx_weight_copy": ["auto", "off", "on"][args.dx_weight_copy]},
        "roofline": roof,
        "cpu_baseline": None,
        "detail": {"kept_rows": kept, "executed_rows": executed, "status": status,
                   "gemm_tflops": gemm, "gemm_share": gshare,
                   "input_gen_s": round(t_gen, 1), "kernels": detail},
    }
    if graph is not None:
        out["config"]["launch"] = "HIP graph replay of one captured step"
        out["detail"]["kernel_timing"] = (f"{args.steps} instrumented eager steps after the "
                                          f"timed replays ({kern_ms / args.steps:.4f} ms/step)")
    if variant != "base":
        out["config"]["variant"] = variant
    if variant == "balance":
        out["config"]["lambda"] = args.lam
        out["detail"]["balance_loss"] = float(L.balance_loss.item())
    if variant == "spec":
        out["detail"]["spec_loss"] = float(L.spec_loss_value.item())
    if variant == "cached":
        n = warmup + args.steps
        out["detail"]["unchanged_fraction"] = round(
            int(extra["unchanged"].item()) / (n * wl.T), 4)
    if variant == "policy":
        st = extra["policy"].state()
        out["detail"]["policy"] = {"delta_launch": args.delta, "recompiles": st["recompiles"],
                                   "capacity": st["cap"],
                                   "capacity_factor": round(sum(st["cap"]) / (wl.T * wl.k), 4)}
        extra["policy"].close()
    log(f"{ms_step:.3f} ms/step")
    del L, step, extra
    torch.cuda.empty_cache()

    headline_default = (args.workload == "c5" and variant == "base" and args.rows == "fill"
                        and not args.capacity and not args.graph)
    if args.configs or (headline_default and not args.no_configs):
        out["detail"]["configs"] = median_runs(args, dev)
    if not args.no_cpu_baseline:
        log("oracle baseline")
        out["cpu_baseline"] = cpu_baseline(wl, I, cap_rule, CPU_SAMPLE[args.workload])
    print(json.dumps(out))


if __name__ == "__main__":
    main()
