#!/usr/bin/env python3
"""Throughput of the Adaptive SGD hot path on one MI355X.

One step = one SGD step of one replica on one batch of the workload: the
first-layer gather, the radix sort of the batch's feature and label ids, the
output-layer forward (online softmax over all labels), the per-row combine
(loss, dH1), the output-layer backward with the in-place W2/b2 update, the b1
update and the sparse W1 update.  The dataset is staged in HBM before timing;
batches are zero-copy row slices.  Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--workload wide-label|wide-feature|mid|tiny|elastic]

With --workload elastic a step is one round of configuration 5 (4 replicas of
the wide-label model on 4 HIP streams: dynamic dispatch of a mega-batch, merge,
batch-size scaling).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

METRIC = "training samples/sec at 1 GPU + % of HBM/MFMA roofline per kernel"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}
H = 128
# on the library's second stream (beside the output layer) or inside another launch
OVERLAPPED = ("gather", "sort", "labels", "hidden", "dense_fwd", "dense_bwd", "w1_update")

# HBM traffic of a kernel from `rocprofv3 --pmc FETCH_SIZE` and `--pmc WRITE_SIZE` runs of this bench
# (KiB per dispatch, averaged; profiles/wide_label_hbm_counters.md), scaled by what the same counters
# read for a plain device copy of 256 MiB: fetched bytes = 2.0 x FETCH_SIZE, written = 1.0 x WRITE_SIZE.
# A figure holds only for the kernel sources it was measured on (their sha256); otherwise it is null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
PMC_TRAFFIC = {
    ("wide-label", 256, "out_bwd"): dict(
        sources=('csrc/k_out_bwd.hip', 'csrc/asgd_dev.h', 'csrc/asgd_kernels.h'),
        sha256="bd515fcc493667e9f5aed09b57095f2055fc1c03542cdaac00d2cd86aa7de0a9",
        fetch_kib=169819.5, write_kib=337663.1),
    ("wide-label", 1024, "out_bwd"): dict(
        sources=('csrc/k_out_bwd.hip', 'csrc/asgd_dev.h', 'csrc/asgd_kernels.h'),
        sha256="bd515fcc493667e9f5aed09b57095f2055fc1c03542cdaac00d2cd86aa7de0a9",
        fetch_kib=177337.2, write_kib=337920.8),
    ("wide-feature", 128, "out_bwd"): dict(
        sources=('csrc/k_out_bwd.hip', 'csrc/asgd_dev.h', 'csrc/asgd_kernels.h'),
        sha256="bd515fcc493667e9f5aed09b57095f2055fc1c03542cdaac00d2cd86aa7de0a9",
        fetch_kib=52256.6, write_kib=103524.0),
    ("elastic", 4, "merge"): dict(
        sources=('csrc/k_merge.hip', 'csrc/asgd_dev.h', 'csrc/asgd_kernels.h'),
        sha256="76e8aa214af20f11e78470a2185c4c56fa9aadc98d47c7ddc7b4e6ab63479ba6",
        fetch_kib=1216912.0, write_kib=2028091.2),
}


def measured_traffic(workload: str, batch: int, kernel: str):
    """HBM bytes per launch from the counters, or None if none were taken on these sources."""
    import hashlib
    rec = PMC_TRAFFIC.get((workload, batch, kernel))
    if rec is None:
        return None
    pkg = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2110_07029_amd")
    h = hashlib.sha256()
    for rel in rec["sources"]:
        with open(os.path.join(pkg, rel), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != rec["sha256"]:
        return None
    return (rec["fetch_kib"] * FETCH_SCALE + rec["write_kib"] * WRITE_SCALE) * 1024.0


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="wide-label")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's batch size (e.g. 1024, the elastic b_max)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run 10 plain device copies of 256 MiB (scale for the HBM byte counters)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="budget of the oracle CPU baseline (0 disables it)")
    ap.add_argument("--unfused", action="store_true",
                    help="the output layer with stored logits and a standalone softmax / cross-entropy pass "
                         "(ASGD_UNFUSED_OUTPUT) instead of the fused one")
    ap.add_argument("--extra-hidden", action="store_true",
                    help="the model with a second dense hidden layer (extra_hidden_layers = 1)")
    ap.add_argument("--ramp", type=int, default=0,
                    help="only time N steps one by one from an idle GPU (per-step HIP events) and print "
                         "the step times by window: how long the clocks take to reach their loaded state")
    ap.add_argument("--settle-ms", type=float, default=400.0,
                    help="untimed load before the warm-up steps, so that the GPU's clocks have left "
                         "their idle state (0 disables it)")
    return ap.parse_args()


def settle(step, ms: float) -> int:
    """Run `step(i)` untimed until `ms` milliseconds of wall time have passed.

    After idle the GPU takes tens of milliseconds of load to reach its loaded
    clocks: per-step event times of the wide-label step measured from a cold
    start were 0.35 ms for steps 5-25, 0.31 ms for 25-50 and 0.27 ms after
    step 100, and a 20-step window taken after 0.5 s of idle ran at 0.34 ms.
    A short timed region right after data generation would measure that ramp,
    not the kernels, so the warm-up steps start from a loaded GPU."""
    import torch
    if ms <= 0:
        return 0
    n, t0 = 0, time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(8):
            step(n)
            n += 1
        torch.cuda.synchronize()
    return n


def kernel_model(w, B, nnz, lnnz, uniq, splits):
    """Algorithmic bytes and flops of one launch of each kernel group."""
    F, L = w.n_features, w.n_labels
    op = 2 if w.gemm_bf16 else 4
    ldz = -(-L // 32) * 32          # stored logits: whole 32-label tiles per row
    return {
        # unfused output: reads W2 and b2 once, writes Z [B x ldz] fp32
        "logits": dict(bytes=4.0 * L * (H + 1) + 4.0 * B * ldz, flops=2.0 * B * H * L),
        # unfused output: reads Z once (the online-max pass) and the target logits; writes lse, loss
        "softmax": dict(bytes=4.0 * B * ldz + 4.0 * lnnz + 8.0 * B, flops=0.0),
        # unfused output: reads Z and W2 once, writes the split partials of P W2, then dA
        "dh": dict(bytes=4.0 * B * ldz + 4.0 * L * (H + 1) + splits * B * H * 4.0 + lnnz * H * 4.0 + B * H * 8.0,
                   flops=2.0 * B * H * L),
        # second hidden layer: A1 and Wh read, A2 and H2 written; backward reads dA2, A1, Wh, writes dA1, Wh
        "dense_fwd": dict(bytes=B * H * 4.0 + H * H * 4.0 + B * H * (4.0 + op), flops=2.0 * B * H * H),
        "dense_bwd": dict(bytes=3 * B * H * 4.0 + 3 * H * H * 4.0, flops=4.0 * B * H * H),
        # reads the touched W1 rows once, the batch's (id, value) pairs; writes A1 (fp32) and H1
        # in the operand type (and its transpose, for fp32 operands only)
        "gather": dict(bytes=uniq * H * 4 + nnz * 8 + B * H * (4 + op * (1 if w.gemm_bf16 else 2)),
                       flops=2.0 * nnz * H),
        # two radix passes over (key, position) of every feature entry
        "sort": dict(bytes=2 * nnz * 4 * 5, flops=0.0),
        # label entries: read (label, row), write the grouped pairs and the block offsets
        "labels": dict(bytes=lnnz * 12 + (L // 32 + 1) * 4, flops=0.0),
        # reads W2 and b2 once; Z = H1 W2^T and O = P W2 (the dense part of dH1)
        "out_fwd": dict(bytes=4.0 * L * (H + 1), flops=4.0 * B * H * L),
        # reads the forward's per-(split, row) maxima and sums and the target rows of W2; writes
        # lse, the loss rows and the rows' mean target weights
        "out_combine": dict(bytes=splits * B * 2 * 4 + lnnz * H * 4 + B * H * 4, flops=2.0 * lnnz * H),
        # reads the forward's partials (max, sum, O), the mean target weights and A1; writes dA1
        "hidden": dict(bytes=splits * B * (H + 2) * 4 + B * H * 4 * 3, flops=0.0),
        # reads and writes W2 and b2 once; the logits recomputed (Z = H1 W2^T) and dW2 = dZ^T H1
        "out_bwd": dict(bytes=8.0 * L * (H + 1), flops=4.0 * B * H * L),
        # reads and writes the touched W1 rows once, the sorted (key, position) pairs, the
        # entries' rows and values; its last workgroup reads dA1 for the b1 update
        "w1_update": dict(bytes=uniq * H * 8 + nnz * 16 + B * H * 4, flops=2.0 * nnz * H + B * H),
    }


def measured_peaks(n_floats: int, stream):
    """What this GPU sustains, measured in the same run beside the datasheet peaks:
    an in-place streaming update of n_floats fp32 (read and write the same
    addresses, like the backward's W2 update), and a large bf16 GEMM by the
    vendor library (a practical matrix-core rate)."""
    import torch
    a = torch.ones(n_floats, dtype=torch.float32, device="cuda")
    x = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")
    y = torch.randn(8192, 8192, dtype=torch.bfloat16, device="cuda")

    def timed(fn, reps):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3 / reps

    t_up = timed(lambda: a.mul_(1.0000001), 20)
    t_mm = timed(lambda: torch.matmul(x, y), 10)
    del a, x, y
    return {"hbm_inplace_update_GBs": round(8.0 * n_floats / t_up / 1e9, 1),
            "bf16_gemm_TFLOPs": round(2.0 * 8192 ** 3 / t_mm / 1e12, 1),
            "how": "torch mul_ in place over a W2-sized fp32 tensor; torch.matmul 8192^3 bf16"}


def measure_gather_saturating(w, stream, rows=16384, reps=10):
    """The first-layer gather at a shape that fills the GPU: top-k prediction over
    `rows` rows of the workload (the library's largest prediction batch: one
    workgroup of 8 waves per row, 16 waves of workgroups per CU; its gather is the
    training step's kernel without the label work), timed with the library's
    events.  At the training batch the gather is latency-bound; here its rate shows
    what the kernel sustains."""
    import torch
    import paper_2110_07029_amd as asgd
    from paper_2110_07029_amd import synth
    ds = synth.generate(w, n_samples=rows)
    ip = np.asarray(ds.x.indptr)
    nnz = int(ip[-1] - ip[0])
    uniq = len(np.unique(ds.x.indices))
    dx = asgd.DeviceCSR(ds.x)
    m = asgd.asgd_model_init(w.n_features, w.n_labels, rows, nnz, 1, gemm_bf16=w.gemm_bf16,
                             seed=w.init_seed, stream=stream)
    try:
        ids = torch.empty((rows, 1), dtype=torch.int32, device="cuda")
        xb = dx.batch(0, rows)
        asgd.asgd_predict_topk(m, xb, 1, ids)
        torch.cuda.synchronize()
        k = asgd.KERNELS.index("gather")
        asgd.asgd_model_set_timing(m, True)
        asgd.asgd_model_get_timing(m, k)
        for _ in range(reps):
            asgd.asgd_predict_topk(m, xb, 1, ids)
        torch.cuda.synchronize()
        tot, n = asgd.asgd_model_get_timing(m, k)
        asgd.asgd_model_set_timing(m, False)
    finally:
        asgd.asgd_model_free(m)
    avg_s = tot / n * 1e-3
    op = 2 if w.gemm_bf16 else 4
    out_b = rows * H * (4 + op * (1 if w.gemm_bf16 else 2))
    compulsory = uniq * H * 4 + nnz * 8 + out_b
    logical = nnz * H * 4 + nnz * 8 + out_b
    return {"rows": rows, "nnz": nnz, "unique_features": uniq, "avg_us": round(avg_s * 1e6, 2),
            "launches": n, "logical_bytes": logical, "logical_GB/s": round(logical / avg_s / 1e9, 1),
            "logical_hbm_frac": round(logical / avg_s / 1e9 / HBM_PEAK_GBS, 4),
            "compulsory_bytes": compulsory, "compulsory_GB/s": round(compulsory / avg_s / 1e9, 1),
            "how": "asgd_predict_topk(k=1) over the rows; logical = every entry's W1 row read once"}


def measure_merge(w, n_rep, reps_iters, stream):
    """Normalized merge of n_rep replicas of the workload's model (with momentum and
    broadcast, as in the elastic configuration), timed with the library's events."""
    import paper_2110_07029_amd as asgd
    mk = lambda s: asgd.asgd_model_init(w.n_features, w.n_labels, 8, 64, 64, gemm_bf16=w.gemm_bf16,
                                        seed=s, stream=stream)
    g, gp = mk(1), mk(2)
    reps = [mk(10 + i) for i in range(n_rep)]
    try:
        alpha = [1.0 / n_rep] * n_rep
        for _ in range(3):
            asgd.asgd_merge(g, gp, reps, alpha, 0.9, True)
        asgd.asgd_model_set_timing(g, True)
        asgd.asgd_model_get_timing(g, asgd.KERNELS.index("merge"))
        for _ in range(reps_iters):
            asgd.asgd_merge(g, gp, reps, alpha, 0.9, True)
        tot, n = asgd.asgd_model_get_timing(g, asgd.KERNELS.index("merge"))
        P = asgd.asgd_model_num_params(g)
    finally:
        for m in [g, gp] + reps:
            asgd.asgd_model_free(m)
    avg = tot / n
    # reads the n replicas, w and w_prev; writes w' and n broadcast copies
    byts = (n_rep + 2) * P * 4.0 + (n_rep + 1) * P * 4.0
    gbs = byts / (avg * 1e-3) / 1e9
    return {"avg_us": round(avg * 1e3, 2), "launches": n, "alg_bytes": byts, "alg_flops": 0.0,
            "GB/s": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "replicas": n_rep}


def run_elastic(args):
    """Configuration 5: 4 replicas of the wide-label model on 4 HIP streams, timed dynamic
    dispatch, merge every ~8 steps per replica (mega-batch 8 x 4 x b_max samples),
    weights from samples processed, momentum 0.9, Alg. 1 with b in [64, 1024]."""
    import torch
    import paper_2110_07029_amd as asgd
    from paper_2110_07029_amd import synth
    cfg5 = synth.ELASTIC
    w = synth.WORKLOADS[cfg5["base"]]
    n, b_min, b_max = cfg5["n_replicas"], cfg5["b_min"], cfg5["b_max"]
    mega = cfg5["steps_per_round"] * n * b_max
    K, W = args.steps, args.warmup
    n_samples = min(w.n_samples, max(mega * (K + W), 4 * b_max))
    log(f"elastic: {n} replicas of {w.name}, b in [{b_min}, {b_max}], mega-batch {mega}; {n_samples} samples")
    ds = synth.generate(w, n_samples=n_samples)
    ipx = np.asarray(ds.x.indptr, np.int64)
    ipy = np.asarray(ds.y.indptr, np.int64)
    max_nnz = int(np.max(ipx[b_max:] - ipx[:-b_max]))
    max_lnnz = int(np.max(ipy[b_max:] - ipy[:-b_max]))
    dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
    xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
    mcfg = asgd.asgd_config(n_features=w.n_features, n_labels=w.n_labels, hidden=H, max_batch=b_max,
                            max_nnz=max_nnz, max_label_nnz=max_lnnz, gemm_bf16=1 if w.gemm_bf16 else 0)
    ec = asgd.asgd_elastic_config()
    ec.n_replicas, ec.b_min, ec.b_max, ec.beta = n, b_min, b_max, b_min / 2.0
    ec.lr, ec.gamma, ec.weight_mode, ec.perturb = w.lr, 0.9, asgd.ASGD_WEIGHTS_SAMPLES, 0
    ec.pert_thr, ec.delta, ec.megabatch, ec.clock = 0.1, 0.1, mega, asgd.ASGD_CLOCK_TIMED
    streams = [torch.cuda.Stream() for _ in range(n)]
    gstream = torch.cuda.current_stream()
    e = asgd.asgd_elastic_create(ec, mcfg, cfg5["index"] + 2000, streams, gstream)
    xi, yi = ipx.astype(np.int32), ipy.astype(np.int32)
    try:
        n_settle = settle(lambda i: asgd.asgd_elastic_round(e, xa, ya, xi, yi), args.settle_ms)
        for _ in range(W):
            asgd.asgd_elastic_round(e, xa, ya, xi, yi)
        torch.cuda.synchronize()
        log(f"settle ({n_settle} rounds) and warmup ({W} rounds) done")
        t0 = time.perf_counter()
        samples, bs = 0, []
        for r in range(K):
            lg = asgd.asgd_elastic_round(e, xa, ya, xi, yi)
            samples += sum(lg["samples"][:n])
            bs.append(lg["b_next"][:n])
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
    finally:
        asgd.asgd_elastic_free(e)
    log(f"timed {K} rounds: {el * 1e3:.1f} ms, final batch sizes {bs[-1] if bs else None}")
    merge = measure_merge(w, n, 10, gstream)
    cpu = None
    if args.cpu_seconds > 0:
        log(f"oracle CPU baseline, ~{args.cpu_seconds:.0f} s budget")
        cpu = cpu_baseline_elastic(w, ds, b_max, n, mega, args.cpu_seconds)
    return {
        "metric": METRIC, "value": round(samples / el, 1), "unit": "samples/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": round(el * 1e3 / K, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if w.gemm_bf16 else "fp32", "data": "synthetic",
        "config": {"workload": "elastic-4x-wide-label", "n_features": w.n_features, "n_labels": w.n_labels,
                   "hidden": H, "replicas": n, "b_min": b_min, "b_max": b_max, "megabatch": mega,
                   "global_batch": mega, "clock": "timed", "weights": "samples", "momentum": 0.9,
                   "parallelism": "4 replicas on 4 HIP streams", "step": "one round (dispatch + merge)",
                   "hw_queues": os.environ.get("GPU_MAX_HW_QUEUES")},
        "roofline": {"kernel": "merge", "bound": "hbm", "achieved": merge["GB/s"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": merge["hbm_frac"], "traffic": measured_traffic("elastic", n, "merge")},
        "cpu_baseline": cpu,
        "settle": {"ms": args.settle_ms, "rounds": n_settle},
        "kernels": {"merge": merge},
        "batch_sizes_per_round": bs,
    }


def _oracle_steps(w, ds, B, budget_s, max_steps):
    from oracle import model as om
    p = om.init_params(w.n_features, w.n_labels, H, w.init_seed)
    ops = "bf16" if w.gemm_bf16 else "fp32"
    n_steps, samples, r0 = 0, 0, 0
    t0 = time.perf_counter()
    while True:
        r1 = min(r0 + B, ds.x.n_rows)
        p, *_ = om.train_step(p, ds.x.rows(r0, r1), ds.y.rows(r0, r1), w.lr, ops)
        n_steps += 1
        samples += r1 - r0
        r0 = r1 % ds.x.n_rows
        el = time.perf_counter() - t0
        log(f"oracle step {n_steps}: {el:.1f} s")
        if el >= budget_s or n_steps >= max_steps:
            return n_steps, samples, el


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:  # pragma: no cover - not Linux
        pass
    return None


def ramp(m, xs, ys, lr, n, stream, idle_s=2.0):
    """Step times from an idle GPU: after `idle_s` seconds without work, n steps
    each bracketed by HIP events on the model's stream."""
    import torch
    import paper_2110_07029_amd as asgd
    torch.cuda.synchronize()
    time.sleep(idle_s)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record(stream)
    for i in range(n):
        asgd.asgd_train_step(m, xs[i % len(xs)], ys[i % len(xs)], lr)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    t = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(n)])
    edges = [e for e in (0, 5, 25, 50, 100, 200, 400, 800, 1600) if e < n] + [n]
    return {"idle_s": idle_s, "steps": n, "first_10_ms": [round(v, 4) for v in t[:10]],
            "windows_ms": {f"{a}-{b}": round(float(t[a:b].mean()), 4) for a, b in zip(edges, edges[1:])}}


def cpu_baseline_elastic(w, ds, b, n_rep, mega, budget_s):
    """The oracle on a bounded sample of an elastic round: steps of one replica at
    batch b (the replicas' starting size) within most of the budget, and one
    oracle merge of n_rep replicas with momentum; a round of `mega` samples is
    then mega/b such steps plus one merge."""
    from oracle import elastic as oe
    from oracle import model as om
    n_steps, samples, el = _oracle_steps(w, ds, b, 0.75 * budget_s, 4)
    g = om.flat_params(om.init_params(w.n_features, w.n_labels, H, w.init_seed))
    reps = [g.copy() for _ in range(n_rep)]
    t0 = time.perf_counter()
    oe.merge(g, g, reps, [1.0 / n_rep] * n_rep, 0.9)
    t_merge = time.perf_counter() - t0
    t_step = el / n_steps
    t_round = (mega / b) * t_step + t_merge
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        cores = os.cpu_count() or 1
    return {"value": mega / t_round, "unit": "samples/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n_steps} oracle steps x {b} rows of {w.name} ({t_step:.1f} s each) and one oracle "
                      f"merge of {n_rep} replicas ({t_merge:.1f} s), scaled to a round of {mega} samples",
            "cpu_model": _cpu_model(), "host_cpus": os.cpu_count()}


def cpu_baseline(w, ds, B, budget_s):
    """The oracle as it stands, timed on this host on a bounded sample of the
    workload: with every thread its BLAS starts, then with one thread."""
    n_steps, samples, el = _oracle_steps(w, ds, B, budget_s, 64)
    try:  # threads of the BLAS the oracle's products ran on (loaded by now)
        from threadpoolctl import threadpool_info, threadpool_limits
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threadpool_limits = None
        cores = os.cpu_count() or 1
    out = {"value": samples / el, "unit": "samples/s", "cores": int(cores), "kind": "oracle",
           "sample": f"{n_steps} oracle steps x {B} rows of {w.name} ({samples} samples, {el:.1f} s)",
           "cpu_model": _cpu_model(), "host_cpus": os.cpu_count()}
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            n1, s1, e1 = _oracle_steps(w, ds, B, budget_s / 2, 64)
        out["one_thread"] = {"value": s1 / e1, "cores": 1,
                             "sample": f"{n1} oracle steps x {B} rows ({s1} samples, {e1:.1f} s)"}
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the replicas of the elastic "
              f"configuration share a single MI355X, and the multi-GPU merge is a design, not a measured path.",
              file=sys.stderr)
        sys.exit(2)
    if args.workload == "elastic" and int(os.environ.get("GPU_MAX_HW_QUEUES", "0") or 0) < 16:
        # The elastic round runs every replica on a model stream and an internal
        # stream of its own.  With the runtime's default of 4 hardware queues,
        # several of those streams share a queue, and the order in which a shared
        # queue serves them, not the replicas' speed, decides which replica is
        # free first: Alg. 1 then drives two of the four batch sizes to b_min.
        # One hardware queue per stream (read when the runtime starts) avoids it.
        os.environ["GPU_MAX_HW_QUEUES"] = "16"
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        # a copy kernel of known size: FETCH_SIZE / WRITE_SIZE per dispatch against 256 MiB
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 10 copies of 256 MiB done")
        return
    import paper_2110_07029_amd as asgd
    from paper_2110_07029_amd import synth

    asgd.load()
    if args.workload == "elastic":
        print(json.dumps(run_elastic(args)), flush=True)
        return
    w = synth.WORKLOADS[args.workload]
    B = args.batch or w.batch
    K, W = args.steps, args.warmup
    if args.ramp:
        K, W = args.ramp, 0
    n_samples = min(w.n_samples, (K + W) * B)
    log(f"workload {w.name}: F={w.n_features} L={w.n_labels} B={B}; generating {n_samples} samples")
    ds = synth.generate(w, n_samples=n_samples)
    n_full = ds.x.n_rows // B
    bounds = [(i * B, (i + 1) * B) for i in range(n_full)]
    ipx, ipy = np.asarray(ds.x.indptr), np.asarray(ds.y.indptr)
    nnz = [int(ipx[b] - ipx[a]) for a, b in bounds]
    lnnz = [int(ipy[b] - ipy[a]) for a, b in bounds]
    dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
    xs = [dx.batch(a, b) for a, b in bounds]
    ys = [dy.batch(a, b) for a, b in bounds]
    stream = torch.cuda.current_stream()
    flags = asgd.ASGD_UNFUSED_OUTPUT if args.unfused else 0
    m = asgd.asgd_model_init(w.n_features, w.n_labels, B, max(nnz), max(lnnz), gemm_bf16=w.gemm_bf16,
                             seed=w.init_seed, stream=stream, flags=flags,
                             extra_hidden_layers=1 if args.extra_hidden else 0)
    try:
        lr = w.lr
        if args.ramp:
            print(json.dumps(ramp(m, xs, ys, lr, args.ramp, stream)), flush=True)
            return
        n_settle = settle(lambda i: asgd.asgd_train_step(m, xs[i % n_full], ys[i % n_full], lr), args.settle_ms)
        for i in range(W):
            asgd.asgd_train_step(m, xs[i % n_full], ys[i % n_full], lr)
        torch.cuda.synchronize()
        log(f"settle ({n_settle} steps, {args.settle_ms:.0f} ms) and warmup ({W} steps) done")
        # timed region: K steps with no per-kernel events on the stream
        t_start = torch.cuda.Event(enable_timing=True)
        t_end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_start.record(stream)
        used = []
        h0 = time.perf_counter()
        n_host = min(K, 16)
        for i in range(K):
            j = (W + i) % n_full
            used.append(j)
            asgd.asgd_train_step(m, xs[j], ys[j], lr)
            if i + 1 == n_host:
                # the host's own time to issue a step, taken over the first steps only (later
                # calls can wait for room in the device queue)
                host_ms = (time.perf_counter() - h0) * 1e3 / n_host
        t_end.record(stream)
        torch.cuda.synchronize()
        ms = t_start.elapsed_time(t_end)
        loss = asgd.asgd_model_last_loss(m)
        log(f"timed {K} steps: {ms:.2f} ms, last loss {loss:.4f}")
        # per-kernel durations: a second pass with the library's HIP events around
        # every launch (recorded on the stream each kernel runs on)
        KT = min(K, 100)
        asgd.asgd_model_set_timing(m, True)
        for k in range(len(asgd.KERNELS)):
            asgd.asgd_model_get_timing(m, k)
        for i in range(KT):
            j = (W + i) % n_full
            asgd.asgd_train_step(m, xs[j], ys[j], lr)
        torch.cuda.synchronize()
        kt = {}
        for k, name in enumerate(asgd.KERNELS):
            tot, n = asgd.asgd_model_get_timing(m, k)
            if n:
                kt[name] = (tot, n)
        asgd.asgd_model_set_timing(m, False)
    finally:
        asgd.asgd_model_free(m)

    samples = K * B
    value = samples / (ms / 1e3)
    mean_nnz = float(np.mean([nnz[j] for j in used]))
    mean_lnnz = float(np.mean([lnnz[j] for j in used]))
    uniq = float(np.mean([len(np.unique(ds.x.indices[ipx[bounds[j][0]]:ipx[bounds[j][1]]]))
                          for j in used[:32]]))
    # label splits of the forward (and of the unfused path's P W2): one persistent workgroup per CU
    # but 16, shared by the 256-row blocks
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    splits = min((w.n_labels + 31) // 32, -(-(n_cu - 16) // -(-B // 256)))
    model = kernel_model(w, B, mean_nnz, mean_lnnz, uniq, splits)
    dtype = "bf16" if w.gemm_bf16 else "fp32"
    kernels = {}
    for name, (tot, n) in kt.items():
        avg = tot / n
        km = model.get(name, dict(bytes=0.0, flops=0.0))
        gbs = km["bytes"] / (avg * 1e-3) / 1e9
        tfs = km["flops"] / (avg * 1e-3) / 1e12
        kernels[name] = {"avg_us": round(avg * 1e3, 2), "launches": n,
                         "alg_bytes": km["bytes"], "alg_flops": km["flops"],
                         "GB/s": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                         "TFLOP/s": round(tfs, 2), "mfma_frac": round(tfs / MFMA_PEAK_TFLOPS[dtype], 4),
                         "share_of_step": round(tot / KT / (ms / K), 4)}
        if name in OVERLAPPED:
            kernels[name]["overlapped"] = True
    # the sort and the W1 update run on the library's second stream, overlapped with
    # the output layer (their event spans include time spent waiting for CUs), and the
    # label grouping is a workgroup of the forward launch: none is a candidate
    dom = max((k for k in kt if k not in OVERLAPPED), key=lambda k: kt[k][0])
    if args.workload == "wide-label":
        # the merge of the elastic configuration: 4 replicas of this model
        kernels["merge"] = measure_merge(w, 4, 10, stream)
        kernels["gather_saturating"] = measure_gather_saturating(w, stream)
    d = kernels[dom]
    traffic = measured_traffic(w.name, B, dom)
    # the dominant kernel against the resource it uses the larger share of: HBM
    # (algorithmic bytes) or the matrix cores (algorithmic flops, at the dtype's peak)
    mfma_bound = d["mfma_frac"] > d["hbm_frac"]
    if mfma_bound:
        roofline = {"kernel": dom, "bound": "mfma", "achieved": d["TFLOP/s"], "peak": MFMA_PEAK_TFLOPS[dtype],
                    "unit": "TFLOP/s", "frac": d["mfma_frac"]}
    else:
        roofline = {"kernel": dom, "bound": "hbm", "achieved": d["GB/s"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": d["hbm_frac"]}
    roofline["traffic"] = None if traffic is None else round(traffic / 1e9, 4)
    if traffic is not None:
        roofline["traffic_unit"] = "GB per launch"
    meas = measured_peaks(w.n_labels * H, stream)
    roofline["measured_peaks"] = meas
    # (the measured matrix-core rate is a bf16 GEMM's: no figure for fp32 operands)
    roofline["frac_of_measured"] = (None if mfma_bound and dtype != "bf16" else
                                    round(d["TFLOP/s"] / meas["bf16_gemm_TFLOPs"] if mfma_bound
                                          else d["GB/s"] / meas["hbm_inplace_update_GBs"], 4))
    cpu = None
    if args.cpu_seconds > 0:
        log(f"oracle CPU baseline, ~{args.cpu_seconds:.0f} s budget")
        cpu = cpu_baseline(w, ds, B, args.cpu_seconds)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1, "steps": K,
        "warmup": W, "ms_per_step": round(ms / K, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": w.name, "n_features": w.n_features, "n_labels": w.n_labels,
                   "hidden": H, "batch": B, "global_batch": B, "mean_nnz_per_batch": round(mean_nnz, 1),
                   "mean_labels_per_batch": round(mean_lnnz, 1), "master_weights": "fp32",
                   "output_layer": "unfused (stored logits)" if args.unfused else "fused",
                   "hidden_layers": 2 if args.extra_hidden else 1,
                   "parallelism": "single replica"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "settle": {"ms": args.settle_ms, "steps": n_settle,
                   "why": "untimed load before the warm-up steps: the GPU's clocks ramp for tens of ms after idle"},
        # host time to issue one step's launches: when it reaches ms_per_step the GPU waits for the host
        "host_ms_per_step": round(host_ms, 4),
        "kernels": kernels,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
