"""Time-to-accuracy runs of Adaptive SGD and the paper's baselines (Sec. 5.2
setting, on synthetic data with planted label structure).

Each round of ``asgd_elastic_round`` trains the replicas on one mega-batch and
merges them into the global model; after every round the global model's top-1
accuracy on held-out rows is measured with ``asgd_predict_topk`` (the label
with the highest score counts as correct when it is one of the row's labels),
as the paper measures after every mega-batch.  Evaluation time is excluded from
the clocks, as in the paper.

Modes (Sec. 2.2, Sec. 3, Sec. 5.1):

* ``adaptive``: dynamic dispatch, Alg. 1 batch scaling, Alg. 2 weights with the
  perturbation, momentum merge;
* ``elastic``: elastic model averaging: a static schedule (batch k to replica
  k mod n), equal fixed batches, uniform weights, no momentum;
* ``ga``: gradient aggregation: the elastic schedule with one batch per
  replica per round.

The replicas share one GPU, so their speeds differ only through the virtual
clock: replica i's step costs ``slow[i] * (c0 + c1 * rows + c2 * nnz)``
virtual seconds, and a round lasts until its last replica finishes.  Both the
virtual time (heterogeneous GPUs, modelled) and the measured GPU time of the
rounds are reported.

    python -m paper_2110_07029_amd.tta --mode all --budget 0.5
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import _binding as B
from . import synth

MODES = ("adaptive", "elastic", "ga")


def elastic_config(mode: str, n: int, b_min: int, b_max: int, lr: float, megabatch: int,
                   slow, cost, gamma: float = 0.5) -> B.asgd_elastic_config:
    c = B.asgd_elastic_config()
    c.n_replicas, c.b_min, c.b_max, c.lr = n, b_min, b_max, lr
    c.clock = B.ASGD_CLOCK_VIRTUAL
    c.c0, c.c1, c.c2 = cost
    for i, v in enumerate(slow):
        c.slow[i] = v
    if mode == "adaptive":
        c.dispatch, c.weight_mode, c.perturb = B.ASGD_DISPATCH_DYNAMIC, B.ASGD_WEIGHTS_ALG2, 1
        c.beta, c.gamma, c.pert_thr, c.delta = b_min / 2.0, gamma, 0.1, 0.1
        c.megabatch = megabatch
    elif mode in ("elastic", "ga"):
        c.dispatch, c.weight_mode, c.perturb = B.ASGD_DISPATCH_STATIC, B.ASGD_WEIGHTS_UNIFORM, 0
        c.beta, c.gamma = 0.0, 0.0
        c.megabatch = megabatch if mode == "elastic" else n * b_max
    else:
        raise ValueError(mode)
    return c


def round_virtual_time(log: dict, indptr: np.ndarray, slow, cost) -> float:
    """Virtual duration of a round: the largest per-replica sum of step costs."""
    t = [0.0] * 16
    for w, r0, r1 in log["schedule"]:
        nnz = int(indptr[r1] - indptr[r0])
        t[w] += slow[w] * (cost[0] + cost[1] * (r1 - r0) + cost[2] * nnz)
    return max(t)


def top1_accuracy(model: int, dx, test_y: synth.CSR, max_batch: int) -> float:
    import torch
    n = dx.n_rows
    ids = torch.empty((max_batch, 1), dtype=torch.int32, device="cuda")
    hit = 0
    for r0 in range(0, n, max_batch):
        r1 = min(n, r0 + max_batch)
        B.asgd_predict_topk(model, dx.batch(r0, r1), 1, ids[: r1 - r0])
        pred = ids[: r1 - r0, 0].cpu().numpy()
        for i, p in enumerate(pred):
            lab = test_y.indices[test_y.indptr[r0 + i]:test_y.indptr[r0 + i + 1]]
            hit += int(p in lab)
    return hit / n


def run(mode: str, planted: synth.Planted = synth.PLANTED_SMALL, budget_s: float = 0.5,
        n_train: int = 60_000, n_test: int = 4_000, n_replicas: int = 4, b_max: int = 128, lr: float = 1.0,
        gamma: float = 0.5, batches_per_round: int = 16, slow=(1.0, 1.3, 1.6, 2.0), cost=(1e-4, 2e-6, 2e-8),
        seed: int = 1, evals: int = 40, max_rounds: int = 100_000, out=None):
    """Train until the virtual clock reaches ``budget_s`` (every mode gets the same
    time, as in the paper); the accuracy is measured after the first round that
    crosses each of ``evals`` evenly spaced times.  Returns one record per
    measurement."""
    import torch
    from .device_data import DeviceCSR
    train = synth.generate_planted(planted, n_train)
    test = synth.generate_planted(planted, n_test, seed_offset=1)
    dx, dy, tx = DeviceCSR(train.x), DeviceCSR(train.y), DeviceCSR(test.x)
    ip, lp = np.asarray(train.x.indptr, np.int64), np.asarray(train.y.indptr, np.int64)
    win = lambda a, b: int(np.max(a[b:] - a[:-b])) if len(a) > b else int(a[-1] - a[0])
    max_nnz = max(win(ip, b_max), win(np.asarray(test.x.indptr, np.int64), b_max), 1)
    mcfg = B.asgd_config(n_features=planted.n_features, n_labels=planted.n_labels, hidden=synth.HIDDEN,
                         max_batch=b_max, max_nnz=max_nnz, max_label_nnz=max(win(lp, b_max), 1), gemm_bf16=1)
    slow = list(slow)[:n_replicas]
    cfg = elastic_config(mode, n_replicas, max(1, b_max // 8), b_max, lr,
                         batches_per_round * n_replicas * b_max, slow, cost, gamma)
    streams = [torch.cuda.Stream() for _ in range(n_replicas)]
    e = B.asgd_elastic_create(cfg, mcfg, seed, streams, torch.cuda.current_stream())
    recs = []
    try:
        xa, ya = dx.batch(0, train.x.n_rows), dy.batch(0, train.y.n_rows)
        g = B.asgd_elastic_model(e, -1)
        acc0 = top1_accuracy(g, tx, test.y, b_max)
        vt, gt, samples, next_eval = 0.0, 0.0, 0, budget_s / evals
        recs.append(dict(mode=mode, round=0, virtual_s=0.0, gpu_s=0.0, samples=0, top1=acc0))
        for r in range(1, max_rounds + 1):
            if vt >= budget_s:
                break
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            log = B.asgd_elastic_round(e, xa, ya, train.x.indptr, train.y.indptr)
            torch.cuda.synchronize()
            gt += time.perf_counter() - t0
            vt += round_virtual_time(log, ip, slow, cost)
            samples += int(sum(log["samples"][:n_replicas]))
            if vt < next_eval and vt < budget_s:
                continue
            while next_eval <= vt:
                next_eval += budget_s / evals
            rec = dict(mode=mode, round=r, virtual_s=round(vt, 6), gpu_s=round(gt, 6), samples=samples,
                       top1=top1_accuracy(g, tx, test.y, b_max),
                       b=[int(v) for v in log["b_next"][:n_replicas]],
                       u=[int(v) for v in log["u"][:n_replicas]])
            recs.append(rec)
            if out is not None:
                print(json.dumps(rec), file=out, flush=True)
    finally:
        B.asgd_elastic_free(e)
    return recs


def time_to_accuracy(recs, target: float, clock: str = "virtual_s"):
    """First time (on ``clock``) the top-1 accuracy reaches ``target``, or None."""
    for r in recs:
        if r["top1"] >= target:
            return r[clock]
    return None


def main(argv=None):
    ap = argparse.ArgumentParser(description="time-to-accuracy of Adaptive SGD and its baselines")
    ap.add_argument("--mode", choices=MODES + ("all",), default="all")
    ap.add_argument("--data", choices=("small", "wide"), default="small")
    ap.add_argument("--budget", type=float, default=0.5, help="virtual seconds per mode")
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--b-max", type=int, default=128)
    ap.add_argument("--lr", type=float, default=1.0)
    ap.add_argument("--gamma", type=float, default=0.5, help="merge momentum of the adaptive mode")
    ap.add_argument("--batches-per-round", type=int, default=16)
    ap.add_argument("--n-train", type=int, default=60_000)
    ap.add_argument("--target", type=float, default=0.55)
    a = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        raise SystemExit("time-to-accuracy runs need the GPU")
    B.load(build_if_missing=False)
    planted = synth.PLANTED_SMALL if a.data == "small" else synth.PLANTED_WIDE
    modes = MODES if a.mode == "all" else (a.mode,)
    summary = {}
    for m in modes:
        recs = run(m, planted, a.budget, a.n_train, n_replicas=a.replicas, b_max=a.b_max, lr=a.lr,
                   gamma=a.gamma, batches_per_round=a.batches_per_round, out=sys.stdout)
        summary[m] = dict(final_top1=recs[-1]["top1"], best_top1=max(r["top1"] for r in recs),
                          virtual_s_to_target=time_to_accuracy(recs, a.target),
                          gpu_s_to_target=time_to_accuracy(recs, a.target, "gpu_s"))
    print(json.dumps(dict(target=a.target, summary=summary)), flush=True)


if __name__ == "__main__":
    main()
