"""Oracle for Adaptive SGD's elastic part (test infrastructure only).

* ``scale_batches``  - batch-size scaling, Alg. 1 (Sec. 3.2): linear in the
                       deviation of a worker's update count from the mean,
                       applied only when the result stays inside
                       [b_min, b_max]; learning rate scaled linearly with b.
* ``merge_weights``  - normalized merge weights, Alg. 2 (Sec. 3.3): by batch
                       size when every worker made the same number of
                       updates, by update count otherwise; the alternative
                       normalization by samples processed that Sec. 3.3
                       mentions; and the optional perturbation of the weights
                       of the most and least updated replicas, gated by the
                       L2 norm per parameter of every replica.
* ``merge``          - the momentum merge closing Alg. 2:
                       w' = sum_i alpha_i w_i + gamma (w - w_prev); w_prev <- w; w <- w'.
* ``dispatch_round`` - dynamic scheduling of one mega-batch (Sec. 3.1): batches
                       go one by one to whichever worker is free first, until
                       the fixed sample budget is spent; worker speed comes
                       from a deterministic virtual clock.  With ``static``
                       the k-th batch goes to worker k mod n instead: the
                       fixed schedule of the paper's baselines (elastic model
                       averaging; gradient aggregation when the budget is one
                       batch per worker, Sec. 2.2), whose uniform weights are
                       ``MODE_UNIFORM``.

Readings where the paper is silent: the scaled batch size is rounded to the
nearest integer (halves away from zero) after the bound test on the exact
value, and the learning rate is scaled by the rounded ratio; ties in the
argmax / argmin of the update counts are broken by batch size, then by index
(lowest index for the max, highest for the min); a batch never wraps past the
end of the dataset and the last batch of a mega-batch is cut to the remaining
budget.
"""
from __future__ import annotations

import math
from typing import List, Sequence

import numpy as np

MODE_ALG2 = 0      # Alg. 2: by batch size if all update counts are equal, else by update count
MODE_SAMPLES = 1   # by samples processed (the alternative named in Sec. 3.3)
MODE_UNIFORM = 2   # 1/n: the plain model average of the baselines (Sec. 2.2)


def _round_half_away(v: float) -> int:
    return int(math.floor(v + 0.5)) if v >= 0 else -int(math.floor(-v + 0.5))


def scale_batches(u: Sequence[int], b: Sequence[int], lr: Sequence[float],
                  b_min: int, b_max: int, beta: float):
    """Alg. 1.  Returns new (b, lr) lists; lr values are rounded to float32."""
    n = len(u)
    mu = float(sum(u)) / n
    nb, nlr = list(int(v) for v in b), [float(np.float32(v)) for v in lr]
    for i in range(n):
        up = float(b[i]) + beta * (float(u[i]) - mu)      # faster worker: grow
        down = float(b[i]) - beta * (mu - float(u[i]))    # slower worker: shrink
        if u[i] > mu and up <= b_max:
            new_b = _round_half_away(up)
        elif u[i] < mu and down >= b_min:
            new_b = _round_half_away(down)
        else:
            continue
        nlr[i] = float(np.float32(float(np.float32(lr[i])) * new_b / b[i]))
        nb[i] = new_b
    return nb, nlr


def merge_weights(u: Sequence[int], b: Sequence[int], samples: Sequence[int], mode: int,
                  l2_per_param: Sequence[float] = None, pert_thr: float = 0.1,
                  delta: float = 0.1) -> np.ndarray:
    """Alg. 2 weight computation.  ``l2_per_param[i]`` = ||w_i||_2 / |w| (None: no perturbation)."""
    n = len(u)
    if mode == MODE_ALG2:
        if all(v == u[0] for v in u):
            tot = float(sum(b))
            alpha = [float(v) / tot for v in b]
        else:
            tot = float(sum(u))
            alpha = [float(v) / tot for v in u]
    elif mode == MODE_SAMPLES:
        tot = float(sum(samples))
        alpha = [float(v) / tot for v in samples]
    elif mode == MODE_UNIFORM:
        alpha = [1.0 / n] * n
    else:
        raise ValueError(mode)
    if l2_per_param is not None and n > 1 and all(v < pert_thr for v in l2_per_param):
        key = [(u[i], b[i]) for i in range(n)]
        r = max(range(n), key=lambda i: (key[i], -i))     # most updated; lowest index on ties
        s = min(range(n), key=lambda i: (key[i], -i))     # least updated; highest index on ties
        alpha[r] *= (1.0 + delta)
        alpha[s] *= (1.0 - delta)
    return np.array(alpha, np.float64).astype(np.float32)


def merge(global_w: np.ndarray, prev_w: np.ndarray, replicas: List[np.ndarray],
          alpha: Sequence[float], gamma: float):
    """Momentum merge in float64, rounded once.  Returns (new global, new previous global)."""
    acc = np.zeros(global_w.shape, np.float64)
    for a, w in zip(alpha, replicas):
        acc += np.float64(np.float32(a)) * w.astype(np.float64)
    acc += np.float64(np.float32(gamma)) * (global_w.astype(np.float64) - prev_w.astype(np.float64))
    return acc.astype(np.float32), global_w.copy()


def step_cost(c0: float, c1: float, c2: float, slow: float, rows: int, nnz: int) -> float:
    """Virtual-clock duration of one step: slow * (c0 + c1 * rows + c2 * nnz)."""
    return slow * (c0 + c1 * rows + c2 * nnz)


def dispatch_round(indptr: np.ndarray, cursor: int, b: Sequence[int], budget: int,
                   clock: Sequence[float], cost=(0.0, 0.0, 0.0), slow=None, static: bool = False):
    """Dynamic dispatch of one mega-batch of ``budget`` samples over n workers.

    Each batch goes to the worker whose clock is smallest (lowest index on ties);
    its clock advances by ``step_cost``.  A batch is ``b[w]`` consecutive rows
    from ``cursor``, cut at the dataset end (the cursor then wraps to 0) and at
    the remaining budget.  Returns (schedule, new cursor, new clocks, u, samples),
    where schedule entries are (worker, r0, r1).
    """
    n = len(b)
    n_rows = len(indptr) - 1
    slow = [1.0] * n if slow is None else list(slow)
    clock = [float(c) for c in clock]
    sched, u, samples = [], [0] * n, [0] * n
    left = int(budget)
    while left > 0:
        w = len(sched) % n if static else min(range(n), key=lambda i: (clock[i], i))
        take = min(int(b[w]), left, n_rows - cursor)
        r0, r1 = cursor, cursor + take
        sched.append((w, r0, r1))
        nnz = int(indptr[r1] - indptr[r0])
        clock[w] += step_cost(cost[0], cost[1], cost[2], slow[w], take, nnz)
        u[w] += 1
        samples[w] += take
        left -= take
        cursor = r1 if r1 < n_rows else 0
    return sched, cursor, clock, u, samples
