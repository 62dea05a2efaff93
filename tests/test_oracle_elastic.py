"""Pins of the oracle's elastic part: Alg. 1 (batch-size scaling), Alg. 2
(normalized merge weights, perturbation, momentum merge) and the dynamic
mega-batch dispatch of Sec. 3.1."""
import os

import numpy as np
import pytest

from oracle import elastic as oe

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    out = {}
    for line in open(os.path.join(GOLDEN, name)):
        if line.startswith("#") or not line.strip():
            continue
        k, *v = line.split()
        out[k] = [float(t) for t in v]
    return out


# --------------------------------------------------------------------------- Alg. 1
def test_alg1_worked_case_of_section_3_1():
    g = _golden("alg1_fig4_case.txt")
    b, lr = oe.scale_batches([int(v) for v in g["u"]], [int(v) for v in g["b"]], g["lr"],
                             int(g["b_min"][0]), int(g["b_max"][0]), g["beta"][0])
    assert b == [int(v) for v in g["b_new"]]
    # the learning rates are float32: within one float32 ulp of the exact values
    for got, want in zip(lr, g["lr_new"]):
        assert abs(got - want) <= float(np.spacing(np.float32(want)))


def test_alg1_conserves_total_and_lr_per_sample_when_no_bound_bites():
    rng = np.random.default_rng(0)
    for _ in range(200):
        n = int(rng.integers(2, 9))
        u = list(rng.integers(1, 20, n))
        # choose beta so that every increment beta*(u_i - mean) is an integer
        beta = float(n * rng.integers(1, 4))
        b = list(rng.integers(400, 600, n))
        lr = [0.01 * bi / 512 for bi in b]
        nb, nlr = oe.scale_batches(u, b, lr, 1, 10_000, beta)
        assert sum(nb) == sum(b)
        for i in range(n):
            assert abs(nlr[i] / nb[i] - lr[i] / b[i]) <= 1e-6 * lr[i] / b[i]
            mu = sum(u) / n
            if u[i] > mu:
                assert nb[i] > b[i]
            elif u[i] < mu:
                assert nb[i] < b[i]
            else:
                assert nb[i] == b[i]


def test_alg1_skips_rather_than_clamps_at_the_bounds():
    # u = (10, 0): mean 5; +-beta*5 with beta=20 -> 200 and -100 ; bounds [50, 150]
    b, lr = oe.scale_batches([10, 0], [100, 100], [0.1, 0.1], 50, 150, 20.0)
    assert b == [100, 100] and lr == [float(np.float32(0.1))] * 2
    # only the side that stays inside moves
    b, lr = oe.scale_batches([10, 0], [100, 120], [0.1, 0.1], 50, 250, 20.0)
    assert b == [200, 120]


def test_alg1_equal_updates_is_identity():
    b, lr = oe.scale_batches([4, 4, 4], [64, 128, 1024], [0.1, 0.2, 0.3], 64, 1024, 32.0)
    assert b == [64, 128, 1024]


def test_alg1_rounds_half_away_and_scales_lr_by_rounded_ratio():
    # u = (2, 1): mean 1.5 ; beta = 3 -> 100 +- 1.5 = 101.5 and 98.5 -> 102 and 99
    b, lr = oe.scale_batches([2, 1], [100, 100], [0.5, 0.5], 1, 1000, 3.0)
    assert b == [102, 99]
    assert lr == [float(np.float32(0.5 * 102 / 100)), float(np.float32(0.5 * 99 / 100))]


# --------------------------------------------------------------------------- Alg. 2 weights
def test_alg2_equal_updates_weights_by_batch_size():
    a = oe.merge_weights([3, 3, 3], [100, 200, 100], [0, 0, 0], oe.MODE_ALG2)
    assert np.allclose(a, [0.25, 0.5, 0.25]) and a.dtype == np.float32


def test_alg2_unequal_updates_weights_by_update_count():
    a = oe.merge_weights([3, 2, 5], [100, 200, 100], [0, 0, 0], oe.MODE_ALG2)
    assert np.allclose(a, [0.3, 0.2, 0.5])


def test_samples_mode_and_its_agreement_with_alg2_for_constant_batches():
    u, b = [3, 2, 5], [64, 64, 64]
    s = [ui * bi for ui, bi in zip(u, b)]
    a = oe.merge_weights(u, b, s, oe.MODE_SAMPLES)
    assert abs(float(np.sum(a.astype(np.float64))) - 1) < 1e-7
    assert np.allclose(a, oe.merge_weights(u, b, s, oe.MODE_ALG2))


def test_perturbation_closed_form_and_gate():
    u, b = [5, 2, 3, 2], [100, 100, 100, 90]
    base = oe.merge_weights(u, b, [0] * 4, oe.MODE_ALG2).astype(np.float64)
    pert = oe.merge_weights(u, b, [0] * 4, oe.MODE_ALG2, l2_per_param=[0.01] * 4,
                            pert_thr=0.1, delta=0.1).astype(np.float64)
    # r = most updates (index 0); s = fewest updates, then smaller batch (index 3)
    assert np.isclose(pert[0], 1.1 * base[0]) and np.isclose(pert[3], 0.9 * base[3])
    assert np.allclose(pert[1:3], base[1:3])
    assert np.isclose(pert.sum(), 1 + 0.1 * (base[0] - base[3]))
    # gate: one replica not regularized -> no perturbation
    gated = oe.merge_weights(u, b, [0] * 4, oe.MODE_ALG2, l2_per_param=[0.01, 0.2, 0.01, 0.01])
    assert np.allclose(gated, base)


# --------------------------------------------------------------------------- merge
def test_merge_identical_replicas_dyadic_weights_is_identity_bit_exact():
    w = np.random.default_rng(1).normal(size=1000).astype(np.float32)
    new, prev = oe.merge(w, w, [w, w, w, w], [0.25] * 4, 0.9)
    assert np.array_equal(new.view(np.uint32), w.view(np.uint32))
    assert np.array_equal(prev, w)


def test_merge_linearity_and_momentum_term():
    rng = np.random.default_rng(2)
    g, gp = rng.normal(size=500).astype(np.float32), rng.normal(size=500).astype(np.float32)
    reps = [rng.normal(size=500).astype(np.float32) for _ in range(3)]
    a = [0.5, 0.25, 0.25]
    new0, _ = oe.merge(g, g, reps, a, 0.9)          # w = w_prev: no momentum
    new1, prev = oe.merge(g, gp, reps, a, 0.9)
    direct = sum(np.float64(ai) * r.astype(np.float64) for ai, r in zip(a, reps))
    assert np.allclose(new0, direct, rtol=1e-7, atol=1e-7)
    mom = new1.astype(np.float64) - new0.astype(np.float64)
    assert np.allclose(mom, np.float64(np.float32(0.9)) * (g.astype(np.float64) - gp), rtol=1e-6, atol=1e-6)
    assert np.array_equal(prev, g)


# --------------------------------------------------------------------------- dispatch
def test_dispatch_reproduces_three_vs_two_updates():
    # Sec. 3.1 / Fig. "adaptive-elastic-sgd": a mega-batch of 5 equal batches on two
    # GPUs where GPU 2 is 1.5x slower: GPU 1 makes 3 updates, GPU 2 makes 2.
    indptr = np.arange(0, 1001)
    sched, cur, clock, u, s = oe.dispatch_round(indptr, 0, [100, 100], 500, [0.0, 0.0],
                                                cost=(0.0, 1.0, 0.0), slow=[1.0, 1.5])
    assert u == [3, 2] and s == [300, 200]
    assert [w for w, *_ in sched] == [0, 1, 0, 1, 0]
    assert cur == 500
    # Alg. 1 then gives the faster GPU the larger batch
    b, _ = oe.scale_batches(u, [100, 100], [0.1, 0.1], 10, 1000, 10.0)
    assert b[0] > 100 > b[1]


def test_dispatch_budget_wrap_and_cut():
    indptr = np.arange(0, 11)      # 10 rows
    sched, cur, clock, u, s = oe.dispatch_round(indptr, 7, [4, 4], 9, [0.0, 0.0], cost=(1.0, 0, 0))
    # rows 7..10 cut at the end (3 rows), wrap, 4 rows, then the last batch is cut to 2
    assert [(r0, r1) for _, r0, r1 in sched] == [(7, 10), (0, 4), (4, 6)]
    assert sum(s) == 9 and cur == 6 and sum(u) == 3


# --------------------------------------------------------------------------- baselines
def test_uniform_weights_are_one_over_n_whatever_the_counts():
    for n in (1, 3, 4, 7):
        u = list(range(1, n + 1))
        a = oe.merge_weights(u, [64] * n, [10 * v for v in u], oe.MODE_UNIFORM)
        assert np.array_equal(a, np.full(n, np.float32(1.0 / n)))


def test_static_dispatch_is_round_robin_whatever_the_speeds():
    # the baselines' fixed schedule: a 3x slower worker still gets every n-th batch,
    # where dynamic dispatch would give most batches to the fast one
    indptr = np.arange(0, 1001)
    kw = dict(cost=(0.0, 1.0, 0.0), slow=[1.0, 3.0])
    sched, cur, clock, u, s = oe.dispatch_round(indptr, 0, [100, 100], 600, [0.0, 0.0], static=True, **kw)
    assert [w for w, *_ in sched] == [0, 1, 0, 1, 0, 1] and u == [3, 3] and s == [300, 300]
    assert clock == [300.0, 900.0]          # the round waits for the slower worker
    _, _, _, ud, _ = oe.dispatch_round(indptr, 0, [100, 100], 600, [0.0, 0.0], **kw)
    assert ud == [4, 2]                  # dynamic: the fast worker takes more


def test_gradient_aggregation_mode_is_one_step_on_the_whole_mega_batch():
    # Sec. 2.2 (merging after every batch turns model averaging into gradient
    # aggregation) through the driver's pieces: static dispatch of a budget of one
    # batch per worker, uniform weights, no momentum.
    from oracle import model as om
    from paper_2110_07029_amd import synth
    w = synth.TINY
    ds = synth.generate(w, n_samples=300)
    p = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
    n, b, lr = 3, 40, 0.05
    sched, cur, _, u, s = oe.dispatch_round(ds.x.indptr, 0, [b] * n, n * b, [0.0] * n, static=True)
    assert [x[0] for x in sched] == [0, 1, 2] and cur == n * b
    reps = [om.flat_params(om.train_step(p, ds.x.rows(r0, r1), ds.y.rows(r0, r1), lr)[0])
            for _, r0, r1 in sched]
    alpha = oe.merge_weights(u, [b] * n, s, oe.MODE_UNIFORM)
    g0 = om.flat_params(p)
    merged, _ = oe.merge(g0, g0, reps, alpha, 0.0)
    big = om.flat_params(om.train_step(p, ds.x.rows(0, n * b), ds.y.rows(0, n * b), lr)[0])
    d_m, d_b = merged.astype(np.float64) - g0, big.astype(np.float64) - g0
    # equal up to the float32 storage of the replicas, of 1/3 and of the merge
    assert np.linalg.norm(d_m - d_b) <= 1e-6 * np.linalg.norm(d_b) + 4 * np.linalg.norm(np.spacing(np.abs(g0)))
