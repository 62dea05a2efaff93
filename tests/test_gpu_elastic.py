"""GPU parity of the elastic round driver (replicas on HIP streams, dynamic
dispatch of a mega-batch, Alg. 2 merge, Alg. 1 scaling) against the oracle:
in virtual-clock mode the schedule and every host decision are bit-exact, and
replaying the logged schedule through the oracle reproduces the models."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import elastic as oe
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import assert_update_close, flush, read_params

pytestmark = pytest.mark.gpu

W = synth.TINY
N_REP, B_MIN, B_MAX, BETA = 3, 16, 64, 8.0
COST = (1.0, 0.01, 0.001)
SLOW = (1.0, 1.5, 2.0)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


def _make(ds, clock, perturb, mode, megabatch, dispatch=asgd.ASGD_DISPATCH_DYNAMIC, beta=BETA, gamma=0.9):
    import torch
    ip = np.asarray(ds.x.indptr, np.int64)
    lp = np.asarray(ds.y.indptr, np.int64)
    max_nnz = int(max(ip[i + B_MAX] - ip[i] for i in range(len(ip) - B_MAX)))
    max_lnnz = int(max(lp[i + B_MAX] - lp[i] for i in range(len(lp) - B_MAX)))
    mcfg = asgd.asgd_config(W.n_features, W.n_labels, 128, B_MAX, max_nnz, max_lnnz, 0, 0)
    cfg = asgd.asgd_elastic_config()
    cfg.n_replicas, cfg.b_min, cfg.b_max, cfg.beta = N_REP, B_MIN, B_MAX, beta
    cfg.lr, cfg.gamma, cfg.weight_mode, cfg.perturb = 0.05, gamma, mode, perturb
    cfg.dispatch = dispatch
    cfg.pert_thr, cfg.delta, cfg.megabatch, cfg.clock = 0.1, 0.1, megabatch, clock
    cfg.c0, cfg.c1, cfg.c2 = COST
    for i, v in enumerate(SLOW):
        cfg.slow[i] = v
    streams = [torch.cuda.Stream() for _ in range(N_REP)]
    e = asgd.asgd_elastic_create(cfg, mcfg, W.init_seed, streams, torch.cuda.current_stream())
    return e, streams


# (weights, perturbation, dispatch, beta, gamma): Adaptive SGD in both weight modes, and the
# baselines: elastic model averaging (static schedule, uniform weights, fixed batches, no
# momentum) and gradient aggregation (the same with one batch per replica per round)
CASES = [(asgd.ASGD_WEIGHTS_SAMPLES, 0, asgd.ASGD_DISPATCH_DYNAMIC, BETA, 0.9, 8),
         (asgd.ASGD_WEIGHTS_ALG2, 1, asgd.ASGD_DISPATCH_DYNAMIC, BETA, 0.9, 8),
         (asgd.ASGD_WEIGHTS_UNIFORM, 0, asgd.ASGD_DISPATCH_STATIC, 0.0, 0.0, 8),
         (asgd.ASGD_WEIGHTS_UNIFORM, 0, asgd.ASGD_DISPATCH_STATIC, 0.0, 0.0, 1)]


@pytest.mark.parametrize("mode,perturb,dispatch,beta,gamma,batches", CASES)
def test_virtual_clock_rounds_match_oracle_replay(mode, perturb, dispatch, beta, gamma, batches):
    import torch
    flush(f"elastic virtual clock: mode={mode} perturb={perturb} dispatch={dispatch} batches/replica={batches}")
    ds = synth.generate(W, n_samples=2000)
    megabatch = batches * N_REP * B_MAX
    static = dispatch == asgd.ASGD_DISPATCH_STATIC
    e, _ = _make(ds, asgd.ASGD_CLOCK_VIRTUAL, perturb, mode, megabatch, dispatch, beta, gamma)
    try:
        dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
        xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
        g0 = om.init_params(W.n_features, W.n_labels, 128, W.init_seed)
        ref_g, ref_prev = om.flat_params(g0), om.flat_params(g0)
        b, lr, cursor = [B_MAX] * N_REP, [0.05] * N_REP, 0
        for rnd in range(3):
            log = asgd.asgd_elastic_round(e, xa, ya, ds.x.indptr, ds.y.indptr)
            torch.cuda.synchronize()
            sched, cursor2, _, u, samples = oe.dispatch_round(ds.x.indptr, cursor, b, megabatch,
                                                              [0.0] * N_REP, COST, SLOW, static=static)
            assert log["schedule"] == sched, rnd
            assert log["u"][:N_REP] == u and log["samples"][:N_REP] == samples
            assert log["cursor"] == cursor2
            assert log["b_used"][:N_REP] == b
            # replay the schedule through the oracle from the current global model
            reps = [om.unflat_params(ref_g, W.n_features, W.n_labels, 128) for _ in range(N_REP)]
            for w, r0, r1 in sched:
                reps[w], *_ = om.train_step(reps[w], ds.x.rows(r0, r1), ds.y.rows(r0, r1), lr[w], "fp32")
            flat = [om.flat_params(p) for p in reps]
            l2 = None
            if perturb:
                l2 = [float(np.sqrt(np.sum(f.astype(np.float64) ** 2)) / f.size) for f in flat]
                assert np.allclose(log["l2_per_param"][:N_REP], l2, rtol=1e-3)
                l2 = log["l2_per_param"][:N_REP]  # the gate's inputs are the library's norms
            alpha = oe.merge_weights(u, b, samples, mode, l2, 0.1, 0.1)
            assert np.array_equal(log["alpha"][:N_REP], alpha)
            ref_g_new, ref_prev = oe.merge(ref_g, ref_prev, flat, alpha, gamma)
            ref_g = ref_g_new
            b, lr = oe.scale_batches(u, b, lr, B_MIN, B_MAX, beta)
            assert log["b_next"][:N_REP] == b
            assert [float(np.float32(v)) for v in log["lr_next"][:N_REP]] == [float(np.float32(v)) for v in lr]
            cursor = cursor2
        # the global model and every replica (broadcast) agree with the replay
        got = om.flat_params(read_params(asgd.asgd_elastic_model(e, -1), W.n_features, W.n_labels))
        init = om.flat_params(g0)
        # free-running over ~30 steps and 3 merges: rounding drift is bounded by the
        # typical size of the update, so the elementwise floor is its RMS
        d_ref = ref_g.astype(np.float64) - init
        rms = float(np.sqrt(np.mean(d_ref ** 2)))
        assert_update_close("global", init, got, ref_g, 1e-3, mag=np.full(d_ref.shape, rms))
        for i in range(N_REP):
            rep = om.flat_params(read_params(asgd.asgd_elastic_model(e, i), W.n_features, W.n_labels))
            assert np.array_equal(rep.view(np.uint32), got.view(np.uint32))
        if static:      # the baselines keep equal batches and give every replica its share
            uu = log["u"][:N_REP]   # (a batch cut at the dataset's end adds one dispatch)
            assert b == [B_MAX] * N_REP and min(uu) >= batches and max(uu) - min(uu) <= 1
        else:           # heterogeneous clocks moved the batch sizes: fastest replica largest
            assert b[0] >= b[-1]
    finally:
        asgd.asgd_elastic_free(e)


def test_timed_rounds_invariants():
    import torch
    flush("elastic timed clock: invariants")
    ds = synth.generate(W, n_samples=2000)
    megabatch = 8 * N_REP * B_MAX
    e, _ = _make(ds, asgd.ASGD_CLOCK_TIMED, 0, asgd.ASGD_WEIGHTS_SAMPLES, megabatch)
    try:
        dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
        xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
        cursor = 0
        for rnd in range(3):
            log = asgd.asgd_elastic_round(e, xa, ya, ds.x.indptr, ds.y.indptr)
            sched = log["schedule"]
            assert sum(r1 - r0 for _, r0, r1 in sched) == megabatch
            for w, r0, r1 in sched:     # consecutive rows, wrapping at the dataset end
                assert r0 == cursor and 0 < r1 - r0 <= log["b_used"][w]
                cursor = r1 if r1 < ds.x.n_rows else 0
            assert abs(float(np.sum(log["alpha"][:N_REP].astype(np.float64))) - 1.0) < 1e-6
            for i in range(N_REP):
                assert B_MIN <= log["b_next"][i] <= B_MAX
                assert abs(log["lr_next"][i] / log["b_next"][i] - 0.05 / B_MAX) < 1e-6 * 0.05 / B_MAX + 1e-12
        torch.cuda.synchronize()
        g = read_params(asgd.asgd_elastic_model(e, -1), W.n_features, W.n_labels)
        assert all(np.all(np.isfinite(v)) for v in g.values())
    finally:
        asgd.asgd_elastic_free(e)
