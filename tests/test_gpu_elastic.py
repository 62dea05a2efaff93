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

from gpu_util import RTOL_BF16, assert_update_close, flush, read_params

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


def _make(ds, clock, perturb, mode, megabatch, dispatch=asgd.ASGD_DISPATCH_DYNAMIC, beta=BETA, gamma=0.9,
          pert_thr=0.1, w=W, n_rep=N_REP, b_min=B_MIN, b_max=B_MAX, lr=0.05, slow=SLOW):
    import torch
    ip = np.asarray(ds.x.indptr, np.int64)
    lp = np.asarray(ds.y.indptr, np.int64)
    max_nnz = int(max(ip[i + b_max] - ip[i] for i in range(len(ip) - b_max)))
    max_lnnz = int(max(lp[i + b_max] - lp[i] for i in range(len(lp) - b_max)))
    mcfg = asgd.asgd_config(n_features=w.n_features, n_labels=w.n_labels, hidden=128, max_batch=b_max,
                            max_nnz=max_nnz, max_label_nnz=max_lnnz, gemm_bf16=1 if w.gemm_bf16 else 0)
    cfg = asgd.asgd_elastic_config()
    cfg.n_replicas, cfg.b_min, cfg.b_max, cfg.beta = n_rep, b_min, b_max, beta
    cfg.lr, cfg.gamma, cfg.weight_mode, cfg.perturb = lr, gamma, mode, perturb
    cfg.dispatch = dispatch
    cfg.pert_thr, cfg.delta, cfg.megabatch, cfg.clock = pert_thr, 0.1, megabatch, clock
    cfg.c0, cfg.c1, cfg.c2 = COST
    for i, v in enumerate(slow):
        cfg.slow[i] = v
    streams = [torch.cuda.Stream() for _ in range(n_rep)]
    e = asgd.asgd_elastic_create(cfg, mcfg, w.init_seed, streams, torch.cuda.current_stream())
    return e, streams


class Replay:
    """The oracle's side of a run: the global and previous global models, the
    batch sizes and learning rates, replayed round by round from the schedule
    the library logged.  Every host decision of the round (update counts,
    samples, Alg. 2 weights from the oracle's own replica norms, Alg. 1 batch
    sizes and learning rates) is compared bit-exactly with the library's log."""

    def __init__(self, w, n_rep, b_max, lr, mode, perturb, pert_thr, gamma, beta, b_min, ops="fp32"):
        self.w, self.n = w, n_rep
        self.g0 = om.flat_params(om.init_params(w.n_features, w.n_labels, 128, w.init_seed))
        self.g, self.prev = self.g0, self.g0
        self.b, self.lr = [b_max] * n_rep, [lr] * n_rep
        self.mode, self.perturb, self.pert_thr, self.gamma = mode, perturb, pert_thr, gamma
        self.beta, self.b_min, self.b_max, self.ops = beta, b_min, b_max, ops
        self.gates = []

    def round(self, ds, log):
        w, n = self.w, self.n
        sched = log["schedule"]
        assert log["b_used"][:n] == self.b
        assert [np.float32(v) for v in log["lr_used"][:n]] == [np.float32(v) for v in self.lr]
        u, samples = [0] * n, [0] * n
        for r, r0, r1 in sched:
            assert 0 < r1 - r0 <= self.b[r]
            u[r] += 1
            samples[r] += r1 - r0
        assert log["u"][:n] == u and log["samples"][:n] == samples
        reps = [om.unflat_params(self.g, w.n_features, w.n_labels, 128) for _ in range(n)]
        for r, r0, r1 in sched:
            reps[r], *_ = om.train_step(reps[r], ds.x.rows(r0, r1), ds.y.rows(r0, r1), self.lr[r], self.ops)
        flat = [om.flat_params(p) for p in reps]
        l2 = None
        if self.perturb:
            # the oracle's own norms decide its gate; the library's (over its own
            # replicas, which differ from these by rounding only) must agree closely
            # and sit on the same side of the threshold
            l2 = [float(np.sqrt(np.sum(f.astype(np.float64) ** 2)) / f.size) for f in flat]
            got = log["l2_per_param"][:n]
            assert np.allclose(got, l2, rtol=1e-6, atol=0), (got, l2)
            assert all((a < self.pert_thr) == (b < self.pert_thr) for a, b in zip(got, l2))
            self.gates.append(all(v < self.pert_thr for v in l2))
        alpha = oe.merge_weights(u, self.b, samples, self.mode, l2, self.pert_thr, 0.1)
        assert np.array_equal(log["alpha"][:n], alpha)
        self.g, self.prev = oe.merge(self.g, self.prev, flat, alpha, self.gamma)
        self.b, self.lr = oe.scale_batches(u, self.b, self.lr, self.b_min, self.b_max, self.beta)
        assert log["b_next"][:n] == self.b
        assert [np.float32(v) for v in log["lr_next"][:n]] == [np.float32(v) for v in self.lr]
        return u

    def check_models(self, e, rtol):
        """The global model and every replica (broadcast) agree with the replay.
        Free-running over several steps and merges, rounding differences are
        carried from step to step, so the elementwise floor is the RMS of the
        reference update."""
        w = self.w
        got = om.flat_params(read_params(asgd.asgd_elastic_model(e, -1), w.n_features, w.n_labels))
        d_ref = self.g.astype(np.float64) - self.g0
        rms = float(np.sqrt(np.mean(d_ref ** 2)))
        assert_update_close("global", self.g0, got, self.g, rtol, mag=np.full(d_ref.shape, rms))
        for i in range(self.n):
            rep = om.flat_params(read_params(asgd.asgd_elastic_model(e, i), w.n_features, w.n_labels))
            assert np.array_equal(rep.view(np.uint32), got.view(np.uint32))


# (weights, perturbation, dispatch, beta, gamma, batches per replica, pert_thr): Adaptive SGD in
# both weight modes, with the perturbation gate on (threshold above every replica's L2 norm per
# parameter, ~2e-5 here) and off (threshold below it); and the baselines: elastic model averaging
# (static schedule, uniform weights, fixed batches, no momentum) and gradient aggregation (the same
# with one batch per replica per round)
CASES = [(asgd.ASGD_WEIGHTS_SAMPLES, 0, asgd.ASGD_DISPATCH_DYNAMIC, BETA, 0.9, 8, 0.1),
         (asgd.ASGD_WEIGHTS_ALG2, 1, asgd.ASGD_DISPATCH_DYNAMIC, BETA, 0.9, 8, 0.1),
         (asgd.ASGD_WEIGHTS_ALG2, 1, asgd.ASGD_DISPATCH_DYNAMIC, BETA, 0.9, 8, 1e-6),
         (asgd.ASGD_WEIGHTS_UNIFORM, 0, asgd.ASGD_DISPATCH_STATIC, 0.0, 0.0, 8, 0.1),
         (asgd.ASGD_WEIGHTS_UNIFORM, 0, asgd.ASGD_DISPATCH_STATIC, 0.0, 0.0, 1, 0.1)]


@pytest.mark.parametrize("mode,perturb,dispatch,beta,gamma,batches,pert_thr", CASES)
def test_virtual_clock_rounds_match_oracle_replay(mode, perturb, dispatch, beta, gamma, batches, pert_thr):
    import torch
    flush(f"elastic virtual clock: mode={mode} perturb={perturb} pert_thr={pert_thr} dispatch={dispatch} "
          f"batches/replica={batches}")
    ds = synth.generate(W, n_samples=2000)
    megabatch = batches * N_REP * B_MAX
    static = dispatch == asgd.ASGD_DISPATCH_STATIC
    e, _ = _make(ds, asgd.ASGD_CLOCK_VIRTUAL, perturb, mode, megabatch, dispatch, beta, gamma, pert_thr)
    try:
        dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
        xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
        rp = Replay(W, N_REP, B_MAX, 0.05, mode, perturb, pert_thr, gamma, beta, B_MIN)
        cursor = 0
        for rnd in range(3):
            b_before = list(rp.b)
            log = asgd.asgd_elastic_round(e, xa, ya, ds.x.indptr, ds.y.indptr)
            torch.cuda.synchronize()
            # the dispatch itself: the oracle's virtual clock gives the same schedule
            sched, cursor2, _, u, samples = oe.dispatch_round(ds.x.indptr, cursor, b_before, megabatch,
                                                              [0.0] * N_REP, COST, SLOW, static=static)
            assert log["schedule"] == sched, rnd
            assert log["cursor"] == cursor2
            rp.round(ds, log)
            cursor = cursor2
        rp.check_models(e, 1e-3)
        if perturb:     # the gate is on for a threshold above the norms, off below them
            assert rp.gates == [pert_thr > 1e-3] * 3
        uu = log["u"][:N_REP]
        if static:      # the baselines keep equal batches and give every replica its share
            assert rp.b == [B_MAX] * N_REP and min(uu) >= batches and max(uu) - min(uu) <= 1
        else:           # heterogeneous clocks moved the batch sizes: fastest replica largest
            assert rp.b[0] >= rp.b[-1]
    finally:
        asgd.asgd_elastic_free(e)


@pytest.mark.timeout(900)
def test_wide_label_bf16_replicas_match_oracle_replay():
    """The elastic configuration at its own model shape: four replicas of the
    wide-label model (F = 135,909, L = 670,091, bf16 operands, fp32 master
    weights) on four streams, weights from samples processed, momentum 0.9,
    Alg. 1 on the replicas' virtual clocks.  The batch bounds and the
    mega-batch are scaled down ([16, 64], 2 batches per replica per round) so
    that the oracle's replay of three rounds stays within about a minute; the
    schedule and every host decision are bit-exact, the global model is
    within the bf16 bar of the exact-product oracle."""
    import torch
    w = synth.WIDE_LABEL
    n, b_min, b_max, beta = 4, 16, 64, 8.0
    slow = (1.0, 1.5, 2.5, 4.0)
    megabatch = 2 * n * b_max
    flush(f"elastic wide-label bf16: {n} replicas, b in [{b_min}, {b_max}], mega-batch {megabatch}")
    ds = synth.generate(w, n_samples=4 * megabatch)
    e, _ = _make(ds, asgd.ASGD_CLOCK_VIRTUAL, 0, asgd.ASGD_WEIGHTS_SAMPLES, megabatch, w=w, n_rep=n,
                 b_min=b_min, b_max=b_max, beta=beta, lr=0.01, slow=slow)
    try:
        dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
        xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
        rp = Replay(w, n, b_max, 0.01, asgd.ASGD_WEIGHTS_SAMPLES, 0, 0.1, 0.9, beta, b_min)
        cursor = 0
        for rnd in range(3):
            b_before = list(rp.b)
            log = asgd.asgd_elastic_round(e, xa, ya, ds.x.indptr, ds.y.indptr)
            torch.cuda.synchronize()
            sched, cursor2, _, u, samples = oe.dispatch_round(ds.x.indptr, cursor, b_before, megabatch,
                                                              [0.0] * n, COST, slow)
            assert log["schedule"] == sched, rnd
            assert log["cursor"] == cursor2
            assert abs(float(np.sum(log["alpha"][:n].astype(np.float64))) - 1.0) < 1e-6
            rp.round(ds, log)
            flush(f"  round {rnd}: u {log['u'][:n]} b_next {log['b_next'][:n]}")
            cursor = cursor2
        assert rp.b != [b_max] * n       # the heterogeneous clocks moved the batch sizes
        rp.check_models(e, RTOL_BF16)
    finally:
        asgd.asgd_elastic_free(e)


def test_timed_rounds_replay_logged_schedule():
    """Timed clock: the replica that takes the next batch is whichever stream
    finished first, so the schedule is not reproducible; every round's logged
    schedule is replayed through the oracle instead, which must reproduce the
    host decisions bit-exactly and the models within the bar."""
    import torch
    flush("elastic timed clock: replay of the logged schedules")
    ds = synth.generate(W, n_samples=2000)
    megabatch = 8 * N_REP * B_MAX
    e, _ = _make(ds, asgd.ASGD_CLOCK_TIMED, 0, asgd.ASGD_WEIGHTS_SAMPLES, megabatch)
    try:
        dx, dy = asgd.DeviceCSR(ds.x), asgd.DeviceCSR(ds.y)
        xa, ya = dx.batch(0, ds.x.n_rows), dy.batch(0, ds.y.n_rows)
        rp = Replay(W, N_REP, B_MAX, 0.05, asgd.ASGD_WEIGHTS_SAMPLES, 0, 0.1, 0.9, BETA, B_MIN)
        cursor = 0
        for rnd in range(3):
            log = asgd.asgd_elastic_round(e, xa, ya, ds.x.indptr, ds.y.indptr)
            torch.cuda.synchronize()
            sched = log["schedule"]
            assert sum(r1 - r0 for _, r0, r1 in sched) == megabatch
            for _, r0, r1 in sched:     # consecutive rows, wrapping at the dataset end
                assert r0 == cursor
                cursor = r1 if r1 < ds.x.n_rows else 0
            assert log["cursor"] == cursor
            rp.round(ds, log)
        rp.check_models(e, 1e-3)
    finally:
        asgd.asgd_elastic_free(e)
