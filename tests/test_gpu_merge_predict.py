"""GPU parity of the normalized merge (Alg. 2), the regularization gate,
top-k prediction, and replica streams against the CPU oracle."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import elastic as oe
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import Setup, flush, h1_flip_logit_bound, read_params, write_params

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


def _models(n, w, seed0=10):
    import torch
    hs = []
    for i in range(n):
        hs.append(asgd.asgd_model_init(w.n_features, w.n_labels, 8, 64, 16, gemm_bf16=w.gemm_bf16,
                                       seed=seed0 + i, stream=torch.cuda.current_stream()))
    return hs


def _flat(m, w):
    return om.flat_params(read_params(m, w.n_features, w.n_labels))


def test_merge_parity_with_momentum_and_buffer_swap():
    flush("merge: 4 replicas + momentum vs oracle")
    w = synth.TINY
    g, gp, *reps = _models(6, w)
    try:
        fg, fgp = _flat(g, w), _flat(gp, w)
        freps = [_flat(r, w) for r in reps]
        alpha = np.array([0.4, 0.3, 0.2, 0.1], np.float32)
        asgd.asgd_merge(g, gp, reps, alpha, 0.9, broadcast=False)
        want, want_prev = oe.merge(fg, fgp, freps, alpha, 0.9)
        got, got_prev = _flat(g, w), _flat(gp, w)
        assert np.array_equal(got_prev.view(np.uint32), want_prev.view(np.uint32))
        ulp = np.spacing(np.abs(want)).astype(np.float64)
        assert np.all(np.abs(got.astype(np.float64) - want) <= ulp)
        assert np.mean(got != want) < 1e-3
        for r, fr in zip(reps, freps):   # replicas untouched without broadcast
            assert np.array_equal(_flat(r, w), fr)
    finally:
        for m in (g, gp, *reps):
            asgd.asgd_model_free(m)


def test_merge_identity_and_broadcast():
    flush("merge: identity (bit exact) and broadcast")
    w = synth.TINY
    g, a, b, c, d = _models(5, w)
    try:
        fa = _flat(a, w)
        for r in (b, c, d):
            write_params(r, read_params(a, w.n_features, w.n_labels))
        asgd.asgd_merge(g, None, [a, b, c, d], [0.25] * 4, 0.9, broadcast=True)
        assert np.array_equal(_flat(g, w).view(np.uint32), fa.view(np.uint32))
        for r in (a, b, c, d):
            assert np.array_equal(_flat(r, w).view(np.uint32), fa.view(np.uint32))
    finally:
        for m in (g, a, b, c, d):
            asgd.asgd_model_free(m)


def test_merge_rejects_bad_arguments():
    flush("merge: argument errors")
    w = synth.TINY
    g, a = _models(2, w)
    other = asgd.asgd_model_init(10, 5, 8, 16, 8, gemm_bf16=False, seed=1)
    try:
        with pytest.raises(asgd.AsgdError):
            asgd.asgd_merge(g, None, [g], [1.0], 0.0, False)        # replica aliases global
        with pytest.raises(asgd.AsgdError):
            asgd.asgd_merge(g, None, [other], [1.0], 0.0, False)    # shape mismatch
        with pytest.raises(asgd.AsgdError):
            asgd.asgd_merge(g, None, [a] * 17, [0.1] * 17, 0.0, False)
    finally:
        for m in (g, a, other):
            asgd.asgd_model_free(m)


def test_l2_per_param_matches_numpy():
    flush("l2 per parameter")
    w = synth.TINY
    (m,) = _models(1, w)
    try:
        f = _flat(m, w).astype(np.float64)
        want = np.sqrt(np.sum(f * f)) / f.size
        got = asgd.asgd_model_l2_per_param(m)
        assert abs(got - want) <= 1e-12 * want
    finally:
        asgd.asgd_model_free(m)


def test_l2_per_param_of_several_models_in_one_call():
    """The perturbation gate's norms for all replicas at once (one launch, one
    synchronization): equal to NumPy's float64 norms and to the one-model call."""
    import torch
    flush("l2 per parameter, several models")
    w = synth.TINY
    ms = _models(3, w)
    try:
        rng = np.random.default_rng(3)
        for i, m in enumerate(ms):   # make the models differ
            asgd.asgd_model_set_params(m, asgd.ASGD_PARAM_B2, rng.normal(0, 1 + i, w.n_labels).astype(np.float32))
        torch.cuda.synchronize()
        got = asgd.asgd_models_l2_per_param(ms)
        for m, g in zip(ms, got):
            f = _flat(m, w).astype(np.float64)
            want = np.sqrt(np.sum(f * f)) / f.size
            assert abs(g - want) <= 1e-12 * want
            assert abs(g - asgd.asgd_model_l2_per_param(m)) <= 1e-13 * want
        assert asgd.asgd_models_l2_per_param(ms[1:2]) == got[1:2]
        with pytest.raises(asgd.AsgdError):
            asgd.asgd_models_l2_per_param([ms[0]] * 17)
    finally:
        for m in ms:
            asgd.asgd_model_free(m)


# min_frac: share of the rows whose top k + 1 logits must be far enough apart
# to be compared id by id; at k = 32 all 32 consecutive gaps must clear the
# bound, which ~10-15 % of these rows do (every row's scores are checked anyway)
@pytest.mark.parametrize("w,bf16,k,min_frac", [(synth.TINY, False, 5, 0.5), (synth.TINY, True, 1, 0.5),
                                               (synth.MID, True, 8, 0.5), (synth.TINY, False, 32, 0.1),
                                               (synth.TINY, True, 32, 0.1)])
def test_topk_ids_bit_exact_on_tie_free_rows(w, bf16, k, min_frac):
    import torch
    flush(f"top-k: {w.name} bf16={bf16} k={k}")
    s = Setup(w, 300, 300, bf16=bf16)
    try:
        # make the logits row-dependent and spread out (|Z| ~ 1), so that most rows'
        # top k+1 logits are separated by far more than the kernel's rounding
        rng = np.random.default_rng(0)
        p0 = s.params()
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_W1, p0["W1"] * 30.0)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_W2, p0["W2"] * 60.0)
        b2 = rng.normal(0, 0.1, w.n_labels).astype(np.float32)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_B2, b2)
        B = 300
        ids = torch.empty((B, k), dtype=torch.int32, device="cuda")
        sc = torch.empty((B, k), dtype=torch.float32, device="cuda")
        asgd.asgd_predict_topk(s.m, s.xb(0, B), k, ids, sc)
        torch.cuda.synchronize()
        xh, _ = s.host_batch(0, B)
        p = s.params()
        ops = "bf16" if bf16 else "fp32"
        fw = om.forward(p, xh, None, ops)
        Z = fw["Z"]
        rid, rsc = om.predict_topk(p, xh, k, ops)
        gi, gs = ids.cpu().numpy(), sc.cpu().numpy()
        tol = 1e-5
        # bf16 operands: a float32 A1 next to a bf16 rounding boundary may round
        # the other way in the kernel; fb bounds what that does to each logit
        fb = h1_flip_logit_bound(p, xh, fw) if bf16 else np.zeros_like(Z)
        checked = 0
        for i in range(B):
            row = np.sort(Z[i])[::-1]
            gaps = -np.diff(row[:k + 1])
            if np.all(gaps > 50 * tol * max(1.0, abs(row[0])) + 2.0 * fb[i].max()):
                assert np.array_equal(gi[i], rid[i]), i
                checked += 1
            # every returned id is a valid label with its own logit
            zi = Z[i, gi[i]]
            assert np.all(np.abs(gs[i] - zi) <= tol * (1.0 + np.abs(zi)) + fb[i, gi[i]]), i
            assert np.all(np.diff(gs[i]) <= 0)
        assert checked > B * min_frac
    finally:
        s.free()


def test_replicas_on_streams_equal_serial_execution():
    import torch
    flush("streams: 4 replicas on 4 streams vs one stream")
    w = synth.TINY
    ds = synth.generate(w, n_samples=1024)
    streams = [torch.cuda.Stream() for _ in range(4)]
    par = [Setup(w, 0, 128, ds=ds) for _ in range(4)]
    ser = [Setup(w, 0, 128, ds=ds) for _ in range(4)]
    try:
        for i, s in enumerate(par):
            asgd.asgd_model_set_stream(s.m, streams[i])
        for step in range(2):
            for i in range(4):
                r0 = (step * 4 + i) * 128
                asgd.asgd_train_step(par[i].m, par[i].xb(r0, r0 + 128), par[i].yb(r0, r0 + 128), 0.05)
        for step in range(2):
            for i in range(4):
                r0 = (step * 4 + i) * 128
                asgd.asgd_train_step(ser[i].m, ser[i].xb(r0, r0 + 128), ser[i].yb(r0, r0 + 128), 0.05)
        torch.cuda.synchronize()
        for a, b in zip(par, ser):
            pa, pb = a.params(), b.params()
            for k in pa:
                assert np.array_equal(pa[k].view(np.uint32), pb[k].view(np.uint32)), k
    finally:
        for s in par + ser:
            s.free()
