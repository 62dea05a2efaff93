"""GPU parity at the benchmark's full sizes (Table 1 shapes of the paper's two
datasets, synthetic): one SGD step per configuration, teacher-forced from the
same initial model, every parameter tensor compared with the oracle; the
B = 1024 batch of the elastic configuration; top-1 prediction; and the merge
of four full-size replicas."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import elastic as oe
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import (RTOL_BF16, Setup, assert_update_close, flush, h1_flip_logit_bound, read_params,
                      step_magnitudes, write_params)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("name,B", [("wide-label", 256), ("wide-feature", 128), ("mid", 256),
                                    ("wide-label", 1024)])
def test_full_size_step(name, B):
    w = synth.WORKLOADS[name]
    flush(f"full-size step: {name} B={B}")
    s = Setup(w, 2 * B, B)
    try:
        before = s.params()
        r0, r1 = B // 2, B // 2 + B   # a batch that starts mid-dataset (indptr[0] > 0)
        if r1 > s.ds.x.n_rows:
            r0, r1 = 0, B
        loss = asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), w.lr, want_loss=True)
        after = s.params()
        xh, yh = s.host_batch(r0, r1)
        ref, ref_loss, g, fw = om.train_step(before, xh, yh, w.lr, "fp32")
        flush(f"  loss gpu {loss:.6f} oracle {ref_loss:.6f}")
        assert abs(loss - ref_loss) <= 1e-3 * abs(ref_loss)
        mag = step_magnitudes(before, xh, yh, g, fw, w.lr)
        for k in ("b1", "W2", "b2"):
            assert_update_close(k, before[k], after[k], ref[k], RTOL_BF16, mag[k])
        t = g["touched"]
        assert_update_close("W1[touched]", before["W1"][t], after["W1"][t], ref["W1"][t], RTOL_BF16, mag["W1"])
        untouched = np.ones(w.n_features, bool)
        untouched[t] = False
        assert np.array_equal(after["W1"][untouched].view(np.uint32), before["W1"][untouched].view(np.uint32))
    finally:
        s.free()


def test_full_size_step_after_training():
    """The same comparison from a trained model instead of the initial one: 49
    steps at lr 20 on distinct batches move the weights well away from their
    small initial values (sharper softmax rows, larger W1 rows for hot
    features), then one step at the workload's lr is compared with the oracle
    started from the GPU's state."""
    w = synth.WIDE_LABEL
    B, n_pre = 256, 49
    flush(f"full-size step after {n_pre} training steps: wide-label B={B}")
    s = Setup(w, (n_pre + 1) * B, B)
    try:
        p0 = s.params()
        for i in range(n_pre):
            asgd.asgd_train_step(s.m, s.xb(i * B, (i + 1) * B), s.yb(i * B, (i + 1) * B), 20.0)
        before = s.params()
        assert all(np.all(np.isfinite(v)) for v in before.values())
        moved = np.linalg.norm(before["W2"] - p0["W2"]) / np.linalg.norm(p0["W2"])
        flush(f"  W2 moved by {moved:.3f} of its initial norm")
        assert moved > 1e-2
        r0, r1 = n_pre * B, (n_pre + 1) * B
        loss = asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), w.lr, want_loss=True)
        after = s.params()
        xh, yh = s.host_batch(r0, r1)
        ref, ref_loss, g, fw = om.train_step(before, xh, yh, w.lr, "fp32")
        flush(f"  loss gpu {loss:.6f} oracle {ref_loss:.6f}")
        assert abs(loss - ref_loss) <= 1e-3 * abs(ref_loss)
        mag = step_magnitudes(before, xh, yh, g, fw, w.lr)
        for k in ("b1", "W2", "b2"):
            assert_update_close(k, before[k], after[k], ref[k], RTOL_BF16, mag[k])
        t = g["touched"]
        assert_update_close("W1[touched]", before["W1"][t], after["W1"][t], ref["W1"][t], RTOL_BF16, mag["W1"])
    finally:
        s.free()


def test_full_size_top1():
    import torch
    w = synth.WIDE_LABEL
    flush("full-size top-1: wide-label")
    s = Setup(w, 256, 256)
    try:
        p0 = s.params()
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_W1, p0["W1"] * 30.0)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_W2, p0["W2"] * 60.0)
        ids = torch.empty((256, 1), dtype=torch.int32, device="cuda")
        sc = torch.empty((256, 1), dtype=torch.float32, device="cuda")
        asgd.asgd_predict_topk(s.m, s.xb(0, 256), 1, ids, sc)
        torch.cuda.synchronize()
        xh, _ = s.host_batch(0, 256)
        p = s.params()
        fw = om.forward(p, xh, None, "bf16")
        Z = fw["Z"]
        gi, gs = ids.cpu().numpy()[:, 0], sc.cpu().numpy()[:, 0]
        # a float32 A1 next to a bf16 rounding boundary may round the other way
        # in the kernel; fb bounds what that does to each logit
        fb = h1_flip_logit_bound(p, xh, fw)
        top2 = -np.sort(-Z, axis=1)[:, :2]
        clear = (top2[:, 0] - top2[:, 1]) > 1e-3 * np.maximum(1.0, np.abs(top2[:, 0])) + 2.0 * fb.max(axis=1)
        assert clear.sum() > 200
        assert np.array_equal(gi[clear], np.argmax(Z[clear], axis=1))
        zi = Z[np.arange(256), gi]
        assert np.all(np.abs(gs - zi) <= 1e-5 * (1.0 + np.abs(zi)) + fb[np.arange(256), gi])
    finally:
        s.free()


def test_full_size_merge_of_four_replicas():
    import torch
    w = synth.WIDE_LABEL
    flush("full-size merge: 4 replicas of wide-label")
    mk = lambda seed: asgd.asgd_model_init(w.n_features, w.n_labels, 8, 64, 64, gemm_bf16=True, seed=seed,
                                           stream=torch.cuda.current_stream())
    g, gp = mk(1), mk(2)
    reps = [mk(10 + i) for i in range(4)]
    try:
        flat = lambda m: om.flat_params(read_params(m, w.n_features, w.n_labels))
        fg, fgp = flat(g), flat(gp)
        fr = [flat(r) for r in reps]
        alpha = np.array([0.31, 0.27, 0.23, 0.19], np.float32)
        asgd.asgd_merge(g, gp, reps, alpha, 0.9, True)
        want, want_prev = oe.merge(fg, fgp, fr, alpha, 0.9)
        got = flat(g)
        assert np.array_equal(flat(gp).view(np.uint32), want_prev.view(np.uint32))
        ulp = np.spacing(np.abs(want)).astype(np.float64)
        assert np.all(np.abs(got.astype(np.float64) - want) <= ulp)
        for r in reps:
            assert np.array_equal(flat(r).view(np.uint32), got.view(np.uint32))
    finally:
        for m in [g, gp] + reps:
            asgd.asgd_model_free(m)
