"""GPU parity of the per-replica step (HIP path through the C ABI) against the
CPU oracle on the same seeded inputs: initialisation, the first-layer gather,
the output-layer forward (log-sum-exp, loss), the touched-row set, and the
full SGD update of every parameter tensor."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import (RTOL_BF16, RTOL_EMU_ELEM, RTOL_EMU_NORM, RTOL_FP32, Setup, a1_bound, assert_rel_close,
                      assert_update_close,
                      flush, read_params, step_magnitudes)

pytestmark = pytest.mark.gpu

SMALL_MID = synth.Workload("mid-small", 20_000, 3_000, 4_000, 256, 0.01, True, "lognormal", 4.0,
                           0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)
# feature ids up to 2^22 - 1, the library's limit: the feature sort then runs two
# passes of 11-bit digits, its widest (the largest LDS counter arrays)
WIDE_IDS = synth.Workload("ids-22-bit", (1 << 22) - 1, 500, 512, 256, 0.01, True, "lognormal", 4.0,
                          0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


def test_init_bit_exact_against_oracle():
    flush("init: tiny fp32 and mid-small bf16")
    for w in (synth.TINY, SMALL_MID):
        s = Setup(w, 256, 128)
        try:
            got = s.params()
            ref = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
            for k in ("W1", "b1", "W2", "b2"):
                assert np.array_equal(got[k].view(np.uint32), ref[k].view(np.uint32)), (w.name, k)
        finally:
            s.free()


@pytest.mark.parametrize("w,B,rows", [(synth.TINY, 128, (0, 128)), (synth.TINY, 128, (1920, 2000)),
                                      (SMALL_MID, 256, (0, 256)), (SMALL_MID, 256, (256, 333)),
                                      (SMALL_MID, 256, (7, 8))])
def test_forward_parity(w, B, rows):
    import torch
    r0, r1 = rows
    flush(f"forward: {w.name} rows {r0}..{r1}")
    s = Setup(w, max(r1, 512), B)
    try:
        n = r1 - r0
        a1 = torch.empty((n, 128), dtype=torch.float32, device="cuda")
        lse = torch.empty(n, dtype=torch.float32, device="cuda")
        lr_ = torch.empty(n, dtype=torch.float32, device="cuda")
        asgd.asgd_debug_forward(s.m, s.xb(r0, r1), s.yb(r0, r1), a1_dev=a1, lse_dev=lse, loss_rows_dev=lr_)
        torch.cuda.synchronize()
        xh, yh = s.host_batch(r0, r1)
        p = s.params()
        ops = "bf16" if s.bf16 else "fp32"
        ref = om.forward(p, xh, yh, ops)
        # A1 is a float32 fma chain: within n*u*(|b1| + |X||W1|) of the exact value
        err = np.abs(a1.cpu().numpy().astype(np.float64) - ref["A1"])
        assert np.all(err <= a1_bound(p, xh) + 1e-7 * np.abs(ref["A1"]))
        rt = RTOL_FP32 if not s.bf16 else 1e-3
        assert_rel_close("lse", lse.cpu().numpy(), ref["lse"], rt, floor_frac=0.0)
        assert_rel_close("loss_rows", lr_.cpu().numpy(), ref["loss_rows"], rt, floor_frac=0.0)
        if s.bf16:  # against the exact (non-emulated) definition, the bf16 bar
            ex = om.forward(p, xh, yh, "fp32")
            assert_rel_close("loss_rows(exact)", lr_.cpu().numpy(), ex["loss_rows"], RTOL_BF16, 0.0)
    finally:
        s.free()


def test_one_hot_rows_are_exact_rows_of_w1():
    import torch
    flush("forward: one-hot rows")
    w = synth.TINY
    F = w.n_features
    fs = np.array([0, 17, 4999, 2500, 17], np.int32)
    x = synth.CSR(np.arange(6), fs, np.ones(5, np.float32), F)
    y = synth.CSR(np.arange(6), np.array([1, 2, 3, 4, 5], np.int32), None, w.n_labels)
    ds = synth.Dataset(w, x, y)
    s = Setup(w, 0, 8, ds=ds)
    try:
        b1 = np.linspace(-0.5, 0.5, 128).astype(np.float32)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_B1, b1)
        a1 = torch.empty((5, 128), dtype=torch.float32, device="cuda")
        asgd.asgd_debug_forward(s.m, s.xb(0, 5), None, a1_dev=a1)
        torch.cuda.synchronize()
        W1 = s.params()["W1"]
        want = (W1[fs].astype(np.float64) + b1.astype(np.float64)).astype(np.float32)
        assert np.array_equal(a1.cpu().numpy().view(np.uint32), want.view(np.uint32))
    finally:
        s.free()


@pytest.mark.parametrize("w,rows", [(synth.TINY, (0, 128)), (SMALL_MID, (0, 256)), (SMALL_MID, (100, 101)),
                                    (WIDE_IDS, (0, 256))])
def test_touched_rows_bit_exact(w, rows):
    import torch
    flush(f"touched rows: {w.name} {rows}")
    s = Setup(w, 512, 256)
    try:
        r0, r1 = rows
        ids = torch.empty(s.dx.nnz(r0, r1) + 1, dtype=torch.int32, device="cuda")
        c = asgd.asgd_debug_touched_rows(s.m, s.xb(r0, r1), ids)
        xh, _ = s.host_batch(r0, r1)
        ref = om.touched_features(xh)
        assert c == len(ref)
        assert np.array_equal(ids[:c].cpu().numpy(), ref)
    finally:
        s.free()


def _step_parity(s, r0, r1, lr, rtol, ops):
    before = s.params()
    loss = asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), lr, want_loss=True)
    after = s.params()
    xh, yh = s.host_batch(r0, r1)
    ref, ref_loss, g, fw = om.train_step(before, xh, yh, lr, ops)
    assert abs(loss - ref_loss) <= max(rtol, 1e-5) * abs(ref_loss), (loss, ref_loss)
    mag = step_magnitudes(before, xh, yh, g, fw, lr)
    for k in ("b1", "W2", "b2"):
        assert_update_close(k, before[k], after[k], ref[k], rtol, mag[k])
    t = g["touched"]
    assert_update_close("W1[touched]", before["W1"][t], after["W1"][t], ref["W1"][t], rtol, mag["W1"])
    untouched = np.setdiff1d(np.arange(s.F), t)
    assert np.array_equal(after["W1"][untouched].view(np.uint32), before["W1"][untouched].view(np.uint32))
    return before, after, ref


@pytest.mark.parametrize("rows", [(0, 128), (1920, 2000), (5, 6)])
def test_step_parity_fp32(rows):
    flush(f"step fp32 tiny rows {rows}")
    s = Setup(synth.TINY, 2000, 128)
    try:
        _step_parity(s, rows[0], rows[1], 0.01, RTOL_FP32, "fp32")
    finally:
        s.free()


@pytest.mark.parametrize("rows,B", [((0, 256), 256), ((256, 389), 256), ((0, 600), 600),
                                    ((3, 4), 256), ((0, 128), 256), ((100, 197), 256)])
def test_step_parity_bf16(rows, B):
    flush(f"step bf16 mid-small rows {rows} max_batch {B}")
    s = Setup(SMALL_MID, 1024, B)
    try:
        before, after, ref_exact = _step_parity(s, rows[0], rows[1], 0.05, RTOL_BF16, "fp32")
        # tighter against the oracle with bf16-rounded operands
        xh, yh = s.host_batch(*rows)
        ref_emu, _, g, fw = om.train_step(before, xh, yh, 0.05, "bf16")
        mag = step_magnitudes(before, xh, yh, g, fw, 0.05)
        assert_update_close("W2(bf16 operands)", before["W2"], after["W2"], ref_emu["W2"], RTOL_EMU_ELEM,
                            mag["W2"], norm_rtol=RTOL_EMU_NORM)
        assert_update_close("b2(bf16 operands)", before["b2"], after["b2"], ref_emu["b2"], RTOL_EMU_ELEM,
                            mag["b2"], norm_rtol=RTOL_EMU_NORM)
    finally:
        s.free()


@pytest.mark.parametrize("bf16", [True, False])
def test_step_parity_at_the_largest_batch(bf16):
    """The library's largest batch, 2048 rows: eight 256-row blocks in the
    forward, the backward over 256-row H1 chunks (bf16) or with every row's
    operands in global memory (fp32), and a sort and W1 update over ~150k
    entries."""
    flush(f"step mid-small rows 0..2048 max_batch 2048 bf16={bf16}")
    s = Setup(SMALL_MID, 2048, 2048, bf16=bf16)
    try:
        _step_parity(s, 0, 2048, 0.05, RTOL_BF16 if bf16 else RTOL_FP32, "fp32")
    finally:
        s.free()


def test_step_parity_with_22_bit_feature_ids():
    """F = 2^22 - 1 (W1 is 2 GiB): the batch's ids spread over the whole 22-bit
    range, so both 11-bit digit passes of the feature sort are exercised."""
    flush("step: 22-bit feature ids, F = 2^22 - 1, rows 0..256")
    s = Setup(WIDE_IDS, 512, 256)
    try:
        xh, _ = s.host_batch(0, 256)
        ids = np.asarray(xh.indices[int(xh.indptr[0]):int(xh.indptr[-1])])
        assert ids.max() >= 1 << 21 and ids.min() < 1 << 11
        _step_parity(s, 0, 256, 0.05, RTOL_BF16, "fp32")
    finally:
        s.free()


# rows of about 400 entries (lognormal, some thousands long): batches averaging
# 160 entries or more per row split every row over several gather workgroups
LONG_ROWS = synth.Workload("long-rows", 20_000, 3_000, 1_000, 128, 0.01, True, "lognormal", 5.6,
                           0.9, 5_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)


@pytest.mark.parametrize("rows,bf16", [((0, 128), True), ((128, 161), True), ((0, 128), False)])
def test_step_parity_with_rows_split_over_gather_workgroups(rows, bf16):
    """The gather's split path: every row over four workgroups, their partial
    sums added by a second launch; A1 within its summation bound, the step's
    updates within the parity bar."""
    import torch
    r0, r1 = rows
    flush(f"step: long rows {rows} bf16={bf16}")
    s = Setup(LONG_ROWS, 512, 128, bf16=bf16)
    try:
        xh, _ = s.host_batch(r0, r1)
        assert (int(xh.indptr[-1]) - int(xh.indptr[0])) >= 160 * (r1 - r0)   # the split path runs
        a1 = torch.empty((r1 - r0, 128), dtype=torch.float32, device="cuda")
        asgd.asgd_debug_forward(s.m, s.xb(r0, r1), s.yb(r0, r1), a1_dev=a1)
        torch.cuda.synchronize()
        p = s.params()
        ref = om.forward(p, xh, None, "fp32")
        err = np.abs(a1.cpu().numpy().astype(np.float64) - ref["A1"])
        assert np.all(err <= a1_bound(p, xh) + 1e-7 * np.abs(ref["A1"]))
        _step_parity(s, r0, r1, 0.05, RTOL_BF16 if bf16 else RTOL_FP32, "fp32")
    finally:
        s.free()


def test_split_gather_with_empty_and_very_long_rows():
    """A long-row batch (so the gather splits rows) whose rows are empty, one
    entry, 4,000 entries and lengths that do not divide evenly over the 32
    wavefronts of a split row: A1 within its bound, the step within the bar."""
    import torch
    flush("step: split gather, empty and very long rows")
    w = LONG_ROWS
    rng = np.random.default_rng(11)
    lens = [0, 1, 4000, 37, 0, 1001, 2, 333]
    ip, ind, val = [0], [], []
    for n in lens:
        f = np.sort(rng.choice(w.n_features, n, replace=False)).astype(np.int32)
        ind.append(f)
        val.append(rng.uniform(0.1, 1.0, n).astype(np.float32))
        ip.append(ip[-1] + n)
    x = synth.CSR(np.array(ip), np.concatenate(ind), np.concatenate(val), w.n_features)
    lab = [np.sort(rng.choice(w.n_labels, 1 + i % 3, replace=False)).astype(np.int32) for i in range(len(lens))]
    lip = np.concatenate([[0], np.cumsum([len(a) for a in lab])])
    y = synth.CSR(lip, np.concatenate(lab), None, w.n_labels)
    assert ip[-1] >= 160 * len(lens)   # the split path runs
    s = Setup(w, 0, 128, ds=synth.Dataset(w, x, y))
    try:
        n = len(lens)
        a1 = torch.empty((n, 128), dtype=torch.float32, device="cuda")
        asgd.asgd_debug_forward(s.m, s.xb(0, n), s.yb(0, n), a1_dev=a1)
        torch.cuda.synchronize()
        p = s.params()
        xh, _ = s.host_batch(0, n)
        ref = om.forward(p, xh, None, "fp32")
        err = np.abs(a1.cpu().numpy().astype(np.float64) - ref["A1"])
        assert np.all(err <= a1_bound(p, xh) + 1e-7 * np.abs(ref["A1"]))
        # empty rows: A1 = b1 exactly
        for r in (0, 4):
            assert np.array_equal(a1.cpu().numpy()[r].view(np.uint32), p["b1"].view(np.uint32))
        _step_parity(s, 0, n, 0.05, RTOL_BF16, "fp32")
    finally:
        s.free()


# more 32-label blocks than the forward launch's LDS holds counters for: the
# label grouping then counts in global memory
MANY_LABELS = synth.Workload("labels-1m", 5_000, 1_000_003, 128, 64, 0.01, True, "lognormal", 4.0,
                             0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)


def test_step_parity_with_label_counters_in_global_memory():
    """L = 1,000,003 (ragged last tile): 31,251 label blocks do not fit the
    forward's LDS, so the label grouping takes its global-memory path."""
    flush("step: L = 1,000,003, rows 0..64")
    s = Setup(MANY_LABELS, 128, 64)
    try:
        _step_parity(s, 0, 64, 0.05, RTOL_BF16, "fp32")
    finally:
        s.free()


# 40 labels: two label blocks (the second holds 8), each with hundreds of a
# batch's (row, label) pairs
FEW_LABELS = synth.Workload("labels-40", 5_000, 40, 600, 256, 0.01, True, "lognormal", 4.0,
                            0.8, 2_000, 1.05, "uniform", "poisson", 4.0, None, 2)


@pytest.mark.parametrize("rows", [(0, 256), (256, 455), (455, 555)])
def test_step_parity_with_dense_label_blocks(rows):
    """Every label block holds far more than 64 of the batch's (row, label)
    pairs, so the backward reads a block's pairs past the first 64 from memory
    (the first 64 arrive with the block's weights); 40 labels are two tiles,
    so each of the forward's two splits holds one."""
    flush(f"step: 40 labels, rows {rows}")
    s = Setup(FEW_LABELS, 600, 256)
    try:
        xh, yh = s.host_batch(*rows)
        lab = np.asarray(yh.indices[int(yh.indptr[0]):int(yh.indptr[-1])])
        assert np.bincount(lab // 32, minlength=2).min() > 64
        before, after, _ = _step_parity(s, rows[0], rows[1], 0.05, RTOL_BF16, "fp32")
        ref_emu, _, g, fw = om.train_step(before, xh, yh, 0.05, "bf16")
        mag = step_magnitudes(before, xh, yh, g, fw, 0.05)
        assert_update_close("W2(bf16 operands)", before["W2"], after["W2"], ref_emu["W2"], RTOL_EMU_ELEM,
                            mag["W2"], norm_rtol=RTOL_EMU_NORM)
        assert_update_close("b2(bf16 operands)", before["b2"], after["b2"], ref_emu["b2"], RTOL_EMU_ELEM,
                            mag["b2"], norm_rtol=RTOL_EMU_NORM)
    finally:
        s.free()


def test_step_parity_when_the_running_maximum_rises():
    """Biases rising by 6 per 32-label tile: on every tile of a split the row
    maximum exceeds the forward's running reference by more than its lazy
    rescale margin (8 in base 2, about 5.5), so the rescale of the running sum
    and of the O accumulators runs on every tile."""
    flush("step: rising biases (forward rescale path), mid rows 0..256")
    w = synth.MID
    s = Setup(w, 256, 256)
    try:
        b2 = (6.0 * (np.arange(w.n_labels) // 32)).astype(np.float32)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_B2, b2)
        _step_parity(s, 0, 256, 0.05, RTOL_BF16, "fp32")
    finally:
        s.free()


def test_step_with_empty_feature_row_and_single_label_rows():
    flush("step: empty feature rows")
    w = synth.TINY
    x = synth.CSR(np.array([0, 2, 2, 5, 5]), np.array([3, 9, 1, 2, 4999], np.int32),
                  np.array([0.6, 0.8, 0.5, 0.5, 0.7], np.float32), w.n_features)
    y = synth.CSR(np.array([0, 1, 3, 4, 5]), np.array([0, 5, 999, 7, 7], np.int32), None, w.n_labels)
    s = Setup(w, 0, 8, ds=synth.Dataset(w, x, y))
    try:
        _step_parity(s, 0, 4, 0.1, RTOL_FP32, "fp32")
    finally:
        s.free()


def test_step_w1_segments_across_windows():
    """The sparse W1 update sums each feature's entries window by window (32
    sorted entries per wavefront) and joins the pieces of features that cross
    windows: one feature in every row (a segment of B entries), features with
    tens of entries, and many features seen once, at a batch above 256 rows."""
    flush("step: W1 segments across windows, B=520")
    w = synth.TINY
    rng = np.random.default_rng(11)
    B = 520
    ind, val, ip = [], [], [0]
    lab, lip = [], [0]
    for i in range(B):
        f = {0, 1 + i % 7, 100 + i % 40} | set(rng.choice(np.arange(1000, w.n_features), 3, replace=False).tolist())
        f = np.array(sorted(f), np.int32)
        ind.append(f)
        val.append(rng.uniform(0.1, 1.0, len(f)).astype(np.float32))
        ip.append(ip[-1] + len(f))
        lb = np.sort(rng.choice(w.n_labels, int(rng.integers(1, 4)), replace=False)).astype(np.int32)
        lab.append(lb)
        lip.append(lip[-1] + len(lb))
    x = synth.CSR(np.array(ip), np.concatenate(ind), np.concatenate(val), w.n_features)
    y = synth.CSR(np.array(lip), np.concatenate(lab), None, w.n_labels)
    s = Setup(w, 0, B, ds=synth.Dataset(w, x, y))
    try:
        _step_parity(s, 0, B, 0.1, RTOL_FP32, "fp32")
    finally:
        s.free()


def test_epoch_free_running_fp32():
    flush("epoch: tiny fp32, 16 steps free running")
    w = synth.TINY
    s = Setup(w, 2000, 128)
    try:
        ref = s.params()
        for r0, r1 in synth.batches(s.ds, 128):
            asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), w.lr)
            xh, yh = s.host_batch(r0, r1)
            ref, *_ = om.train_step(ref, xh, yh, w.lr, "fp32")
        got = s.params()
        init = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
        for k in ("W1", "b1", "W2", "b2"):
            assert_update_close(k, init[k], got[k], ref[k], 1e-3)
    finally:
        s.free()


def test_step_is_deterministic():
    flush("determinism: same step twice")
    s = Setup(SMALL_MID, 512, 256)
    try:
        p0 = s.params()
        asgd.asgd_train_step(s.m, s.xb(0, 256), s.yb(0, 256), 0.05)
        p1 = s.params()
        from gpu_util import write_params
        write_params(s.m, p0)
        asgd.asgd_train_step(s.m, s.xb(0, 256), s.yb(0, 256), 0.05)
        p2 = s.params()
        for k in p1:
            assert np.array_equal(p1[k].view(np.uint32), p2[k].view(np.uint32)), k
    finally:
        s.free()


def test_argument_errors_leave_model_unchanged():
    flush("errors: host-side argument checks and device validation")
    w = synth.TINY
    s = Setup(w, 512, 64, flags=asgd.ASGD_VALIDATE)
    try:
        p0 = s.params()
        with pytest.raises(asgd.AsgdError) as e:          # batch beyond max_batch
            asgd.asgd_train_step(s.m, s.xb(0, 100), s.yb(0, 100), 0.1)
        assert e.value.status in (asgd.ASGD_ERANGE,)
        with pytest.raises(asgd.AsgdError) as e:          # row count mismatch
            asgd.asgd_train_step(s.m, s.xb(0, 10), s.yb(0, 11), 0.1)
        assert e.value.status == asgd.ASGD_EINVAL
        with pytest.raises(asgd.AsgdError):               # k out of range
            asgd.asgd_predict_topk(s.m, s.xb(0, 10), 33, 0)
        # malformed content caught on the device: feature id out of range, duplicate ids,
        # empty label row -> EINVAL and nothing updated
        bad_x = synth.CSR(np.array([0, 2, 4]), np.array([1, 5000, 3, 3], np.int32),
                          np.ones(4, np.float32), w.n_features)
        bad_y = synth.CSR(np.array([0, 1, 1]), np.array([2], np.int32), None, w.n_labels)
        bx, by = asgd.DeviceCSR(bad_x), asgd.DeviceCSR(bad_y)
        with pytest.raises(asgd.AsgdError) as e:
            asgd.asgd_train_step(s.m, bx.batch(0, 2), by.batch(0, 2), 0.1)
        assert e.value.status == asgd.ASGD_EINVAL
        msg = asgd.asgd_last_error()
        assert "0x1" in msg or "0x" in msg
        p1 = s.params()
        for k in p0:
            assert np.array_equal(p0[k].view(np.uint32), p1[k].view(np.uint32)), k
    finally:
        s.free()


# many labels per batch entry (L / max_nnz ~ 35): the library runs the gather on its
# internal stream, beside the previous step's backward
WIDE_SMALL = synth.Workload("wide-small", 20_000, 200_003, 2_000, 256, 0.01, True, "lognormal", 3.0,
                            0.7, 500, 1.05, "uniform", "poisson", 4.0, 1.2, 2)


@pytest.mark.parametrize("w,bf16", [(WIDE_SMALL, True), (WIDE_SMALL, False), (SMALL_MID, True)])
def test_consecutive_steps_match_the_oracle_sequence(w, bf16):
    """Steps issued back to back, with batches of different sizes, a
    prediction and a parameter write in between: the model after every step
    follows the oracle's sequence.  With many labels (WIDE_SMALL) the next
    step's gather runs on the internal stream beside the previous backward,
    on the other copy of H1, and after a call other than a step it must wait
    for the model's stream again; otherwise the gather stays on the model's
    stream."""
    import torch
    flush(f"consecutive steps {w.name} bf16={bf16}")
    s = Setup(w, 2000, 256, bf16=bf16)
    try:
        p = s.params()
        bounds = [(0, 256), (256, 300), (300, 556), (556, 557), (557, 813), (813, 1000), (1000, 1256)]
        ids = torch.empty((256, 1), dtype=torch.int32, device="cuda")
        # free-running over seven steps, rounding differences carry from step to step: the
        # elementwise floor is the RMS of the reference update (as for the elastic rounds)
        rt = RTOL_BF16 if bf16 else 1e-3
        for k, (r0, r1) in enumerate(bounds):
            asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), 0.05)
            xh, yh = s.host_batch(r0, r1)
            p, *_ = om.train_step(p, xh, yh, 0.05, "fp32")
            if k == 2:   # a prediction between two steps
                asgd.asgd_predict_topk(s.m, s.xb(0, 256), 1, ids)
            if k == 4:   # a parameter write between two steps (the same values)
                asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_B1, s.params()["b1"])
        torch.cuda.synchronize()
        got = s.params()
        init = om.init_params(w.n_features, w.n_labels, 128, s.seed)
        for k in ("W1", "b1", "W2", "b2"):
            d_ref = p[k].astype(np.float64) - init[k]
            rms = float(np.sqrt(np.mean(d_ref ** 2)))
            assert_update_close(k, init[k], got[k], p[k], rt, mag=np.full(d_ref.shape, rms))
    finally:
        s.free()
