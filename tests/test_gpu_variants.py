"""GPU parity of the model and output-layer variants against the oracle: the
second dense hidden layer (the other reading of the paper's "3-layer MLP",
Sec. 5.1), the output layer with stored logits and a standalone softmax /
cross-entropy pass (ASGD_UNFUSED_OUTPUT), and the logits returned by
asgd_debug_forward.  Same bar as the plain step: every parameter's update
against the exact-product oracle (1e-4 for fp32 operands, 2e-2 for bf16),
untouched W1 rows bit-exact."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import (RTOL_BF16, RTOL_FP32, Setup, a1_bound, assert_rel_close, assert_update_close, flush,
                      h1_flip_logit_bound, step_magnitudes)

pytestmark = pytest.mark.gpu

SMALL_MID = synth.Workload("mid-small", 20_000, 3_000, 4_000, 256, 0.01, True, "lognormal", 4.0,
                           0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)
# L = 1,001 = 31 * 32 + 9: the last label tile is ragged (stored logits past L are padding)
RAGGED_L = synth.Workload("ragged-labels", 5_000, 1_001, 2_000, 128, 0.01, False, "poisson", 20.0, 0.0, 5_000,
                          1.1, "uniform", "uniform5", 0.0, None, 1)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


def _step_parity(s, r0, r1, lr, rtol):
    before = s.params()
    loss = asgd.asgd_train_step(s.m, s.xb(r0, r1), s.yb(r0, r1), lr, want_loss=True)
    after = s.params()
    xh, yh = s.host_batch(r0, r1)
    ref, ref_loss, g, fw = om.train_step(before, xh, yh, lr, "fp32")
    assert abs(loss - ref_loss) <= max(rtol, 1e-5) * abs(ref_loss), (loss, ref_loss)
    mag = step_magnitudes(before, xh, yh, g, fw, lr)
    for k in before:
        if k == "W1":
            continue
        assert_update_close(k, before[k], after[k], ref[k], rtol, mag[k])
    t = g["touched"]
    assert_update_close("W1[touched]", before["W1"][t], after["W1"][t], ref["W1"][t], rtol, mag["W1"])
    untouched = np.setdiff1d(np.arange(s.F), t)
    assert np.array_equal(after["W1"][untouched].view(np.uint32), before["W1"][untouched].view(np.uint32))


def test_extra_layer_init_bit_exact_against_oracle():
    flush("extra layer: init")
    s = Setup(synth.TINY, 256, 128, extra=1)
    try:
        got = s.params()
        ref = om.init_params(s.F, s.L, 128, s.seed, extra_hidden_layers=1)
        assert list(got) == list(ref)
        for k in ref:
            assert np.array_equal(got[k].view(np.uint32), ref[k].view(np.uint32)), k
        assert asgd.asgd_model_num_params(s.m) == om.flat_params(ref).size
    finally:
        s.free()


@pytest.mark.parametrize("w,bf16,rows,flags", [
    (synth.TINY, False, (0, 128), 0), (synth.TINY, False, (1920, 2000), 0), (synth.TINY, False, (5, 6), 0),
    (SMALL_MID, True, (0, 256), 0), (SMALL_MID, True, (300, 377), 0),
    (synth.TINY, False, (0, 128), asgd.ASGD_UNFUSED_OUTPUT), (SMALL_MID, True, (0, 256), asgd.ASGD_UNFUSED_OUTPUT)])
def test_extra_layer_step_parity(w, bf16, rows, flags):
    flush(f"extra layer step: {w.name} bf16={bf16} rows {rows} flags {flags}")
    s = Setup(w, 2000, 256, bf16=bf16, extra=1, flags=flags)
    try:
        # biases away from zero so that both ReLU masks are exercised on both sides
        rng = np.random.default_rng(5)
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_BH, rng.normal(0, 0.05, 128).astype(np.float32))
        asgd.asgd_model_set_params(s.m, asgd.ASGD_PARAM_B1, rng.normal(0, 0.02, 128).astype(np.float32))
        _step_parity(s, rows[0], rows[1], 0.05, RTOL_BF16 if bf16 else RTOL_FP32)
    finally:
        s.free()


@pytest.mark.parametrize("w,bf16,rows,B", [
    (synth.TINY, False, (0, 128), 128), (synth.TINY, False, (1920, 2000), 128), (RAGGED_L, False, (7, 8), 128),
    (RAGGED_L, False, (0, 128), 128), (SMALL_MID, True, (0, 256), 256), (SMALL_MID, True, (256, 389), 256),
    (SMALL_MID, True, (0, 600), 600)])
def test_unfused_step_parity(w, bf16, rows, B):
    flush(f"unfused step: {w.name} bf16={bf16} rows {rows} max_batch {B}")
    s = Setup(w, 2000, B, bf16=bf16, flags=asgd.ASGD_UNFUSED_OUTPUT)
    try:
        _step_parity(s, rows[0], rows[1], 0.05, RTOL_BF16 if bf16 else RTOL_FP32)
    finally:
        s.free()


@pytest.mark.parametrize("w,bf16,flags,rows", [
    (synth.TINY, False, 0, (0, 128)), (RAGGED_L, False, asgd.ASGD_UNFUSED_OUTPUT, (3, 131)),
    (SMALL_MID, True, 0, (0, 256)), (SMALL_MID, True, asgd.ASGD_UNFUSED_OUTPUT, (11, 267))])
def test_logits_lse_and_loss_against_oracle(w, bf16, flags, rows):
    """Z from asgd_debug_forward in both output modes (the stored logits of the
    unfused step, or the logits kernel writing the caller's [B x L] buffer), and
    lse and the loss rows of the softmax / cross-entropy pass over them."""
    import torch
    r0, r1 = rows
    n = r1 - r0
    flush(f"logits: {w.name} bf16={bf16} flags {flags} rows {rows}")
    s = Setup(w, 2000, 256, bf16=bf16, flags=flags)
    try:
        z = torch.full((n, s.L), float("nan"), dtype=torch.float32, device="cuda")
        lse = torch.empty(n, dtype=torch.float32, device="cuda")
        lrows = torch.empty(n, dtype=torch.float32, device="cuda")
        asgd.asgd_debug_forward(s.m, s.xb(r0, r1), s.yb(r0, r1), z_dev=z, lse_dev=lse, loss_rows_dev=lrows)
        torch.cuda.synchronize()
        p = s.params()
        xh, yh = s.host_batch(r0, r1)
        ops = "bf16" if bf16 else "fp32"
        ref = om.forward(p, xh, yh, ops)
        Z = z.cpu().numpy().astype(np.float64)
        assert np.all(np.isfinite(Z))
        # per logit, a float32 sum of 128 products and the bias: |err| <= 130 u (|H| |W2| + |b2|);
        # plus what the kernel's float32 A1 carries in (fp32 operands: its summation bound
        # times |W2|; bf16 operands: a flipped rounding of H1 near a rounding boundary)
        aw = np.abs(om._operand(p["W2"], ops))
        Hm = np.abs(om._operand(ref["H1"], ops)) @ aw.T
        allow = 130 * 2.0 ** -24 * (Hm + np.abs(p["b2"])) + 1e-30
        allow = allow + (h1_flip_logit_bound(p, xh, ref) if bf16 else a1_bound(p, xh) @ aw.T)
        err = np.abs(Z - ref["Z"])
        assert np.all(err <= allow), float(np.max(err / allow))
        rt = RTOL_FP32 if not bf16 else 1e-3
        assert_rel_close("lse", lse.cpu().numpy(), ref["lse"], rt, floor_frac=0.0)
        assert_rel_close("loss_rows", lrows.cpu().numpy(), ref["loss_rows"], rt, floor_frac=0.0)
    finally:
        s.free()


def test_extra_layer_merge_identity_and_topk():
    """Models with the second hidden layer merge as one flat vector (identical
    replicas with weights 1/4 give the identity bit-exactly), and predict with
    it (top-1 ids equal to the oracle's on rows whose top gap is wide)."""
    import torch
    flush("extra layer: merge identity and top-1")
    w = synth.TINY
    mk = lambda: asgd.asgd_model_init(w.n_features, w.n_labels, 128, 4000, 1000, gemm_bf16=False, seed=w.init_seed,
                                      stream=torch.cuda.current_stream(), extra_hidden_layers=1)
    g, reps = mk(), [mk() for _ in range(4)]
    try:
        from gpu_util import read_params
        before = read_params(g, w.n_features, w.n_labels, True)
        asgd.asgd_merge(g, None, reps, [0.25] * 4, 0.0, True)
        torch.cuda.synchronize()
        after = read_params(g, w.n_features, w.n_labels, True)
        for k in before:
            assert np.array_equal(after[k].view(np.uint32), before[k].view(np.uint32)), k
        ds = synth.generate(w, n_samples=128)
        dx = asgd.DeviceCSR(ds.x)
        ids = torch.empty((128, 1), dtype=torch.int32, device="cuda")
        asgd.asgd_predict_topk(g, dx.batch(0, 128), 1, ids)
        torch.cuda.synchronize()
        ref = om.forward(before, ds.x, None, "fp32")["Z"]
        top2 = np.sort(ref, axis=1)[:, -2:]
        clear = (top2[:, 1] - top2[:, 0]) > 1e-4 * (1 + np.abs(top2[:, 1]))
        assert clear.mean() > 0.5
        want = np.argmax(ref, axis=1)
        assert np.array_equal(ids.cpu().numpy()[clear, 0], want[clear])
    finally:
        for m in [g] + reps:
            asgd.asgd_model_free(m)


def test_variant_arguments_are_checked():
    with pytest.raises(asgd.AsgdError):
        asgd.asgd_model_init(100, 10, 8, 16, 8, extra_hidden_layers=2)
    m = asgd.asgd_model_init(100, 10, 8, 16, 8)
    try:
        with pytest.raises(asgd.AsgdError):   # no second hidden layer in this model
            asgd.asgd_model_get_params(m, asgd.ASGD_PARAM_WH, (128, 128))
    finally:
        asgd.asgd_model_free(m)
