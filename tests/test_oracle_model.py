"""Pins of the CPU oracle's model step against values fixed outside the oracle.

Each test checks the oracle against something other than itself: published
generator outputs, textbook identities (log-sum-exp, softmax cross-entropy),
closed forms, dense-matrix equivalents, central finite differences and
invariants that hold for any input.
"""
import math
import os

import numpy as np
import pytest

from oracle import model as om
from paper_2110_07029_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_problem(seed=0, B=6, F=12, L=7, H=5, nnz=(1, 5), labels=(1, 3), scale=1.0):
    """A small random CSR batch and parameters (float64 storage for FD tests)."""
    rng = np.random.default_rng(seed)
    indptr = [0]
    idx, val = [], []
    for _ in range(B):
        k = int(rng.integers(nnz[0], nnz[1] + 1))
        f = np.sort(rng.choice(F, k, replace=False))
        idx += list(f)
        val += list(rng.uniform(0.2, 1.0, k))
        indptr.append(len(idx))
    x = synth.CSR(np.array(indptr), np.array(idx, np.int32), np.array(val, np.float32), F)
    yptr = [0]
    yidx = []
    for _ in range(B):
        k = int(rng.integers(labels[0], labels[1] + 1))
        yidx += list(np.sort(rng.choice(L, k, replace=False)))
        yptr.append(len(yidx))
    y = synth.CSR(np.array(yptr), np.array(yidx, np.int32), None, L)
    p = dict(W1=rng.normal(0, scale, (F, H)), b1=rng.normal(0, 0.1, H),
             W2=rng.normal(0, scale, (L, H)), b2=rng.normal(0, 0.1, L))
    return x, y, p


def dense_x(x):
    B = len(x.indptr) - 1
    X = np.zeros((B, x.n_cols))
    for i in range(B):
        for p in range(x.indptr[i], x.indptr[i + 1]):
            X[i, x.indices[p]] += float(x.values[p])
    return X


# --------------------------------------------------------------------------- init
def test_splitmix64_published_outputs():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64_seed0.txt")) if not l.startswith("#")]
    states = np.array([int(r[0], 16) for r in rows], np.uint64)
    want = [int(r[1], 16) for r in rows]
    got = [int(v) for v in om.splitmix64(states)]
    assert got == want


def test_init_uniform_grid_and_moments():
    F, L, H = 3000, 500, 128
    p = om.init_params(F, L, H, seed=1234)
    a1 = float(om.xavier_bound(F, H))
    a2 = float(om.xavier_bound(H, L))
    assert math.isclose(a1, math.sqrt(6 / (F + H)), rel_tol=1e-7)
    for w, a in ((p["W1"], a1), (p["W2"], a2)):
        assert w.dtype == np.float32
        assert np.all(np.abs(w) <= a)
        # uniform on [-a, a): mean 0, variance a^2/3 (n ~ 10^5 draws)
        assert abs(float(w.mean())) < 0.01 * a
        assert abs(float(w.var()) / (a * a / 3) - 1) < 0.01
        # every value is fl32(k * 2^-23 - 1) * a for an integer k: (w/a + 1) * 2^23 close to an integer
        k = (w.astype(np.float64) / a + 1.0) * 2.0 ** 23
        assert np.max(np.abs(k - np.rint(k))) < 2.0 ** -1
    assert np.all(p["b1"] == 0) and np.all(p["b2"] == 0)
    # different tensors / seeds give different streams
    q = om.init_params(F, L, H, seed=1235)
    assert not np.array_equal(p["W1"], q["W1"])
    u0 = om.init_uniform24(7, 0, 1000)
    u1 = om.init_uniform24(7, 1, 1000)
    assert not np.array_equal(u0, u1)


def test_init_element_formula():
    # element e of tensor t: u = (splitmix64(seed ^ (t << 56) ^ e) >> 40) * 2^-24
    seed, t, e = 99, 1, 12345
    z = int(om.splitmix64(np.array([seed ^ (t << 56) ^ e], np.uint64))[0])
    want = (z >> 40) / 2.0 ** 24
    assert om.init_uniform24(seed, t, 1, start=e)[0] == want


# --------------------------------------------------------------------------- bf16
def test_round_bf16_textbook_cases():
    one = 1.0
    cases = [
        (one, one),
        (one + 2.0 ** -8, one),                      # halfway, ties to even (down)
        (one + 3 * 2.0 ** -8, one + 2.0 ** -6),      # halfway, ties to even (up)
        (one + 2.0 ** -8 + 2.0 ** -20, one + 2.0 ** -7),  # just above halfway
        (-(one + 2.0 ** -9), -one),
    ]
    for v, want in cases:
        got = float(om.round_bf16(np.array([v], np.float32))[0])
        assert got == want, (v, got, want)
    assert np.isnan(om.round_bf16(np.array([np.nan], np.float32))[0])
    assert om.round_bf16(np.array([np.inf], np.float32))[0] == np.inf


def test_round_bf16_is_nearest_ties_even_brute_force():
    # bf16 values are float32 values with 16 zero low bits: the result must be the
    # nearer of the two bracketing bf16 values (ties: even last kept bit).
    v = np.random.default_rng(0).normal(size=20000).astype(np.float32)
    v[:50] = (v[:50].view(np.uint32) & 0xFFFF0000 | 0x8000).view(np.float32)  # exact ties
    r = om.round_bf16(v)
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    lo = (v.view(np.uint32) & 0xFFFF0000).view(np.float32).astype(np.float64)   # toward zero
    step = np.ldexp(1.0, np.frexp(np.abs(lo))[1] - 8)                            # bf16 ulp at |lo|
    hi = lo + np.sign(v.astype(np.float64)) * step                                 # away from zero
    x = v.astype(np.float64)
    dlo, dhi = np.abs(x - lo), np.abs(x - hi)
    lo_even = ((v.view(np.uint32) >> 16) & 1) == 0
    want = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo_even, lo, hi)))
    assert np.array_equal(r.astype(np.float64), want)


# --------------------------------------------------------------------------- forward
def test_forward_matches_dense_and_library_logsumexp():
    import scipy.special
    x, y, p = tiny_problem(seed=1)
    fw = om.forward(p, x, y)
    X = dense_x(x)
    A1 = X @ p["W1"] + p["b1"]
    Z = np.maximum(A1, 0) @ p["W2"].T + p["b2"]
    assert np.allclose(fw["A1"], A1, rtol=1e-13, atol=1e-13)
    assert np.allclose(fw["Z"], Z, rtol=1e-13, atol=1e-13)
    assert np.allclose(fw["lse"], scipy.special.logsumexp(Z, axis=1), rtol=1e-13)


def test_loss_equals_torch_cross_entropy_with_probability_targets():
    import torch
    x, y, p = tiny_problem(seed=2, labels=(1, 4))
    fw = om.forward(p, x, y)
    T = om.targets(y, 7)
    ref = torch.nn.functional.cross_entropy(torch.tensor(fw["Z"]), torch.tensor(T), reduction="mean")
    assert math.isclose(fw["loss"], float(ref), rel_tol=1e-12)


def test_single_label_reduces_to_textbook_softmax_ce():
    x, y, p = tiny_problem(seed=3, labels=(1, 1))
    fw = om.forward(p, x, y)
    Z = fw["Z"]
    for i in range(Z.shape[0]):
        t = y.indices[i]
        sm = np.exp(Z[i] - Z[i].max()) / np.exp(Z[i] - Z[i].max()).sum()
        assert math.isclose(fw["loss_rows"][i], -math.log(sm[t]), rel_tol=1e-12)


def test_zero_output_layer_closed_form():
    x, y, p = tiny_problem(seed=4, L=7, labels=(1, 3))
    p["W2"][:] = 0
    p["b2"][:] = 0
    fw = om.forward(p, x, y)
    assert np.allclose(fw["loss_rows"], math.log(7), rtol=0, atol=1e-15)
    g = om.backward(p, x, y, fw)
    B = 6
    assert np.allclose(g["dZ"], (1.0 / 7 - om.targets(y, 7)) / B, atol=1e-16)
    assert np.all(g["dH1"] == 0)


def test_one_hot_rows_gather_exact_rows():
    # rows with a single entry of value 1 give A1 = W1[f] + b1 exactly (float32 params)
    F, H = 50, 128
    p = om.init_params(F, 10, H, seed=5)
    p["b1"] = np.linspace(-0.1, 0.1, H).astype(np.float32)
    fs = np.array([3, 17, 49, 0], np.int32)
    x = synth.CSR(np.arange(5), fs, np.ones(4, np.float32), F)
    fw = om.forward(p, x)
    want = p["W1"][fs].astype(np.float64) + p["b1"].astype(np.float64)
    assert np.array_equal(fw["A1"], want)


# --------------------------------------------------------------------------- backward
def _loss_of(p, x, y):
    return om.forward(p, x, y)["loss"]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_gradients_match_central_finite_differences(seed):
    x, y, p = tiny_problem(seed=seed + 10)
    fw = om.forward(p, x, y)
    assert np.min(np.abs(fw["A1"])) > 1e-3      # away from the ReLU kink
    g = om.backward(p, x, y, fw)
    eps = 1e-6
    dense_dW1 = np.zeros_like(p["W1"])
    dense_dW1[g["touched"]] = g["dW1_rows"]
    for name, ana in (("W1", dense_dW1), ("b1", g["db1"]), ("W2", g["dW2"]), ("b2", g["db2"])):
        num = np.zeros_like(p[name])
        it = np.nditer(p[name], flags=["multi_index"])
        for _ in it:
            j = it.multi_index
            q = {k: v.copy() for k, v in p.items()}
            q[name][j] += eps
            lp = _loss_of(q, x, y)
            q[name][j] -= 2 * eps
            lm = _loss_of(q, x, y)
            num[j] = (lp - lm) / (2 * eps)
        err = np.max(np.abs(num - ana)) / max(np.max(np.abs(ana)), 1e-12)
        assert err < 1e-6, (name, err)


def _with_extra_layer(p, seed, H, scale=1.0):
    rng = np.random.default_rng(seed)
    q = {k: p[k] for k in ("W1", "b1")}
    q["Wh"] = rng.normal(0, scale, (H, H))
    q["bh"] = rng.normal(0, 0.1, H)
    q["W2"], q["b2"] = p["W2"], p["b2"]
    return q


@pytest.mark.parametrize("seed", [0, 1])
def test_extra_hidden_layer_gradients_match_central_finite_differences(seed):
    # the other reading of the "3-layer MLP": F -> H (ReLU) -> H (ReLU) -> L
    x, y, p = tiny_problem(seed=seed + 40)
    p = _with_extra_layer(p, seed + 50, 5)
    fw = om.forward(p, x, y)
    assert np.min(np.abs(fw["A1"])) > 1e-3 and np.min(np.abs(fw["A2"])) > 1e-3   # away from the kinks
    g = om.backward(p, x, y, fw)
    eps = 1e-6
    dense_dW1 = np.zeros_like(p["W1"])
    dense_dW1[g["touched"]] = g["dW1_rows"]
    for name, ana in (("W1", dense_dW1), ("b1", g["db1"]), ("Wh", g["dWh"]), ("bh", g["dbh"]),
                      ("W2", g["dW2"]), ("b2", g["db2"])):
        num = np.zeros_like(p[name])
        it = np.nditer(p[name], flags=["multi_index"])
        for _ in it:
            j = it.multi_index
            q = {k: v.copy() for k, v in p.items()}
            q[name][j] += eps
            lp = _loss_of(q, x, y)
            q[name][j] -= 2 * eps
            lm = _loss_of(q, x, y)
            num[j] = (lp - lm) / (2 * eps)
        err = np.max(np.abs(num - ana)) / max(np.max(np.abs(ana)), 1e-12)
        assert err < 1e-6, (name, err)


def test_extra_hidden_layer_dense_form_and_identity_reduction():
    x, y, p = tiny_problem(seed=45)
    q = _with_extra_layer(p, 46, 5)
    fw = om.forward(q, x, y)
    X = dense_x(x)
    H1 = np.maximum(X @ p["W1"] + p["b1"], 0)
    H2 = np.maximum(H1 @ q["Wh"].T + q["bh"], 0)
    assert np.allclose(fw["Z"], H2 @ p["W2"].T + p["b2"], rtol=1e-13, atol=1e-13)
    # Wh = I, bh = 0: H2 = ReLU(H1) = H1, so the model is the two-matrix one; its
    # gradients carry over, and dWh = dA2^T H1 with dA2 = dH1 [H1 > 0]
    q["Wh"] = np.eye(5)
    q["bh"] = np.zeros(5)
    f3, f2 = om.forward(q, x, y), om.forward(p, x, y)
    assert np.allclose(f3["loss_rows"], f2["loss_rows"], rtol=1e-14, atol=1e-15)
    g3, g2 = om.backward(q, x, y, f3), om.backward(p, x, y, f2)
    for k in ("dW2", "db2", "db1", "dW1_rows"):
        assert np.allclose(g3[k], g2[k], rtol=1e-13, atol=1e-15), k
    dA2 = g2["dH1"] * (H1 > 0)
    assert np.allclose(g3["dWh"], dA2.T @ H1, rtol=1e-13, atol=1e-15)
    assert np.allclose(g3["dbh"], dA2.sum(axis=0), rtol=1e-13, atol=1e-15)


def test_extra_hidden_layer_init_and_flat_order():
    p = om.init_params(40, 9, 128, seed=7, extra_hidden_layers=1)
    assert list(p) == ["W1", "b1", "Wh", "bh", "W2", "b2"]
    a = float(om.xavier_bound(128, 128))
    assert math.isclose(a, math.sqrt(6 / 256), rel_tol=1e-7)
    assert np.all(np.abs(p["Wh"]) <= a) and np.all(p["bh"] == 0)
    # tensor 2 of the same seed; the other tensors are those of the two-matrix model
    u = om.init_uniform24(7, 2, 128 * 128)
    assert np.array_equal(p["Wh"].ravel(), (2.0 * u - 1.0).astype(np.float32) * np.float32(a))
    p2 = om.init_params(40, 9, 128, seed=7)
    assert all(np.array_equal(p[k], p2[k]) for k in p2)
    v = om.flat_params(p)
    assert v.size == 40 * 128 + 128 + 128 * 128 + 128 + 9 * 128 + 9
    back = om.unflat_params(v, 40, 9, 128, extra_hidden_layers=1)
    assert all(np.array_equal(back[k], p[k]) for k in p)
    # an SGD step updates Wh and bh against their gradients
    x = synth.CSR(np.array([0, 2]), np.array([3, 7], np.int32), np.array([0.6, 0.8], np.float32), 40)
    y = synth.CSR(np.array([0, 1]), np.array([4], np.int32), None, 9)
    q, loss, g, _ = om.train_step(p, x, y, 0.5)
    d = q["Wh"].astype(np.float64) - p["Wh"]
    ulp = np.spacing(np.maximum(np.abs(p["Wh"]), np.abs(q["Wh"]))).astype(np.float64)
    assert np.all(np.abs(d + 0.5 * g["dWh"]) <= ulp)


def test_gradient_invariants():
    x, y, p = tiny_problem(seed=20, B=9, F=30, L=11)
    fw = om.forward(p, x, y)
    g = om.backward(p, x, y, fw)
    # softmax minus a probability distribution sums to zero in every row
    assert np.allclose(g["dZ"].sum(axis=1), 0, atol=1e-15)
    assert abs(g["db2"].sum()) < 1e-14
    # db1 = column sums of dA1 ; dW1 = X^T dA1 on touched rows, zero elsewhere
    assert np.allclose(g["db1"], g["dA1"].sum(axis=0))
    full = dense_x(x).T @ g["dA1"]
    assert np.allclose(full[g["touched"]], g["dW1_rows"], rtol=1e-12, atol=1e-15)
    untouched = np.setdiff1d(np.arange(30), g["touched"])
    assert np.all(full[untouched] == 0)
    assert np.array_equal(g["touched"], np.unique(x.indices))


def test_update_touches_only_batch_rows_and_moves_against_gradient():
    w = synth.TINY
    ds = synth.generate(w, n_samples=256)
    p = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
    xb, yb = ds.x.rows(0, 128), ds.y.rows(0, 128)
    q, loss, g, fw = om.train_step(p, xb, yb, 0.01)
    untouched = np.setdiff1d(np.arange(w.n_features), g["touched"])
    assert np.array_equal(q["W1"][untouched].view(np.uint32), p["W1"][untouched].view(np.uint32))
    t = g["touched"]
    dW1 = q["W1"][t].astype(np.float64) - p["W1"][t]
    ulp = np.spacing(np.maximum(np.abs(p["W1"][t]), np.abs(q["W1"][t]))).astype(np.float64)
    assert np.all(np.abs(dW1 + 0.01 * g["dW1_rows"]) <= ulp)
    assert math.isclose(loss, fw["loss"])
    # a small step lowers the loss on the same batch
    assert om.forward(q, xb, yb)["loss"] < loss


def test_bf16_operands_close_to_exact():
    w = synth.TINY
    ds = synth.generate(w, n_samples=128)
    p = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
    f32 = om.forward(p, ds.x, ds.y, "fp32")
    b16 = om.forward(p, ds.x, ds.y, "bf16")
    rel = np.linalg.norm(b16["Z"] - f32["Z"]) / np.linalg.norm(f32["Z"])
    assert 1e-5 < rel < 1e-2


def _one_row_problem(w1_row, w2):
    """F = 1, H = 2, L = 3, B = 1: one feature of value 1, label {0}, b1 = b2 = 0."""
    x = synth.CSR(np.array([0, 1]), np.array([0], np.int32), np.array([1.0], np.float32), 1)
    y = synth.CSR(np.array([0, 1]), np.array([0], np.int32), None, 3)
    p = dict(W1=np.array([w1_row], np.float32), b1=np.zeros(2, np.float32),
             W2=np.array(w2, np.float32), b2=np.zeros(3, np.float32))
    return x, y, p


# Hand-derived values for the bf16 pins.  With Z = 0 over L = 3 labels the softmax
# is 1/3 everywhere, so dZ = (1/3 - 1, 1/3, 1/3) for the target {0}.  As float32
# these are 0xBF2AAAAB and 0x3EAAAAAB; rounded to nearest bf16 (ties to even) they
# become 0xBF2B = -171/256 and 0x3EAB = 171/512 (truncation would give 0xBF2A =
# -170/256 and 0x3EAA = 170/512).  The hidden value 1.005859375 = 0x3F80C000
# rounds up to 0x3F81 = 129/128 (truncation: 1.0); 0.5 is a bf16 value.
DZ0_B, DZ1_B, H_B = -171 / 256, 171 / 512, 129 / 128


def test_bf16_backward_rounds_dz_h1_and_w2_to_nearest_even_dw2():
    # W2 = 0 and H1 = (1.005859375, 0.5): dW2 = bf16(dZ)^T bf16(H1), exactly
    x, y, p = _one_row_problem([1.005859375, 0.5], np.zeros((3, 2)))
    fw = om.forward(p, x, y, "bf16")
    assert np.all(fw["Z"] == 0.0)
    g = om.backward(p, x, y, fw, "bf16")
    want = np.array([[DZ0_B * H_B, DZ0_B * 0.5], [DZ1_B * H_B, DZ1_B * 0.5], [DZ1_B * H_B, DZ1_B * 0.5]])
    assert np.array_equal(g["dW2"], want)
    assert want[1, 0] == 22059 / 65536           # 0.3365936279296875 (no rounding: 0.33528...)
    # the bias gradient is the unrounded dZ; the update with lr = 1 stores -dW2
    assert np.allclose(g["db2"], [-2 / 3, 1 / 3, 1 / 3], rtol=0, atol=1e-15)
    q, *_ = om.train_step(p, x, y, 1.0, "bf16")
    assert np.array_equal(q["W2"].astype(np.float64), -want)
    # fp32 operands: the exact products
    g32 = om.backward(p, x, y, om.forward(p, x, y, "fp32"), "fp32")
    assert np.allclose(g32["dW2"][1], [1.005859375 / 3, 0.5 / 3], rtol=1e-15, atol=0)


def test_bf16_backward_rounds_dz_and_w2_in_dh1():
    # H1 = 0 (both pre-activations negative), so Z = b2 = 0 whatever W2 is; then
    # dH1 = bf16(dZ) bf16(W2) with W2 row 0 = (1.005859375, 0.5), the others 0
    x, y, p = _one_row_problem([-1.0, -2.0], [[1.005859375, 0.5], [0.0, 0.0], [0.0, 0.0]])
    fw = om.forward(p, x, y, "bf16")
    assert np.all(fw["H1"] == 0.0) and np.all(fw["Z"] == 0.0)
    g = om.backward(p, x, y, fw, "bf16")
    assert np.array_equal(g["dH1"], [[DZ0_B * H_B, DZ0_B * 0.5]])
    assert g["dH1"][0, 0] == -22059 / 32768       # -0.673187255859375 (no rounding: -0.67057...)
    assert np.all(g["dA1"] == 0.0)                # ReLU'(A1 < 0) = 0
    g32 = om.backward(p, x, y, om.forward(p, x, y, "fp32"), "fp32")
    assert np.allclose(g32["dH1"], [[-2 / 3 * 1.005859375, -1 / 3]], rtol=1e-15, atol=0)


def test_gradient_aggregation_equals_model_averaging_after_one_step():
    # Sec. 2.2: averaging after every batch makes model averaging equal gradient
    # aggregation: n replicas, one step each on disjoint batches of size b, merged
    # with alpha = 1/n and no momentum, equal one step on the n*b concatenation.
    from oracle import elastic as oe
    w = synth.TINY
    ds = synth.generate(w, n_samples=512)
    p = om.init_params(w.n_features, w.n_labels, 128, w.init_seed)
    n, b, lr = 4, 64, 0.05
    reps = []
    for i in range(n):
        q, *_ = om.train_step(p, ds.x.rows(i * b, (i + 1) * b), ds.y.rows(i * b, (i + 1) * b), lr)
        reps.append(om.flat_params(q))
    g0 = om.flat_params(p)
    merged, prev = oe.merge(g0, g0, reps, [1.0 / n] * n, 0.0)
    big, *_ = om.train_step(p, ds.x.rows(0, n * b), ds.y.rows(0, n * b), lr)
    big = om.flat_params(big)
    d_m = merged.astype(np.float64) - g0
    d_b = big.astype(np.float64) - g0
    # mathematically equal; each side stores float32 once per step and once per merge,
    # so elements may differ by those roundings: <= 1.5 ulp of the largest value stored
    mag = np.maximum.reduce([np.abs(g0), np.abs(merged), np.abs(big)] + [np.abs(r) for r in reps])
    ulp = np.spacing(mag).astype(np.float64)
    assert np.all(np.abs(d_m - d_b) <= 2 * ulp)
    assert np.linalg.norm(d_m - d_b) <= 1e-3 * np.linalg.norm(d_b)
    assert np.array_equal(prev, g0)


# --------------------------------------------------------------------------- top-k
def test_topk_brute_force():
    x, y, p = tiny_problem(seed=30, B=5, L=9)
    ids, sc = om.predict_topk(p, x, 4)
    Z = om.forward(p, x)["Z"]
    for i in range(5):
        pairs = sorted(((-Z[i, j], j) for j in range(9)))
        assert list(ids[i]) == [j for _, j in pairs[:4]]
        assert np.allclose(sc[i], [-v for v, _ in pairs[:4]])


def test_topk_ties_prefer_smaller_label():
    x, y, p = tiny_problem(seed=31, B=3, L=6)
    p["W2"][:] = 0
    p["b2"] = np.array([0.5, 1.0, 1.0, 0.2, 1.0, 0.0])
    ids, _ = om.predict_topk(p, x, 4)
    assert np.all(ids == np.array([1, 2, 4, 0]))


def test_touched_features_brute_force():
    x, y, p = tiny_problem(seed=32, B=8, F=40)
    assert list(om.touched_features(x)) == sorted(set(int(v) for v in x.indices))


def test_flat_roundtrip():
    p = om.init_params(20, 9, 128, 3)
    v = om.flat_params(p)
    assert v.size == 20 * 128 + 128 + 9 * 128 + 9
    q = om.unflat_params(v, 20, 9, 128)
    for k in p:
        assert np.array_equal(p[k], q[k])
