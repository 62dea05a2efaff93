"""Helpers shared by the GPU parity tests: stage a synthetic dataset on the
device, build models through the C ABI, read parameters back and compare
parameter updates with the oracle's."""
from __future__ import annotations

import numpy as np

import paper_2110_07029_amd as asgd
from paper_2110_07029_amd import synth

H = asgd.HIDDEN

# Tolerances of the parity bar: relative 1e-4 for fp32 products and 2e-2 for
# bf16-operand products.  Elementwise the bound is rtol * (|ref| + mag), where
# mag is the same sum taken over absolute values (|a|^T |b| for a product):
# the standard forward-error bound of a dot product, which stays meaningful for
# entries that cancel to near zero; plus two float32 ulps of the stored weight
# for the final rounding of the update.  Normwise: ||err|| <= rtol ||ref||.
RTOL_FP32 = 1e-4
RTOL_BF16 = 2e-2


def flush(msg: str):
    print(msg, flush=True)


SELECT = {"W1": asgd.ASGD_PARAM_W1, "b1": asgd.ASGD_PARAM_B1, "Wh": asgd.ASGD_PARAM_WH,
          "bh": asgd.ASGD_PARAM_BH, "W2": asgd.ASGD_PARAM_W2, "b2": asgd.ASGD_PARAM_B2}


def read_params(m, F, L, extra=False) -> dict:
    """Parameters in the oracle's order (W1, b1, [Wh, bh,] W2, b2)."""
    shapes = {"W1": (F, H), "b1": (H,), "Wh": (H, H), "bh": (H,), "W2": (L, H), "b2": (L,)}
    names = ["W1", "b1"] + (["Wh", "bh"] if extra else []) + ["W2", "b2"]
    return {k: asgd.asgd_model_get_params(m, SELECT[k], shapes[k]) for k in names}


def write_params(m, p: dict):
    for k, v in p.items():
        asgd.asgd_model_set_params(m, SELECT[k], v)


def max_batch_nnz(csr, batch: int) -> int:
    """Largest nnz of any window of `batch` consecutive rows (batches may start
    at any row, e.g. in the elastic dispatch)."""
    ip = np.asarray(csr.indptr, np.int64)
    n = len(ip) - 1
    b = min(batch, n)
    return int(np.max(ip[b:] - ip[:n - b + 1])) if n else 0


class Setup:
    """A dataset staged on the device plus a model sized for it."""

    def __init__(self, w: synth.Workload, n_samples: int, batch: int, bf16=None, flags=0, seed=None,
                 ds=None, max_batch=None, extra=0):
        import torch
        self.w = w
        self.ds = ds if ds is not None else synth.generate(w, n_samples=n_samples)
        self.batch = batch
        self.bf16 = w.gemm_bf16 if bf16 is None else bf16
        self.F, self.L = w.n_features, w.n_labels
        self.dx = asgd.DeviceCSR(self.ds.x)
        self.dy = asgd.DeviceCSR(self.ds.y)
        mb = max_batch or batch
        self.max_nnz = max(max_batch_nnz(self.ds.x, mb), 1)
        self.max_lnnz = max(max_batch_nnz(self.ds.y, mb), 1)
        self.seed = w.init_seed if seed is None else seed
        self.extra = extra
        self.m = asgd.asgd_model_init(self.F, self.L, mb, self.max_nnz, self.max_lnnz,
                                      gemm_bf16=self.bf16, seed=self.seed, flags=flags,
                                      stream=torch.cuda.current_stream(), extra_hidden_layers=extra)
        self.stream = torch.cuda.current_stream()

    def free(self):
        if self.m:
            asgd.asgd_model_free(self.m)
            self.m = None

    def xb(self, r0, r1):
        return self.dx.batch(r0, r1)

    def yb(self, r0, r1):
        return self.dy.batch(r0, r1)

    def host_batch(self, r0, r1):
        return self.ds.x.rows(r0, r1), self.ds.y.rows(r0, r1)

    def params(self):
        return read_params(self.m, self.F, self.L, self.extra)


def update_error(before, gpu, ref):
    """(max elementwise excess ratio, normwise relative error) of the update gpu-before vs ref-before."""
    b = before.astype(np.float64)
    d_g = gpu.astype(np.float64) - b
    d_r = ref.astype(np.float64) - b
    mag = np.maximum.reduce([np.abs(before), np.abs(gpu), np.abs(ref)]).astype(np.float32)
    ulp = np.spacing(mag).astype(np.float64)
    rms = float(np.sqrt(np.mean(d_r * d_r))) if d_r.size else 0.0
    err = np.abs(d_g - d_r)
    return err, d_r, ulp, rms


def assert_update_close(name, before, gpu, ref, rtol, mag=None, norm_rtol=None):
    """Elementwise |err| <= rtol (|ref| + mag) + 2 ulp and normwise ||err|| <= norm_rtol ||ref||
    (norm_rtol defaults to rtol)."""
    err, d_r, ulp, rms = update_error(before, gpu, ref)
    floor = 0.1 * rms if mag is None else np.asarray(mag, np.float64)
    bound = rtol * (np.abs(d_r) + floor) + 2.0 * ulp
    bad = err > bound
    nref = float(np.linalg.norm(d_r))
    nerr = float(np.linalg.norm(err))
    if bad.any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())} of {err.size} elements outside the bound; worst "
                             f"at {i}: err {err[i]:.3e} bound {bound[i]:.3e} ref {d_r[i]:.3e}")
    nr = rtol if norm_rtol is None else norm_rtol
    assert nerr <= nr * nref + 2.0 * float(np.linalg.norm(ulp)), (name, nerr, nref)


# Against the oracle that rounds the same operands to bf16: the kernel's fp32
# accumulation order differs, which can move a value across a bf16 rounding
# boundary; a flipped rounding of one dZ or H1 operand changes that product term
# by at most 2^-7 of its magnitude, so elementwise the bound is 2 * 2^-7 * mag;
# normwise (rare flips, no systematic error) it stays 2e-3.
RTOL_EMU_ELEM = 2.0 * 2.0 ** -7
RTOL_EMU_NORM = 2e-3


def assert_rel_close(name, got, ref, rtol, floor_frac=0.1):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    err = np.abs(got - ref)
    bound = rtol * (np.abs(ref) + floor_frac * rms) + 1e-30
    if (err > bound).any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{name}: worst at {i}: got {got[i]!r} ref {ref[i]!r} err {err[i]:.3e} "
                             f"bound {bound[i]:.3e}")


def step_magnitudes(p, x, y, g, fw, lr):
    """|lr| times each parameter gradient evaluated on absolute values along the whole
    chain: |dZ| <= (P + T)/B, |dH| <= (P + T)|W2|/B at the output layer's input; with
    the second hidden layer |dA2| <= |dH| [A2 > 0] and |dH1| <= |dA2||Wh|; |dA1| <=
    |dH1| [A1 > 0], then |X|^T |dA1| for W1 and sums over rows for the biases."""
    from oracle.model import row_ids, targets
    s0, e0 = int(x.indptr[0]), int(x.indptr[-1])
    ind = np.asarray(x.indices[s0:e0], np.int64)
    val = np.abs(np.asarray(x.values[s0:e0], np.float64))
    rows = row_ids(np.asarray(x.indptr, np.int64) - s0)
    B, L = fw["Z"].shape
    P = np.exp(fw["Z"] - fw["lse"][:, None])
    PT = (P + targets(y, L)) / B
    dHm = PT @ np.abs(p["W2"]).astype(np.float64)
    lr = abs(float(lr))
    out = {}
    Hin = fw["H1"]
    if "Wh" in p:
        dA2m = dHm * (fw["A2"] > 0)
        out.update(Wh=lr * (dA2m.T @ np.abs(fw["H1"])), bh=lr * dA2m.sum(0))
        dHm = dA2m @ np.abs(p["Wh"]).astype(np.float64)
        Hin = fw["H2"]
    dA1m = dHm * (fw["A1"] > 0)
    inv = np.searchsorted(g["touched"], ind)
    mW1 = np.zeros((len(g["touched"]), dA1m.shape[1]))
    np.add.at(mW1, inv, val[:, None] * dA1m[rows])
    out.update(W2=lr * (PT.T @ np.abs(Hin)), b2=lr * PT.sum(0), b1=lr * dA1m.sum(0), W1=lr * mW1)
    return out


def a1_bound(p, x):
    """Rigorous bound for A1 = b1 + X W1 summed in float32 in any order, products
    exact inside fma: row i has n_i + 1 terms, so |err| <= gamma_{n_i} (|b1| + |X| |W1|)
    <= (n_i + 2) u (|b1| + |X| |W1|) per row."""
    from oracle.model import row_ids
    s0, e0 = int(x.indptr[0]), int(x.indptr[-1])
    ind = np.asarray(x.indices[s0:e0], np.int64)
    val = np.abs(np.asarray(x.values[s0:e0], np.float64))
    rows = row_ids(np.asarray(x.indptr, np.int64) - s0)
    B = len(x.indptr) - 1
    mag = np.tile(np.abs(p["b1"]).astype(np.float64), (B, 1))
    np.add.at(mag, rows, val[:, None] * np.abs(p["W1"][ind]).astype(np.float64))
    n = np.diff(np.asarray(x.indptr, np.int64)).astype(np.float64)
    return ((n + 2.0) * 2.0 ** -24)[:, None] * mag


def h1_flip_logit_bound(p, x, fw, labels=None):
    """Largest change of a logit that rounding H1 to bf16 can make between the
    kernel and the oracle.  The kernel's float32 A1 lies within a1_bound of the
    exact A1, and ReLU, float32 and bf16 rounding are monotonic, so its bf16 H1
    lies between the roundings of the interval's ends; d = the larger distance
    from the oracle's bf16 H1 (zero unless the interval straddles a rounding
    boundary).  Returns d |W2_bf16|^T, (B, L) or (B, len(labels))."""
    from oracle.model import round_bf16
    A1 = np.asarray(fw["A1"], np.float64)
    e = a1_bound(p, x)
    rb = lambda a: round_bf16(np.maximum(a, 0.0).astype(np.float32)).astype(np.float64)
    h = rb(A1)
    d = np.maximum(np.abs(rb(A1 + e) - h), np.abs(rb(A1 - e) - h))
    W2 = p["W2"] if labels is None else p["W2"][labels]
    aw = np.abs(round_bf16(np.asarray(W2, np.float32)).astype(np.float64))
    out = np.zeros((A1.shape[0], aw.shape[0]))
    rows = np.flatnonzero(d.any(axis=1))
    if rows.size:
        out[rows] = d[rows] @ aw.T
    return out
