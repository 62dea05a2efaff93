"""Oracle for one replica's SGD step on the sparse MLP (test infrastructure only).

The model is the paper's 3-layer MLP for extreme multi-label classification
(Sec. 5.1, "Datasets and Model"): a sparse input layer of F features, one
dense ReLU hidden layer of H units, and an output layer of L labels with
softmax and cross-entropy.  One SGD step is the three passes of Sec. 2.1
("Stochastic Gradient Descent"): forward, backward (chain rule) and a model
update with the learning rate.

Readings where the paper is silent (each is listed in the design notes):
* two weight matrices, F -> H (ReLU) -> L, with biases b1 and b2 (zero init);
  the other reading of "3-layer MLP", a second dense hidden layer H -> H
  (ReLU) with weights Wh [H x H] and bias bh, is available with
  ``extra_hidden_layers=1`` (its product is always exact: the bf16 rounding
  applies to the output layer only);
* multi-label target distribution T[i, y] = 1/|Y_i| on the true labels, loss
  = mean over the batch of the cross-entropy between T and the softmax;
* gradients averaged over the batch (mean), ReLU'(0) = 0;
* Xavier-uniform init from a counter-based splitmix64 stream (the paper's
  "std = number of units" init is not usable as written);
* only W1 rows whose feature occurs in the batch are written by the update.

Arithmetic is float64 on float32-stored parameters; each updated parameter is
rounded to float32 once.  With ``operands="bf16"`` the three products of the
output layer take bfloat16-rounded operands (round-to-nearest-even of the
float32 value) and are still summed in float64: Z = bf16(H1) bf16(W2)^T + b2,
dW2 = bf16(dZ)^T bf16(H1) and dH1 = bf16(dZ) bf16(W2).  Nothing else is
rounded: the softmax, the loss, dZ itself, db2 and the first layer stay in
float64.
"""
from __future__ import annotations

import numpy as np

F64 = np.float64
F32 = np.float32

# ----------------------------------------------------------------------------
# Counter-based init generator: splitmix64 (Steele, Lea & Flood, OOPSLA 2014;
# the 64-bit finalizer constants are those of the published generator).
# ----------------------------------------------------------------------------
_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

TENSOR_W1 = 0
TENSOR_W2 = 1
TENSOR_WH = 2


def splitmix64(x: np.ndarray) -> np.ndarray:
    """Output of splitmix64 for the state ``x`` (state advanced by gamma, then mixed)."""
    z = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = z + _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def init_uniform24(seed: int, tensor: int, count: int, start: int = 0) -> np.ndarray:
    """u_e = top 24 bits of splitmix64(seed ^ (tensor << 56) ^ e) times 2^-24, in [0, 1)."""
    e = np.arange(start, start + count, dtype=np.uint64)
    key = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) ^ (np.uint64(tensor) << np.uint64(56))
    z = splitmix64(e ^ key)
    return (z >> np.uint64(40)).astype(F64) * (2.0 ** -24)


def xavier_bound(fan_in: int, fan_out: int) -> np.float32:
    """Xavier-uniform half-width a = sqrt(6 / (fan_in + fan_out)), rounded to float32."""
    return F32(np.sqrt(6.0 / (fan_in + fan_out)))


def _xavier_tensor(seed: int, tensor: int, fan_in: int, fan_out: int, count: int) -> np.ndarray:
    a = xavier_bound(fan_in, fan_out)
    u = init_uniform24(seed, tensor, count)
    return (2.0 * u - 1.0).astype(F32) * a   # 2u-1 is exact in float32; one rounding in the product


def init_params(n_features: int, n_labels: int, hidden: int, seed: int, extra_hidden_layers: int = 0) -> dict:
    """W1 [F,H], W2 [L,H] (and Wh [H,H]) Xavier-uniform; biases zero.  w = fl32(fl32(2u-1) * a)."""
    p = dict(W1=_xavier_tensor(seed, TENSOR_W1, n_features, hidden, n_features * hidden).reshape(n_features, hidden),
             b1=np.zeros(hidden, F32))
    if extra_hidden_layers:
        p["Wh"] = _xavier_tensor(seed, TENSOR_WH, hidden, hidden, hidden * hidden).reshape(hidden, hidden)
        p["bh"] = np.zeros(hidden, F32)
    p["W2"] = _xavier_tensor(seed, TENSOR_W2, hidden, n_labels, n_labels * hidden).reshape(n_labels, hidden)
    p["b2"] = np.zeros(n_labels, F32)
    return p


# ----------------------------------------------------------------------------
# bfloat16 rounding (round to nearest, ties to even; NaN kept quiet)
# ----------------------------------------------------------------------------
def round_bf16(a: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 value (ties to even), returned as float32."""
    a = np.ascontiguousarray(a, dtype=F32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    r = ((bits + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = (bits[nan].astype(np.uint32) | np.uint32(0x00400000)) & np.uint32(0xFFFF0000)
    return r.view(F32)


def _operand(a: np.ndarray, operands: str) -> np.ndarray:
    if operands == "bf16":
        return round_bf16(a.astype(F32)).astype(F64)
    if operands == "fp32":
        return np.asarray(a, F64)
    raise ValueError(operands)


# ----------------------------------------------------------------------------
# CSR helpers (absolute indptr offsets, as a row slice of a larger matrix)
# ----------------------------------------------------------------------------
def row_ids(indptr: np.ndarray) -> np.ndarray:
    """Row index of every stored entry."""
    return np.repeat(np.arange(len(indptr) - 1), np.diff(np.asarray(indptr, np.int64)))


def touched_features(x) -> np.ndarray:
    """Sorted distinct feature ids occurring in the batch (the rows of W1 a step writes)."""
    s, e = int(x.indptr[0]), int(x.indptr[-1])
    return np.unique(np.asarray(x.indices[s:e], np.int64)).astype(np.int32)


def _entries(x):
    s, e = int(x.indptr[0]), int(x.indptr[-1])
    ind = np.asarray(x.indices[s:e], np.int64)
    val = None if x.values is None else np.asarray(x.values[s:e], F64)
    return ind, val, row_ids(np.asarray(x.indptr, np.int64) - s)


def targets(y, n_labels: int) -> np.ndarray:
    """Dense target distribution T [B, L]: 1/|Y_i| on each true label of row i."""
    B = len(y.indptr) - 1
    ind, _, rows = _entries(y)
    cnt = np.diff(np.asarray(y.indptr, np.int64)).astype(F64)
    T = np.zeros((B, n_labels), F64)
    np.add.at(T, (rows, ind), 1.0 / cnt[rows])
    return T


# ----------------------------------------------------------------------------
# Forward, backward, update
# ----------------------------------------------------------------------------
def forward(p: dict, x, y=None, operands: str = "fp32") -> dict:
    """A1 = X W1 + b1; H1 = ReLU(A1); [A2 = H1 Wh^T + bh; H2 = ReLU(A2)]; Z = H W2^T + b2
    with H the last hidden activation; lse; per-row and mean loss."""
    B = len(x.indptr) - 1
    ind, val, rows = _entries(x)
    A1 = np.tile(p["b1"].astype(F64), (B, 1))
    np.add.at(A1, rows, val[:, None] * p["W1"][ind].astype(F64))
    H1 = np.maximum(A1, 0.0)
    out = dict(A1=A1, H1=H1)
    Hout = H1
    if "Wh" in p:
        A2 = H1 @ p["Wh"].astype(F64).T + p["bh"].astype(F64)
        Hout = np.maximum(A2, 0.0)
        out.update(A2=A2, H2=Hout)
    Z = _operand(Hout, operands) @ _operand(p["W2"], operands).T + p["b2"].astype(F64)
    m = Z.max(axis=1)
    lse = m + np.log(np.exp(Z - m[:, None]).sum(axis=1))
    out.update(Z=Z, lse=lse)
    if y is not None:
        L = Z.shape[1]
        yind, _, yrows = _entries(y)
        cnt = np.diff(np.asarray(y.indptr, np.int64)).astype(F64)
        tz = np.zeros(B, F64)
        np.add.at(tz, yrows, Z[yrows, yind] / cnt[yrows])
        out["loss_rows"] = lse - tz
        out["loss"] = float(out["loss_rows"].mean())
    return out


def backward(p: dict, x, y, fw: dict, operands: str = "fp32") -> dict:
    """Gradients of the mean loss (chain rule through softmax-CE, W2, ReLU, W1)."""
    B, L = fw["Z"].shape
    P = np.exp(fw["Z"] - fw["lse"][:, None])
    T = targets(y, L)
    dZ = (P - T) / B
    # the two products of the output layer take their operands in `operands`:
    # with bf16, dZ (stored as float32 first), H1 and the pre-update W2 are
    # rounded; the bias gradient is a plain sum of the unrounded dZ
    dZo = _operand(dZ.astype(F32), operands) if operands == "bf16" else dZ
    extra = "Wh" in p
    dW2 = dZo.T @ _operand(fw["H2"] if extra else fw["H1"], operands)
    db2 = dZ.sum(axis=0)
    dHo = dZo @ _operand(p["W2"], operands)    # at the output layer's input; the pre-update W2
    g = dict(dZ=dZ, dW2=dW2, db2=db2)
    if extra:
        dA2 = dHo * (fw["A2"] > 0.0)
        g.update(dH2=dHo, dA2=dA2, dWh=dA2.T @ fw["H1"], dbh=dA2.sum(axis=0))
        dH1 = dA2 @ p["Wh"].astype(F64)          # the pre-update Wh
    else:
        dH1 = dHo
    dA1 = dH1 * (fw["A1"] > 0.0)
    db1 = dA1.sum(axis=0)
    ind, val, rows = _entries(x)
    T_ids, inv = np.unique(ind, return_inverse=True)
    dW1 = np.zeros((len(T_ids), p["W1"].shape[1]), F64)
    np.add.at(dW1, inv, val[:, None] * dA1[rows])
    g.update(dH1=dH1, dA1=dA1, db1=db1, touched=T_ids.astype(np.int32), dW1_rows=dW1)
    return g


def sgd_update(p: dict, g: dict, lr) -> dict:
    """theta <- fl32(theta - lr * g); W1 rows outside the touched set are not written."""
    lr = F64(F32(lr))
    q = {k: v.copy() for k, v in p.items()}
    t = g["touched"]
    q["W1"][t] = (p["W1"][t].astype(F64) - lr * g["dW1_rows"]).astype(F32)
    q["b1"] = (p["b1"].astype(F64) - lr * g["db1"]).astype(F32)
    if "Wh" in p:
        q["Wh"] = (p["Wh"].astype(F64) - lr * g["dWh"]).astype(F32)
        q["bh"] = (p["bh"].astype(F64) - lr * g["dbh"]).astype(F32)
    q["W2"] = (p["W2"].astype(F64) - lr * g["dW2"]).astype(F32)
    q["b2"] = (p["b2"].astype(F64) - lr * g["db2"]).astype(F32)
    return q


def train_step(p: dict, x, y, lr, operands: str = "fp32"):
    """One SGD step: returns (new params, mean loss before the update, grads, forward)."""
    fw = forward(p, x, y, operands)
    g = backward(p, x, y, fw, operands)
    return sgd_update(p, g, lr), fw["loss"], g, fw


def predict_topk(p: dict, x, k: int, operands: str = "fp32"):
    """Top-k labels per row ordered by (-score, label id); scores are the logits Z."""
    Z = forward(p, x, None, operands)["Z"]
    B, L = Z.shape
    ids = np.empty((B, k), np.int32)
    sc = np.empty((B, k), F64)
    lab = np.arange(L)
    for i in range(B):
        order = np.lexsort((lab, -Z[i]))[:k]
        ids[i] = order
        sc[i] = Z[i, order]
    return ids, sc


PARAM_ORDER = ("W1", "b1", "Wh", "bh", "W2", "b2")


def flat_params(p: dict) -> np.ndarray:
    """The model as one float32 vector in the order W1, b1, [Wh, bh,] W2, b2."""
    return np.concatenate([p[k].ravel() for k in PARAM_ORDER if k in p]).astype(F32)


def unflat_params(v: np.ndarray, n_features: int, n_labels: int, hidden: int,
                  extra_hidden_layers: int = 0) -> dict:
    o = 0
    out = {}
    shapes = [("W1", (n_features, hidden)), ("b1", (hidden,))]
    if extra_hidden_layers:
        shapes += [("Wh", (hidden, hidden)), ("bh", (hidden,))]
    shapes += [("W2", (n_labels, hidden)), ("b2", (n_labels,))]
    for name, shape in shapes:
        n = int(np.prod(shape))
        out[name] = np.asarray(v[o:o + n], F32).reshape(shape).copy()
        o += n
    return out
