"""Seeded synthetic sparse extreme-multi-label datasets.

This module only draws inputs; it holds none of the training method's
arithmetic, so both the HIP path and the CPU oracle consume its output.

The shapes follow the paper's two datasets (Table 1: Amazon-670k with 135,909
features / 670,091 labels, ~76 features and ~5 labels per sample; Delicious-200k
with 782,585 features / 205,443 labels, ~302 features and ~75 labels per
sample) and two smaller cases.  The real datasets are not used; these draws
stand in for them.

Recipe, per configuration ``c`` (data seed ``1000 + c``):

* nnz per row: ``max(Poisson(20), 1)`` (tiny) or ``round(lognormal(mu, sigma))``
  clipped to ``[1, nnz_max]``;
* feature ids per row: distinct, drawn from a bounded Zipf(s) law on ranks
  ``1..F`` by inverse CDF, mapped through a seeded permutation of ``0..F-1`` so
  that hot features are scattered over W1, then sorted ascending;
* values: ``U(0,1)`` or ``exp(N(0,1))``, then L2-normalised per row (float32);
* labels: a count per row (uniform in ``1..5`` or ``1 + Poisson(lam)``, capped at
  L), distinct ids drawn uniformly or from a permuted bounded Zipf law, sorted.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

HIDDEN = 128


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_features: int
    n_labels: int
    n_samples: int
    batch: int
    lr: float
    gemm_bf16: bool
    nnz_kind: str          # "poisson" | "lognormal"
    nnz_mu: float
    nnz_sigma: float
    nnz_max: int
    feat_zipf: float
    value_kind: str        # "uniform" | "lognormal"
    label_count_kind: str  # "uniform5" | "poisson"
    label_lam: float
    label_zipf: Optional[float]  # None = uniform label ids
    index: int             # configuration number (1-based); seeds derive from it

    @property
    def data_seed(self) -> int:
        return 1000 + self.index

    @property
    def init_seed(self) -> int:
        return 2000 + self.index


TINY = Workload("tiny", 5_000, 1_000, 2_000, 128, 0.01, False,
                "poisson", 20.0, 0.0, 5_000, 1.1, "uniform", "uniform5", 0.0, None, 1)
MID = Workload("mid", 100_000, 30_000, 50_000, 256, 0.01, True,
               "lognormal", 4.0, 0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)
WIDE_FEATURE = Workload("wide-feature", 782_585, 205_443, 100_000, 128, 0.01, True,
                        "lognormal", 5.4, 0.9, 5_000, 1.05, "lognormal", "poisson", 74.0, 1.1, 3)
WIDE_LABEL = Workload("wide-label", 135_909, 670_091, 200_000, 256, 0.01, True,
                      "lognormal", 4.1, 0.7, 1_500, 1.05, "uniform", "poisson", 4.5, 1.2, 4)

WORKLOADS = {w.name: w for w in (TINY, MID, WIDE_FEATURE, WIDE_LABEL)}

# Elastic replicas: four replicas of the wide-label model, batch sizes in
# [64, 1024], merge every ~8 steps per replica, 50 rounds.
ELASTIC = dict(base="wide-label", n_replicas=4, b_min=64, b_max=1024,
               steps_per_round=8, rounds=50, index=5)


@dataclasses.dataclass
class CSR:
    """Host CSR matrix; ``indptr`` is int64 absolute offsets starting at 0."""
    indptr: np.ndarray
    indices: np.ndarray   # int32
    values: Optional[np.ndarray]  # float32 or None (label matrices)
    n_cols: int

    @property
    def n_rows(self) -> int:
        return len(self.indptr) - 1

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1] - self.indptr[0])

    def rows(self, r0: int, r1: int) -> "CSR":
        """Row slice [r0, r1) re-based to start at offset 0 (a copy)."""
        s, e = int(self.indptr[r0]), int(self.indptr[r1])
        return CSR(self.indptr[r0:r1 + 1] - s, self.indices[s:e].copy(),
                   None if self.values is None else self.values[s:e].copy(), self.n_cols)


@dataclasses.dataclass
class Dataset:
    workload: Workload
    x: CSR
    y: CSR


class _BoundedZipf:
    """Inverse-CDF sampler of P(rank r) ~ r^-s on r = 1..n, returned as 0-based
    ids through a seeded permutation."""

    def __init__(self, n: int, s: float, rng: np.random.Generator):
        w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
        cdf = np.cumsum(w)
        cdf /= cdf[-1]
        self.cdf = cdf
        self.perm = rng.permutation(n).astype(np.int64)
        self.n = n

    def draw(self, count: int, rng: np.random.Generator) -> np.ndarray:
        u = rng.random(count)
        r = np.searchsorted(self.cdf, u, side="right")
        np.minimum(r, self.n - 1, out=r)
        return self.perm[r]


def _distinct_rows(counts: np.ndarray, n_ids: int, draw, rng: np.random.Generator) -> tuple:
    """Per row i, ``counts[i]`` distinct ids from ``draw``; rows sorted ascending.

    Ids are kept in draw order (first occurrences) before the final sort, so the
    selection is not biased toward small ids.  Returns (indptr int64, ids int32).
    """
    n_rows = len(counts)
    counts = np.minimum(counts, n_ids).astype(np.int64)
    got_rows = [np.zeros(0, np.int64)] * n_rows
    need = counts.copy()
    pending = np.nonzero(need > 0)[0]
    chunks_r, chunks_i = [], []
    have = np.zeros(n_rows, np.int64)
    rounds = 0
    while len(pending):
        rounds += 1
        over = np.maximum((need[pending] * 1.25).astype(np.int64) + 4, 4)
        rows = np.repeat(pending, over)
        ids = draw(int(over.sum()))
        chunks_r.append(rows)
        chunks_i.append(ids)
        r_all = np.concatenate(chunks_r)
        i_all = np.concatenate(chunks_i)
        order_key = np.arange(len(r_all), dtype=np.int64)
        # unique (row, id) keeping the first draw
        key = r_all * n_ids + i_all
        srt = np.lexsort((order_key, key))
        ks = key[srt]
        first = np.ones(len(ks), bool)
        first[1:] = ks[1:] != ks[:-1]
        keep = srt[first]
        keep.sort()  # back to draw order
        kr = r_all[keep]
        have = np.bincount(kr, minlength=n_rows)
        need = counts - have
        pending = np.nonzero(need > 0)[0]
        chunks_r, chunks_i = [kr], [i_all[keep]]
        if rounds > 200:
            raise RuntimeError("distinct-id sampling did not converge")
    r_all, i_all = chunks_r[0], chunks_i[0]
    # take the first counts[i] draws of each row (draw order), then sort by (row, id)
    order = np.argsort(r_all, kind="stable")
    r_all, i_all = r_all[order], i_all[order]
    starts = np.zeros(n_rows + 1, np.int64)
    np.cumsum(np.bincount(r_all, minlength=n_rows), out=starts[1:])
    pos_in_row = np.arange(len(r_all), dtype=np.int64) - starts[r_all]
    sel = pos_in_row < counts[r_all]
    r_all, i_all = r_all[sel], i_all[sel]
    final = np.lexsort((i_all, r_all))
    ids = i_all[final].astype(np.int32)
    indptr = np.zeros(n_rows + 1, np.int64)
    np.cumsum(counts, out=indptr[1:])
    return indptr, ids


def _nnz_counts(w: Workload, n: int, rng: np.random.Generator) -> np.ndarray:
    if w.nnz_kind == "poisson":
        c = np.maximum(rng.poisson(w.nnz_mu, n), 1)
    else:
        c = np.rint(rng.lognormal(w.nnz_mu, w.nnz_sigma, n))
        c = np.clip(c, 1, w.nnz_max)
    return np.minimum(c.astype(np.int64), w.n_features)


def _label_counts(w: Workload, n: int, rng: np.random.Generator) -> np.ndarray:
    if w.label_count_kind == "uniform5":
        c = rng.integers(1, 6, n)
    else:
        c = 1 + rng.poisson(w.label_lam, n)
    return np.minimum(c.astype(np.int64), w.n_labels)


def generate(w: Workload, n_samples: Optional[int] = None, seed: Optional[int] = None) -> Dataset:
    """Draw the dataset of workload ``w`` (``n_samples`` overrides the size)."""
    n = w.n_samples if n_samples is None else int(n_samples)
    rng = np.random.default_rng(w.data_seed if seed is None else seed)
    fz = _BoundedZipf(w.n_features, w.feat_zipf, rng)
    counts = _nnz_counts(w, n, rng)
    indptr, ids = _distinct_rows(counts, w.n_features, lambda k: fz.draw(k, rng), rng)
    if w.value_kind == "uniform":
        vals = rng.random(len(ids))
    else:
        vals = np.exp(rng.standard_normal(len(ids)))
    row = np.repeat(np.arange(n), np.diff(indptr))
    norms = np.sqrt(np.bincount(row, weights=vals * vals, minlength=n))
    vals = (vals / norms[row]).astype(np.float32)
    x = CSR(indptr, ids, vals, w.n_features)

    lcounts = _label_counts(w, n, rng)
    if w.label_zipf is None:
        ldraw = lambda k: rng.integers(0, w.n_labels, k)
    else:
        lz = _BoundedZipf(w.n_labels, w.label_zipf, rng)
        ldraw = lambda k: lz.draw(k, rng)
    lindptr, lids = _distinct_rows(lcounts, w.n_labels, ldraw, rng)
    y = CSR(lindptr, lids, None, w.n_labels)
    return Dataset(w, x, y)


def batches(ds: Dataset, batch: int):
    """Consecutive row slices [r0, r1) covering the dataset (last may be short)."""
    n = ds.x.n_rows
    for r0 in range(0, n, batch):
        yield r0, min(n, r0 + batch)


# ---------------------------------------------------------------------------
# Planted label structure, for time-to-accuracy runs: the draws above have no
# relation between features and labels, so no model can learn them.  Here
# every label owns a signature of `sig` feature ids (drawn from the feature
# Zipf law); a row's labels are drawn as above, its features are each of its
# labels' signature features kept with probability `keep`, plus `noise`
# features from the Zipf law; values U(0,1), L2-normalised.  Top-1 accuracy
# (the best-scoring label is one of the row's labels) is then learnable.
# ---------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class Planted:
    name: str
    n_features: int
    n_labels: int
    feat_zipf: float
    label_zipf: float
    label_lam: float     # labels per row: 1 + Poisson(label_lam)
    sig: int             # signature features per label
    keep: float          # probability a signature feature appears in a row
    noise: int           # noise features per row: Poisson(noise)
    seed: int


PLANTED_SMALL = Planted("planted-small", 20_000, 2_000, 1.05, 1.1, 1.0, 8, 0.7, 12, 3001)
PLANTED_WIDE = Planted("planted-wide", 135_909, 670_091, 1.05, 1.2, 4.5, 8, 0.7, 40, 3004)


def generate_planted(p: Planted, n_samples: int, seed_offset: int = 0) -> Dataset:
    """Rows of the planted-structure dataset (``seed_offset`` draws a disjoint
    sample set, e.g. held-out rows, from the same signatures)."""
    rng_sig = np.random.default_rng(p.seed)
    fz = _BoundedZipf(p.n_features, p.feat_zipf, rng_sig)
    sig = fz.draw(p.n_labels * p.sig, rng_sig).reshape(p.n_labels, p.sig)
    lz = _BoundedZipf(p.n_labels, p.label_zipf, rng_sig)
    rng = np.random.default_rng(p.seed + 7919 * (1 + seed_offset))
    n = int(n_samples)
    lcounts = np.minimum(1 + rng.poisson(p.label_lam, n), p.n_labels).astype(np.int64)
    lindptr, lids = _distinct_rows(lcounts, p.n_labels, lambda k: lz.draw(k, rng), rng)
    row_l = np.repeat(np.arange(n), np.diff(lindptr))
    cand_f = sig[lids].reshape(-1)
    cand_r = np.repeat(row_l, p.sig)
    kept = rng.random(len(cand_f)) < p.keep
    nz = rng.poisson(p.noise, n)
    noise_r = np.repeat(np.arange(n), nz)
    noise_f = fz.draw(int(nz.sum()), rng)
    r_all = np.concatenate([cand_r[kept], noise_r])
    f_all = np.concatenate([cand_f[kept], noise_f]).astype(np.int64)
    # distinct (row, feature), sorted; rows left empty get one noise feature
    key = np.unique(r_all * p.n_features + f_all)
    rows, feats = key // p.n_features, key % p.n_features
    empty = np.setdiff1d(np.arange(n), rows)
    if len(empty):
        extra = fz.draw(len(empty), rng)
        key = np.unique(np.concatenate([key, empty * p.n_features + extra]))
        rows, feats = key // p.n_features, key % p.n_features
    indptr = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(rows, minlength=n), out=indptr[1:])
    vals = rng.random(len(feats))
    norms = np.sqrt(np.bincount(rows, weights=vals * vals, minlength=n))
    vals = (vals / norms[rows]).astype(np.float32)
    x = CSR(indptr, feats.astype(np.int32), vals, p.n_features)
    y = CSR(lindptr, lids, None, p.n_labels)
    w = Workload(p.name, p.n_features, p.n_labels, n, 256, 0.01, True, "planted", 0.0, 0.0, 0,
                 p.feat_zipf, "uniform", "poisson", p.label_lam, p.label_zipf, 0)
    return Dataset(w, x, y)
