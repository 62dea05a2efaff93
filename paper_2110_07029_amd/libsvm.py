"""Datasets from files of the Extreme Classification Repository (libSVM-style
text, the format of the paper's datasets, Sec. 5.1), parsed by the library's
native reader (``asgd_libsvm_scan`` / ``asgd_libsvm_read``), as the same host
CSR structures the synthetic generator returns; ``DeviceCSR`` then stages them
in HBM.  The real datasets are not shipped; this is for users who have them.
"""
from __future__ import annotations

import numpy as np

from . import _binding as B
from . import synth


def load(path: str, one_based: bool = False, lr: float = 0.01, batch: int = 256,
         unlabeled: str = "drop") -> synth.Dataset:
    """Read a dataset file into host CSR structures.

    Rows without labels are valid in the file format, but the training step's
    loss is undefined for them (the target distribution puts 1/|Y_i| on each
    true label), and the library rejects such a batch with ``ASGD_EINVAL``
    under ``ASGD_VALIDATE``.  ``unlabeled`` says what happens to them:
    ``"drop"`` (default) leaves them out, ``"error"`` raises ``ValueError``
    naming how many there are and the first one, ``"keep"`` keeps them (for
    prediction only).  The row count of the returned dataset is after dropping.
    """
    if unlabeled not in ("drop", "error", "keep"):
        raise ValueError(f"unlabeled must be 'drop', 'error' or 'keep', not {unlabeled!r}")
    info = B.asgd_libsvm_scan(path, one_based)
    ip, ix, va, lp, lx = B.asgd_libsvm_read(path, info, one_based)
    F, L = int(info.n_features), int(info.n_labels)
    empty = np.flatnonzero(np.diff(lp) == 0)
    if empty.size and unlabeled == "error":
        raise ValueError(f"{path}: {empty.size} rows have no labels (first: data row {int(empty[0])})")
    if empty.size and unlabeled == "drop":
        keep = np.ones(len(ip) - 1, bool)
        keep[empty] = False
        ip, ix, va = _take_rows(ip, ix, va, keep)
        lp, lx, _ = _take_rows(lp, lx, None, keep)
    w = synth.Workload(path, F, L, len(ip) - 1, batch, lr, True, "file", 0.0, 0.0, 0, 0.0, "file",
                       "file", 0.0, None, 0)
    return synth.Dataset(w, synth.CSR(ip, ix, va, F), synth.CSR(lp, lx, None, L))


def _take_rows(indptr, indices, values, keep):
    """The rows of a CSR where ``keep`` is true, in order."""
    counts = np.diff(indptr)[keep]
    entry_keep = np.repeat(keep, np.diff(indptr))
    out_ptr = np.zeros(len(counts) + 1, np.int64)
    np.cumsum(counts, out=out_ptr[1:])
    return out_ptr, indices[entry_keep], None if values is None else values[entry_keep]


def save(ds: synth.Dataset, path: str, header: bool = True):
    """Write a dataset in the repository's format (0-based ids)."""
    x, y = ds.x, ds.y
    with open(path, "w") as f:
        if header:
            f.write(f"{x.n_rows} {x.n_cols} {y.n_cols}\n")
        for i in range(x.n_rows):
            labs = ",".join(str(int(v)) for v in y.indices[y.indptr[i]:y.indptr[i + 1]])
            s, e = int(x.indptr[i]), int(x.indptr[i + 1])
            feats = " ".join(f"{int(a)}:{float(b):.9g}" for a, b in zip(x.indices[s:e], x.values[s:e]))
            f.write(f"{labs} {feats}\n" if feats else f"{labs}\n")
