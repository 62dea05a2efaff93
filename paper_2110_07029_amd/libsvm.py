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


def load(path: str, one_based: bool = False, lr: float = 0.01, batch: int = 256) -> synth.Dataset:
    info = B.asgd_libsvm_scan(path, one_based)
    ip, ix, va, lp, lx = B.asgd_libsvm_read(path, info, one_based)
    F, L = int(info.n_features), int(info.n_labels)
    w = synth.Workload(path, F, L, int(info.n_rows), batch, lr, True, "file", 0.0, 0.0, 0, 0.0, "file",
                       "file", 0.0, None, 0)
    return synth.Dataset(w, synth.CSR(ip, ix, va, F), synth.CSR(lp, lx, None, L))


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
