"""Device-resident CSR datasets whose batches are zero-copy row slices.

The whole synthetic dataset is staged once in HBM (torch tensors are used only
as device memory); a batch handed to the library is a pointer into the
dataset's indptr plus the host's nnz count for that slice.
"""
from __future__ import annotations

import numpy as np

from ._binding import asgd_csr


class DeviceCSR:
    def __init__(self, csr, device="cuda"):
        import torch
        indptr = np.asarray(csr.indptr, np.int64)
        if indptr[-1] >= 2 ** 31:
            raise ValueError("dataset has more than 2^31 entries")
        self.indptr_host = indptr
        self.n_cols = int(csr.n_cols)
        self.n_rows = len(indptr) - 1
        self.indptr = torch.from_numpy(indptr.astype(np.int32)).to(device)
        self.indices = torch.from_numpy(np.asarray(csr.indices, np.int32)).to(device)
        self.values = None if csr.values is None else torch.from_numpy(
            np.asarray(csr.values, np.float32)).to(device)

    def batch(self, r0: int, r1: int) -> asgd_csr:
        """Rows [r0, r1) as an asgd_csr (indptr offsets stay absolute)."""
        if not (0 <= r0 < r1 <= self.n_rows):
            raise ValueError("row range out of bounds")
        nnz = int(self.indptr_host[r1] - self.indptr_host[r0])
        return asgd_csr(r1 - r0, self.n_cols, nnz, self.indptr.data_ptr() + 4 * r0,
                        self.indices.data_ptr(),
                        None if self.values is None else self.values.data_ptr())

    def nnz(self, r0: int, r1: int) -> int:
        return int(self.indptr_host[r1] - self.indptr_host[r0])
