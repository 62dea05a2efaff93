"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, rejects bad host arguments, and its host-only Alg. 1 / Alg. 2
functions agree exactly with the oracle.  No GPU work is issued here."""
import os
import re

import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import elastic as oe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    text = open(os.path.join(ROOT, "include", "asgd.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(asgd_[a-z0-9_]+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    lib = asgd.load()
    declared = header_symbols()
    assert len(declared) >= 15
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(asgd.EXPORTS) == declared


def test_exported_symbols_are_plain_c():
    # extern "C": unmangled names in the dynamic symbol table
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", asgd.library_path()],
                         capture_output=True, text=True).stdout
    names = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for s in header_symbols():
        assert s in names


def test_host_argument_errors_without_gpu():
    with pytest.raises(asgd.AsgdError) as e:
        asgd.asgd_scale_batches([1, 2], [10, 10], [0.1, 0.1], 20, 10, 1.0)
    assert e.value.status == asgd.ASGD_EINVAL
    with pytest.raises(asgd.AsgdError):
        asgd.asgd_merge_weights([1, 1], [0, 0])          # batch sizes sum to zero
    with pytest.raises(asgd.AsgdError):
        asgd.asgd_merge_weights([1, 2], [1, 1], mode=asgd.ASGD_WEIGHTS_SAMPLES)  # no samples
    assert "samples" in asgd.asgd_last_error()


def test_alg1_library_equals_oracle():
    rng = np.random.default_rng(5)
    for _ in range(500):
        n = int(rng.integers(1, 9))
        u = [int(v) for v in rng.integers(0, 30, n)]
        b = [int(v) for v in rng.integers(64, 1025, n)]
        lr = [float(np.float32(v)) for v in rng.uniform(1e-3, 1e-1, n)]
        beta = float(rng.choice([32.0, 64.0, 7.5, 0.5]))
        nb_o, nlr_o = oe.scale_batches(u, b, lr, 64, 1024, beta)
        nb_l, nlr_l = asgd.asgd_scale_batches(u, b, lr, 64, 1024, beta)
        assert nb_l == nb_o
        assert nlr_l == nlr_o


def test_alg2_library_equals_oracle():
    rng = np.random.default_rng(6)
    for _ in range(500):
        n = int(rng.integers(1, 9))
        u = [int(v) for v in rng.integers(1, 6, n)]
        b = [int(v) for v in rng.integers(64, 1025, n)]
        s = [int(ui * bi) for ui, bi in zip(u, b)]
        mode = int(rng.integers(0, 2))
        g = None if rng.random() < 0.3 else [float(v) for v in rng.uniform(0, 0.15, n)]
        a_o = oe.merge_weights(u, b, s, mode, g, 0.1, 0.1)
        a_l = asgd.asgd_merge_weights(u, b, s, mode, g, 0.1, 0.1)
        assert np.array_equal(a_o, a_l), (u, b, mode, g, a_o, a_l)
