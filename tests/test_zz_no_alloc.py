"""The allocation-free norms entry point against the allocating one, through
the C ABI: the same float64 norms for two calls in a row on the library's
fixed device array, the second with fewer and smaller models (so the array
still holds the first call's partials when the second starts)."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from oracle import model as om
from paper_2110_07029_amd import synth

from gpu_util import flush, read_params

pytestmark = pytest.mark.gpu


def _models(n, F, L, seed0):
    import torch
    ms = [asgd.asgd_model_init(F, L, 8, 64, 16, gemm_bf16=False, seed=seed0 + i, stream=torch.cuda.current_stream())
          for i in range(n)]
    rng = np.random.default_rng(seed0)
    for i, m in enumerate(ms):   # models that differ in more than their seed
        asgd.asgd_model_set_params(m, asgd.ASGD_PARAM_B2, rng.normal(0, 1 + i, L).astype(np.float32))
    return ms


def test_noalloc_norms_equal_the_allocating_entry_point():
    import torch
    asgd.load()
    for n, F, L, seed0 in ((4, synth.TINY.n_features, synth.TINY.n_labels, 40), (2, 300, 70, 80)):
        flush(f"no-alloc norms: {n} models, F={F} L={L}")
        ms = _models(n, F, L, seed0)
        try:
            out = torch.full((n,), float("nan"), dtype=torch.float64, device="cuda")
            asgd.asgd_models_l2_per_param_noalloc(ms, out)
            torch.cuda.synchronize()
            got = out.cpu().numpy()
            ref = np.array(asgd.asgd_models_l2_per_param(ms))
            # same kernels and summation order; the last division runs on the device here
            assert np.all(np.abs(got - ref) <= 1e-15 * ref), (got, ref)
            for m, g in zip(ms, got):
                f = om.flat_params(read_params(m, F, L)).astype(np.float64)
                want = np.sqrt(np.sum(f * f)) / f.size
                assert abs(g - want) <= 1e-12 * want
        finally:
            for m in ms:
                asgd.asgd_model_free(m)
    m = asgd.asgd_model_init(100, 10, 8, 16, 8, gemm_bf16=False)
    try:
        out = torch.empty(17, dtype=torch.float64, device="cuda")
        with pytest.raises(asgd.AsgdError):   # beyond the array's 16 models
            asgd.asgd_models_l2_per_param_noalloc([m] * 17, out)
    finally:
        asgd.asgd_model_free(m)
