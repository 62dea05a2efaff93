"""Per-kernel timing through the C ABI: the output layer's forward and backward
(timed by events that their launch completes at the kernel's own start and
end) and the gather (timed by events recorded around its launch) each report
one positive duration per timed launch, shorter than the wall time of the
steps; reading a group resets it, and no launch is timed once timing is off."""
import time

import pytest

import paper_2110_07029_amd as asgd
from paper_2110_07029_amd import synth

from gpu_util import Setup, flush

pytestmark = pytest.mark.gpu

# bf16 operands; B = 256 runs the staged backward, B = 384 the chunked one
TIMED = synth.Workload("timing-mid", 20_000, 3_000, 2_048, 384, 0.01, True, "lognormal", 4.0,
                       0.8, 2_000, 1.05, "uniform", "poisson", 4.0, 1.2, 2)


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("B", [256, 384])
def test_kernel_timing_counts_and_resets(B):
    import torch
    flush(f"timing: three steps of {B} rows")
    s = Setup(TIMED, 2_048, B)
    try:
        groups = [asgd.KERNELS.index(k) for k in ("out_fwd", "out_bwd", "gather")]
        asgd.asgd_train_step(s.m, s.xb(0, B), s.yb(0, B), 0.01)  # untimed first step
        torch.cuda.synchronize()
        asgd.asgd_model_set_timing(s.m, True)
        t0 = time.perf_counter()
        for i in range(3):
            asgd.asgd_train_step(s.m, s.xb(B * (i + 1), B * (i + 2)), s.yb(B * (i + 1), B * (i + 2)), 0.01)
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        for k in groups:
            tot, n = asgd.asgd_model_get_timing(s.m, k)
            assert n == 3, (asgd.KERNELS[k], n)
            assert 0.0 < tot < wall_ms, (asgd.KERNELS[k], tot, wall_ms)
            assert asgd.asgd_model_get_timing(s.m, k) == (0.0, 0), asgd.KERNELS[k]
        asgd.asgd_model_set_timing(s.m, False)
        asgd.asgd_train_step(s.m, s.xb(0, B), s.yb(0, B), 0.01)
        torch.cuda.synchronize()
        for k in groups:
            assert asgd.asgd_model_get_timing(s.m, k) == (0.0, 0), asgd.KERNELS[k]
    finally:
        s.free()
