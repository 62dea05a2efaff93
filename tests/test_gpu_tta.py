"""Time-to-accuracy harness on the GPU: the global model learns the planted
labels under Adaptive SGD and the elastic-averaging baseline within a short
virtual-time budget, and the records are consistent."""
import pytest

import paper_2110_07029_amd as asgd
from paper_2110_07029_amd import tta

from gpu_util import flush

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    asgd.load()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("mode", ["adaptive", "elastic"])
def test_planted_labels_are_learned_within_the_budget(mode):
    flush(f"time-to-accuracy: {mode}")
    recs = tta.run(mode, budget_s=0.25, n_train=40_000, n_test=2_000, evals=5)
    assert recs[0]["top1"] < 0.05                       # untrained: about 1 / n_labels
    assert max(r["top1"] for r in recs[-2:]) > 0.45     # well above the 0.3 of the most frequent label
    assert recs[-1]["virtual_s"] >= 0.25
    assert all(a["virtual_s"] <= b["virtual_s"] and a["samples"] <= b["samples"] for a, b in zip(recs, recs[1:]))
    if mode == "adaptive":                              # slower virtual replicas end with smaller batches
        assert recs[-1]["b"][0] >= recs[-1]["b"][-1]
    else:
        assert recs[-1]["b"] == [128] * 4
