"""Per-layer launches of base decode attention, eager and replayed from a
captured HIP graph, against the layer-batched call (layerbench.run on a small
shape): bit-equal outputs, and every one of three graph replays (eager launches
and synchronisations between them) equal to the eager per-layer result."""
import pytest
import torch

from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("D", [128, 64])
def test_per_layer_and_graph_match_batched(D):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import layerbench
    from paper_2608_15797_amd.workloads import BaseShape
    b = BaseShape(S=4, L=3, Hq=8, Hkv=2, D=D, B=16, W=4, buffer=16, prompt=0)
    r = layerbench.run(reps=3, base=b)
    say(" ", r)
    assert r["n"] == 16 + 9
    assert r["per_layer_same_as_batched"]
    assert r["graph_replays_match"]
