"""A probe + refresh step recorded into a HIP graph (driver.capture) and
replayed: every replay, with eager steps and host synchronisations between
the replays, reproduces the eager step's anchors, scores and refreshed rows
bit for bit (same kernels, same inputs, fixed summation orders)."""

import pytest
import torch

import workloads as W
from paper_2608_26140_amd import driver as D
from paper_2608_26140_amd import workload as WL
from tests.oracle_side import anchor_count

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["mini-stack", "tiny-f32"])
def test_graph_replay_matches_eager(name):
    torch.cuda.set_device(0)
    w = W.get_config(name)
    batch = WL.build(w, keep_host=False).batch
    k = anchor_count(w)

    def step():
        anchors, scores = batch.select_anchors(k)
        x, _ = batch.refresh(anchors, k)
        return anchors, scores, x

    def eager():
        a, sc, x = step()
        torch.cuda.synchronize()
        return a.clone(), sc.clone(), x.clone()

    ref = eager()
    again = eager()  # the step reads nothing it writes: two eager steps agree
    for r, g in zip(ref, again):
        assert torch.equal(r, g)

    graph, out = D.capture(step)
    torch.cuda.synchronize()
    for i in range(3):
        for t in out:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        for what, r, g in zip(("anchors", "scores", "rows"), ref, out):
            assert torch.equal(r, g), f"replay {i}: {what} differ from the eager step"
        mid = eager()  # eager work between replays
        for r, g in zip(ref, mid):
            assert torch.equal(r, g)
