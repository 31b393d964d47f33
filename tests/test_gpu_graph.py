"""The whole predict -> route -> prioritize step captured into a HIP graph (torch's graph capture
of the C-ABI calls on the current stream): every replay, each after the outputs were
overwritten and with eager steps and synchronisations in between, reproduces the eager step's
outputs bit for bit. Nothing in the step allocates or records a memset, so it is capturable."""
import pytest
import torch

from paper_2606_12950_amd import pipeline
from paper_2606_12950_amd import workload as W

pytestmark = pytest.mark.gpu


def _outputs(o):
    return [o.pred_len, o.kv_bytes, o.node_idx, o.score, o.remaining_us, o.slack_key, o.order]


def test_step_replays_from_a_graph_bit_for_bit():
    b = pipeline.to_device(W.workload("c3"))
    o = pipeline.allocate_outputs(b)
    pipeline.run_step(b, o)
    torch.cuda.synchronize()
    ref = [t.clone() for t in _outputs(o)]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):               # warm-up off the default stream, as capture needs
        pipeline.run_step(b, o)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        pipeline.run_step(b, o)
    torch.cuda.synchronize()

    for rep in range(4):
        for t in _outputs(o):                   # stale values must not survive a replay
            t.fill_(-1)
        if rep % 2:
            pipeline.run_step(b, o)             # eager work between replays
            torch.cuda.synchronize()
            for t in _outputs(o):
                t.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for got, want, name in zip(_outputs(o), ref, ["pred_len", "kv_bytes", "node_idx", "score", "remaining_us",
                                                       "slack_key", "order"]):
            assert torch.equal(got, want), f"replay {rep}: {name} differs from the eager step"
