"""One step of the hot path captured into a HIP graph (torch.cuda.CUDAGraph):
the library allocates nothing and records no memset, so the step replays.
At 52,000 nodes the placer's two-part schedule forks to its second stream
and joins back inside the capture.
Every replay, with eager work of another seed between replays, must give the
eager step's logits, placements and log-probs bit for bit."""
import sys

import pytest

from paper_1910_01578_amd import workloads as W
from tests.parity import workload

pytestmark = pytest.mark.gpu


def _bits(t):
    import torch
    return t.detach().contiguous().cpu().view(torch.uint8).numpy().tobytes()


@pytest.mark.parametrize("name", ["tiny_layered_256", "superposition_4x", "gnmt8_52000"])
def test_step_graph_replays_equal_eager(name):
    import torch
    from paper_1910_01578_amd import gdp
    cfg, g, w = workload(name)
    print("graph replay", name, flush=True)
    sys.stdout.flush()
    r = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), cfg.k_samples)
    seed = cfg.sample_seed
    r.forward(seed)
    torch.cuda.synchronize()
    ref = (_bits(r.logits), _bits(r.placements), _bits(r.logp), _bits(r.node_emb))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        r.forward(seed)                     # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        r.forward(seed)
    torch.cuda.synchronize()
    for rep in range(3):
        r.forward(seed + 1 + rep)            # eager work between replays overwrites the outputs
        torch.cuda.synchronize()
        assert _bits(r.placements) != ref[1]
        graph.replay()
        torch.cuda.synchronize()
        got = (_bits(r.logits), _bits(r.placements), _bits(r.logp), _bits(r.node_emb))
        assert got == ref, rep
