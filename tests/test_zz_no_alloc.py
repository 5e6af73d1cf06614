"""gdp_sample_noalloc (the allocation-free variant of gdp_sample, scratch in the
library's own per-device array) against gdp_sample through the C ABI: placements
and log-probs bit for bit on two calls in a row, the second on a smaller input,
then the first input again (the array keeps the previous call's contents)."""
import numpy as np
import pytest

from paper_1910_01578_amd import workloads as W

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.detach().contiguous().cpu().numpy().tobytes()


def _runner(name, **over):
    from paper_1910_01578_amd import gdp
    cfg = W.get_config(name).replace(**over)
    g, w = W.make_graph(cfg), W.make_weights(cfg)
    r = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), cfg.k_samples)
    r.embed()
    r.place()
    return cfg, r


def _compare(cfg, r, seed, use_lse=True):
    import torch
    r.sample(seed, use_lse=use_lse)
    ref_p, ref_l = r.placements.clone(), r.logp.clone()
    p = torch.full_like(r.placements, -1)
    lp = torch.full_like(r.logp, float("nan"))
    r.sample_noalloc(seed, placements=p, logp=lp, use_lse=use_lse)
    torch.cuda.synchronize()
    print(f"noalloc {cfg.name} N={r.graph.n_nodes} K={r.k} G={r.graph.n_graphs} seed={seed}", flush=True)
    assert _bits(p) == _bits(ref_p)
    assert _bits(lp) == _bits(ref_l)
    assert np.isfinite(lp.cpu().numpy()).all()


def test_noalloc_equals_sample_two_calls_second_smaller():
    big_cfg, big = _runner("superposition_4x")          # 29,000 nodes in 4 graphs, K = 16
    small_cfg, small = _runner("inception_2500")       # 2,500 nodes, K = 16
    _compare(big_cfg, big, 11)
    _compare(small_cfg, small, 12)                     # smaller: part of the array keeps the big call's sums
    _compare(big_cfg, big, 13, use_lse=False)


def test_noalloc_at_the_largest_workload():
    cfg, r = _runner("gnmt8_52000")                    # 52,000 nodes, K = 64
    _compare(cfg, r, cfg.sample_seed)
