"""The two-part layer schedule of gdp_place (rows below and above a segment
start on two streams, with the next layer's QKV in a second buffer) against
the one-stream schedule, bit for bit.

A batch of two copies of one graph (same node and graph embeddings) is large
enough to take the two-part schedule, while one copy alone takes the one-
stream schedule.  Every step of the placer is row-local or local to a graph's
segments, so each copy's logits, lse and final activations must equal the
single graph's exactly, whichever stream computed them."""
import ctypes

import numpy as np
import pytest

from paper_1910_01578_amd import workloads as W

pytestmark = pytest.mark.gpu

SPLIT_ROWS = 256 * 128      # part A's target size; the schedule needs N >= 1.25 x this


def _log(*a):
    print(*a, flush=True)


def _bits(t):
    import torch
    t = t.detach().contiguous().cpu()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).numpy().tobytes()


def _edgeless(sizes, feat_dim, dtype):
    n = int(sum(sizes))
    gp = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    x = np.zeros((n, feat_dim))
    xdev = np.zeros((n, feat_dim), np.uint16 if dtype == "bf16" else np.float32)
    return W.Graph(gp, np.zeros(n + 1, np.int32), np.zeros(0, np.int32), x, xdev)


def _place(cfg, w, sizes, node_emb, graph_emb, train):
    import torch
    from paper_1910_01578_amd import gdp
    r = gdp.Runner(gdp.DeviceGraph(_edgeless(sizes, cfg.feat_dim, cfg.dtype), cfg.dtype),
                   gdp.DevicePolicy(cfg, w), 1)
    r.node_emb.copy_(node_emb)
    r.graph_emb.copy_(graph_emb)
    r.logits.fill_(float("nan"))
    r.lse.fill_(float("nan"))
    x = r.place_train() if train else None
    if not train:
        r.place()
    torch.cuda.synchronize()
    return r.logits, r.lse, x


@pytest.mark.parametrize("base,n,n_dev,mem_len,train,over", [
    ("gnmt8_52000", 36000, 8, 512, False, {}),      # part A ends inside the first copy
    ("gnmt8_52000", 36000, 20, 512, True, {}),      # head in its own kernel; final activations kept
    ("gnmt8_52000", 36000, 8, 1024, False, {}),     # part B's memory reaches two segments into part A
    ("gnmt8_52000", 32768, 8, 512, True, {}),       # part A ends at the second copy's first row
    ("gnmt8_52000", 36000, 8, 0, False, {"film": False}),   # no memory, no conditioning
    ("tiny_layered_256", 36000, 4, 64, True, {"seg_len": 256}),   # fp32, d = 64
])
def test_two_part_schedule_equals_one_stream(base, n, n_dev, mem_len, train, over):
    import torch
    assert n < SPLIT_ROWS + SPLIT_ROWS // 4 <= 2 * n
    cfg = W.get_config(base).replace(graph_sizes=(n,), n_devices=n_dev, mem_len=mem_len, **over)
    w = W.make_weights(cfg)
    _log("split schedule", base, n, n_dev, mem_len, train, over)
    gen = torch.Generator().manual_seed(n + n_dev + mem_len)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    emb = torch.rand((n, cfg.hidden), generator=gen).to(tdt).cuda()
    gemb = torch.randn((1, cfg.hidden), generator=gen).cuda()
    one = _place(cfg, w, (n,), emb, gemb, train)
    two = _place(cfg, w, (n, n), torch.cat([emb, emb]), torch.cat([gemb, gemb]), train)
    for a, b in zip(one, two):
        if a is None:
            continue
        assert torch.isfinite(b).all()
        assert _bits(b[:n]) == _bits(a)
        assert _bits(b[n:]) == _bits(a)


def test_schedules_agree_on_the_52000_node_workload():
    """gdp_set_place_streams(1) against the default two-part schedule on the
    whole 52,000-node workload (embeddings from gdp_embed): logits, lse and
    the final activations bit for bit, twice in a row each."""
    import torch
    from paper_1910_01578_amd import gdp
    from tests.parity import workload
    cfg, g, w = workload("gnmt8_52000")
    _log("schedules", cfg.name)
    r = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), 1)
    r.embed()
    out = {}
    try:
        for n in (2, 1, 2, 1):
            gdp.set_place_streams(n)
            r.logits.fill_(float("nan"))
            x = r.place_train()
            torch.cuda.synchronize()
            got = (_bits(r.logits), _bits(r.lse), _bits(x))
            assert out.setdefault(n, got) == got, n
    finally:
        gdp.set_place_streams(2)
    assert out[1] == out[2]


@pytest.mark.parametrize("call", ["place", "place_sample"])
def test_first_call_under_capture_keeps_one_stream(call):
    """A thread whose first two-part gdp_place (or gdp_place_sample) call is
    captured into a HIP graph creates no stream and keeps every launch on the
    capturing stream; the replay equals the eager two-part result bit for bit."""
    import threading
    import torch
    from paper_1910_01578_amd import gdp
    from tests.parity import workload
    cfg, g, w = workload("gnmt8_52000")
    _log("capture in a fresh thread", cfg.name, call)
    r = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), 4)
    r.embed()
    run = (lambda: r.place()) if call == "place" else (lambda: r.place_sample(cfg.sample_seed))
    outs = (r.logits, r.lse) if call == "place" else (r.logits, r.lse, r.placements, r.logp)
    run()
    torch.cuda.synchronize()
    want = tuple(_bits(t) for t in outs)
    res = {}

    def work():
        try:
            torch.cuda.set_device(0)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                run()
            torch.cuda.synchronize()
            r.logits.fill_(float("nan"))
            r.placements.fill_(-1)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            res["got"] = tuple(_bits(t) for t in outs)
        except Exception as e:   # reported in the main thread
            res["err"] = e

    t = threading.Thread(target=work)
    t.start()
    t.join()
    assert "err" not in res, res.get("err")
    assert res["got"] == want
