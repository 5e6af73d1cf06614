"""CPU checks of bench.py's host logic: the one-GPU guard, the algorithmic work
model the roofline figures divide by, and the staleness rule for the recorded
HBM counters."""
import json
import os
import subprocess
import sys
import types

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1910_01578_amd import workloads as W  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def _keys_brute(gp, S, M):
    """Keys of every query, one query at a time: the band [max(g0, q0 - M), q1)."""
    total = 0
    for gi in range(len(gp) - 1):
        g0, g1 = int(gp[gi]), int(gp[gi + 1])
        for q in range(g0, g1):
            q0 = g0 + ((q - g0) // S) * S
            q1 = min(q0 + S, g1)
            total += q1 - max(g0, q0 - M)
    return total


def test_attention_keys_match_per_query_count():
    cfg = W.get_config("tiny_layered_256").replace(graph_sizes=(300, 57, 1, 130), seg_len=64, mem_len=40)
    gp = np.concatenate([[0], np.cumsum(cfg.graph_sizes)])
    g = types.SimpleNamespace(n_nodes=int(gp[-1]), graph_ptr=gp)
    work, keys = bench.flop_model(cfg, g, {"sum_s": 0})
    assert keys == _keys_brute(gp, 64, 40)
    assert work["seg_attention"] == ("mfma", 4.0 * cfg.d_model * keys)


def test_headline_workload_work_model():
    """The figures the kernel table quotes for the 52,000-node workload."""
    cfg = W.get_config("gnmt8_52000")
    gp = np.array([0, 52000])
    g = types.SimpleNamespace(n_nodes=52000, graph_ptr=gp)
    work, keys = bench.flop_model(cfg, g, {"sum_s": 207816})
    assert keys == 52921344 == _keys_brute(gp, cfg.seg_len, cfg.mem_len)
    N, d, dff, L = 52000, cfg.d_model, cfg.d_ff, cfg.placer_layers
    assert abs(work["post_attn"][1] / 1e9 - 78.4) < 0.05
    want = 2.0 * N * d * d + 4.0 * N * d * dff + (L - 1) / L * 6.0 * N * d * d
    assert abs(work["post_attn"][1] - want) <= 1e-12 * want
    assert work["gather_max"][0] == "hbm" and abs(work["gather_max"][1] / 1e6 - 134.07) < 0.005


def test_split_layer_work_model():
    """With each layer's kernels launched over two row ranges (the GNN's layer-0
    transform stays one launch), the work per launch is the step's work over
    twice the launches: totals are unchanged."""
    cfg = W.get_config("gnmt8_52000")
    g = types.SimpleNamespace(n_nodes=52000, graph_ptr=np.array([0, 52000]))
    L = cfg.placer_layers
    G = cfg.gnn_layers
    one, _ = bench.flop_model(cfg, g, {"sum_s": 1000}, fused_gnn=True)
    two, _ = bench.flop_model(cfg, g, {"sum_s": 1000}, fused_gnn=True,
                              launches={"pre_layer": 2, "seg_attention": 2 * L, "post_attn": 2 * L,
                                        "gather_max": 2 * G, "gemm_update_pool": 2 * (G - 1), "gemm_update_relu": 2})
    for k in ("pre_layer", "seg_attention", "post_attn", "gather_max", "gemm_update_pool", "gemm_update_relu"):
        assert abs(2 * two[k][1] - one[k][1]) <= 1e-12 * one[k][1]
    assert two["gemm_pool_sigmoid"] == one["gemm_pool_sigmoid"]


def test_fused_gnn_work_model():
    """With the update of layer l fused to the transform of layer l + 1, the
    three GNN kinds together still count every layer's products once."""
    cfg = W.get_config("gnmt8_52000")
    g = types.SimpleNamespace(n_nodes=52000, graph_ptr=np.array([0, 52000]))
    N, H, F, L = 52000, cfg.hidden, cfg.feat_dim, cfg.gnn_layers
    plain, _ = bench.flop_model(cfg, g, {"sum_s": 0})
    fused, _ = bench.flop_model(cfg, g, {"sum_s": 0}, fused_gnn=True)
    total_plain = L * (plain["gemm_pool_sigmoid"][1] + plain["gemm_update_relu"][1])
    total_fused = fused["gemm_pool_sigmoid"][1] + fused["gemm_update_relu"][1] + (L - 1) * fused["gemm_update_pool"][1]
    assert abs(total_fused - total_plain) <= 1e-6 * total_plain
    assert fused["gemm_pool_sigmoid"][1] == 2.0 * N * F * H                       # layer 0 only
    # launch l: layer l's update (layer 0 reads the F input features) and layer l + 1's transform
    per_launch = [2.0 * N * ((F if l == 0 else H) + H) * H + 2.0 * N * H * H for l in range(L - 1)]
    assert abs(fused["gemm_update_pool"][1] - sum(per_launch) / (L - 1)) <= 1e-9 * per_launch[0]


def test_recorded_traffic_goes_stale_with_its_source(monkeypatch):
    rec = bench.measured_traffic("post_attn")
    if rec is not None:
        assert abs(rec["bytes_per_launch"] - rec["fetch_bytes"] - rec["write_bytes"]) <= 1   # each rounded
    # the same record checked against another source file no longer applies
    monkeypatch.setitem(bench.KERNEL_SOURCES, "post_attn", "ppo.hip")
    assert bench.measured_traffic("post_attn") is None
    assert bench.measured_traffic("no_such_kernel") is None
