"""The GNN with each layer's update fused to the next layer's transform
(gdp_embed on an L-layer network) against the same layers run one at a time
(L one-layer gdp_embed calls, each a separate transform, gather and update,
the previous call's node embeddings as the next call's features): node
embeddings and graph embeddings bit for bit.  The neighbour sample S(v)
depends only on the graph and the seed, so every call sees the same one."""
import numpy as np
import pytest

from paper_1910_01578_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _bits(t):
    import torch
    t = t.detach().contiguous().cpu()
    return (t.view(torch.int16) if t.dtype == torch.bfloat16 else t).numpy().tobytes()


def _embed(cfg, g, w, layers):
    from paper_1910_01578_amd import gdp
    c = cfg.replace(gnn_layers=len(layers), feat_dim=int(g.x_dev.shape[1]))
    wl = W.Weights(gnn=layers, placer=w.placer, head=w.head)
    r = gdp.Runner(gdp.DeviceGraph(g, c.dtype), gdp.DevicePolicy(c, wl), 1)
    r.embed()
    return r


def _as_features(cfg, g, node_emb):
    """The node embeddings (device, dtype of cfg) as the features of the same graph."""
    import torch
    if cfg.dtype == "bf16":
        bits = node_emb.detach().cpu().view(torch.int16).numpy().view(np.uint16).copy()
        x64, xdev = W.bf16_to_f64(bits), bits
    else:
        xdev = node_emb.detach().cpu().numpy().astype(np.float32)
        x64 = xdev.astype(np.float64)
    return W.Graph(g.graph_ptr, g.row_ptr, g.col_idx, x64, xdev)


@pytest.mark.parametrize("name", ["tiny_layered_256", "inception_2500", "superposition_4x", "gnmt8_52000"])
def test_fused_gnn_equals_layer_by_layer(name):
    import torch
    cfg = W.get_config(name)
    g, w = W.make_graph(cfg), W.make_weights(cfg)
    _log("gnn fusion", name, cfg.dtype, "H", cfg.hidden, "layers", cfg.gnn_layers)
    whole = _embed(cfg, g, w, w.gnn)
    torch.cuda.synchronize()
    gl = g
    for l in range(cfg.gnn_layers):
        one = _embed(cfg, gl, w, [w.gnn[l]])
        torch.cuda.synchronize()
        if l + 1 < cfg.gnn_layers:
            gl = _as_features(cfg, g, one.node_emb)
    assert _bits(one.node_emb) == _bits(whole.node_emb)
    assert _bits(one.graph_emb) == _bits(whole.graph_emb)
