"""Pins of the gradient oracle (oracle/policy_grad.py) to things other than
itself: central finite differences of the float64 numpy forward oracle (with
the memory rows frozen at their recorded values, the stop-gradient of Section
3.2), the forward oracle's own logits, the chain rule between the stages, and
torch.optim.Adam for the update step."""
import numpy as np
import pytest
import torch

from oracle import gdp_oracle as O
from oracle import policy_grad as PG
from paper_1910_01578_amd import workloads as W


def _small(**over):
    c = W.get_config("tiny_layered_256").replace(**over)
    g = W.make_graph(c)
    w = W.make_weights(c)
    gnn, pl, hd = w.f64()
    return c, g, gnn, pl, hd


def _placer_numpy(node_emb, x0, gp, pl, hd, heads, S, M, film, mems_in=None, record=None, attention=True):
    """The forward oracle's segment loop with the memory read from mems_in when given
    (frozen), recording what each (graph, segment, layer) used."""
    gamma, beta = O.film_params(x0, pl, film)
    N, d = node_emb.shape
    out = np.zeros((N, d))
    for g in range(len(gp) - 1):
        gs, ge = int(gp[g]), int(gp[g + 1])
        if not attention:
            x = node_emb[gs:ge]
            for l, lw in enumerate(pl):
                y = gamma[g, l] * x + beta[g, l]
                x = O.layer_norm(y + O.ffn(y, lw), lw["ln2_g"], lw["ln2_b"])
            out[gs:ge] = x
            continue
        cache = [np.zeros((0, d)) for _ in pl]
        for q0 in range(gs, ge, S):
            q1 = min(q0 + S, ge)
            x = node_emb[q0:q1]
            for l, lw in enumerate(pl):
                y = gamma[g, l] * x + beta[g, l]
                mem = mems_in[(g, q0, l)] if mems_in is not None else cache[l]
                if record is not None:
                    record[(g, q0, l)] = mem.copy()
                ctx = np.concatenate([cache[l], y], axis=0)
                cache[l] = ctx[max(0, len(ctx) - M):] if M > 0 else np.zeros((0, d))
                x = O.transformer_block(y, np.concatenate([mem, y], axis=0), lw, heads)
            out[q0:q1] = x
    return out @ hd["w_out"].T + hd["b_out"]


def _fd_check(loss, params, grads, rng, eps=1e-6, n_dirs=2, rtol=1e-6):
    """Central differences along random directions of every parameter tensor (a
    small step: larger ones cross ReLU kinks of the feed-forward layers)."""
    for key in params:
        for _ in range(n_dirs):
            base = params[key].copy()
            delta = rng.normal(size=base.shape)
            params[key] = base + eps * delta
            lp = loss()
            params[key] = base - eps * delta
            lm = loss()
            params[key] = base
            fd = (lp - lm) / (2 * eps)
            an = float((grads[key] * delta).sum())
            assert abs(fd - an) <= rtol * max(1.0, abs(an)), (key, fd, an)


@pytest.mark.parametrize("S,M,film", [(16, 16, True), (16, 40, False), (24, 8, True)])
def test_placer_gradient_equals_finite_differences_with_frozen_memory(S, M, film):
    c, g, gnn, pl, hd = _small(placer_layers=2)
    rng = np.random.default_rng(0)
    N, d = 70, c.d_model
    gp = np.array([0, 45, N])
    ne = rng.normal(size=(N, d))
    x0 = rng.normal(size=(2, d)) * 0.5
    dl = rng.normal(size=(N, c.n_devices))
    rec = {}
    logits = _placer_numpy(ne, x0, gp, pl, hd, c.heads, S, M, film, record=rec)
    out = PG.placer_backward(ne, x0, gp, pl, hd["w_out"], hd["b_out"], dl, n_heads=c.heads, seg_len=S, mem_len=M,
                             film=film)
    np.testing.assert_allclose(out["logits"], logits, rtol=0, atol=1e-11)
    # every weight of both layers, the head, the node and graph embeddings
    params = {}
    grads = {}
    for l, lw in enumerate(pl):
        for k in lw:
            if not film and k.startswith("film"):
                continue
            params[(l, k)] = lw[k]
            grads[(l, k)] = out["placer"][l][k]
    params["w_out"], grads["w_out"] = hd["w_out"], out["head"]["w_out"]
    params["ne"], grads["ne"] = ne, out["dnode_emb"]
    if film:
        params["x0"], grads["x0"] = x0, out["dgraph_emb"]

    def loss():
        pls = [{k: params.get((l, k), lw[k]) for k in lw} for l, lw in enumerate(pl)]
        hds = {"w_out": params["w_out"], "b_out": hd["b_out"]}
        return float((_placer_numpy(params["ne"], params.get("x0", x0), gp, pls, hds, c.heads, S, M, film,
                                    mems_in=rec) * dl).sum())
    _fd_check(loss, params, grads, rng)


def test_memory_is_detached():
    """With memory the gradient differs from the derivative of the unfrozen forward
    (the plain derivative would pass gradient into earlier segments)."""
    c, g, gnn, pl, hd = _small(placer_layers=1)
    rng = np.random.default_rng(1)
    N, d = 40, c.d_model
    gp = np.array([0, N])
    ne = rng.normal(size=(N, d))
    x0 = np.zeros((1, d))
    dl = np.zeros((N, c.n_devices))
    dl[30:] = rng.normal(size=(10, c.n_devices))      # only the last segment's logits matter
    out = PG.placer_backward(ne, x0, gp, pl, hd["w_out"], hd["b_out"], dl, n_heads=c.heads, seg_len=10,
                             mem_len=20, film=False)
    # rows 0..29 feed the last segment only as memory: no gradient reaches them
    assert np.all(out["dnode_emb"][:30] == 0.0)
    assert np.abs(out["dnode_emb"][30:]).max() > 0
    # but the memory's keys and values still carry gradient into W_qkv's K and V rows
    eps, base = 1e-6, pl[0]["w_qkv"].copy()
    delta = np.zeros_like(base)
    delta[d:3 * d] = rng.normal(size=(2 * d, d))
    rec = {}
    _placer_numpy(ne, x0, gp, pl, hd, c.heads, 10, 20, False, record=rec)

    def loss(wq):
        p2 = [dict(pl[0], w_qkv=wq)]
        return float((_placer_numpy(ne, x0, gp, p2, hd, c.heads, 10, 20, False, mems_in=rec) * dl).sum())
    fd = (loss(base + eps * delta) - loss(base - eps * delta)) / (2 * eps)
    an = float((out["placer"][0]["w_qkv"] * delta).sum())
    assert abs(fd - an) <= 2e-6 * max(1, abs(an)) and abs(an) > 1e-3


def test_no_attention_placer_gradient_equals_finite_differences():
    c, g, gnn, pl, hd = _small(placer_layers=3)
    rng = np.random.default_rng(2)
    N, d = 30, c.d_model
    gp = np.array([0, 12, N])
    ne, x0 = rng.normal(size=(N, d)), rng.normal(size=(2, d))
    dl = rng.normal(size=(N, c.n_devices))
    out = PG.placer_backward(ne, x0, gp, pl, hd["w_out"], hd["b_out"], dl, n_heads=c.heads, seg_len=8, mem_len=8,
                             film=True, attention=False)
    ref = O.place(ne, x0, gp, pl, hd["w_out"], hd["b_out"], c.heads, 8, 8, film=True, attention=False)
    np.testing.assert_allclose(out["logits"], ref["logits"], rtol=0, atol=1e-11)
    params = {(l, k): pl[l][k] for l in range(3) for k in ("film_wg", "film_wb", "w_1", "b_1", "w_2", "ln2_g")}
    grads = {key: out["placer"][key[0]][key[1]] for key in params}
    params["x0"], grads["x0"] = x0, out["dgraph_emb"]

    def loss():
        pls = [{k: params.get((l, k), lw[k]) for k in lw} for l, lw in enumerate(pl)]
        return float((_placer_numpy(ne, params["x0"], gp, pls, hd, c.heads, 8, 8, True, attention=False) * dl).sum())
    _fd_check(loss, params, grads, rng)


def test_gnn_gradient_equals_finite_differences():
    c, g, gnn, pl, hd = _small(gnn_layers=2, fanout=3)
    rng = np.random.default_rng(3)
    N, H = g.n_nodes, c.hidden
    G = 1
    dn = rng.normal(size=(N, H))
    dg = rng.normal(size=(G, H))
    out = PG.gnn_backward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, dn, dg, fanout=c.fanout, nb_seed=c.nb_seed)
    e = O.embed(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, c.fanout, c.nb_seed)
    np.testing.assert_allclose(out["node_emb"], e["node_emb"], rtol=0, atol=1e-12)
    params = {(l, k): gnn[l][k] for l in range(2) for k in gnn[l]}
    grads = {key: out["gnn"][key[0]][key[1]] for key in params}

    def loss():
        layers = [{k: params[(l, k)] for k in gnn[l]} for l in range(2)]
        ee = O.embed(g.graph_ptr, g.row_ptr, g.col_idx, g.x, layers, c.fanout, c.nb_seed)
        return float((ee["node_emb"] * dn).sum() + (ee["graph_emb"] * dg).sum())
    _fd_check(loss, params, grads, rng, eps=1e-8, n_dirs=1, rtol=1e-5)   # kinks: a tiny step


def test_whole_chain_equals_its_stages_and_the_forward_oracle():
    c, g, gnn, pl, hd = _small(gnn_layers=2, placer_layers=2)
    rng = np.random.default_rng(4)
    dl = rng.normal(size=(g.n_nodes, c.n_devices))
    kw = dict(n_heads=c.heads, seg_len=64, mem_len=64, film=True)
    full = PG.policy_backward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, pl, hd["w_out"], hd["b_out"], dl,
                              fanout=c.fanout, nb_seed=c.nb_seed, **kw)
    ref = O.policy_forward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, pl, hd["w_out"], hd["b_out"], fanout=c.fanout,
                           nb_seed=c.nb_seed, n_heads=c.heads, seg_len=64, mem_len=64, k_samples=1, sample_seed=1)
    np.testing.assert_allclose(full["logits"], ref["logits"], rtol=0, atol=1e-11)
    p = PG.placer_backward(ref["node_emb"], ref["graph_emb"], g.graph_ptr, pl, hd["w_out"], hd["b_out"], dl, **kw)
    n = PG.gnn_backward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, p["dnode_emb"], p["dgraph_emb"],
                        fanout=c.fanout, nb_seed=c.nb_seed)
    for l in range(2):
        for k in gnn[l]:
            np.testing.assert_allclose(full["gnn"][l][k], n["gnn"][l][k], rtol=1e-9, atol=1e-12)
        for k in pl[l]:
            np.testing.assert_allclose(full["placer"][l][k], p["placer"][l][k], rtol=1e-9, atol=1e-12)


def test_adam_against_torch_and_first_step_closed_form():
    rng = np.random.default_rng(5)
    p0 = rng.normal(size=(7, 5))
    lr, b1, b2, eps = 3e-3, 0.9, 0.999, 1e-8
    t = torch.tensor(p0, requires_grad=True)
    opt = torch.optim.Adam([t], lr=lr, betas=(b1, b2), eps=eps)
    p, m, v = p0.copy(), np.zeros_like(p0), np.zeros_like(p0)
    for step in range(1, 6):
        gr = rng.normal(size=p0.shape)
        if step == 1:
            first = p0 - lr * gr / (np.abs(gr) + eps)
        t.grad = torch.tensor(gr)
        opt.step()
        p, m, v = PG.adam_step(p, gr, m, v, step, lr, b1, b2, eps)
        if step == 1:
            np.testing.assert_allclose(p, first, rtol=0, atol=1e-15)
        np.testing.assert_allclose(p, t.detach().numpy(), rtol=0, atol=1e-14)


def test_decisions_from_the_same_run_change_nothing():
    """Fixing the ReLU signs and max-pool winners to the forward's own choices
    reproduces the free forward and its gradients (the decision path is the same
    function where the decisions agree)."""
    c, g, gnn, pl, hd = _small(gnn_layers=2, placer_layers=2, fanout=3)
    rng = np.random.default_rng(9)
    dl = rng.normal(size=(g.n_nodes, c.n_devices))
    kw = dict(fanout=c.fanout, nb_seed=c.nb_seed, n_heads=c.heads, seg_len=64, mem_len=64, film=True)
    free = PG.policy_backward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, pl, hd["w_out"], hd["b_out"], dl, **kw)
    # the forward's own decisions, from the numpy oracle
    S = O.sample_neighbours(O.neighbour_lists(g.row_ptr, g.col_idx), g.graph_ptr, c.fanout, c.nb_seed)
    h = g.x
    dec_gnn = []
    for lw in gnn:
        A, P = O.aggregate_maxpool(h, S, lw["w_pool"], lw["b_pool"])
        arg = np.full(A.shape, -1, np.int64)
        for v, s in enumerate(S):
            if len(s):
                s = np.sort(np.asarray(s))
                arg[v] = s[np.argmax(P[s], axis=0)]           # first maximum in ascending order
        pre = h @ lw["w_self"].T + A @ lw["w_neigh"].T + lw["b_upd"]
        dec_gnn.append((arg, pre > 0))
        h = O.relu(pre)
    e = O.embed(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, c.fanout, c.nb_seed)
    gamma, beta = O.film_params(e["graph_emb"], pl, True)
    x = e["node_emb"]
    dec_ffn = []
    for l, lw in enumerate(pl):                      # one segment of 64 with memory 64 == the band form
        y = gamma[0, l] * x + beta[0, l]
        nxt = np.zeros_like(x)
        mask = np.zeros((g.n_nodes, c.d_ff), bool)
        for q0 in range(0, g.n_nodes, 64):
            q1 = min(q0 + 64, g.n_nodes)
            k0 = max(0, q0 - 64)
            z = O.layer_norm(y[q0:q1] + O.attention(y[q0:q1], y[k0:q1], lw, c.heads), lw["ln1_g"], lw["ln1_b"])
            u = z @ lw["w_1"].T + lw["b_1"]
            mask[q0:q1] = u > 0
            nxt[q0:q1] = O.layer_norm(z + O.relu(u) @ lw["w_2"].T + lw["b_2"], lw["ln2_g"], lw["ln2_b"])
        dec_ffn.append(mask)
        x = nxt
    fixed = PG.policy_backward(g.graph_ptr, g.row_ptr, g.col_idx, g.x, gnn, pl, hd["w_out"], hd["b_out"], dl, **kw,
                               decisions={"gnn": dec_gnn, "ffn": dec_ffn})
    np.testing.assert_allclose(fixed["logits"], free["logits"], rtol=0, atol=1e-12)
    for l in range(2):
        for k in gnn[l]:
            np.testing.assert_allclose(fixed["gnn"][l][k], free["gnn"][l][k], rtol=1e-10, atol=1e-12)
        for k in pl[l]:
            np.testing.assert_allclose(fixed["placer"][l][k], free["placer"][l][k], rtol=1e-10, atol=1e-12)
