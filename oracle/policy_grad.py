"""Gradients of the GDP policy for its update step (Section 3: Eq. 1's objective
optimised with PPO; Section 3.1: the graph embedding network is trained jointly
with the placement network; Section 3.2: the cached segment memory passes no
gradient).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import or run this module.  It shares no code
with the HIP path.

The gradient of a loss has a plain definition: the derivative of the forward
pass.  Here the forward pass is written out once more with plain PyTorch CPU
ops in float64, step by step in the order of the forward oracle
(``gdp_oracle``), and torch.autograd (a library primitive) differentiates it.
The only modelling choice is the memory's stop-gradient: as in Transformer-XL,
the rows cached from earlier segments enter a layer as constants (their
queries, keys and values still use the layer's weights, so the weights receive
gradient through them; the earlier segments' activations do not).  The cache
holds each layer's conditioned input (after FiLM), the quantity the forward
oracle caches.

Every function takes an upstream gradient ``dlogits`` and returns the
vector-Jacobian product, i.e. the gradient of sum(dlogits * logits).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np
import torch

from . import gdp_oracle as O

F64 = torch.float64


def _t(a, grad=False):
    t = torch.as_tensor(np.asarray(a, np.float64), dtype=F64).clone()
    t.requires_grad_(grad)
    return t


def _layer_norm(x, g, b):
    mu = x.mean(dim=-1, keepdim=True)
    var = ((x - mu) ** 2).mean(dim=-1, keepdim=True)
    return (x - mu) / torch.sqrt(var + O.LN_EPS) * g + b


def _attention(yq, ykv, lw, n_heads):
    d = yq.shape[1]
    dh = d // n_heads
    w, b = lw["w_qkv"], lw["b_qkv"]
    q = yq @ w[:d].T + b[:d]
    k = ykv @ w[d:2 * d].T + b[d:2 * d]
    v = ykv @ w[2 * d:].T + b[2 * d:]
    heads = []
    for h in range(n_heads):
        sl = slice(h * dh, (h + 1) * dh)
        p = torch.softmax(q[:, sl] @ k[:, sl].T / np.sqrt(dh), dim=-1)
        heads.append(p @ v[:, sl])
    return torch.cat(heads, dim=1) @ lw["w_o"].T + lw["b_o"]


def _relu(u, mask=None):
    """ReLU; with mask (the sign decisions of a run to compare against) the
    decision is taken from the mask instead of from u's sign."""
    return torch.relu(u) if mask is None else u * torch.as_tensor(mask, dtype=F64)


def _ffn(z, lw, mask=None):
    return _relu(z @ lw["w_1"].T + lw["b_1"], mask) @ lw["w_2"].T + lw["b_2"]


def _block(y, mem, lw, n_heads, mask=None):
    """Post-LN layer on the segment rows y with the cached rows mem (constants)."""
    ctx = torch.cat([mem, y], dim=0)
    z = _layer_norm(y + _attention(y, ctx, lw, n_heads), lw["ln1_g"], lw["ln1_b"])
    return _layer_norm(z + _ffn(z, lw, mask), lw["ln2_g"], lw["ln2_b"])


def _film(x0, placer, film):
    G = x0.shape[0]
    out = []
    for lw in placer:
        if film:
            out.append((1.0 + x0 @ lw["film_wg"].T + lw["film_bg"], x0 @ lw["film_wb"].T + lw["film_bb"]))
        else:
            d = lw["ln2_g"].shape[0]
            out.append((torch.ones(G, d, dtype=F64), torch.zeros(G, d, dtype=F64)))
    return out


def _placer_forward(node_emb, x0, graph_ptr, placer, head, n_heads, seg_len, mem_len, film, attention,
                    ffn_masks=None):
    """Formulation A (segment loop, per-graph memory caches of each layer's
    conditioned input, detached), or the ablation's row-local layers.
    ffn_masks: optional per-layer [N, d_ff] sign decisions of the FFN's ReLU."""
    N, d = node_emb.shape
    cond = _film(x0, placer, film)
    fm = (lambda l, a, b: None) if ffn_masks is None else (lambda l, a, b: ffn_masks[l][a:b])
    rows = []
    for g in range(len(graph_ptr) - 1):
        gs, ge = int(graph_ptr[g]), int(graph_ptr[g + 1])
        if not attention:
            x = node_emb[gs:ge]
            for l, lw in enumerate(placer):
                y = cond[l][0][g] * x + cond[l][1][g]
                x = _layer_norm(y + _ffn(y, lw, fm(l, gs, ge)), lw["ln2_g"], lw["ln2_b"])
            rows.append(x)
            continue
        mems = [torch.zeros(0, d, dtype=F64) for _ in placer]
        for q0 in range(gs, ge, seg_len):
            q1 = min(q0 + seg_len, ge)
            x = node_emb[q0:q1]
            for l, lw in enumerate(placer):
                y = cond[l][0][g] * x + cond[l][1][g]
                new_mem = torch.cat([mems[l], y], dim=0)
                x_next = _block(y, mems[l], lw, n_heads, fm(l, q0, q1))
                mems[l] = new_mem[max(0, new_mem.shape[0] - mem_len):].detach() if mem_len > 0 \
                    else torch.zeros(0, d, dtype=F64)
                x = x_next
            rows.append(x)
    x = torch.cat(rows, dim=0)
    return x @ head["w_out"].T + head["b_out"]


def _gnn_forward(x, S, gnn, decisions=None):
    """Eq. 2 and Eq. 3; the max over S(v) takes, per element, the first maximal
    row of S(v) in ascending node order (torch.max's documented tie rule), and
    an empty S(v) aggregates to 0.  decisions: optional per-layer (arg [N, H],
    relu mask [N, H]) -- the winning neighbour of every element (-1: none) and
    the update's ReLU signs of a run to compare against."""
    N = x.shape[0]
    width = max(1, max((len(s) for s in S), default=0))
    idx = np.full((N, width), N, np.int64)            # pad with the row index N (-inf below)
    for v, s in enumerate(S):
        idx[v, :len(s)] = np.sort(np.asarray(s, np.int64))
    has = torch.as_tensor(np.array([len(s) > 0 for s in S]))[:, None]
    idx_t = torch.as_tensor(idx)
    h = x
    for l, lw in enumerate(gnn):
        P = torch.sigmoid(h @ lw["w_pool"].T + lw["b_pool"])
        if decisions is None:
            pad = torch.cat([P, torch.full((1, P.shape[1]), -np.inf, dtype=F64)], dim=0)
            A, _ = torch.max(pad[idx_t], dim=1)
            A = torch.where(has, A, torch.zeros_like(A))
            mask = None
        else:
            arg, mask = decisions[l]
            arg = np.asarray(arg, np.int64)
            cols = np.broadcast_to(np.arange(P.shape[1]), arg.shape)
            A = P[torch.as_tensor(np.maximum(arg, 0)), torch.as_tensor(np.array(cols))]
            A = torch.where(torch.as_tensor(arg >= 0), A, torch.zeros_like(A))
        h = _relu(h @ lw["w_self"].T + A @ lw["w_neigh"].T + lw["b_upd"], mask)
    return h


def _leaves(layers: List[Dict[str, np.ndarray]]):
    return [{k: _t(v, True) for k, v in lw.items()} for lw in layers]


def _grads(layers):
    return [{k: (v.grad.numpy().copy() if v.grad is not None else np.zeros(tuple(v.shape))) for k, v in lw.items()}
            for lw in layers]


def placer_backward(node_emb, graph_emb, graph_ptr, placer_layers, w_out, b_out, dlogits, *, n_heads, seg_len,
                    mem_len, film=True, attention=True):
    """Gradient of sum(dlogits * logits) with respect to every placer and head
    weight, to the node embeddings and to the pooled graph embeddings."""
    ne = _t(node_emb, True)
    x0 = _t(graph_emb, True)
    pl = _leaves(placer_layers)
    hd = {"w_out": _t(w_out, True), "b_out": _t(b_out, True)}
    logits = _placer_forward(ne, x0, graph_ptr, pl, hd, n_heads, seg_len, mem_len, film, attention)
    (logits * _t(dlogits)).sum().backward()
    return {"logits": logits.detach().numpy(), "placer": _grads(pl),
            "head": {k: v.grad.numpy().copy() for k, v in hd.items()},
            "dnode_emb": ne.grad.numpy().copy(),
            "dgraph_emb": x0.grad.numpy().copy() if x0.grad is not None else np.zeros(tuple(x0.shape))}


def gnn_backward(graph_ptr, row_ptr, col_idx, x, gnn_layers, dnode_emb, dgraph_emb, *, fanout, nb_seed):
    """Gradient of sum(dnode_emb * h) + sum(dgraph_emb * x0) with respect to the
    GNN weights, where h are the final node embeddings and x0 their per-graph
    means (the two ways the placer reads the GNN)."""
    S = O.sample_neighbours(O.neighbour_lists(row_ptr, col_idx), graph_ptr, fanout, nb_seed)
    gnn = _leaves(gnn_layers)
    h = _gnn_forward(_t(x), S, gnn)
    G = len(graph_ptr) - 1
    x0 = torch.stack([h[graph_ptr[g]:graph_ptr[g + 1]].mean(dim=0) for g in range(G)])
    ((h * _t(dnode_emb)).sum() + (x0 * _t(dgraph_emb)).sum()).backward()
    return {"node_emb": h.detach().numpy(), "graph_emb": x0.detach().numpy(), "gnn": _grads(gnn)}


def policy_backward(graph_ptr, row_ptr, col_idx, x, gnn_layers, placer_layers, w_out, b_out, dlogits, *, fanout,
                    nb_seed, n_heads, seg_len, mem_len, film=True, attention=True, decisions=None):
    """The whole chain in one graph: gradient of sum(dlogits * logits) with
    respect to every weight of the GNN, the placer and the head.

    decisions (optional) fixes the forward's discrete choices -- each ReLU's
    sign and each max-pool element's winning neighbour -- to those of another
    run: {"gnn": [(arg, mask)] per GNN layer, "ffn": [mask] per placer layer}.
    Where a pre-activation lies within rounding of zero, or two neighbours
    within rounding of each other, the two runs may decide differently, and
    the gradient jumps there; with the same decisions the comparison measures
    the arithmetic alone."""
    S = O.sample_neighbours(O.neighbour_lists(row_ptr, col_idx), graph_ptr, fanout, nb_seed)
    gnn = _leaves(gnn_layers)
    pl = _leaves(placer_layers)
    hd = {"w_out": _t(w_out, True), "b_out": _t(b_out, True)}
    dec = decisions or {}
    h = _gnn_forward(_t(x), S, gnn, dec.get("gnn"))
    G = len(graph_ptr) - 1
    x0 = torch.stack([h[graph_ptr[g]:graph_ptr[g + 1]].mean(dim=0) for g in range(G)])
    logits = _placer_forward(h, x0, graph_ptr, pl, hd, n_heads, seg_len, mem_len, film, attention, dec.get("ffn"))
    (logits * _t(dlogits)).sum().backward()
    return {"logits": logits.detach().numpy(), "gnn": _grads(gnn), "placer": _grads(pl),
            "head": {k: v.grad.numpy().copy() for k, v in hd.items()}}


def adam_step(param, grad, m, v, step, lr, beta1, beta2, eps):
    """One Adam update (Kingma and Ba, 2015) of a parameter array: the moment
    estimates, their bias corrections at step t (1-based) and the step."""
    param = np.asarray(param, np.float64)
    g = np.asarray(grad, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** step)
    vhat = v / (1.0 - beta2 ** step)
    return param - lr * mhat / (np.sqrt(vhat) + eps), m, v
