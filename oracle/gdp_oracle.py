"""Plain float64 CPU oracle of the GDP placement policy's forward pass + sampling.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check and the
benchmark's CPU-baseline leg may import or run this module.  It shares no code
with the HIP path (no kernels, headers, tables or helpers); both sides only
consume the same seeded input arrays.

Everything is written the slow, obvious way in numpy float64, following the
paper's order and notation:

* Graph embedding network (Section 3.1).  For iteration l, every node v
  aggregates its neighbours' representations with a max-pool of
  sigmoid(W h_u + b) over u in N(v)  (Eq. 2), concatenates the result with
  its own representation and feeds it through a fully connected layer f
  (Eq. 3).
* Placement network (Section 3.2).  A Transformer without positional
  embedding, run over the node sequence with Transformer-XL segment-level
  recurrence: the previous positions' hidden states of each layer are cached
  and reused as extra context for the next segment.
* Superposition (Section 3.3, Eq. 4).  The dense layers of the placement
  network see their input multiplied element-wise by a conditioning c(x0) of
  the pooled graph representation x0.
* The policy emits a placement for every op of the graph at once (Section 2,
  Section 3), drawn here by Gumbel-max from the per-node device logits.

Readings of points the paper leaves open (all listed in the design notes):
neighbours are in- and out-neighbours; above ``fanout`` neighbours a
deterministic, order-invariant hash sample is taken; an empty neighbourhood
aggregates to 0; f is a ReLU dense layer; layers are post-LN with a ReLU FFN;
attention is bidirectional inside a segment plus the cached memory; the
conditioning is a FiLM scale (1 + W x0 + b) and shift (W x0 + b) per placer
layer; the residual adds to the conditioned input.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from .philox import philox4x64_10

LN_EPS = 1e-5


# ----------------------------------------------------------------------------
# Elementary functions (definitions, float64).
# ----------------------------------------------------------------------------

def sigmoid(z):
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    ez = np.exp(z[~pos])
    out[~pos] = ez / (1.0 + ez)
    return out


def relu(z):
    return np.maximum(z, 0.0)


def layer_norm(x, g, b, eps=LN_EPS):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def logsumexp_rows(s):
    m = s.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(s - m).sum(axis=-1, keepdims=True)))[..., 0]


# ----------------------------------------------------------------------------
# Section 3.1: neighbourhoods, sampling, Eq. 2 and Eq. 3.
# ----------------------------------------------------------------------------

def neighbour_lists(row_ptr, col_idx) -> List[np.ndarray]:
    """N(v) = successors(v) union predecessors(v) (data dependencies in both
    directions).  In a DAG without duplicate edges the two sets are disjoint."""
    n = len(row_ptr) - 1
    pred: List[List[int]] = [[] for _ in range(n)]
    for u in range(n):
        for v in col_idx[row_ptr[u]:row_ptr[u + 1]]:
            pred[int(v)].append(u)
    return [np.concatenate([np.asarray(col_idx[row_ptr[v]:row_ptr[v + 1]], np.int64),
                            np.asarray(pred[v], np.int64)]) for v in range(n)]


def neighbour_keys(v_local, u_local, nb_seed):
    """64-bit sampling key of the (v, u) pair: word 0 of
    Philox4x64-10(counter = (v, u, 1, 0), key = (nb_seed, 0)), graph-local ids."""
    w0, _, _, _ = philox4x64_10(
        (np.asarray(v_local, np.uint64), np.asarray(u_local, np.uint64),
         np.uint64(1), np.uint64(0)),
        (np.uint64(nb_seed), np.uint64(0)))
    return w0


def sample_neighbours(nb: Sequence[np.ndarray], graph_ptr, fanout: int, nb_seed: int):
    """S(v): all of N(v) when |N(v)| <= fanout, otherwise the ``fanout``
    members with the smallest (key, u) -- independent of neighbour order.
    Returned sorted by node id."""
    n = len(nb)
    gid = np.searchsorted(np.asarray(graph_ptr), np.arange(n), side="right") - 1
    out = []
    for v in range(n):
        cand = np.asarray(nb[v], np.int64)
        if cand.size > fanout:
            g0 = int(graph_ptr[gid[v]])
            keys = neighbour_keys(np.full(cand.size, v - g0, np.uint64),
                                  (cand - g0).astype(np.uint64), nb_seed)
            order = np.lexsort((cand, keys))      # primary: key, tie: u
            cand = cand[order[:fanout]]
        out.append(np.sort(cand))
    return out


def aggregate_maxpool(h, S, w_pool, b_pool):
    """Eq. 2: h_N(v) = max_{u in S(v)} sigmoid(W h_u + b); 0 when S(v) is empty.
    sigmoid(W h_u + b) depends on u only, so it is formed once per node."""
    P = sigmoid(h @ w_pool.T + b_pool)
    A = np.zeros((h.shape[0], w_pool.shape[0]))
    for v, s in enumerate(S):
        if len(s):
            A[v] = P[np.asarray(s)].max(axis=0)
    return A, P


def node_update(h, A, w_self, w_neigh, b_upd):
    """Eq. 3 with f = ReLU dense layer on concat(h_v, h_N(v)); the weight of f is
    [w_self | w_neigh]."""
    return relu(h @ w_self.T + A @ w_neigh.T + b_upd)


def embed(graph_ptr, row_ptr, col_idx, x, gnn_layers, fanout, nb_seed, keep=False):
    """Graph embedding network: node embeddings [N, H] and per-graph mean-pooled
    graph embeddings x0 [G, H]."""
    nb = neighbour_lists(row_ptr, col_idx)
    S = sample_neighbours(nb, graph_ptr, fanout, nb_seed)
    h = np.asarray(x, dtype=np.float64)
    trace = []
    for lw in gnn_layers:
        A, P = aggregate_maxpool(h, S, lw["w_pool"], lw["b_pool"])
        h = node_update(h, A, lw["w_self"], lw["w_neigh"], lw["b_upd"])
        if keep:
            trace.append({"P": P, "A": A, "h": h})
    G = len(graph_ptr) - 1
    x0 = np.stack([h[graph_ptr[g]:graph_ptr[g + 1]].mean(axis=0) for g in range(G)])
    return {"node_emb": h, "graph_emb": x0, "S": S, "trace": trace}


# ----------------------------------------------------------------------------
# Section 3.3, Eq. 4: feature conditioning of the placer layers.
# ----------------------------------------------------------------------------

def film_params(x0, placer_layers, film=True):
    """gamma[g, l] = 1 + W_g x0_g + b_g and beta[g, l] = W_b x0_g + b_b per
    placer layer; identity conditioning when ``film`` is off."""
    G = x0.shape[0]
    L = len(placer_layers)
    d = placer_layers[0]["w_o"].shape[0]
    gamma = np.ones((G, L, d))
    beta = np.zeros((G, L, d))
    if film:
        for l, lw in enumerate(placer_layers):
            gamma[:, l] = 1.0 + x0 @ lw["film_wg"].T + lw["film_bg"]
            beta[:, l] = x0 @ lw["film_wb"].T + lw["film_bb"]
    return gamma, beta


# ----------------------------------------------------------------------------
# Section 3.2: Transformer layer without positional terms.
# ----------------------------------------------------------------------------

def attention(yq, ykv, lw, n_heads, probs_out: Optional[list] = None):
    """Multi-head attention of the query rows ``yq`` over the context rows ``ykv``
    (no mask, no positional terms); output projection included."""
    d = yq.shape[1]
    dh = d // n_heads
    wq, wk, wv = lw["w_qkv"][:d], lw["w_qkv"][d:2 * d], lw["w_qkv"][2 * d:]
    bq, bk, bv = lw["b_qkv"][:d], lw["b_qkv"][d:2 * d], lw["b_qkv"][2 * d:]
    q = yq @ wq.T + bq
    k = ykv @ wk.T + bk
    v = ykv @ wv.T + bv
    heads = []
    for hd in range(n_heads):
        sl = slice(hd * dh, (hd + 1) * dh)
        p = softmax_rows(q[:, sl] @ k[:, sl].T / np.sqrt(dh))
        if probs_out is not None:
            probs_out.append(p)
        heads.append(p @ v[:, sl])
    o = np.concatenate(heads, axis=1)
    return o @ lw["w_o"].T + lw["b_o"]


def ffn(z, lw):
    return relu(z @ lw["w_1"].T + lw["b_1"]) @ lw["w_2"].T + lw["b_2"]


def transformer_block(y, ctx, lw, n_heads, probs_out=None):
    """Post-LN layer: z = LN(y + Attn(y, ctx)); out = LN(z + FFN(z))."""
    z = layer_norm(y + attention(y, ctx, lw, n_heads, probs_out), lw["ln1_g"], lw["ln1_b"])
    return layer_norm(z + ffn(z, lw), lw["ln2_g"], lw["ln2_b"])


def placer_recurrent(node_emb, graph_ptr, gamma, beta, placer_layers, n_heads,
                     seg_len, mem_len, probs_out=None):
    """Formulation A: Transformer-XL segment loop.  For every graph, segments of
    ``seg_len`` nodes are processed in node-id order; each layer keeps a cache
    of the last ``mem_len`` inputs it has seen in this graph and attends over
    [cache ; current segment].  The cache is per graph (it starts empty)."""
    N, d = node_emb.shape
    out = np.zeros((N, d))
    L = len(placer_layers)
    for g in range(len(graph_ptr) - 1):
        gs, ge = int(graph_ptr[g]), int(graph_ptr[g + 1])
        mems = [np.zeros((0, d)) for _ in range(L)]
        for q0 in range(gs, ge, seg_len):
            q1 = min(q0 + seg_len, ge)
            x = node_emb[q0:q1]
            for l, lw in enumerate(placer_layers):
                y = gamma[g, l] * x + beta[g, l]
                ctx = np.concatenate([mems[l], y], axis=0)
                mems[l] = ctx[max(0, len(ctx) - mem_len):] if mem_len > 0 else np.zeros((0, d))
                x = transformer_block(y, ctx, lw, n_heads, probs_out)
            out[q0:q1] = x
    return out


def placer_band(node_emb, graph_ptr, gamma, beta, placer_layers, n_heads, seg_len, mem_len):
    """Formulation B: layer by layer over all nodes.  The query rows of segment
    [q0, q1) of graph g attend to the rows [max(g_start, q0 - mem_len), q1)
    of the same layer's input."""
    N, d = node_emb.shape
    x = np.array(node_emb, dtype=np.float64)
    gid = np.searchsorted(np.asarray(graph_ptr), np.arange(N), side="right") - 1
    for l, lw in enumerate(placer_layers):
        y = gamma[gid, l] * x + beta[gid, l]
        nxt = np.zeros_like(x)
        for g in range(len(graph_ptr) - 1):
            gs, ge = int(graph_ptr[g]), int(graph_ptr[g + 1])
            for q0 in range(gs, ge, seg_len):
                q1 = min(q0 + seg_len, ge)
                k0 = max(gs, q0 - mem_len)
                nxt[q0:q1] = transformer_block(y[q0:q1], y[k0:q1], lw, n_heads)
        x = nxt
    return x


# ----------------------------------------------------------------------------
# Section 4.4 (ablation): the placement network with no attention.
# ----------------------------------------------------------------------------

def placer_no_attention(node_emb, graph_ptr, gamma, beta, placer_layers):
    """Every placer layer without its attention sublayer: the conditioned input
    y = gamma * x + beta goes straight to the feed-forward sublayer,
    x <- LN(y + FFN(y)) with the layer's second LayerNorm.  Each node's result
    depends only on its own row and its graph's conditioning."""
    N, d = node_emb.shape
    x = np.array(node_emb, dtype=np.float64)
    gid = np.searchsorted(np.asarray(graph_ptr), np.arange(N), side="right") - 1
    for l, lw in enumerate(placer_layers):
        y = gamma[gid, l] * x + beta[gid, l]
        x = layer_norm(y + ffn(y, lw), lw["ln2_g"], lw["ln2_b"])
    return x


def head(x, w_out, b_out):
    """Per-node device logits (Fig. 1: N x d output) and their log-sum-exp."""
    logits = x @ w_out.T + b_out
    return logits, logsumexp_rows(logits)


def place(node_emb, graph_emb, graph_ptr, placer_layers, w_out, b_out, n_heads,
          seg_len, mem_len, film=True, formulation="recurrent", attention=True):
    """The placement network and head; attention=False is the ablation's
    placer without attention (n_heads, seg_len and mem_len then unused)."""
    gamma, beta = film_params(graph_emb, placer_layers, film)
    if not attention:
        x = placer_no_attention(node_emb, graph_ptr, gamma, beta, placer_layers)
    else:
        fn = placer_recurrent if formulation == "recurrent" else placer_band
        x = fn(node_emb, graph_ptr, gamma, beta, placer_layers, n_heads, seg_len, mem_len)
    logits, lse = head(x, w_out, b_out)
    return {"x": x, "logits": logits, "lse": lse, "gamma": gamma, "beta": beta}


# ----------------------------------------------------------------------------
# Whole-graph sampling (Gumbel-max) and log-probabilities.
# ----------------------------------------------------------------------------

def gumbel_uniforms(seed: int, n_nodes: int, k_samples: int, n_devices: int):
    """u[k, v, j] in (0, 1): Philox4x64-10 with key (seed, 0) and counter
    (v, k, 2, j >> 3); the 64-bit word (j & 7) >> 1 is split into 32-bit halves
    (half j & 1, 0 = low), and u = (2 * (half >> 9) + 1) * 2^-24 (exactly
    representable in float32 and float64)."""
    v = np.arange(n_nodes, dtype=np.uint64)[None, :]
    k = np.arange(k_samples, dtype=np.uint64)[:, None]
    u = np.empty((k_samples, n_nodes, n_devices))
    for blk in range((n_devices + 7) // 8):
        words = philox4x64_10((v, k, np.uint64(2), np.uint64(blk)), (np.uint64(seed), np.uint64(0)))
        for j in range(blk * 8, min(n_devices, blk * 8 + 8)):
            w = words[(j & 7) >> 1]
            half = (w >> np.uint64(32)) if (j & 1) else (w & np.uint64(0xFFFFFFFF))
            u[:, :, j] = (2.0 * (half >> np.uint64(9)).astype(np.float64) + 1.0) * 2.0 ** -24
    return u


def sample(logits, lse, graph_ptr, k_samples: int, seed: int, uniforms=None):
    """placements[k, v] = argmax_j (logits[v, j] - ln(-ln u[k, v, j])), ties to the
    lowest j; logp[g, k] = sum over v in g of (logits[v, p] - lse[v])."""
    N, D = logits.shape
    u = gumbel_uniforms(seed, N, k_samples, D) if uniforms is None else np.asarray(uniforms, np.float64)
    g = -np.log(-np.log(u))
    scores = logits[None, :, :] + g
    placements = np.argmax(scores, axis=-1).astype(np.int32)
    lp = log_prob_of(logits, lse, graph_ptr, placements)
    return {"placements": placements, "logp": lp, "scores": scores}


def log_prob_of(logits, lse, graph_ptr, placements):
    """log pi(D | G) of given placements: sum over the graph's nodes of the
    per-node log-softmax at the chosen device; shape [G, K]."""
    K, N = placements.shape
    per = logits[np.arange(N)[None, :], placements] - lse[None, :]
    G = len(graph_ptr) - 1
    return np.stack([per[:, graph_ptr[g]:graph_ptr[g + 1]].sum(axis=1) for g in range(G)])


def policy_forward(graph_ptr, row_ptr, col_idx, x, gnn_layers, placer_layers, w_out, b_out, *,
                   fanout, nb_seed, n_heads, seg_len, mem_len, k_samples, sample_seed,
                   film=True, uniforms=None):
    """embed -> place -> sample, as one call."""
    e = embed(graph_ptr, row_ptr, col_idx, x, gnn_layers, fanout, nb_seed)
    p = place(e["node_emb"], e["graph_emb"], graph_ptr, placer_layers, w_out, b_out,
              n_heads, seg_len, mem_len, film)
    s = sample(p["logits"], p["lse"], graph_ptr, k_samples, sample_seed, uniforms)
    out = {}
    out.update(e)
    out.update(p)
    out.update(s)
    return out


# ----------------------------------------------------------------------------
# Section 3 (Eq. 1, optimised with PPO): the clipped surrogate over the K
# sampled placements of every graph and its gradient with respect to the
# device logits -- where the update path starts its backward pass.
# ----------------------------------------------------------------------------

def ppo_clipped_surrogate(logits, lse, graph_ptr, placements, logp, logp_old, adv, clip_eps):
    """Per graph g, with ratio r = exp(logp - logp_old) of each sample k:
        L_g = -(1/K) sum_k min(r A, clip(r, 1 - eps, 1 + eps) A)
    (PPO's clipped objective, negated to a loss), and the gradient of the batch
    loss L = (1/G) sum_g L_g (Eq. 1 averages over graphs) with respect to the
    logits.  logp[g, k] = sum over v in g of log_softmax(logits_v)[p_kv], so
    d logp[g, k] / d logits[v, j] = 1[p_kv = j] - softmax(logits_v)_j; the
    min takes the unclipped branch's slope r A where that branch attains it
    and 0 where the clipped constant does."""
    logits = np.asarray(logits, np.float64)
    N, D = logits.shape
    G = len(graph_ptr) - 1
    K = placements.shape[0]
    r = np.exp(np.asarray(logp, np.float64) - np.asarray(logp_old, np.float64))
    A = np.asarray(adv, np.float64)
    unclipped = r * A
    clipped = np.clip(r, 1.0 - clip_eps, 1.0 + clip_eps) * A
    loss = -np.minimum(unclipped, clipped).mean(axis=1)
    slope = np.where(unclipped <= clipped, r * A, 0.0)        # d min / d logp
    coef = -slope / K / G                                      # dL / dlogp[g, k]
    soft = np.exp(logits - np.asarray(lse, np.float64)[:, None])
    dlogits = np.zeros((N, D))
    for g in range(G):
        gs, ge = int(graph_ptr[g]), int(graph_ptr[g + 1])
        for k in range(K):
            for v in range(gs, ge):
                dlogits[v, placements[k, v]] += coef[g, k]
            dlogits[gs:ge] -= coef[g, k] * soft[gs:ge]
    return {"loss": loss, "coef": coef, "dlogits": dlogits}


def rewards_advantages(run_time, valid, reward_sum, trial_count):
    """Section 4's reward and advantage for measured run times t[g, k] of the
    K placements of every graph: r = -sqrt(t) for a valid placement and -10
    for an invalid one (out of memory, a broken co-location constraint); the
    bias term is the average reward of all previous trials of the same graph,
    and the advantage is r minus it.  Readings: the K trials of one batch are
    not previous to each other, and a graph with no previous trial takes its
    batch's own mean reward as the bias.  Returns the rewards, advantages and
    bias terms, and the per-graph running state (sum of rewards, number of
    trials) updated with this batch."""
    t = np.asarray(run_time, np.float64)
    G, K = t.shape
    ok = np.ones((G, K), bool) if valid is None else np.asarray(valid, bool)
    r = np.where(ok, -np.sqrt(np.where(ok, t, 0.0)), -10.0)
    s = np.array(reward_sum, np.float64)
    n = np.array(trial_count, np.int64)
    base = np.empty(G)
    for g in range(G):
        base[g] = s[g] / n[g] if n[g] > 0 else r[g].mean()
    adv = r - base[:, None]
    return {"reward": r, "advantage": adv, "baseline": base, "reward_sum": s + r.sum(axis=1),
            "trial_count": n + K}


def head_backward(x, w_out, dlogits):
    """The head's backward pass (logits = x W_out^T + b_out): the gradients with
    respect to its input, weight and bias for a given dL/dlogits."""
    x = np.asarray(x, np.float64)
    dl = np.asarray(dlogits, np.float64)
    return {"dx": dl @ np.asarray(w_out, np.float64), "dw_out": dl.T @ x, "db_out": dl.sum(axis=0)}


# ----------------------------------------------------------------------------
# Section 4.1 (a placement's run time and its validity) and Section 2 (graph
# placement "with and without simulation"): a simulated step time of each
# sampled placement, the input of the reward.  The paper measures run times
# on hardware and defines no simulator; this is the reading used here.
# ----------------------------------------------------------------------------

def simulate_placements(graph_ptr, row_ptr, col_idx, placements, n_devices, op_cost, out_xfer, op_mem, mem_cap):
    """In-order list scheduling of every graph under each of the K placements.

    Every device runs its ops one at a time in node-id order (a topological
    order).  Op v may start once its device has finished the device's previous
    op and every input has arrived: the output of a predecessor u is available
    on u's own device when u finishes and on any other device out_xfer[u] later
    (transfers overlap with compute and with each other).  Then
        ready(v)  = max over predecessors u of finish(u) + (p_u != p_v) * out_xfer[u]   (0 without one)
        start(v)  = max(ready(v), free[p_v]),  finish(v) = start(v) + op_cost[v],  free[p_v] = finish(v)
    and the graph's run time is its largest finish time.  A placement is valid
    when every device holds at most mem_cap[g] of memory, the sum of op_mem over
    the ops placed on it (out of memory makes it invalid).  All arithmetic is on
    Python / numpy integers, so results are exact.

    Returns makespan [G, K] int64, valid [G, K] bool and device_mem [G, K, D]."""
    placements = np.asarray(placements, np.int64)
    K, N = placements.shape
    G = len(graph_ptr) - 1
    cost = np.asarray(op_cost, np.int64)
    xfer = np.asarray(out_xfer, np.int64)
    mem = np.asarray(op_mem, np.int64)
    pred: List[List[int]] = [[] for _ in range(N)]
    for u in range(N):
        for v in col_idx[row_ptr[u]:row_ptr[u + 1]]:
            pred[int(v)].append(u)
    makespan = np.zeros((G, K), np.int64)
    device_mem = np.zeros((G, K, n_devices), np.int64)
    ks = np.arange(K)
    for g in range(G):
        gs, ge = int(graph_ptr[g]), int(graph_ptr[g + 1])
        finish = np.zeros((ge - gs, K), np.int64)
        free = np.zeros((K, n_devices), np.int64)
        for v in range(gs, ge):
            pv = placements[:, v]
            ready = np.zeros(K, np.int64)
            for u in pred[v]:
                arrive = finish[u - gs] + np.where(placements[:, u] != pv, xfer[u], 0)
                ready = np.maximum(ready, arrive)
            start = np.maximum(ready, free[ks, pv])
            finish[v - gs] = start + cost[v]
            free[ks, pv] = finish[v - gs]
            device_mem[g, ks, pv] += mem[v]
        makespan[g] = finish.max(axis=0)
    valid = (device_mem <= np.asarray(mem_cap, np.int64)[:, None, None]).all(axis=2)
    return {"makespan": makespan, "valid": valid, "device_mem": device_mem}
