"""Seeded synthetic workloads: dataflow DAGs, node features and policy weights.

This module only *generates inputs*.  It holds none of the policy's arithmetic
(no aggregation, attention, normalisation or sampling), so that the CPU oracle
under ``oracle/`` and the HIP path can both consume its arrays without sharing
any computation.

The paper's workloads (TensorFlow graphs of Inception, RNNLM, GNMT, ...; §4.2)
are not available, so five seeded generator families stand in for them.  All
generators emit *topological* node ids (every edge u -> v has u < v) and an
out-edge CSR with sorted column lists.

Node features follow the paper's description of per-op meta features
(§3.1: op type and output shape): a one-hot op type plus log-normal size
features.  Raw node ids are not used as features (they would break the
topology invariance the paper asks of the policy, §3).

Weights are Xavier-uniform; biases and LayerNorm parameters are small
non-trivial perturbations so that bias and normalisation mistakes are visible.
For bf16 configurations every weight and feature is rounded once,
round-to-nearest-even, and both the oracle (widened to float64) and the
device path (as raw bf16 bit patterns) see the same rounded values.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# Configurations (sizes of the five workloads).
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class Config:
    cfg_id: int
    name: str
    family: str                 # generator family
    graph_sizes: Tuple[int, ...]  # nodes per graph of the (ragged) batch
    feat_dim: int
    n_types: int
    hidden: int                 # GNN hidden width H (= placer d_model)
    gnn_layers: int
    fanout: int
    placer_layers: int
    heads: int
    d_ff: int
    seg_len: int
    mem_len: int
    n_devices: int
    k_samples: int
    dtype: str                  # "f32" or "bf16"
    film: bool = True
    attention: bool = True      # False: the ablation's placer without attention (Section 4.4)

    @property
    def n_nodes(self) -> int:
        return int(sum(self.graph_sizes))

    @property
    def d_model(self) -> int:
        return self.hidden

    @property
    def d_head(self) -> int:
        return self.hidden // self.heads

    @property
    def nb_seed(self) -> int:
        return 1000 + self.cfg_id

    @property
    def sample_seed(self) -> int:
        return 2000 + self.cfg_id

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, Config] = {
    "tiny_layered_256": Config(
        0, "tiny_layered_256", "layered", (256,), 32, 16, 64, 2, 8,
        2, 4, 256, 64, 64, 4, 4, "f32"),
    "inception_2500": Config(
        1, "inception_2500", "inception", (2500,), 64, 32, 128, 3, 10,
        4, 8, 512, 128, 128, 8, 16, "bf16"),
    "recurrent_12000": Config(
        2, "recurrent_12000", "recurrent", (12000,), 64, 32, 128, 3, 10,
        4, 8, 512, 256, 256, 8, 32, "bf16"),
    "superposition_4x": Config(
        3, "superposition_4x", "ragged", (1000, 4000, 8000, 16000), 64, 32, 128,
        3, 10, 4, 8, 512, 256, 256, 8, 16, "bf16"),
    "gnmt8_52000": Config(
        4, "gnmt8_52000", "gnmt", (52000,), 64, 32, 256, 3, 16,
        6, 8, 1024, 512, 512, 8, 64, "bf16"),
}
CONFIG_ORDER = ["tiny_layered_256", "inception_2500", "recurrent_12000",
                "superposition_4x", "gnmt8_52000"]


def get_config(name_or_id) -> Config:
    if isinstance(name_or_id, int):
        return CONFIGS[CONFIG_ORDER[name_or_id]]
    return CONFIGS[name_or_id]


# ----------------------------------------------------------------------------
# bf16 rounding (input preparation only).
# ----------------------------------------------------------------------------

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round to bf16 (round-to-nearest-even) and return the uint16 bit patterns."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return rounded.astype(np.uint16)


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Value of ``a`` after bf16 RNE rounding, as float64."""
    return bf16_to_f64(bf16_bits(a))


# ----------------------------------------------------------------------------
# Edge-list helpers.
# ----------------------------------------------------------------------------

class _Edges:
    def __init__(self):
        self.src: List[int] = []
        self.dst: List[int] = []

    def add(self, u: int, v: int):
        assert u < v, (u, v)
        self.src.append(u)
        self.dst.append(v)


def _to_csr(n: int, src: np.ndarray, dst: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Out-edge CSR with sorted, de-duplicated columns."""
    key = src.astype(np.int64) * n + dst.astype(np.int64)
    key = np.unique(key)
    s = (key // n).astype(np.int32)
    d = (key % n).astype(np.int32)
    row_ptr = np.zeros(n + 1, dtype=np.int32)
    np.add.at(row_ptr, s + 1, 1)
    row_ptr = np.cumsum(row_ptr, dtype=np.int64).astype(np.int32)
    return row_ptr, d


def _layer_sizes(n: int, n_layers: int) -> List[int]:
    base, extra = divmod(n, n_layers)
    return [base + (1 if i < extra else 0) for i in range(n_layers)]


def _layered_edges(rng: np.random.Generator, sizes: List[int], offset: int,
                   edges: _Edges, kmin: int = 1, kmax: int = 3) -> List[List[int]]:
    """Layered DAG: each node of layer >= 1 draws k ~ U{kmin..kmax} distinct
    predecessors uniformly from all earlier layers.  Returns node ids per layer."""
    layers: List[List[int]] = []
    nxt = offset
    for sz in sizes:
        layers.append(list(range(nxt, nxt + sz)))
        nxt += sz
    for li in range(1, len(layers)):
        earlier = np.arange(offset, layers[li][0], dtype=np.int64)
        for v in layers[li]:
            k = int(rng.integers(kmin, kmax + 1))
            k = min(k, earlier.size)
            preds = rng.choice(earlier, size=k, replace=False)
            for u in sorted(int(p) for p in preds):
                edges.add(u, v)
    return layers


# ----------------------------------------------------------------------------
# Generator families.
# ----------------------------------------------------------------------------

def gen_layered(rng: np.random.Generator, n: int, n_layers: int, offset: int,
                edges: _Edges) -> None:
    _layered_edges(rng, _layer_sizes(n, n_layers), offset, edges)


def gen_inception(rng: np.random.Generator, n: int, n_blocks: int, offset: int,
                  edges: _Edges) -> None:
    """Branching DAG: one input op, then ``n_blocks`` blocks of 4 parallel
    branches of U{3..8} skeleton ops joined by a concat op.  Every skeleton
    branch op is a chain of primitive nodes; chain lengths are spread evenly
    (floor, +1 for the first ones in generation order) so that the total node
    count is exactly ``n``."""
    branch_lens = [[int(rng.integers(3, 9)) for _ in range(4)] for _ in range(n_blocks)]
    n_ops = sum(sum(b) for b in branch_lens)
    n_fixed = 1 + n_blocks
    remaining = n - n_fixed
    if remaining < n_ops:
        raise ValueError("inception graph too small for its skeleton")
    base, extra = divmod(remaining, n_ops)
    nxt = offset
    inp = nxt
    nxt += 1
    op_counter = 0
    for b in range(n_blocks):
        branch_tails = []
        for br in range(4):
            prev = inp
            for _ in range(branch_lens[b][br]):
                c = base + (1 if op_counter < extra else 0)
                op_counter += 1
                first = nxt
                edges.add(prev, first)
                for i in range(1, c):
                    edges.add(first + i - 1, first + i)
                nxt += c
                prev = nxt - 1
            branch_tails.append(prev)
        concat = nxt
        nxt += 1
        for t in branch_tails:
            edges.add(t, concat)
        inp = concat
    assert nxt - offset == n, (nxt - offset, n)


def gen_recurrent(rng: np.random.Generator, n_cells: int, cell_size: int,
                  offset: int, edges: _Edges, cell_layers: int = 10,
                  skip_p: float = 0.05, skip_span: int = 3) -> None:
    """Unrolled recurrent cells: each cell is a layered DAG; every first-layer
    node of cell t+1 takes one edge from a uniform last-layer node of cell t;
    every node of cell t >= 1 takes, with probability ``skip_p``, one skip
    predecessor uniform over the nodes of cells [max(0, t-3), t-1]."""
    sizes = _layer_sizes(cell_size, cell_layers)
    cells = []
    for t in range(n_cells):
        base = offset + t * cell_size
        cells.append(_layered_edges(rng, sizes, base, edges))
    extra_src: List[int] = []
    extra_dst: List[int] = []
    for t in range(1, n_cells):
        last = cells[t - 1][-1]
        for v in cells[t][0]:
            u = last[int(rng.integers(0, len(last)))]
            extra_src.append(u)
            extra_dst.append(v)
        lo = offset + max(0, t - skip_span) * cell_size
        hi = offset + t * cell_size
        for v in range(offset + t * cell_size, offset + (t + 1) * cell_size):
            if rng.random() < skip_p:
                u = int(rng.integers(lo, hi))
                extra_src.append(u)
                extra_dst.append(v)
    for u, v in zip(extra_src, extra_dst):
        edges.add(u, v)


def _lstm_template(rng: np.random.Generator):
    """An 80-node LSTM-cell-like template: layer 0 holds the input slots
    (x, h, c), the last layer the outputs (c', h'); the inside is a layered DAG."""
    sizes = [3, 11, 11, 11, 11, 11, 11, 9, 2]
    assert sum(sizes) == 80
    tmp = _Edges()
    _layered_edges(rng, sizes, 0, tmp)
    return list(zip(tmp.src, tmp.dst)), {"x": 0, "h": 1, "c": 2, "c_out": 78, "h_out": 79}


def gen_gnmt(rng: np.random.Generator, offset: int, edges: _Edges,
             n_layers: int = 8, steps: int = 40) -> int:
    """GNMT-like encoder/decoder: 80 embedding nodes, 8 encoder and 8 decoder
    layers of unrolled 80-node cells over 40 steps, 2 attention nodes (score,
    context) per decoder cell whose score node reads all 40 encoder outputs of
    the same layer (plus the decoder's previous hidden state), and two output
    nodes (projection, loss) per decoder step.  52,000 nodes for the default
    sizes."""
    tmpl_edges, slot = _lstm_template(rng)
    nxt = offset
    enc_emb = list(range(nxt, nxt + steps)); nxt += steps
    dec_emb = list(range(nxt, nxt + steps)); nxt += steps

    def cell(base):
        for (a, b) in tmpl_edges:
            edges.add(base + a, base + b)
        return base

    enc = [[0] * steps for _ in range(n_layers)]
    for l in range(n_layers):
        for t in range(steps):
            base = cell(nxt); nxt += 80
            enc[l][t] = base
            if l == 0:
                edges.add(enc_emb[t], base + slot["x"])
            else:
                edges.add(enc[l - 1][t] + slot["h_out"], base + slot["x"])
            if t > 0:
                edges.add(enc[l][t - 1] + slot["h_out"], base + slot["h"])
                edges.add(enc[l][t - 1] + slot["c_out"], base + slot["c"])
    dec = [[0] * steps for _ in range(n_layers)]
    for l in range(n_layers):
        for t in range(steps):
            score = nxt; context = nxt + 1; nxt += 2
            for te in range(steps):
                edges.add(enc[l][te] + slot["h_out"], score)
            if t > 0:
                edges.add(dec[l][t - 1] + slot["h_out"], score)
            edges.add(score, context)
            base = cell(nxt); nxt += 80
            dec[l][t] = base
            edges.add(context, base + slot["x"])
            if l == 0:
                edges.add(dec_emb[t], base + slot["x"])
            else:
                edges.add(dec[l - 1][t] + slot["h_out"], base + slot["x"])
            if t > 0:
                edges.add(dec[l][t - 1] + slot["h_out"], base + slot["h"])
                edges.add(dec[l][t - 1] + slot["c_out"], base + slot["c"])
    for t in range(steps):
        edges.add(dec[n_layers - 1][t] + slot["h_out"], nxt)
        edges.add(nxt, nxt + 1)
        nxt += 2
    return nxt - offset


# ----------------------------------------------------------------------------
# Graph + features.
# ----------------------------------------------------------------------------

@dataclass
class Graph:
    graph_ptr: np.ndarray   # int32 [G+1]
    row_ptr: np.ndarray     # int32 [N+1] out-edge CSR
    col_idx: np.ndarray     # int32 [E]
    x: np.ndarray           # float64 [N, F] (bf16-rounded values for bf16 configs)
    x_dev: np.ndarray       # float32 or uint16 (bf16 bits) [N, F]

    @property
    def n_nodes(self) -> int:
        return int(self.row_ptr.size - 1)

    @property
    def n_edges(self) -> int:
        return int(self.col_idx.size)

    @property
    def n_graphs(self) -> int:
        return int(self.graph_ptr.size - 1)


def _graph_edges(cfg: Config, rng: np.random.Generator) -> Tuple[List[int], _Edges]:
    edges = _Edges()
    sizes = list(cfg.graph_sizes)
    if cfg.family == "layered":
        gen_layered(rng, sizes[0], 6, 0, edges)
    elif cfg.family == "inception":
        gen_inception(rng, sizes[0], 10, 0, edges)
    elif cfg.family == "recurrent":
        gen_recurrent(rng, sizes[0] // 500, 500, 0, edges)
    elif cfg.family == "ragged":
        off = 0
        gen_layered(rng, sizes[0], 10, off, edges); off += sizes[0]
        gen_inception(rng, sizes[1], 16, off, edges); off += sizes[1]
        gen_recurrent(rng, sizes[2] // 500, 500, off, edges); off += sizes[2]
        gen_recurrent(rng, sizes[3] // 500, 500, off, edges); off += sizes[3]
    elif cfg.family == "gnmt":
        n = gen_gnmt(rng, 0, edges)
        assert n == sizes[0], n
    else:
        raise ValueError(cfg.family)
    return sizes, edges


def make_features(cfg: Config, n: int, rng: np.random.Generator) -> np.ndarray:
    t = cfg.n_types
    types = rng.integers(0, t, size=n)
    x = np.zeros((n, cfg.feat_dim), dtype=np.float64)
    x[np.arange(n), types] = 1.0
    x[:, t:] = rng.lognormal(mean=0.0, sigma=1.0, size=(n, cfg.feat_dim - t))
    return x


def _finish(cfg: Config, arr: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """(float64 values seen by the oracle, device array)."""
    if cfg.dtype == "bf16":
        bits = bf16_bits(arr)
        return bf16_to_f64(bits), bits
    f = np.ascontiguousarray(arr, dtype=np.float32)
    return f.astype(np.float64), f


def make_graph(cfg: Config) -> Graph:
    grng = np.random.default_rng(np.random.SeedSequence([cfg.cfg_id, 0]))
    frng = np.random.default_rng(np.random.SeedSequence([cfg.cfg_id, 1]))
    sizes, edges = _graph_edges(cfg, grng)
    n = int(sum(sizes))
    row_ptr, col_idx = _to_csr(n, np.asarray(edges.src, np.int64), np.asarray(edges.dst, np.int64))
    graph_ptr = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    x64, xdev = _finish(cfg, make_features(cfg, n, frng))
    return Graph(graph_ptr, row_ptr, col_idx, x64, xdev)


def graph_from_arrays(cfg: Config, graph_ptr, row_ptr, col_idx, x) -> Graph:
    x64, xdev = _finish(cfg, np.asarray(x, dtype=np.float64))
    return Graph(np.asarray(graph_ptr, np.int32), np.asarray(row_ptr, np.int32),
                 np.asarray(col_idx, np.int32), x64, xdev)


def prefix_graph(g: Graph, n: int) -> Graph:
    """Induced sub-graph on the first ``n`` nodes of a single-graph workload
    (a valid DAG because ids are topological)."""
    assert g.n_graphs == 1
    e_end = int(g.row_ptr[n])
    cols = g.col_idx[:e_end]
    rows = np.repeat(np.arange(n, dtype=np.int32), np.diff(g.row_ptr[: n + 1]))
    keep = cols < n
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    np.add.at(row_ptr, rows[keep] + 1, 1)
    row_ptr = np.cumsum(row_ptr).astype(np.int32)
    return Graph(np.array([0, n], np.int32), row_ptr, cols[keep].astype(np.int32).copy(),
                 g.x[:n].copy(), g.x_dev[:n].copy())


# ----------------------------------------------------------------------------
# Per-op costs for the simulated run time of a placement (inputs only).
# ----------------------------------------------------------------------------

@dataclass
class OpCosts:
    """Integer inputs of the list-scheduling evaluator: per-op compute time,
    time to ship the op's output to another device and memory held on the op's
    device (time in microseconds, memory in KiB), and each graph's per-device
    memory capacity."""
    op_cost: np.ndarray    # [N] int32
    out_xfer: np.ndarray   # [N] int32
    op_mem: np.ndarray     # [N] int32
    mem_cap: np.ndarray    # [G] int64


def make_costs(cfg: Config, g: "Graph", mem_slack: float = 2.8) -> OpCosts:
    """Costs read off each op's first three log-normal size features (the
    output-shape meta features of Section 3.1), so larger tensors cost more to
    compute, move and hold; a device holds mem_slack times an even share of its
    graph's memory."""
    s = g.x[:, cfg.n_types:cfg.n_types + 3]
    op_cost = np.clip(1 + np.floor(20.0 * s[:, 0]), 1, 5000).astype(np.int32)
    out_xfer = np.clip(np.floor(10.0 * s[:, 1]), 0, 5000).astype(np.int32)
    op_mem = np.clip(1 + np.floor(100.0 * s[:, 2]), 1, 100000).astype(np.int32)
    gp = g.graph_ptr
    cap = np.array([int(np.ceil(mem_slack * int(op_mem[gp[i]:gp[i + 1]].astype(np.int64).sum()) / cfg.n_devices))
                    for i in range(len(gp) - 1)], np.int64)
    return OpCosts(op_cost, out_xfer, op_mem, cap)


# ----------------------------------------------------------------------------
# Weights.
# ----------------------------------------------------------------------------

def _xavier(rng, out_dim, in_dim):
    a = np.sqrt(6.0 / (in_dim + out_dim))
    return rng.uniform(-a, a, size=(out_dim, in_dim))


def _bias(rng, n):
    return rng.uniform(-0.05, 0.05, size=n)


@dataclass
class Weights:
    """Each entry maps a name to (float64 values, device array)."""
    gnn: List[Dict[str, Tuple[np.ndarray, np.ndarray]]] = field(default_factory=list)
    placer: List[Dict[str, Tuple[np.ndarray, np.ndarray]]] = field(default_factory=list)
    head: Dict[str, Tuple[np.ndarray, np.ndarray]] = field(default_factory=dict)

    def f64(self):
        """Plain float64 dictionaries (what the oracle consumes)."""
        return ([{k: v[0] for k, v in l.items()} for l in self.gnn],
                [{k: v[0] for k, v in l.items()} for l in self.placer],
                {k: v[0] for k, v in self.head.items()})


GNN_KEYS = ("w_pool", "b_pool", "w_self", "w_neigh", "b_upd")
PLACER_KEYS = ("film_wg", "film_bg", "film_wb", "film_bb", "w_qkv", "b_qkv", "w_o", "b_o",
               "ln1_g", "ln1_b", "w_1", "b_1", "w_2", "b_2", "ln2_g", "ln2_b")


def make_weights(cfg: Config, film_scale: float = 1.0) -> Weights:
    rng = np.random.default_rng(np.random.SeedSequence([cfg.cfg_id, 2]))
    H, F, d, dff, D = cfg.hidden, cfg.feat_dim, cfg.d_model, cfg.d_ff, cfg.n_devices
    w = Weights()
    fin = lambda a: _finish(cfg, a)
    for l in range(cfg.gnn_layers):
        hin = F if l == 0 else H
        w.gnn.append({
            "w_pool": fin(_xavier(rng, H, hin)),
            "b_pool": fin(_bias(rng, H)),
            "w_self": fin(_xavier(rng, H, hin)),
            "w_neigh": fin(_xavier(rng, H, H)),
            "b_upd": fin(_bias(rng, H)),
        })
    for l in range(cfg.placer_layers):
        w.placer.append({
            "film_wg": fin(film_scale * _xavier(rng, d, H)),
            "film_bg": fin(_bias(rng, d)),
            "film_wb": fin(film_scale * _xavier(rng, d, H)),
            "film_bb": fin(_bias(rng, d)),
            "w_qkv": fin(_xavier(rng, 3 * d, d)),
            "b_qkv": fin(_bias(rng, 3 * d)),
            "w_o": fin(_xavier(rng, d, d)),
            "b_o": fin(_bias(rng, d)),
            "ln1_g": fin(1.0 + rng.uniform(-0.1, 0.1, size=d)),
            "ln1_b": fin(rng.uniform(-0.1, 0.1, size=d)),
            "w_1": fin(_xavier(rng, dff, d)),
            "b_1": fin(_bias(rng, dff)),
            "w_2": fin(_xavier(rng, d, dff)),
            "b_2": fin(_bias(rng, d)),
            "ln2_g": fin(1.0 + rng.uniform(-0.1, 0.1, size=d)),
            "ln2_b": fin(rng.uniform(-0.1, 0.1, size=d)),
        })
    w.head = {"w_out": fin(_xavier(rng, D, d)), "b_out": fin(_bias(rng, D))}
    return w


def make_workload(cfg: Config):
    return make_graph(cfg), make_weights(cfg)


def graph_stats(g: Graph, fanout: int) -> Dict[str, float]:
    """Degree statistics used for the algorithmic-bytes model of the gather."""
    n = g.n_nodes
    out_deg = np.diff(g.row_ptr).astype(np.int64)
    in_deg = np.bincount(g.col_idx, minlength=n).astype(np.int64)
    deg = out_deg + in_deg
    s = np.minimum(deg, fanout)
    return {"n": n, "e": g.n_edges, "sum_s": int(s.sum()), "mean_s": float(s.mean()),
            "max_deg": int(deg.max()), "frac_sampled": float((deg > fanout).mean())}
