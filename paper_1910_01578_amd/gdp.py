"""Thin ctypes binding of libgdp (the C ABI in include/gdp.h).

Only argument marshalling happens here: torch tensors provide device memory
and the current HIP stream; every step of the forward pass runs in the
library's HIP kernels.  Importing this module fails loudly when libgdp.so has
not been built -- there is no CPU fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgdp.so")

GDP_OK = 0
GDP_E_INVALID_ARG = -1
GDP_E_BAD_GRAPH = -2
GDP_E_UNSUPPORTED = -3
GDP_E_WORKSPACE = -4
GDP_E_HIP = -5
GDP_F32 = 0
GDP_BF16 = 1
GDP_TOPO_IDS = 1
GDP_MAX_GRAPHS = 128
GDP_NOALLOC_SCRATCH_BYTES = 4 << 20

KERNEL_KINDS = ["graph_prep", "nbr_sample", "gemm_pool_sigmoid", "gather_max", "gemm_update_relu",
                "meanpool", "film", "pre_layer", "seg_attention", "post_attn",
                "head_lse", "gumbel_sample", "logp_reduce", "mlp_placer", "ppo_grad", "head_backward", "advantages",
                "evaluate", "train_forward", "backward", "adam", "log_prob", "gemm_update_pool"]
K_COUNT = len(KERNEL_KINDS)


class GdpError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libgdp error {code}: {msg}")
        self.code = code


class GdpGraph(ctypes.Structure):
    _fields_ = [("n_graphs", c_int32), ("graph_ptr_h", POINTER(c_int32)), ("n_nodes", c_int32),
                ("row_ptr", c_void_p), ("col_idx", c_void_p), ("n_edges", c_int64), ("x", c_void_p),
                ("feat_dim", c_int32), ("dtype", c_int32), ("flags", c_uint32)]


class GdpGnnLayer(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_pool", "b_pool", "w_self", "w_neigh", "b_upd")]


class GdpGnn(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("in_dim", c_int32), ("hidden", c_int32), ("fanout", c_int32),
                ("nbr_seed", c_uint64), ("layers", POINTER(GdpGnnLayer))]


PLACER_LAYER_FIELDS = ("film_wg", "film_bg", "film_wb", "film_bb", "w_qkv", "b_qkv", "w_o", "b_o",
                       "ln1_g", "ln1_b", "w_1", "b_1", "w_2", "b_2", "ln2_g", "ln2_b")


class GdpPlacerLayer(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in PLACER_LAYER_FIELDS]


class GdpPlacer(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("d_ff", c_int32),
                ("seg_len", c_int32), ("mem_len", c_int32), ("n_devices", c_int32), ("film", c_int32),
                ("attention", c_int32),
                ("layers", POINTER(GdpPlacerLayer)), ("w_out", c_void_p), ("b_out", c_void_p)]


class GdpGnnLayerGrad(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_pool", "b_pool", "w_self", "w_neigh", "b_upd")]


class GdpPlacerLayerGrad(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in PLACER_LAYER_FIELDS]


class GdpGrads(ctypes.Structure):
    _fields_ = [("gnn", POINTER(GdpGnnLayerGrad)), ("placer", POINTER(GdpPlacerLayerGrad)), ("w_out", c_void_p),
                ("b_out", c_void_p)]


class GdpAdamTensor(ctypes.Structure):
    _fields_ = [("param", c_void_p), ("master", c_void_p), ("grad", c_void_p), ("m", c_void_p), ("v", c_void_p),
                ("n", c_int64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_1910_01578_amd.build_lib` "
                          "(there is no fallback path)")
    # torch ships its own HIP runtime under the same soname (libamdhip64.so.7).
    # Loading torch first makes libgdp bind to that copy; loaded the other way
    # round the process would hold two runtimes, and pointers and streams from
    # torch would not be valid in the one libgdp calls.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "gdp_workspace_bytes": (c_size_t, [POINTER(GdpGraph), POINTER(GdpGnn), POINTER(GdpPlacer), c_int32]),
        "gdp_embed": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), c_void_p, c_void_p, c_void_p, c_size_t,
                                c_void_p]),
        "gdp_place": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, POINTER(GdpPlacer), c_void_p, c_void_p,
                                c_void_p, c_size_t, c_void_p]),
        "gdp_sample": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, c_int32, c_int32, c_uint64, c_void_p,
                                 c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
        "gdp_place_sample": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, POINTER(GdpPlacer), c_void_p,
                                       c_void_p, c_int32, c_uint64, c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_size_t, c_void_p]),
        "gdp_sample_noalloc": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, c_int32, c_int32, c_uint64,
                                         c_void_p, c_void_p, c_void_p, c_void_p]),
        "gdp_evaluate_workspace_bytes": (c_size_t, [POINTER(GdpGraph), c_int32, c_int32]),
        "gdp_evaluate": (c_int32, [POINTER(GdpGraph), c_int32, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                   POINTER(c_int64), c_double, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                   c_void_p]),
        "gdp_train_sizes": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), POINTER(GdpPlacer), POINTER(c_size_t),
                                      POINTER(c_size_t)]),
        "gdp_forward_train": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), POINTER(GdpPlacer), c_void_p, c_size_t,
                                        c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
        "gdp_backward": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), POINTER(GdpPlacer), c_void_p, c_size_t,
                                   c_void_p, POINTER(GdpGrads), c_void_p, c_size_t, c_void_p]),
        "gdp_log_prob": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                   c_void_p, c_size_t, c_void_p]),
        "gdp_adam_step": (c_int32, [c_int32, POINTER(GdpAdamTensor), c_int32, c_float, c_float, c_float, c_float,
                                    c_int64, c_void_p]),
        "gdp_debug_train_tensor": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), POINTER(GdpPlacer), c_void_p,
                                             c_size_t, c_int32, c_int32, c_void_p, c_size_t, c_void_p]),
        "gdp_validate_graph_host": (c_int32, [c_void_p, c_int32, c_void_p, c_int32, c_void_p, c_int64, c_uint32]),
        "gdp_last_error": (c_char_p, []),
        "gdp_abi_version": (c_int32, []),
        "gdp_advantages": (c_int32, [c_int32, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p]),
        "gdp_place_train": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, POINTER(GdpPlacer), c_void_p, c_void_p,
                                      c_void_p, c_void_p, c_size_t, c_void_p]),
        "gdp_head_backward": (c_int32, [POINTER(GdpGraph), POINTER(GdpPlacer), c_void_p, c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_size_t, c_void_p]),
        "gdp_ppo_grad": (c_int32, [POINTER(GdpGraph), c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                   c_void_p, c_void_p, c_float, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
        "gdp_debug_uniforms": (c_int32, [c_uint64, c_int32, c_int32, c_int32, c_void_p, c_void_p]),
        "gdp_debug_neighbors": (c_int32, [POINTER(GdpGraph), POINTER(GdpGnn), c_void_p, c_void_p, c_int64,
                                          c_void_p, c_size_t, c_void_p]),
        "gdp_set_place_streams": (c_int32, [c_int32]),
        "gdp_timer_begin": (c_int32, [c_uint32]),
        "gdp_timer_end": (c_int32, [POINTER(c_double), POINTER(c_int64)]),
        "gdp_kernel_kind_name": (c_char_p, [c_int32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()


def last_error() -> str:
    return lib.gdp_last_error().decode()


def check(code: int):
    if code != GDP_OK:
        raise GdpError(code, last_error())


def abi_version() -> int:
    return lib.gdp_abi_version()


def validate_graph_host(graph_ptr, row_ptr, col_idx, flags: int = GDP_TOPO_IDS) -> int:
    gp = np.ascontiguousarray(graph_ptr, np.int32)
    rp = np.ascontiguousarray(row_ptr, np.int32)
    ci = np.ascontiguousarray(col_idx, np.int32)
    return lib.gdp_validate_graph_host(gp.ctypes.data, gp.size - 1, rp.ctypes.data, rp.size - 1,
                                       ci.ctypes.data if ci.size else None, ci.size, flags)


# ----------------------------------------------------------------------------
# torch-facing helpers: device memory and the current stream only.
# ----------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream_handle(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def to_device(arr: np.ndarray, dtype: str, device="cuda"):
    """Upload a float32 array (dtype "f32") or uint16 bf16 bit patterns ("bf16")."""
    torch = _torch()
    a = np.ascontiguousarray(arr)
    if dtype == "bf16":
        assert a.dtype == np.uint16
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    assert a.dtype == np.float32
    return torch.from_numpy(a).to(device)


class DeviceGraph:
    """A graph batch resident in device memory plus its C descriptor."""

    def __init__(self, graph, dtype: str, device="cuda", flags: int = GDP_TOPO_IDS):
        torch = _torch()
        self.dtype = dtype
        self.graph_ptr = np.ascontiguousarray(graph.graph_ptr, np.int32)
        self.row_ptr = torch.from_numpy(np.ascontiguousarray(graph.row_ptr, np.int32)).to(device)
        ci = np.ascontiguousarray(graph.col_idx, np.int32)
        self.col_idx = torch.from_numpy(ci if ci.size else np.zeros(1, np.int32)).to(device)
        self.x = to_device(graph.x_dev, dtype, device)
        self.n_nodes = int(graph.row_ptr.size - 1)
        self.n_edges = int(ci.size)
        self.feat_dim = int(graph.x_dev.shape[1])
        self.n_graphs = int(self.graph_ptr.size - 1)
        self.c = GdpGraph(self.n_graphs, self.graph_ptr.ctypes.data_as(POINTER(c_int32)), self.n_nodes,
                          self.row_ptr.data_ptr(), self.col_idx.data_ptr(), self.n_edges, self.x.data_ptr(),
                          self.feat_dim, GDP_BF16 if dtype == "bf16" else GDP_F32, flags)


class DevicePolicy:
    """Policy weights resident in device memory plus the C descriptors."""

    def __init__(self, cfg, weights, device="cuda", film: Optional[bool] = None,
                 attention: Optional[bool] = None):
        self.cfg = cfg
        dt = cfg.dtype
        up = lambda pair: to_device(pair[1], dt, device)
        self.gnn_t = [{k: up(v) for k, v in l.items()} for l in weights.gnn]
        self.placer_t = [{k: up(v) for k, v in l.items()} for l in weights.placer]
        self.head_t = {k: up(v) for k, v in weights.head.items()}
        L = len(self.gnn_t)
        self._gl = (GdpGnnLayer * L)(*[GdpGnnLayer(*[l[k].data_ptr() for k in ("w_pool", "b_pool", "w_self",
                                                                              "w_neigh", "b_upd")])
                                       for l in self.gnn_t])
        self.gnn = GdpGnn(L, cfg.feat_dim, cfg.hidden, cfg.fanout, cfg.nb_seed, self._gl)
        P = len(self.placer_t)
        self._pl = (GdpPlacerLayer * P)(*[GdpPlacerLayer(*[l[k].data_ptr() for k in PLACER_LAYER_FIELDS])
                                          for l in self.placer_t])
        use_film = cfg.film if film is None else film
        use_attention = cfg.attention if attention is None else attention
        self.placer = GdpPlacer(P, cfg.d_model, cfg.heads, cfg.d_ff, cfg.seg_len, cfg.mem_len, cfg.n_devices,
                                1 if use_film else 0, 1 if use_attention else 0, self._pl,
                                self.head_t["w_out"].data_ptr(), self.head_t["b_out"].data_ptr())


class Runner:
    """Owns the outputs and the workspace of one (graph, policy, K) problem."""

    def __init__(self, graph: DeviceGraph, policy: DevicePolicy, k_samples: int, device="cuda"):
        torch = _torch()
        self.graph, self.policy, self.k = graph, policy, int(k_samples)
        cfg = policy.cfg
        tdt = torch.bfloat16 if graph.dtype == "bf16" else torch.float32
        N, G, H, D = graph.n_nodes, graph.n_graphs, cfg.hidden, cfg.n_devices
        self.ws_bytes = lib.gdp_workspace_bytes(ctypes.byref(graph.c), ctypes.byref(policy.gnn),
                                                ctypes.byref(policy.placer), self.k)
        if self.ws_bytes == 0:
            raise GdpError(GDP_E_INVALID_ARG, last_error())
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.node_emb = torch.empty((N, H), dtype=tdt, device=device)
        self.graph_emb = torch.empty((G, H), dtype=torch.float32, device=device)
        self.logits = torch.empty((N, D), dtype=torch.float32, device=device)
        self.lse = torch.empty((N,), dtype=torch.float32, device=device)
        self.placements = torch.empty((self.k, N), dtype=torch.int32, device=device)
        self.logp = torch.empty((G, self.k), dtype=torch.float32, device=device)

    def embed(self, stream=None):
        check(lib.gdp_embed(ctypes.byref(self.graph.c), ctypes.byref(self.policy.gnn), self.node_emb.data_ptr(),
                            self.graph_emb.data_ptr(), self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))

    def place(self, stream=None):
        check(lib.gdp_place(ctypes.byref(self.graph.c), self.node_emb.data_ptr(), self.graph_emb.data_ptr(),
                            ctypes.byref(self.policy.placer), self.logits.data_ptr(), self.lse.data_ptr(),
                            self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))

    def place_train(self, stream=None):
        """place() that also keeps the placement network's output X [N, d] (fp32),
        the head's input, for head_backward(); returns X."""
        torch = _torch()
        x = torch.empty((self.graph.n_nodes, self.policy.cfg.d_model), dtype=torch.float32, device=self.ws.device)
        check(lib.gdp_place_train(ctypes.byref(self.graph.c), self.node_emb.data_ptr(), self.graph_emb.data_ptr(),
                                  ctypes.byref(self.policy.placer), self.logits.data_ptr(), self.lse.data_ptr(),
                                  x.data_ptr(), self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))
        return x

    def head_backward(self, x, dlogits, stream=None):
        """The head's backward pass for dL/dlogits: returns (dx, dw_out, db_out), fp32."""
        torch = _torch()
        N, d, D = self.graph.n_nodes, self.policy.cfg.d_model, self.policy.cfg.n_devices
        dev = self.ws.device
        dx = torch.empty((N, d), dtype=torch.float32, device=dev)
        dw = torch.empty((D, d), dtype=torch.float32, device=dev)
        db = torch.empty((D,), dtype=torch.float32, device=dev)
        check(lib.gdp_head_backward(ctypes.byref(self.graph.c), ctypes.byref(self.policy.placer), x.data_ptr(),
                                    dlogits.data_ptr(), dx.data_ptr(), dw.data_ptr(), db.data_ptr(),
                                    self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))
        return dx, dw, db

    def sample(self, seed: int, uniforms=None, use_lse: bool = True, stream=None):
        check(lib.gdp_sample(ctypes.byref(self.graph.c), self.logits.data_ptr(),
                             self.lse.data_ptr() if use_lse else None, self.policy.cfg.n_devices, self.k, seed,
                             None if uniforms is None else uniforms.data_ptr(), self.placements.data_ptr(),
                             self.logp.data_ptr(), self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))

    def sample_noalloc(self, seed: int, placements=None, logp=None, uniforms=None, use_lse: bool = True,
                       stream=None):
        """sample() through gdp_sample_noalloc (no workspace: the library's own
        per-device scratch array); writes into the given or the runner's outputs."""
        placements = self.placements if placements is None else placements
        logp = self.logp if logp is None else logp
        check(lib.gdp_sample_noalloc(ctypes.byref(self.graph.c), self.logits.data_ptr(),
                                     self.lse.data_ptr() if use_lse else None, self.policy.cfg.n_devices,
                                     int(placements.shape[0]), seed,
                                     None if uniforms is None else uniforms.data_ptr(), placements.data_ptr(),
                                     logp.data_ptr(), _stream_handle(stream)))

    def place_sample(self, seed: int, uniforms=None, use_lse: bool = True, stream=None):
        """place() then sample() as one call (gdp_place_sample); with use_lse
        False the placer writes no lse and the sampling forms it."""
        check(lib.gdp_place_sample(ctypes.byref(self.graph.c), self.node_emb.data_ptr(), self.graph_emb.data_ptr(),
                                   ctypes.byref(self.policy.placer), self.logits.data_ptr(),
                                   self.lse.data_ptr() if use_lse else None, self.k, seed,
                                   None if uniforms is None else uniforms.data_ptr(), self.placements.data_ptr(),
                                   self.logp.data_ptr(), self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))

    def forward(self, seed: int, stream=None):
        """One pass of the hot path: embed -> place -> sample (the last two as one call)."""
        self.embed(stream)
        self.place_sample(seed, stream=stream)

    def ppo_grad(self, logp_old, advantages, clip_eps: float = 0.2, use_lse: bool = True, stream=None):
        """PPO's clipped surrogate per graph and its gradient with respect to the
        logits, for the placements and log-probs of the last sample() call."""
        torch = _torch()
        G, N, D = self.graph.n_graphs, self.graph.n_nodes, self.policy.cfg.n_devices
        loss = torch.empty((G,), dtype=torch.float32, device=self.ws.device)
        dlogits = torch.empty((N, D), dtype=torch.float32, device=self.ws.device)
        check(lib.gdp_ppo_grad(ctypes.byref(self.graph.c), self.logits.data_ptr(),
                               self.lse.data_ptr() if use_lse else None, D, self.k, self.placements.data_ptr(),
                               self.logp.data_ptr(), logp_old.data_ptr(), advantages.data_ptr(), float(clip_eps),
                               loss.data_ptr(), dlogits.data_ptr(), self.ws.data_ptr(), self.ws_bytes,
                               _stream_handle(stream)))
        return loss, dlogits

    def neighbors(self, stream=None):
        torch = _torch()
        n = self.graph.n_nodes
        cap = max(1, min(2 * self.graph.n_edges, n * self.policy.cfg.fanout))
        s_ptr = torch.empty(n + 1, dtype=torch.int32, device=self.ws.device)
        s_idx = torch.empty(cap, dtype=torch.int32, device=self.ws.device)
        check(lib.gdp_debug_neighbors(ctypes.byref(self.graph.c), ctypes.byref(self.policy.gnn), s_ptr.data_ptr(),
                                      s_idx.data_ptr(), cap, self.ws.data_ptr(), self.ws_bytes,
                                      _stream_handle(stream)))
        return s_ptr, s_idx


class Evaluator:
    """Simulated run time and validity of sampled placements (gdp_evaluate) for
    one graph batch: per-op costs in device memory, the workspace, the outputs."""

    def __init__(self, graph: DeviceGraph, n_devices: int, k_samples: int, costs, device="cuda"):
        torch = _torch()
        self.graph, self.D, self.k = graph, int(n_devices), int(k_samples)
        up = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(device)
        self.op_cost, self.out_xfer, self.op_mem = up(costs.op_cost), up(costs.out_xfer), up(costs.op_mem)
        self.mem_cap = np.ascontiguousarray(costs.mem_cap, np.int64)
        self.ws_bytes = lib.gdp_evaluate_workspace_bytes(ctypes.byref(graph.c), self.D, self.k)
        if self.ws_bytes == 0:
            raise GdpError(GDP_E_INVALID_ARG, last_error())
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        G = graph.n_graphs
        self.makespan = torch.empty((G, self.k), dtype=torch.int64, device=device)
        self.valid = torch.empty((G, self.k), dtype=torch.uint8, device=device)
        self.run_time = torch.empty((G, self.k), dtype=torch.float32, device=device)

    def evaluate(self, placements, time_unit: float = 1e-6, stream=None):
        """placements [K, N] int32 (device); returns (makespan, valid, run_time)."""
        assert tuple(placements.shape) == (self.k, self.graph.n_nodes)
        check(lib.gdp_evaluate(ctypes.byref(self.graph.c), self.D, self.k, placements.data_ptr(),
                               self.op_cost.data_ptr(), self.out_xfer.data_ptr(), self.op_mem.data_ptr(),
                               self.mem_cap.ctypes.data_as(POINTER(c_int64)), float(time_unit),
                               self.makespan.data_ptr(), self.valid.data_ptr(), self.run_time.data_ptr(),
                               self.ws.data_ptr(), self.ws_bytes, _stream_handle(stream)))
        return self.makespan, self.valid, self.run_time


class Trainer:
    """The update step of a policy on one graph batch (Section 3, PPO): the
    training forward that keeps every intermediate in a store, the log-probs of
    given placements, the backward pass into fp32 gradients shaped like the
    weights, and Adam on fp32 master copies (the policy's own device weights,
    in its dtype, are rewritten after every step)."""

    def __init__(self, graph: DeviceGraph, policy: DevicePolicy, k_samples: int, device="cuda"):
        torch = _torch()
        self.graph, self.policy, self.k = graph, policy, int(k_samples)
        sb, wb = c_size_t(0), c_size_t(0)
        check(lib.gdp_train_sizes(ctypes.byref(graph.c), ctypes.byref(policy.gnn), ctypes.byref(policy.placer),
                                  ctypes.byref(sb), ctypes.byref(wb)))
        self.store_bytes, self.ws_bytes = sb.value, wb.value
        self.store = torch.empty(self.store_bytes, dtype=torch.uint8, device=device)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        self.sample_ws_bytes = lib.gdp_workspace_bytes(ctypes.byref(graph.c), None, None, self.k)
        self.sample_ws = torch.empty(max(1, self.sample_ws_bytes), dtype=torch.uint8, device=device)
        N, G, D = graph.n_nodes, graph.n_graphs, policy.cfg.n_devices
        self.logits = torch.empty((N, D), dtype=torch.float32, device=device)
        self.lse = torch.empty((N,), dtype=torch.float32, device=device)
        z = lambda t: torch.zeros(t.shape, dtype=torch.float32, device=device)
        self.grad_gnn = [{k: z(v) for k, v in l.items()} for l in policy.gnn_t]
        self.grad_placer = [{k: z(v) for k, v in l.items()} for l in policy.placer_t]
        self.grad_head = {k: z(v) for k, v in policy.head_t.items()}
        self._gg = (GdpGnnLayerGrad * len(self.grad_gnn))(
            *[GdpGnnLayerGrad(*[l[k].data_ptr() for k in ("w_pool", "b_pool", "w_self", "w_neigh", "b_upd")])
              for l in self.grad_gnn])
        self._gp = (GdpPlacerLayerGrad * len(self.grad_placer))(
            *[GdpPlacerLayerGrad(*[l[k].data_ptr() for k in PLACER_LAYER_FIELDS]) for l in self.grad_placer])
        self.grads = GdpGrads(self._gg, self._gp, self.grad_head["w_out"].data_ptr(),
                              self.grad_head["b_out"].data_ptr())
        # Adam: master copies and moments of every weight, in one list
        pairs = []
        for lw, lg in zip(policy.gnn_t, self.grad_gnn):
            pairs += [(lw[k], lg[k]) for k in lw]
        for lw, lg in zip(policy.placer_t, self.grad_placer):
            pairs += [(lw[k], lg[k]) for k in lw]
        pairs += [(policy.head_t[k], self.grad_head[k]) for k in policy.head_t]
        self._adam = []
        for prm, grd in pairs:
            master = prm.float().clone()
            self._adam.append((prm, master, grd, torch.zeros_like(master), torch.zeros_like(master)))
        self._adam_c = (GdpAdamTensor * len(self._adam))(
            *[GdpAdamTensor(prm.data_ptr(), ms.data_ptr(), grd.data_ptr(), m.data_ptr(), v.data_ptr(), prm.numel())
              for prm, ms, grd, m, v in self._adam])
        self.step_count = 0

    def forward(self, stream=None):
        """The training forward; returns (logits, lse) of the current weights."""
        check(lib.gdp_forward_train(ctypes.byref(self.graph.c), ctypes.byref(self.policy.gnn),
                                    ctypes.byref(self.policy.placer), self.store.data_ptr(), self.store_bytes,
                                    self.logits.data_ptr(), self.lse.data_ptr(), self.ws.data_ptr(), self.ws_bytes,
                                    _stream_handle(stream)))
        return self.logits, self.lse

    def log_prob(self, placements, stream=None):
        """log pi(placements) [G, K] under the last forward's logits."""
        torch = _torch()
        logp = torch.empty((self.graph.n_graphs, int(placements.shape[0])), dtype=torch.float32,
                           device=self.logits.device)
        check(lib.gdp_log_prob(ctypes.byref(self.graph.c), self.logits.data_ptr(), self.lse.data_ptr(),
                               self.policy.cfg.n_devices, int(placements.shape[0]), placements.data_ptr(),
                               logp.data_ptr(), self.sample_ws.data_ptr(), self.sample_ws_bytes,
                               _stream_handle(stream)))
        return logp

    def ppo_grad(self, placements, logp, logp_old, advantages, clip_eps=0.2, stream=None):
        """PPO's clipped surrogate and dL/dlogits at the last forward's logits."""
        torch = _torch()
        G, N, D = self.graph.n_graphs, self.graph.n_nodes, self.policy.cfg.n_devices
        K = int(placements.shape[0])
        loss = torch.empty((G,), dtype=torch.float32, device=self.logits.device)
        dlogits = torch.empty((N, D), dtype=torch.float32, device=self.logits.device)
        check(lib.gdp_ppo_grad(ctypes.byref(self.graph.c), self.logits.data_ptr(), self.lse.data_ptr(), D, K,
                               placements.data_ptr(), logp.data_ptr(), logp_old.data_ptr(), advantages.data_ptr(),
                               float(clip_eps), loss.data_ptr(), dlogits.data_ptr(), self.sample_ws.data_ptr(),
                               self.sample_ws_bytes, _stream_handle(stream)))
        return loss, dlogits

    def backward(self, dlogits, stream=None):
        """Gradients of sum(dlogits * logits) into grad_gnn / grad_placer / grad_head."""
        check(lib.gdp_backward(ctypes.byref(self.graph.c), ctypes.byref(self.policy.gnn),
                               ctypes.byref(self.policy.placer), self.store.data_ptr(), self.store_bytes,
                               dlogits.data_ptr(), ctypes.byref(self.grads), self.ws.data_ptr(), self.ws_bytes,
                               _stream_handle(stream)))

    def decisions(self, stream=None):
        """The last forward's discrete choices, for comparisons that take them the
        same way: {"gnn": [(winning neighbour [N, H], ReLU sign [N, H])] per GNN
        layer, "ffn": [ReLU sign [N, d_ff]] per placer layer} (numpy)."""
        torch = _torch()
        N, H, dff = self.graph.n_nodes, self.policy.cfg.hidden, self.policy.cfg.d_ff
        dev = self.store.device

        def get(which, layer, shape, dtype):
            out = torch.empty(shape, dtype=dtype, device=dev)
            check(lib.gdp_debug_train_tensor(ctypes.byref(self.graph.c), ctypes.byref(self.policy.gnn),
                                             ctypes.byref(self.policy.placer), self.store.data_ptr(), self.store_bytes,
                                             which, layer, out.data_ptr(), out.numel() * out.element_size(),
                                             _stream_handle(stream)))
            return out
        gnn = []
        for l in range(len(self.policy.gnn_t)):
            arg = get(2, l, (N, H), torch.int32).cpu().numpy()
            sign = (get(1, l, (N, H), torch.float32) > 0).cpu().numpy()
            gnn.append((arg, sign))
        ffn = [(get(0, l, (N, dff), torch.float32) > 0).cpu().numpy() for l in range(len(self.policy.placer_t))]
        return {"gnn": gnn, "ffn": ffn}

    def adam(self, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, stream=None):
        """One Adam step on every weight (master copies in fp32)."""
        self.step_count += 1
        dt = GDP_BF16 if self.graph.dtype == "bf16" else GDP_F32
        check(lib.gdp_adam_step(len(self._adam), self._adam_c, dt, float(lr), float(beta1), float(beta2), float(eps),
                                self.step_count, _stream_handle(stream)))


class RewardBaseline:
    """Section 4's reward and advantage with the running average of previous
    trials as the bias, one state per graph (device fp64 sums, int64 counts)."""

    def __init__(self, n_graphs: int, device="cuda"):
        torch = _torch()
        self.reward_sum = torch.zeros(n_graphs, dtype=torch.float64, device=device)
        self.trial_count = torch.zeros(n_graphs, dtype=torch.int64, device=device)

    def advantages(self, run_time, valid=None, stream=None):
        """run_time [G, K] fp32 (device), valid [G, K] uint8 or None; returns
        (reward, advantage), both [G, K] fp32, and advances the state."""
        torch = _torch()
        G, K = run_time.shape
        reward = torch.empty_like(run_time)
        adv = torch.empty_like(run_time)
        check(lib.gdp_advantages(G, K, run_time.data_ptr(), None if valid is None else valid.data_ptr(),
                                 self.reward_sum.data_ptr(), self.trial_count.data_ptr(), reward.data_ptr(),
                                 adv.data_ptr(), _stream_handle(stream)))
        return reward, adv


def debug_uniforms(seed: int, n: int, k: int, d: int, device="cuda", stream=None):
    torch = _torch()
    out = torch.empty((k, n, d), dtype=torch.float32, device=device)
    check(lib.gdp_debug_uniforms(seed, n, k, d, out.data_ptr(), _stream_handle(stream)))
    return out


def set_place_streams(n: int) -> None:
    """gdp_place's stream schedule for this thread: 2 (the default) splits a
    large placer pass into two row parts on two streams, 1 keeps every launch
    on the caller's stream.  The results are the same bit for bit."""
    check(lib.gdp_set_place_streams(int(n)))


def timer_begin(kinds) -> None:
    mask = 0
    for k in kinds:
        mask |= 1 << (KERNEL_KINDS.index(k) if isinstance(k, str) else int(k))
    check(lib.gdp_timer_begin(mask))


def timer_end() -> Dict[str, Dict[str, float]]:
    ms = (c_double * K_COUNT)()
    cnt = (c_int64 * K_COUNT)()
    check(lib.gdp_timer_end(ms, cnt))
    return {KERNEL_KINDS[i]: {"ms": ms[i], "launches": int(cnt[i])} for i in range(K_COUNT) if cnt[i]}
