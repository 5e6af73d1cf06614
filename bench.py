#!/usr/bin/env python3
"""Throughput of the GDP policy hot path on one MI355X.

One step = one full pass of the hot path over the 52,000-node GNMT-8-like
dataflow DAG: gdp_embed (3 GraphSAGE max-pool layers) -> gdp_place (6
segment-recurrent attention layers with FiLM conditioning, device logits) ->
gdp_sample (64 whole-graph placements + log-probs).  Inputs are synthetic and
resident in device memory before the timed region starts.

Prints one JSON line.  `value` is nodes per second (N nodes per step).
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "policy fwd+sample nodes/sec on 50k-node DAG; % HBM / MFMA roofline"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0


def flop_model(cfg, g, stats, fused_gnn=False, launches=None):
    """Algorithmic work per launch of each kernel kind (one layer's launch).

    fused_gnn: the run formed each layer's transform inside the previous
    layer's update (kind gemm_update_pool), so the separate transform ran for
    layer 0 only and the plain update for the last layer only.
    launches: launches per step of each kind, where the run split a layer's
    kernels over two row ranges (two launches each); the work of a step is
    then averaged over its launches.

    GEMMs: 2 * M * K * N.  Attention: 4 * d * sum over queries of the keys it
    attends to (QK^T and PV, all heads).  Gather-max: bytes of the sampled
    neighbour rows and their ids, the pointer array and the output rows."""
    N, H, F, d, dff = g.n_nodes, cfg.hidden, cfg.feat_dim, cfg.d_model, cfg.d_ff
    b = 2 if cfg.dtype == "bf16" else 4
    keys = 0
    gp = g.graph_ptr
    for gi in range(len(gp) - 1):
        gs, ge = int(gp[gi]), int(gp[gi + 1])
        for q0 in range(gs, ge, cfg.seg_len):
            q1 = min(q0 + cfg.seg_len, ge)
            keys += (q1 - q0) * (q1 - max(gs, q0 - cfg.mem_len))
    L = cfg.gnn_layers
    pool = [2.0 * N * (F if l == 0 else H) * H for l in range(L)]
    upd = [2.0 * N * ((F if l == 0 else H) + H) * H for l in range(L)]
    gather_bytes = stats["sum_s"] * (H * b + 4) + N * H * b + 4 * (N + 1)
    fused = [upd[l] + pool[l + 1] for l in range(L - 1)]
    P = cfg.placer_layers
    # per step, with the launch count of the one-stream schedule: the GNN's
    # transforms, gathers and updates (fused: layer l's update with layer
    # l + 1's transform), one projection, P attention and P post-attention
    # passes (W_o, the FFN, and all but the last layer's next QKV projection)
    step = {"gemm_pool_sigmoid": (pool[0], 1) if fused_gnn else (sum(pool), L),
            "gemm_update_relu": (upd[-1], 1) if fused_gnn else (sum(upd), L),
            "gemm_update_pool": (sum(fused), L - 1) if fused_gnn and fused else (0.0, 1),
            "gather_max": (L * gather_bytes, L),
            "pre_layer": (2.0 * N * d * 3 * d, 1),
            "seg_attention": (4.0 * d * keys * P, P),
            "post_attn": (P * (2.0 * N * d * d + 4.0 * N * d * dff) + (P - 1) * 2.0 * N * d * 3 * d, P)}
    per_launch = {k: float(tot) / ((launches or {}).get(k) or n) for k, (tot, n) in step.items()}
    return {
        "gemm_pool_sigmoid": ("mfma", per_launch["gemm_pool_sigmoid"]),
        "gemm_update_relu": ("mfma", per_launch["gemm_update_relu"]),
        "gemm_update_pool": ("mfma", per_launch["gemm_update_pool"]),
        "gather_max": ("hbm", per_launch["gather_max"]),
        "pre_layer": ("mfma", per_launch["pre_layer"]),
        "seg_attention": ("mfma", per_launch["seg_attention"]),
        "post_attn": ("mfma", per_launch["post_attn"]),
        # the ablation's placer without attention: every layer's FFN and the head, one launch
        "mlp_placer": ("mfma", 4.0 * N * d * dff * cfg.placer_layers + 2.0 * N * d * cfg.n_devices),
    }, keys


# Kernel kind -> the source file that defines it (for the staleness check of
# the recorded counter measurements).
KERNEL_SOURCES = {"post_attn": "layer.hip", "seg_attention": "attention.hip", "gather_max": "graph_kernels.hip"}


def measured_traffic(kind):
    """HBM bytes per launch of `kind` from the committed rocprofv3 counter
    summary (FETCH_SIZE and WRITE_SIZE, each scaled by the same counter's
    reading for a plain copy of known size), or None when there is none or
    the kernel's source has changed since the counters were taken."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.json")
    if kind not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(kind)
    if not rec:
        return None
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_1910_01578_amd", "csrc", KERNEL_SOURCES[kind])
    with open(src, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != rec["source_sha256"]:
            return None
    out = {"bytes_per_launch": rec["bytes_per_launch"], "fetch_bytes": rec["fetch_bytes"],
           "write_bytes": rec["write_bytes"], "algorithmic_bytes": rec.get("algorithmic_bytes"),
           "summary": rec["summary"]}
    if "one_stream" in rec:      # the same kernel's launches over all rows (one-stream schedule)
        out["one_stream"] = rec["one_stream"]
    return out


def blas_info():
    """The BLAS numpy uses (threadpoolctl's report) for the oracle's timing."""
    try:
        from threadpoolctl import threadpool_info
        for rec in threadpool_info():
            if rec.get("user_api") == "blas":
                return {"internal_api": rec.get("internal_api"), "version": rec.get("version"),
                        "library": os.path.basename(rec.get("filepath", ""))}
    except Exception:   # reporting only
        pass
    return None


def roofline_of(work, kind, ms_total, launches, dtype):
    if kind not in work or launches == 0:
        return None
    bound, amount = work[kind]
    sec = ms_total / launches / 1e3
    if bound == "mfma":
        ach = amount / sec / 1e12
        peak = PEAK_TFLOPS[dtype]
        return {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s", "frac": round(ach / peak, 4)}
    ach = amount / sec / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4)}


def config_leg(cfg, steps, cores):
    """One workload: the step's nodes/s (K steps bracketed by synchronisation,
    like the headline figure), the median / min / max of per-step events over
    K further steps, the dominant kernel's roofline fraction, and the whole
    oracle on the host cores."""
    import numpy as np
    import torch

    from paper_1910_01578_amd import gdp, workloads as W
    g, w = W.make_graph(cfg), W.make_weights(cfg)
    stats = W.graph_stats(g, cfg.fanout)
    r = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), cfg.k_samples)
    for _ in range(2):
        r.forward(cfg.sample_seed)
    torch.cuda.synchronize()
    gdp.timer_begin(range(gdp.K_COUNT))
    r.forward(cfg.sample_seed)
    bd = gdp.timer_end()
    work, _ = flop_model(cfg, g, stats, "gemm_update_pool" in bd, {k: v["launches"] for k, v in bd.items()})
    dominant = max(bd, key=lambda k: bd[k]["ms"])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        r.forward(cfg.sample_seed)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        r.forward(cfg.sample_seed)
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
    med = float(np.median(ms))
    rec = {"workload": cfg.name, "nodes": g.n_nodes, "dtype": cfg.dtype, "value": round(g.n_nodes / wall, 1),
           "unit": "nodes/s", "ms_per_step": round(1e3 * wall, 4), "median_ms": round(med, 4),
           "min_ms": round(float(ms.min()), 4), "max_ms": round(float(ms.max()), 4), "dominant": dominant,
           "roofline": roofline_of(work, dominant, bd[dominant]["ms"], bd[dominant]["launches"], cfg.dtype)}
    del r
    if cores:
        base = cpu_baseline(cfg, g, w, g.n_nodes, cores)
        rec["oracle"] = {"value": round(base["value"], 1), "unit": "nodes/s", "cores": cores,
                         "seconds": round(g.n_nodes / base["value"], 2)}
    return rec


def training_leg(cfg, g, w, steps):
    """The update step on the headline workload: training forward, backward and
    Adam (median of event-timed calls), and whole GDP iterations."""
    import numpy as np
    import torch

    from paper_1910_01578_amd import gdp, trainer as T, workloads as W
    dg = gdp.DeviceGraph(g, cfg.dtype)
    pol = gdp.DevicePolicy(cfg, w)
    t = gdp.Trainer(dg, pol, cfg.k_samples)
    rng = np.random.default_rng(cfg.cfg_id)
    dl = torch.from_numpy((rng.normal(size=(g.n_nodes, cfg.n_devices)) / np.sqrt(g.n_nodes)).astype(np.float32)).cuda()
    t.forward()
    t.backward(dl)
    torch.cuda.synchronize()
    reps = max(3, min(steps, 5))
    out = {"store_bytes": t.store_bytes, "workspace_bytes": t.ws_bytes}
    for name, fn in (("train_forward", t.forward), ("backward", lambda: t.backward(dl)),
                     ("adam", lambda: t.adam(1e-5))):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record()
        for i in range(reps):
            fn()
            ev[i + 1].record()
        torch.cuda.synchronize()
        ms = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)])
        out[name + "_ms"] = round(float(np.median(ms)), 3)
    gdp.timer_begin(range(gdp.K_COUNT))
    t.forward()
    t.backward(dl)
    bd = gdp.timer_end()
    out["breakdown_ms"] = {k: round(v["ms"], 3) for k, v in bd.items()}
    del t, pol, dg
    b = T.GDPBatch(cfg, g, w, W.make_costs(cfg, g), cfg.k_samples)
    b.step(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    hist = T.train(b, 3, seed0=1)
    torch.cuda.synchronize()
    out["gdp_iteration_ms"] = round(1e3 * (time.perf_counter() - t0) / 3, 2)
    out["gdp_iteration"] = "sample K placements, evaluate, reward, 2 PPO epochs (forward, log-probs, PPO gradient, " \
                           "backward, Adam)"
    out["reward_last"] = [round(float(x), 4) for x in hist[-1]["reward"]]
    del b
    return out


def cpu_baseline(cfg, g, w, n_sample, cores):
    """The fp64 oracle (untuned) on the first n_sample nodes of the same DAG."""
    from threadpoolctl import threadpool_limits

    from oracle import gdp_oracle as O
    from paper_1910_01578_amd import workloads as W
    sub = g if n_sample >= g.n_nodes else W.prefix_graph(g, n_sample)
    gnn, pl, hd = w.f64()
    with threadpool_limits(limits=cores):
        t0 = time.perf_counter()
        O.policy_forward(sub.graph_ptr, sub.row_ptr, sub.col_idx, sub.x, gnn, pl, hd["w_out"], hd["b_out"],
                         fanout=cfg.fanout, nb_seed=cfg.nb_seed, n_heads=cfg.heads, seg_len=cfg.seg_len,
                         mem_len=cfg.mem_len, k_samples=cfg.k_samples, sample_seed=cfg.sample_seed, film=cfg.film)
        dt = time.perf_counter() - t0
    what = (f"the whole {g.n_nodes}-node DAG" if n_sample == g.n_nodes else
            f"first {n_sample} nodes of the {g.n_nodes}-node DAG (induced sub-DAG)")
    return {"value": n_sample / dt, "unit": "nodes/s", "cores": cores, "kind": "oracle",
            "sample": f"{what}, full embed+place+sample with K={cfg.k_samples}, numpy float64, {dt:.1f} s",
            "blas": blas_info()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="gnmt8_52000")
    ap.add_argument("--cpu-sample", type=int, default=-1,
                    help="oracle sample: first N nodes (-1 = the whole workload, 0 = skip)")
    ap.add_argument("--all-configs", type=int, default=1, help="also measure the four smaller workloads")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB before the warm-up (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU only; --gpus must be 1 "
                                   "(multi-GPU sharding is described but not built)"}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1910_01578_amd import gdp, workloads as W

    torch.cuda.set_device(0)
    cfg = W.get_config(args.config)
    g, w = W.make_graph(cfg), W.make_weights(cfg)
    stats = W.graph_stats(g, cfg.fanout)
    runner = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w), cfg.k_samples)
    seed = cfg.sample_seed

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(max(1, args.warmup)):
        runner.forward(seed)
    torch.cuda.synchronize()

    # One extra (untimed) step with an event pair around every launch: the breakdown.
    gdp.timer_begin(range(gdp.K_COUNT))
    runner.forward(seed)
    breakdown = gdp.timer_end()
    work, keys = flop_model(cfg, g, stats, "gemm_update_pool" in breakdown,
                            {k: v["launches"] for k, v in breakdown.items()})
    dominant = max(breakdown, key=lambda k: breakdown[k]["ms"])

    # Timed region: K steps bracketed by synchronisation, with HIP events only
    # around the dominant kernel's launches (on their launch streams, recorded
    # without a system-scope fence).
    torch.cuda.synchronize()
    gdp.timer_begin([dominant])
    t0 = time.perf_counter()
    for i in range(args.steps):
        runner.forward(seed)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    dom = gdp.timer_end()[dominant]
    elapsed = t1 - t0
    ms_per_step = 1e3 * elapsed / args.steps
    value = g.n_nodes * args.steps / elapsed

    # Per-step HIP-event statistics from K further steps: a torch event after
    # every step writes back the caches (about 12 us a step), so it stays out
    # of the timed region.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(args.steps):
        runner.forward(seed)
        ev[i + 1].record()
    torch.cuda.synchronize()
    step_ms = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)])
    step_events = {"median_ms": round(float(np.median(step_ms)), 4), "min_ms": round(float(step_ms.min()), 4),
                   "max_ms": round(float(step_ms.max()), 4),
                   "nodes_per_s_at_median": round(g.n_nodes / (float(np.median(step_ms)) * 1e-3), 1),
                   "note": "K further steps with an event after each, outside the timed region"}

    def roof(kind, ms_total, launches, wk=None):
        wk = work if wk is None else wk
        if kind not in wk or launches == 0:
            return None
        bound, amount = wk[kind]
        sec = ms_total / launches / 1e3
        if bound == "mfma":
            ach = amount / sec / 1e12
            peak = PEAK_TFLOPS[cfg.dtype]
            return {"bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                    "frac": round(ach / peak, 4)}
        ach = amount / sec / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4)}

    roofline = roof(dominant, dom["ms"], dom["launches"])
    if roofline is None:
        roofline = {"bound": "alu", "achieved": None, "peak": None, "unit": None, "frac": None}
    roofline["kernel"] = dominant
    roofline["avg_launch_us"] = round(1e3 * dom["ms"] / dom["launches"], 2)
    roofline["traffic"] = measured_traffic(dominant)

    def kernel_table(bd, wk, one_stream=False):
        rows = []
        for kind, v in sorted(bd.items(), key=lambda kv: -kv[1]["ms"]):
            ent = {"kernel": kind, "ms_per_step": round(v["ms"], 4), "launches": v["launches"]}
            rf = roof(kind, v["ms"], v["launches"], wk)
            if rf:
                ent.update({"achieved": rf["achieved"], "unit": rf["unit"], "frac": rf["frac"], "bound": rf["bound"]})
            # the counted HBM bytes of a launch of this shape, where recorded
            tr = measured_traffic(kind)
            if tr and one_stream and kind != "gather_max":
                tr = tr.get("one_stream")
            if tr:
                ent["traffic_bytes_per_launch"] = tr["bytes_per_launch"]
                if rf and rf["bound"] == "hbm":
                    gbs = tr["bytes_per_launch"] / (v["ms"] / v["launches"] * 1e-3) / 1e9
                    ent["counted_achieved"] = round(gbs, 1)
                    ent["counted_frac"] = round(gbs / PEAK_HBM_GBS, 4)
            rows.append(ent)
        return rows

    kernels = kernel_table(breakdown, work)
    two_part = breakdown.get("post_attn", {}).get("launches", 0) > cfg.placer_layers
    roofline["schedule"] = "two-part" if two_part else "one stream"

    # The same step with every launch on the caller's stream (one launch per
    # kernel and layer, nothing overlapping): each kernel's own duration.  In
    # the two-part schedule a launch shares the chip with the other part's
    # kernels, and its event-timed duration includes that sharing.
    kernels_one_stream = None
    if two_part:
        gdp.set_place_streams(1)
        try:
            runner.forward(seed)
            gdp.timer_begin(range(gdp.K_COUNT))
            runner.forward(seed)
            bd1 = gdp.timer_end()
            work1, _ = flop_model(cfg, g, stats, "gemm_update_pool" in bd1,
                                  {k: v["launches"] for k, v in bd1.items()})
            n_iso = max(1, min(args.steps, 10))
            t0 = time.perf_counter()
            gdp.timer_begin([dominant])
            for _ in range(n_iso):
                runner.forward(seed)
            torch.cuda.synchronize()
            iso = gdp.timer_end()[dominant]
            iso_s = (time.perf_counter() - t0) / n_iso
        finally:
            gdp.set_place_streams(2)
        rf1 = roof(dominant, iso["ms"], iso["launches"], work1) or {}
        roofline["one_stream"] = {"avg_launch_us": round(1e3 * iso["ms"] / iso["launches"], 2),
                                  "launches_per_step": iso["launches"] // n_iso,
                                  "achieved": rf1.get("achieved"), "frac": rf1.get("frac"),
                                  "ms_per_step": round(1e3 * iso_s, 4)}
        kernels_one_stream = kernel_table(bd1, work1, one_stream=True)

    # The same step captured once into a HIP graph and replayed K times (the
    # library allocates nothing and records no memset, so a step can be
    # captured): reported beside the eager figure, which is `value`.
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        runner.forward(seed)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        runner.forward(seed)
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        graph.replay()
    torch.cuda.synchronize()
    graph_s = (time.perf_counter() - t0) / args.steps
    graph_replay = {"ms_per_step": round(1e3 * graph_s, 4), "value": round(g.n_nodes / graph_s, 1), "unit": "nodes/s"}
    del graph

    # The update path's first step on the timed step's samples: PPO's clipped
    # surrogate and its logit gradient (HBM-bound: placements, logits, lse in,
    # the gradient out).
    rng = np.random.default_rng(cfg.cfg_id)
    lp = runner.logp.cpu().numpy()
    logp_old = torch.from_numpy((lp + rng.normal(scale=0.05, size=lp.shape)).astype(np.float32)).cuda()
    adv = torch.from_numpy(rng.normal(size=lp.shape).astype(np.float32)).cuda()
    for _ in range(3):
        runner.ppo_grad(logp_old, adv, 0.2)
    torch.cuda.synchronize()
    gdp.timer_begin(["ppo_grad"])
    for _ in range(args.steps):
        runner.ppo_grad(logp_old, adv, 0.2)
    torch.cuda.synchronize()
    pr = gdp.timer_end()["ppo_grad"]
    ppo_us = 1e3 * pr["ms"] / pr["launches"]
    ppo_bytes = 4.0 * (cfg.k_samples * g.n_nodes + 2 * g.n_nodes * cfg.n_devices + g.n_nodes)
    ppo = {"us_per_call": round(ppo_us, 2), "algorithmic_bytes": int(ppo_bytes),
           "achieved": round(ppo_bytes / (ppo_us * 1e-6) / 1e9, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
           "frac": round(ppo_bytes / (ppo_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}

    # The update path's second step: the head's backward pass on X (kept by
    # place_train) and the PPO logit gradient.  HBM-bound: X and dlogits in,
    # dX out (dW_out, db_out and W_out are a few KB).
    _, dl = runner.ppo_grad(logp_old, adv, 0.2)
    x_keep = runner.place_train()
    for _ in range(3):
        runner.head_backward(x_keep, dl)
    torch.cuda.synchronize()
    gdp.timer_begin(["head_backward"])
    for _ in range(args.steps):
        runner.head_backward(x_keep, dl)
    torch.cuda.synchronize()
    hr = gdp.timer_end()["head_backward"]
    hb_us = 1e3 * hr["ms"] / hr["launches"]
    hb_bytes = 4.0 * (2 * g.n_nodes * cfg.d_model + g.n_nodes * cfg.n_devices + cfg.n_devices * (cfg.d_model + 1))
    head_bwd = {"us_per_call": round(hb_us, 2), "algorithmic_bytes": int(hb_bytes),
                "achieved": round(hb_bytes / (hb_us * 1e-6) / 1e9, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
                "frac": round(hb_bytes / (hb_us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
    del x_keep, dl

    # Section 4's reward and advantage of G x K measured run times (synthetic
    # here), the advantages' producer: one small launch.
    G, K = runner.logp.shape
    rt = torch.from_numpy(rng.lognormal(mean=-1.0, sigma=0.3, size=(G, K)).astype(np.float32)).cuda()
    baseline = gdp.RewardBaseline(G)
    for _ in range(3):
        baseline.advantages(rt)
    torch.cuda.synchronize()
    gdp.timer_begin(["advantages"])
    for _ in range(args.steps):
        baseline.advantages(rt)
    torch.cuda.synchronize()
    ar = gdp.timer_end()["advantages"]
    adv_leg = {"us_per_call": round(1e3 * ar["ms"] / ar["launches"], 2), "values": G * K,
               "note": "one work-group per graph; launch-bound at this size"}
    del baseline

    # The simulated run time of the timed step's K placements (in-order list
    # scheduling with transfer costs, the memory check): latency-bound, one
    # wavefront per graph and block of 64 samples walks the nodes in order.
    costs = W.make_costs(cfg, g)
    ev = gdp.Evaluator(runner.graph, cfg.n_devices, cfg.k_samples, costs)
    for _ in range(2):
        ev.evaluate(runner.placements)
    torch.cuda.synchronize()
    gdp.timer_begin(["evaluate"])
    for _ in range(args.steps):
        ev.evaluate(runner.placements)
    torch.cuda.synchronize()
    evr = gdp.timer_end()["evaluate"]
    valid_frac = float(ev.valid.float().mean().item())
    evaluate_leg = {"us_per_call": round(1e3 * evr["ms"] / args.steps, 2), "placements": cfg.k_samples,
                    "nodes": g.n_nodes, "valid_fraction": round(valid_frac, 4),
                    "ns_per_node": round(1e6 * evr["ms"] / args.steps / g.n_nodes, 2)}
    del ev

    # The ablation's placer without attention (Section 4.4) on the same DAG and
    # weights: the same embed and sample calls around one fused placer kernel.
    ab = gdp.Runner(gdp.DeviceGraph(g, cfg.dtype), gdp.DevicePolicy(cfg, w, attention=False), cfg.k_samples)
    for _ in range(max(1, args.warmup)):
        ab.forward(seed)
    torch.cuda.synchronize()
    gdp.timer_begin(range(gdp.K_COUNT))
    ab.forward(seed)
    ab_breakdown = gdp.timer_end()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ab.forward(seed)
    torch.cuda.synchronize()
    ab_elapsed = time.perf_counter() - t0
    ab_kernels = []
    for kind, v in sorted(ab_breakdown.items(), key=lambda kv: -kv[1]["ms"]):
        ent = {"kernel": kind, "ms_per_step": round(v["ms"], 4), "launches": v["launches"]}
        rf = roof(kind, v["ms"], v["launches"])
        if rf:
            ent.update({"achieved": rf["achieved"], "unit": rf["unit"], "frac": rf["frac"], "bound": rf["bound"]})
        ab_kernels.append(ent)
    ablation = {"placer": "no attention (Section 4.4 ablation), all layers in one kernel",
                "value": round(g.n_nodes * args.steps / ab_elapsed, 1), "unit": "nodes/s",
                "ms_per_step": round(1e3 * ab_elapsed / args.steps, 4), "kernels": ab_kernels}
    del ab

    # The update step on the same DAG and weights: the training forward that
    # keeps every intermediate, the backward pass and Adam (fp32 arithmetic),
    # and one whole GDP iteration (sample, evaluate, reward, two PPO epochs).
    training = training_leg(cfg, g, w, args.steps)

    # Every other workload: nodes/s of the same step, its dominant kernel's
    # roofline fraction, and the oracle's time on the host cores.
    cores = len(os.sched_getaffinity(0))
    configs = []
    if args.all_configs:
        for name in W.CONFIG_ORDER:
            if name != cfg.name:
                configs.append(config_leg(W.get_config(name), args.steps, cores if args.cpu_sample != 0 else 0))

    cpu = None
    if args.cpu_sample != 0:
        n = g.n_nodes if args.cpu_sample < 0 else min(args.cpu_sample, g.n_nodes)
        cpu = cpu_baseline(cfg, g, w, n, cores)

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "nodes/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": f"{cfg.name}: GNMT-8-like DAG, N={g.n_nodes}, E={g.n_edges}, GNN 3x{cfg.hidden} "
                               f"fanout {cfg.fanout}, placer {cfg.placer_layers}x d={cfg.d_model} h={cfg.heads} "
                               f"S=M={cfg.seg_len}, D={cfg.n_devices}, K={cfg.k_samples}",
                   "nodes": g.n_nodes, "edges": g.n_edges, "sum_sampled_neighbours": stats["sum_s"],
                   "attention_keys": keys, "parallelism": "single GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "step_events": step_events,
        "kernels": kernels,
        "kernels_one_stream": kernels_one_stream,
        "configs": configs,
        "training": training,
        "graph_replay": graph_replay,
        "ablation_no_attention": ablation,
        "ppo_grad": ppo,
        "head_backward": head_bwd,
        "advantages": adv_leg,
        "evaluate": evaluate_leg,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
