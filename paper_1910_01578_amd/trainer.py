"""GDP-batch training and fine-tuning (Section 4.3 and Section 4.4's
pre-training): one policy, trained with PPO (Section 3, Eq. 1) over a ragged
batch of graphs with the superposition conditioning of Section 3.3, then
fine-tuned on a target graph starting from the pre-trained weights.

This module only sequences calls of the C ABI (through the binding in gdp.py);
every step of an iteration runs in the library's kernels:

  sample     gdp_embed -> gdp_place -> gdp_sample   K placements of every graph
  evaluate   gdp_evaluate                            simulated run time, validity
  reward     gdp_advantages                          -sqrt(t) (-10 if invalid), running-mean baseline
  update     gdp_forward_train, gdp_log_prob,        PPO epochs on the same samples
             gdp_ppo_grad, gdp_backward, gdp_adam_step

The paper trains on measured run times of real placements; here the
simulated run time of gdp_evaluate stands in for them.  Evaluation and reward
run on a second stream, beside the first epoch's training forward and
log-probs (which need only the placements); the PPO gradient waits for both.
"""
from __future__ import annotations

import dataclasses
import time
from typing import Dict, List, Optional

import numpy as np

from . import gdp
from . import workloads as W


@dataclasses.dataclass
class PPOSettings:
    lr: float = 3e-5           # Adam moves every weight by about lr a step; 3e-4 already collapses
    clip_eps: float = 0.2
    epochs: int = 2            # PPO epochs over one batch of samples
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    time_unit: float = 1e-6    # seconds per time unit of the per-op costs


class GDPBatch:
    """A policy, a ragged batch of graphs and everything one PPO iteration
    needs on the device (sampling, evaluation, reward state, update)."""

    def __init__(self, cfg: W.Config, graph: W.Graph, weights: W.Weights, costs: W.OpCosts, k_samples: int,
                 ppo: Optional[PPOSettings] = None, device="cuda"):
        self.cfg = cfg
        self.ppo = ppo or PPOSettings()
        self.k = int(k_samples)
        self.dg = gdp.DeviceGraph(graph, cfg.dtype, device)
        self.policy = gdp.DevicePolicy(cfg, weights, device)
        self.runner = gdp.Runner(self.dg, self.policy, self.k, device)
        self.trainer = gdp.Trainer(self.dg, self.policy, self.k, device)
        self.evaluator = gdp.Evaluator(self.dg, cfg.n_devices, self.k, costs, device)
        self.baseline = gdp.RewardBaseline(self.dg.n_graphs, device)
        self.history: List[Dict[str, np.ndarray]] = []
        # the simulated run times and rewards run here, beside the first PPO
        # epoch's forward and log-probs, which need only the placements
        self.side = gdp._torch().cuda.Stream(device=device)

    def step(self, seed: int) -> Dict[str, np.ndarray]:
        """One iteration: sample, evaluate, reward, PPO update.  Returns the
        per-graph mean reward, best run time and valid fraction of the samples."""
        torch = gdp._torch()
        r, t, p = self.runner, self.trainer, self.ppo
        r.forward(seed)
        placements = r.placements
        main = torch.cuda.current_stream()
        self.side.wait_stream(main)                 # the placements are complete
        with torch.cuda.stream(self.side):
            mk, valid, run_time = self.evaluator.evaluate(placements, p.time_unit)
            reward, adv = self.baseline.advantages(run_time, valid)
        t.forward()
        logp_old = t.log_prob(placements)
        main.wait_stream(self.side)                 # rewards and advantages are complete
        for x in (reward, adv):
            x.record_stream(main)                   # allocated on the side stream, used on this one
        loss = None
        for e in range(p.epochs):
            if e > 0:
                t.forward()
            logp = logp_old if e == 0 else t.log_prob(placements)
            loss, dl = t.ppo_grad(placements, logp, logp_old, adv, p.clip_eps)
            t.backward(dl)
            t.adam(p.lr, p.beta1, p.beta2, p.eps)
        self.last = {"placements": placements, "logp_old": logp_old, "advantages": adv, "loss": loss}
        rt = run_time.cpu().numpy().astype(np.float64)
        ok = valid.cpu().numpy().astype(bool)
        best = np.where(ok, rt, np.inf).min(axis=1)
        rec = {"reward": reward.cpu().numpy().mean(axis=1), "best_run_time": best, "valid": ok.mean(axis=1),
               "loss": loss.cpu().numpy()}
        self.history.append(rec)
        return rec

    def export_weights(self) -> W.Weights:
        """The current weights (each as (float64 value, dtype array)), e.g. to
        start fine-tuning on another graph from them."""
        dt = self.cfg.dtype

        def pair(t):
            if dt == "bf16":
                bits = t.detach().cpu().view(gdp._torch().int16).numpy().view(np.uint16).copy()
                return W.bf16_to_f64(bits), bits
            a = t.detach().cpu().numpy().astype(np.float32)
            return a.astype(np.float64), a
        return W.Weights(gnn=[{k: pair(v) for k, v in l.items()} for l in self.policy.gnn_t],
                         placer=[{k: pair(v) for k, v in l.items()} for l in self.policy.placer_t],
                         head={k: pair(v) for k, v in self.policy.head_t.items()})


def train(batch: GDPBatch, steps: int, seed0: int = 0, log=None) -> List[Dict[str, np.ndarray]]:
    out = []
    for s in range(steps):
        t0 = time.perf_counter()
        rec = batch.step(seed0 + s)
        rec["seconds"] = time.perf_counter() - t0
        out.append(rec)
        if log:
            log(s, rec)
    return out


def pretrain_then_finetune(cfg: W.Config, pre_graph: W.Graph, target_graph: W.Graph, weights: W.Weights,
                           k_samples: int, pre_steps: int, fine_steps: int, ppo: Optional[PPOSettings] = None,
                           log=None):
    """Section 4.4's pre-training: GDP-batch on pre_graph (a ragged batch that,
    as in the paper, may include the target), then fine-tuning on
    target_graph from the pre-trained weights; returns both histories and the
    fine-tuned batch."""
    pre = GDPBatch(cfg, pre_graph, weights, W.make_costs(cfg, pre_graph), k_samples, ppo)
    h_pre = train(pre, pre_steps, 0, (lambda s, r: log("pre", s, r)) if log else None)
    fine = GDPBatch(cfg, target_graph, pre.export_weights(), W.make_costs(cfg, target_graph), k_samples, ppo)
    h_fine = train(fine, fine_steps, 10_000, (lambda s, r: log("fine", s, r)) if log else None)
    return h_pre, h_fine, fine
