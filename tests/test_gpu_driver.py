"""The GDP-batch training driver (paper_1910_01578_amd/trainer.py) on the GPU:
one PPO iteration lowers the clipped surrogate on its own samples, the
fine-tuning run starts from exactly the pre-trained weights, and a short
training run raises the reward."""
import numpy as np
import pytest

from paper_1910_01578_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _batch(cfg, lr=1e-3, epochs=1):
    from paper_1910_01578_amd import trainer as T
    g, w = W.make_graph(cfg), W.make_weights(cfg)
    return T.GDPBatch(cfg, g, w, W.make_costs(cfg, g), cfg.k_samples, T.PPOSettings(lr=lr, epochs=epochs))


def test_one_update_lowers_the_surrogate():
    import torch
    cfg = W.get_config("tiny_layered_256").replace(graph_sizes=(256, 180, 300), k_samples=16)
    b = _batch(cfg, lr=1e-6)     # Adam moves every weight by about lr: a first-order step
    b.step(1)
    last = b.last
    t = b.trainer
    t.forward()
    logp = t.log_prob(last["placements"])
    after, _ = t.ppo_grad(last["placements"], logp, last["logp_old"], last["advantages"], b.ppo.clip_eps)
    torch.cuda.synchronize()
    before = last["loss"].cpu().numpy()
    after = after.cpu().numpy()
    _log(f"surrogate before {before}  after {after}")
    assert after.mean() < before.mean()


def test_finetune_starts_from_the_pretrained_weights():
    from paper_1910_01578_amd import trainer as T
    cfg = W.get_config("tiny_layered_256").replace(graph_sizes=(120, 200), k_samples=8)
    pre_g = W.make_graph(cfg)
    target = W.make_graph(cfg.replace(cfg_id=7, graph_sizes=(150,)))
    h_pre, h_fine, fine = T.pretrain_then_finetune(cfg, pre_g, target, W.make_weights(cfg), cfg.k_samples, 3, 0)
    assert len(h_pre) == 3 and len(h_fine) == 0
    # rebuild the pre-trained batch's weights independently: the fine-tuning policy holds them bitwise
    pre = T.GDPBatch(cfg, pre_g, W.make_weights(cfg), W.make_costs(cfg, pre_g), cfg.k_samples)
    T.train(pre, 3)
    for a, b in zip(pre.policy.placer_t + pre.policy.gnn_t, fine.policy.placer_t + fine.policy.gnn_t):
        for k in a:
            assert np.array_equal(a[k].cpu().numpy(), b[k].cpu().numpy()), k


def test_training_raises_the_reward():
    """60 GDP-batch iterations on two graphs: the mean reward of the last ten
    iterations beats the first ten's (simulated run times shrink)."""
    from paper_1910_01578_amd import trainer as T
    cfg = W.get_config("tiny_layered_256").replace(graph_sizes=(256, 256), k_samples=16)
    b = _batch(cfg, lr=3e-5, epochs=2)
    hist = T.train(b, 60)
    r = np.array([h["reward"].mean() for h in hist])
    first, last = r[:10].mean(), r[-10:].mean()
    _log(f"mean reward first 10 iterations {first:.4f}  last 10 {last:.4f}")
    assert last > first
