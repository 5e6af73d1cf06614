"""Pins of the oracle's PPO clipped surrogate and its logit gradient (Section 3, Eq. 1)."""
import numpy as np
import pytest
import torch

from oracle import gdp_oracle as O


def _case(seed=0, G=3, sizes=(7, 1, 12), K=5, D=4, spread=0.3):
    rng = np.random.default_rng(seed)
    gp = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(gp[-1])
    logits = rng.normal(size=(N, D))
    lse = O.logsumexp_rows(logits)
    placements = rng.integers(0, D, size=(K, N)).astype(np.int32)
    logp = O.log_prob_of(logits, lse, gp, placements)
    logp_old = logp + rng.normal(scale=spread, size=logp.shape)   # ratios around 1, some clipped
    adv = rng.normal(size=(G, K))
    return gp, logits, lse, placements, logp, logp_old, adv


def _torch_loss(logits, gp, placements, logp_old, adv, eps):
    """The same objective written with torch ops; autograd differentiates it."""
    t = torch.tensor(logits, dtype=torch.float64, requires_grad=True)
    ls = torch.log_softmax(t, dim=1)
    K, N = placements.shape
    G = len(gp) - 1
    pick = ls[torch.arange(N)[None, :].expand(K, N), torch.from_numpy(placements).long()]   # [K, N]
    total = 0.0
    for g in range(G):
        lp = pick[:, gp[g]:gp[g + 1]].sum(dim=1)
        r = torch.exp(lp - torch.from_numpy(logp_old[g]))
        a = torch.from_numpy(adv[g])
        total = total - torch.minimum(r * a, torch.clamp(r, 1 - eps, 1 + eps) * a).mean()
    (total / G).backward()
    return t.grad.numpy()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ppo_gradient_equals_torch_autograd(seed):
    gp, logits, lse, p, logp, logp_old, adv = _case(seed)
    eps = 0.2
    ours = O.ppo_clipped_surrogate(logits, lse, gp, p, logp, logp_old, adv, eps)
    ref = _torch_loss(logits, gp, p, logp_old, adv, eps)
    np.testing.assert_allclose(ours["dlogits"], ref, rtol=0, atol=1e-12)
    r = np.exp(logp - logp_old)
    assert ((r < 1 - eps) | (r > 1 + eps)).any() and ((r > 1 - eps) & (r < 1 + eps)).any()   # both branches


def test_ppo_finite_differences():
    gp, logits, lse, p, logp, logp_old, adv = _case(5, G=2, sizes=(4, 3), K=3, D=3)
    eps = 0.25
    def batch_loss(x):
        lz = O.logsumexp_rows(x)
        lp = O.log_prob_of(x, lz, gp, p)
        return O.ppo_clipped_surrogate(x, lz, gp, p, lp, logp_old, adv, eps)["loss"].mean()
    g = O.ppo_clipped_surrogate(logits, lse, gp, p, logp, logp_old, adv, eps)["dlogits"]
    h = 1e-6
    for v in range(logits.shape[0]):
        for j in range(logits.shape[1]):
            e = np.zeros_like(logits)
            e[v, j] = h
            fd = (batch_loss(logits + e) - batch_loss(logits - e)) / (2 * h)
            assert abs(fd - g[v, j]) < 1e-7


def test_ppo_closed_forms():
    gp, logits, lse, p, logp, _, adv = _case(3)
    out = O.ppo_clipped_surrogate(logits, lse, gp, p, logp, logp, adv, 0.2)
    # ratio 1: the loss is minus the mean advantage of each graph
    np.testing.assert_allclose(out["loss"], -adv.mean(axis=1), rtol=0, atol=1e-15)
    # every node's gradient row sums to zero (softmax rows sum to one)
    np.testing.assert_allclose(out["dlogits"].sum(axis=1), 0.0, atol=1e-15)
    # zero advantages: zero loss and gradient
    z = O.ppo_clipped_surrogate(logits, lse, gp, p, logp, logp + 0.1, np.zeros_like(adv), 0.2)
    assert np.all(z["loss"] == 0) and np.all(z["dlogits"] == 0)


def test_head_backward_equals_torch_autograd():
    rng = np.random.default_rng(9)
    N, d, D = 37, 16, 5
    x = rng.normal(size=(N, d))
    w = rng.normal(size=(D, d))
    b = rng.normal(size=D)
    dl = rng.normal(size=(N, D))
    ours = O.head_backward(x, w, dl)
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    tb = torch.tensor(b, requires_grad=True)
    (torch.nn.functional.linear(tx, tw, tb) * torch.from_numpy(dl)).sum().backward()
    np.testing.assert_allclose(ours["dx"], tx.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(ours["dw_out"], tw.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(ours["db_out"], tb.grad.numpy(), rtol=0, atol=1e-12)
    # a one-hot output gradient selects the weight row and the input row
    e = np.zeros((N, D))
    e[3, 2] = 1.0
    one = O.head_backward(x, w, e)
    np.testing.assert_array_equal(one["dx"][3], w[2])
    np.testing.assert_array_equal(one["dw_out"][2], x[3])


def test_update_chain_equals_torch_autograd():
    """PPO loss -> logits -> head: the oracle's two steps composed equal torch
    autograd through the head and the clipped surrogate."""
    rng = np.random.default_rng(13)
    gp = np.array([0, 9, 21])
    N, d, D, K = 21, 8, 4, 6
    x = rng.normal(size=(N, d))
    w = rng.normal(size=(D, d)) * 0.5
    b = rng.normal(size=D) * 0.1
    logits = x @ w.T + b
    lse = O.logsumexp_rows(logits)
    p = rng.integers(0, D, size=(K, N)).astype(np.int32)
    logp = O.log_prob_of(logits, lse, gp, p)
    logp_old = logp + rng.normal(scale=0.3, size=logp.shape)
    adv = rng.normal(size=logp.shape)
    g = O.ppo_clipped_surrogate(logits, lse, gp, p, logp, logp_old, adv, 0.2)
    hb = O.head_backward(x, w, g["dlogits"])
    tx = torch.tensor(x, requires_grad=True)
    tw = torch.tensor(w, requires_grad=True)
    ls = torch.log_softmax(torch.nn.functional.linear(tx, tw, torch.from_numpy(b)), dim=1)
    pick = ls[torch.arange(N)[None, :].expand(K, N), torch.from_numpy(p).long()]
    total = 0.0
    for gi in range(2):
        r = torch.exp(pick[:, gp[gi]:gp[gi + 1]].sum(dim=1) - torch.from_numpy(logp_old[gi]))
        a = torch.from_numpy(adv[gi])
        total = total - torch.minimum(r * a, torch.clamp(r, 0.8, 1.2) * a).mean()
    (total / 2).backward()
    np.testing.assert_allclose(hb["dx"], tx.grad.numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(hb["dw_out"], tw.grad.numpy(), rtol=0, atol=1e-12)
