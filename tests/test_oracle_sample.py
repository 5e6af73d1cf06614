"""Pins of the oracle's whole-graph Gumbel-max sampling and log-probabilities."""
import math

import numpy as np
import pytest
import torch
from scipy import stats

from oracle import gdp_oracle as O


def test_i5_fixed_uniforms_match_scalar_argmax():
    rng = np.random.default_rng(0)
    N, D, K = 40, 6, 5
    logits = rng.normal(size=(N, D)) * 2
    lse = O.logsumexp_rows(logits)
    u = rng.uniform(1e-6, 1 - 1e-6, size=(K, N, D))
    gp = np.array([0, 15, 40])
    out = O.sample(logits, lse, gp, K, seed=0, uniforms=u)
    for k in range(K):
        for v in range(N):
            best, arg = -math.inf, -1
            for j in range(D):
                s = logits[v, j] - math.log(-math.log(u[k, v, j]))
                if s > best:
                    best, arg = s, j
            assert out["placements"][k, v] == arg
    # log-prob against torch's log_softmax gathered at the placements
    ls = torch.log_softmax(torch.from_numpy(logits), dim=1).numpy()
    for k in range(K):
        for gi in range(2):
            rows = range(gp[gi], gp[gi + 1])
            ref = sum(ls[v, out["placements"][k, v]] for v in rows)
            assert abs(out["logp"][gi, k] - ref) < 1e-11


def test_zero_gumbel_is_argmax_and_ties_go_low():
    rng = np.random.default_rng(1)
    logits = rng.normal(size=(30, 8))
    logits[5] = 0.25                                # all-equal row: tie -> device 0
    logits[6, 3] = logits[6, 6] = logits[6].max() + 1.0
    u = np.full((2, 30, 8), math.exp(-1.0))         # -ln(-ln u) = 0
    out = O.sample(logits, O.logsumexp_rows(logits), np.array([0, 30]), 2, 0, uniforms=u)
    assert np.array_equal(out["placements"][0], np.argmax(logits, axis=1))
    assert out["placements"][0, 5] == 0
    assert out["placements"][1, 6] == 3


def test_i6_gumbel_max_frequencies_match_softmax():
    logits = np.array([[0.3, -1.2, 2.0, 0.0, 0.7, -0.4, 1.1, -2.5]])
    K = 100000
    # one node; the K samples use the counter layout (v = 0, k, 2, 0)
    u = O.gumbel_uniforms(seed=123, n_nodes=1, k_samples=K, n_devices=8)
    out = O.sample(logits, O.logsumexp_rows(logits), np.array([0, 1]), K, 123, uniforms=u)
    counts = np.bincount(out["placements"][:, 0], minlength=8)
    p = np.exp(logits[0] - O.logsumexp_rows(logits)[0])
    res = stats.chisquare(counts, K * p)
    assert res.pvalue > 1e-3


def test_seeded_sampling_is_deterministic_and_uses_philox_layout():
    rng = np.random.default_rng(2)
    logits = rng.normal(size=(64, 8))
    lse = O.logsumexp_rows(logits)
    gp = np.array([0, 64])
    a = O.sample(logits, lse, gp, 4, seed=9)
    b = O.sample(logits, lse, gp, 4, seed=9, uniforms=O.gumbel_uniforms(9, 64, 4, 8))
    assert np.array_equal(a["placements"], b["placements"])
    assert np.array_equal(a["logp"], b["logp"])
    c = O.sample(logits, lse, gp, 4, seed=10)
    assert not np.array_equal(a["placements"], c["placements"])
