"""Pins of the oracle's reward and advantage (Section 4): closed forms, the
invalid-placement constant, the running bias over batches against a direct
average of every previous trial, and the reading for a graph's first batch."""
import numpy as np

from oracle import gdp_oracle as O


def test_closed_forms_and_invalid_constant():
    t = np.array([[1.0, 4.0, 0.25, 9.0]])
    ok = np.array([[True, True, True, False]])
    out = O.rewards_advantages(t, ok, [0.0], [0])
    np.testing.assert_array_equal(out["reward"], [[-1.0, -2.0, -0.5, -10.0]])
    # first batch: the bias is the batch's own mean, so the advantages sum to 0
    assert out["baseline"][0] == -13.5 / 4
    assert abs(out["advantage"].sum()) < 1e-12
    assert out["reward_sum"][0] == -13.5 and out["trial_count"][0] == 4


def test_running_bias_equals_mean_of_all_previous_trials():
    rng = np.random.default_rng(3)
    G, K = 3, 5
    s, n = np.zeros(G), np.zeros(G, np.int64)
    history = [[] for _ in range(G)]
    for step in range(6):
        t = rng.uniform(0.1, 2.0, size=(G, K))
        ok = rng.random((G, K)) > 0.2
        out = O.rewards_advantages(t, ok, s, n)
        for g in range(G):
            expect = np.mean(history[g]) if history[g] else np.mean(out["reward"][g])
            assert abs(out["baseline"][g] - expect) < 1e-12
            for k in range(K):      # each reward by hand
                r = -np.sqrt(t[g, k]) if ok[g, k] else -10.0
                assert out["reward"][g, k] == r
                assert abs(out["advantage"][g, k] - (r - expect)) < 1e-12
            history[g] += list(out["reward"][g])
        s, n = out["reward_sum"], out["trial_count"]
    assert list(n) == [6 * K] * G
    np.testing.assert_allclose(s, [np.sum(h) for h in history], rtol=0, atol=1e-12)


def test_all_valid_when_no_mask_and_state_not_mutated():
    t = np.array([[1.0, 2.0], [3.0, 4.0]])
    s0, n0 = np.array([-1.0, -2.0]), np.array([1, 2])
    a = O.rewards_advantages(t, None, s0, n0)
    b = O.rewards_advantages(t, np.ones((2, 2), bool), s0, n0)
    np.testing.assert_array_equal(a["advantage"], b["advantage"])
    np.testing.assert_array_equal(s0, [-1.0, -2.0])
    np.testing.assert_array_equal(a["baseline"], [-1.0, -1.0])
