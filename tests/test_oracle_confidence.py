"""Pins of the oracle's raw-confidence prefix (CPU only).

Sec. 4.2 defines raw confidence as the drafter probability of the drafted
token, the largest output probability under greedy drafting; Sec. 4.1 gates a
prefix on B_k = min_{j<=k} q_j with K = max{k : B_k >= tau} (max of the empty
set = 0).  Pins: brute force of that max over k with scipy's softmax, closed
forms for flat rows, monotonicity in tau, and the extreme thresholds.
"""
import numpy as np
import pytest
from scipy.special import log_softmax, softmax

import oracle


def _brute_skip(z, gamma, tau):
    q = softmax(z[:gamma].astype(np.float64), axis=-1).max(-1)
    best = 0
    for k in range(1, gamma + 1):
        if q[:k].min() >= tau:
            best = k
    return best


@pytest.mark.parametrize("V", [3, 17, 300])
def test_brute_force_longest_prefix(V):
    g = np.random.default_rng(V)
    B, gamma = 40, 6
    z = (g.standard_normal((B, gamma + 1, V)) * 2).astype(np.float32)
    boost = g.uniform(0, 8, size=(B, gamma))
    z[:, :gamma, 0] += boost.astype(np.float32)
    for tau in [0.05, 0.3, 0.5, 0.7, 0.9]:
        r = oracle.confidence_prefix(z, gamma, tau)
        want = [_brute_skip(z[b], gamma, tau) for b in range(B)]
        # exclude near-ties of q vs tau (the decision is taken in fp32)
        q = softmax(z[:, :gamma].astype(np.float64), -1).max(-1)
        near = (np.abs(np.log(q) - np.log(tau)) < 1e-5).any(-1)
        assert (r["skip_len"][~near] == np.array(want)[~near]).all()
        np.testing.assert_allclose(r["log_conf"], np.log(q), rtol=0, atol=1e-12)


def test_monotone_in_tau():
    g = np.random.default_rng(1)
    z = (g.standard_normal((64, 9, 50)) * 3).astype(np.float32)
    z[:, :8, 3] += g.uniform(0, 10, size=(64, 8)).astype(np.float32)
    taus = [0.0, 0.1, 0.3, 0.5, 0.7, 0.9, 0.95, 1.0]
    prev = None
    for t in taus:
        s = oracle.confidence_prefix(z, 8, t)["skip_len"]
        if prev is not None:
            assert (s <= prev).all()
        prev = s


def test_extreme_thresholds():
    g = np.random.default_rng(2)
    V = 40
    z = (g.standard_normal((8, 5, V)) * 3).astype(np.float32)
    assert (oracle.confidence_prefix(z, 5, 0.5 / V)["skip_len"] == 5).all()  # q_j >= 1/V always
    assert (oracle.confidence_prefix(z, 5, 1.0 + 1e-6)["skip_len"] == 0).all()
    assert (oracle.confidence_prefix(z, 0, 0.5)["skip_len"] == 0).all()


def test_flat_and_one_hot_closed_forms():
    V = 1000
    z = np.zeros((1, 3, V), np.float32)
    r = oracle.confidence_prefix(z, 3, 0.5)
    np.testing.assert_allclose(r["log_conf"][0], -np.log(V), rtol=0, atol=1e-12)
    for delta in [0.5, 3.0, 9.0]:
        z = np.zeros((1, 1, V), np.float32)
        z[0, 0, 17] = delta
        want = 1.0 / (1.0 + (V - 1) * np.exp(-delta))
        r = oracle.confidence_prefix(z, 1, 0.5)
        np.testing.assert_allclose(np.exp(r["log_conf"][0, 0]), want, rtol=1e-12)


def test_nonfinite_stops_prefix_and_p_draft():
    g = np.random.default_rng(3)
    z = (g.standard_normal((2, 5, 20))).astype(np.float32)
    z[:, :, 0] += 20
    z[1, 2, 7] = np.inf
    d = g.integers(0, 20, size=(2, 4)).astype(np.int32)
    r = oracle.confidence_prefix(z, 4, 0.5, draft=d)
    assert r["skip_len"].tolist() == [4, 2]
    want = log_softmax(z[0, :4].astype(np.float64), -1)[np.arange(4), d[0]]
    np.testing.assert_allclose(r["log_p_draft"][0], want, atol=1e-12)
    with pytest.raises(ValueError):
        oracle.confidence_prefix(z, 4, float("nan"))
