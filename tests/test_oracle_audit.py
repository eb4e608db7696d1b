"""Pins of the agreement accounting (Sec. 3.2: strict token agreement and full prefix acceptance over the
rounds that commit an unverified prefix)."""
import numpy as np

import oracle


def test_hand_example():
    # rounds: strict (K=0), a lossless skip (K=4 <= L=6), a lossy skip (K=5 > L=2), a skip equal to L
    K = [0, 4, 5, 3]
    L = [7, 6, 2, 3]
    acc = oracle.audit_accumulate(K, L)
    assert acc.tolist() == [3, 12, 4 + 2 + 3, 2]
    st, fp = oracle.agreement(acc)
    assert st == 9 / 12 and fp == 2 / 3


def test_strict_sdd_is_one_and_lossless_skips_are_one():
    assert oracle.agreement(oracle.audit_accumulate([0, 0, 0], [1, 5, 0])) == (1.0, 1.0)
    rng = np.random.default_rng(0)
    L = rng.integers(0, 33, 500)
    K = np.minimum(L, rng.integers(0, 33, 500))  # never more than strict verification accepts
    assert oracle.agreement(oracle.audit_accumulate(K, L)) == (1.0, 1.0)


def test_brute_force_and_accumulation_over_calls():
    rng = np.random.default_rng(1)
    K = rng.integers(0, 33, 1000)
    L = rng.integers(0, 33, 1000)
    acc = np.zeros(4, np.int64)
    for i in range(0, 1000, 100):  # accumulates across calls
        oracle.audit_accumulate(K[i:i + 100], L[i:i + 100], acc)
    A = K > 0
    assert acc.tolist() == [int(A.sum()), int(K[A].sum()), int(np.minimum(K, L)[A].sum()), int((K <= L)[A].sum())]
    st, fp = oracle.agreement(acc)
    assert 0.0 <= st <= 1.0 and 0.0 <= fp <= 1.0
    # a fully accepted prefix is also fully token-agreed: FullPrefix <= StrictToken for every single round
    for k, l in zip(K[A][:50], L[A][:50]):
        s1, f1 = oracle.agreement(oracle.audit_accumulate([k], [l]))
        assert f1 <= s1
