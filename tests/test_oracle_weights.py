"""Pins of the synthetic weight generator used by the oracle (CPU only).

SplitMix64 is pinned to its published test vectors; the Irwin-Hall(4)
normal approximation to its mean and standard deviation; bf16 outputs must be
representable in bf16.
"""
import os

import numpy as np

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "splitmix64_vectors.txt")
GOLDEN_GAMMA = 0x9E3779B97F4A7C15


def test_splitmix64_published_vectors():
    for line in open(GOLD):
        if line.startswith("#") or not line.strip():
            continue
        i, h = line.split()
        state = (int(i) * GOLDEN_GAMMA) % (1 << 64)
        assert oracle.splitmix64(state) == int(h, 16)


def test_moments_and_bf16_grid():
    w = oracle.weight_values(0, 17, 0, 1 << 20, 0.02, True).astype(np.float64)
    n = w.size
    assert abs(w.mean()) < 4 * 0.02 / np.sqrt(n)
    assert abs(w.std() / 0.02 - 1) < 0.01
    # Irwin-Hall(4) excess kurtosis is -0.3; support is bounded by sqrt(12) sigma
    k = ((w - w.mean()) ** 4).mean() / w.var() ** 2 - 3
    assert -0.4 < k < -0.2
    assert np.abs(w).max() <= 0.02 * np.sqrt(12) * 1.01
    bits = w.astype(np.float32).view(np.uint32)
    assert (bits & 0xFFFF == 0).all()


def test_fp32_variant_and_counter_property():
    a = oracle.weight_values(5, 3, 1000, 64, 0.02, False)
    b = oracle.weight_values(5, 3, 0, 2000, 0.02, False)
    assert np.array_equal(a, b[1000:1064])  # value depends only on (seed, tensor, index)
    c = oracle.weight_values(6, 3, 1000, 64, 0.02, False)
    assert not np.array_equal(a, c)
    assert np.array_equal(oracle.weight_values(5, 3, 0, 64, 0.02, True),
                          (b[:64].view(np.uint32) + 0x7FFF + ((b[:64].view(np.uint32) >> 16) & 1)
                           & 0xFFFF0000).view(np.float32))
