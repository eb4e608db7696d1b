"""Pins of the oracle's survival predictor (Appendix "Predictor Details": normalized 3584 + 19 inputs, MLP
3603 -> 256 -> 256 -> 256 -> 1 with GELU, sigmoid output used as the survival score of Sec. 4.2).

Checked against a composition of torch.nn CPU modules in float64 (a library route used only to check the
oracle), closed forms (zero last layer, zero weights), the erf form of GELU at known values, invariance of
the normalization to a common shift of feature and mean, and log-sigmoid at extreme logits."""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W


def _torch_ref(x):
    hid = torch.from_numpy(W.bf16_bits_to_f32(x.hidden_bits).astype(np.float64))
    sc = torch.from_numpy(x.scalars.astype(np.float64))
    inp = (torch.cat([hid, sc], 1) - torch.from_numpy(x.mu.astype(np.float64))) / torch.from_numpy(
        x.sigma.astype(np.float64))
    H, d_in = x.W1.shape
    net = torch.nn.Sequential(torch.nn.Linear(d_in, H), torch.nn.GELU(), torch.nn.Linear(H, H), torch.nn.GELU(),
                              torch.nn.Linear(H, H), torch.nn.GELU(), torch.nn.Linear(H, 1)).double()
    with torch.no_grad():
        for lin, (w, b) in zip([net[0], net[2], net[4], net[6]],
                               [(x.W1, x.b1), (x.W2, x.b2), (x.W3, x.b3), (x.w4, np.array([x.b4], np.float32))]):
            lin.weight.copy_(torch.from_numpy(w.astype(np.float64)))
            lin.bias.copy_(torch.from_numpy(np.asarray(b, np.float32).astype(np.float64)))
        z = net(inp)[:, 0]
        return torch.nn.functional.logsigmoid(z).numpy(), z.numpy()


def _run(x):
    return oracle.survival_mlp(x.hidden_bits, x.scalars, x.mu, x.sigma, x.W1, x.b1, x.W2, x.b2, x.W3, x.b3,
                               x.w4, x.b4)


@pytest.mark.parametrize("n,d_hid,n_sc,H", [(7, 40, 5, 16), (3, 3584, 19, 256), (1, 1, 0, 1)])
def test_matches_torch_modules(n, d_hid, n_sc, H):
    x = W.survival_inputs(seed=n + d_hid, n=n, d_hid=d_hid, n_sc=n_sc, H=H)
    ls, lg = _run(x)
    rls, rlg = _torch_ref(x)
    assert np.allclose(lg, rlg, rtol=0, atol=1e-12)
    assert np.allclose(ls, rls, rtol=0, atol=1e-12)


def test_zero_last_layer_and_zero_weights():
    x = W.survival_inputs(seed=3, n=5, d_hid=64, n_sc=19, H=32)
    x.w4[:] = 0
    x.b4 = 1.25
    ls, lg = _run(x)
    assert np.all(lg == np.float32(1.25)) and np.allclose(ls, -math.log1p(math.exp(-1.25)), atol=1e-15)
    # zero weights everywhere: h1 = GELU(b1), h2 = GELU(b2), h3 = GELU(b3), z = w4 . h3 + b4 for every row
    y = W.survival_inputs(seed=4, n=4, d_hid=16, n_sc=3, H=8)
    for w in (y.W1, y.W2, y.W3):
        w[:] = 0
    gelu = lambda v: 0.5 * v * (1 + np.vectorize(math.erf)(v / math.sqrt(2)))
    z = float(y.w4[0].astype(np.float64) @ gelu(y.b3.astype(np.float64))) + y.b4
    _, lg = _run(y)
    assert np.allclose(lg, z, atol=1e-15)


def test_gelu_erf_form_at_known_values():
    """One hidden unit, identity-like weights: z = GELU(v); GELU(1) = Phi(1) = 0.841344746068543, GELU(0) = 0,
    GELU(-3) = -3 * Phi(-3) = -0.00404969864023."""
    for v, want in ((1.0, 0.8413447460685429), (0.0, 0.0), (-3.0, -3 * 0.0013498980316301), (2.5, 2.5 * 0.9937903346742238)):
        x = W.survival_inputs(seed=5, n=1, d_hid=1, n_sc=0, H=1)
        x.hidden_bits[:] = W.to_bf16_bits(np.array([[v]], np.float32))
        x.mu[:] = 0
        x.sigma[:] = 1
        x.W1[:] = 1
        x.b1[:] = 0
        # layers 2 and 3: make GELU(GELU(GELU(v))) recoverable -> use w4 on h1 only by a 1-unit chain
        x.W2[:] = 1
        x.b2[:] = 0
        x.W3[:] = 1
        x.b3[:] = 0
        x.w4[:] = 1
        x.b4 = 0.0
        _, lg = _run(x)
        g1 = want
        g2 = 0.5 * g1 * (1 + math.erf(g1 / math.sqrt(2)))
        g3 = 0.5 * g2 * (1 + math.erf(g2 / math.sqrt(2)))
        assert abs(lg[0] - g3) < 1e-12, (v, lg[0], g3)


def test_normalization_shift_invariance():
    x = W.survival_inputs(seed=6, n=6, d_hid=32, n_sc=19, H=16)
    base, _ = _run(x)
    x.scalars = (x.scalars + np.float32(0.5)).astype(np.float32)
    x.mu[32:] = x.mu[32:] + np.float32(0.5)
    shifted, _ = _run(x)
    assert np.allclose(base, shifted, atol=1e-5)  # equal up to the fp32 rounding of the shifted inputs


def test_log_sigmoid_extremes():
    x = W.survival_inputs(seed=7, n=2, d_hid=8, n_sc=0, H=4)
    x.w4[:] = 0
    for b4, want in ((100.0, -math.exp(-100.0)), (-100.0, -100.0), (0.0, -math.log(2.0))):
        x.b4 = b4
        ls, _ = _run(x)
        assert np.all(np.isfinite(ls)) and np.allclose(ls, want, rtol=1e-12, atol=1e-300)
