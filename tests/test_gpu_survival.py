"""GPU parity of sdd_survival_mlp against the oracle's survival predictor, and of the scheduler fed by it.

Tolerance on the logit z and on log sigmoid(z): 1e-4 absolute.  The kernel sums fp32 products in a fixed
order (layer 1: 3603 terms of size ~1e-2 whose partial sums stay O(1), rounding ~sqrt(3603) x 6e-8 ~ 4e-6
typical; layers 2-4: 256 terms each), plus the fp32 erf / exp / log1p of GELU and log-sigmoid (a few ulp);
the bound leaves a margin of about 10x over that.  The scheduler decisions taken on the GPU scores must
equal the oracle's except where an oracle score lies within 1e-4 of a threshold (counted).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu
TOL = 1e-4


@pytest.fixture(scope="module")
def sdd():
    from paper_2608_14787_amd import sdd as S
    assert S.device_ok(), "needs a gfx950 device"
    return S


def _mlp(sdd, x):
    return sdd.SurvivalMLP(x.mu, x.sigma, x.W1, x.b1, x.W2, x.b2, x.W3, x.b3, x.w4, x.b4, d_hid=x.hidden_bits.shape[1])


def _run(sdd, x, mlp=None):
    mlp = mlp or _mlp(sdd, x)
    n = x.hidden_bits.shape[0]
    hid = torch.from_numpy(x.hidden_bits.view(np.int16)).cuda().view(torch.bfloat16)
    sc = torch.from_numpy(np.ascontiguousarray(x.scalars)).cuda() if x.scalars.shape[1] else None
    logit = torch.empty(n, dtype=torch.float32, device="cuda")
    ls = mlp(hid, sc, logit=logit)
    torch.cuda.synchronize()
    return ls.cpu().numpy(), logit.cpu().numpy()


def _ref(x):
    return oracle.survival_mlp(x.hidden_bits, x.scalars, x.mu, x.sigma, x.W1, x.b1, x.W2, x.b2, x.W3, x.b3, x.w4, x.b4)


@pytest.mark.parametrize("n,d_hid,n_sc,H", [(32, 3584, 19, 256), (512, 3584, 19, 256), (100, 3584, 19, 256),
                                            (1, 3584, 19, 256), (7, 40, 5, 16), (70, 300, 0, 48)])
def test_survival_matches_oracle(sdd, n, d_hid, n_sc, H):
    x = W.survival_inputs(seed=n + H, n=n, d_hid=d_hid, n_sc=n_sc, H=H)
    x.w4 *= 20.0  # spread the untrained logits over several units
    print(f"survival n={n} d_in={d_hid + n_sc} H={H}", flush=True)
    ls, lg = _run(sdd, x)
    rls, rlg = _ref(x)
    err_z, err_s = np.abs(lg - rlg).max(), np.abs(ls - rls).max()
    print(f"  max |dz| {err_z:.2e}, max |d log score| {err_s:.2e}", flush=True)
    assert err_z <= TOL and err_s <= TOL


def test_survival_repeatable(sdd):
    x = W.survival_inputs(seed=5, n=64)
    mlp = _mlp(sdd, x)
    a = _run(sdd, x, mlp)
    b = _run(sdd, x, mlp)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


@pytest.mark.parametrize("signal", [oracle.SIG_MARGINAL, oracle.SIG_CONDITIONAL])
def test_survival_feeds_scheduler(sdd, signal):
    """Predictor scores of 8 blocks of 32 positions drive the two-gate scheduler (Sec. 4.2 settings:
    eta_m = 0.90 marginal, (0.90, 0.90) conditional)."""
    B, gamma = 8, 32
    x = W.survival_inputs(seed=11 + signal, n=B * gamma)
    # logit spread and offset chosen so that the blocks' prefixes have different lengths
    scale, offset = (30.0, 2.5) if signal == oracle.SIG_MARGINAL else (100.0, 6.5)
    x.w4 *= scale
    x.b4 = offset
    ls, _ = _run(sdd, x)
    rls, _ = _ref(x)
    eta = 0.90
    lq_gpu = torch.from_numpy(ls.reshape(B, gamma)).cuda()
    D = torch.zeros(B, dtype=torch.int32, device="cuda")
    K, Kh, rs = sdd.schedule(lq_gpu, D, signal, eta, eta, k_min=6, s_max=64)
    torch.cuda.synchronize()
    ref = oracle.schedule(rls.reshape(B, gamma).astype(np.float32), np.zeros(B, np.int32), signal, eta, eta,
                          k_min=6, s_max=64)
    lt = math.log(eta)
    if signal == oracle.SIG_MARGINAL:
        near = np.abs(rls.reshape(B, gamma) - lt).min(1) < TOL
    else:
        near = np.abs(np.cumsum(rls.reshape(B, gamma), 1) - lt).min(1) < TOL * gamma
    same = Kh.cpu().numpy() == ref["K_hat"]
    print(f"K_hat {Kh.cpu().numpy().tolist()} (oracle {ref['K_hat'].tolist()}), near ties {int(near.sum())}", flush=True)
    assert np.all(same | near)
    assert len(set(ref["K_hat"].tolist())) > 2  # prefixes of several lengths: the gates are exercised


def test_survival_argument_errors(sdd):
    x = W.survival_inputs(seed=1, n=4, d_hid=32, n_sc=3, H=16)
    x.W1 = np.zeros((20, 35), np.float32)
    x.b1 = np.zeros(20, np.float32)
    with pytest.raises(sdd.SDDError):
        _run(sdd, x)  # H = 20 is not a multiple of 16
