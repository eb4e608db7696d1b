"""GPU parity of sdd_schedule against the CPU oracle's scheduler.

All outputs are integers decided by fp32 comparisons that both sides take on identical fp32 inputs with the
same left-to-right fp32 sums, so K, K_hat, reason and the updated D must be bit-exact, ties included.
Shapes span several 64-sequence blocks with a ragged last block; gamma 0, 1, 7, 32 and 64; every signal;
special tokens, repetition, shortened blocks, staleness, non-finite scores, scores exactly at the
threshold; multi-round D carried on the device; and the raw-confidence chain fed by sdd_confidence_prefix.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

SIGNALS = [oracle.SIG_RAW, oracle.SIG_MARGINAL, oracle.SIG_CONDITIONAL]


@pytest.fixture(scope="module")
def sdd():
    from paper_2608_14787_amd import sdd as S
    assert S.device_ok(), "needs a gfx950 device"
    return S


def _dev(a, dtype=np.int32):
    return torch.from_numpy(np.ascontiguousarray(a, dtype)).cuda()


def _run_both(sdd, inp, signal, eta_b, eta_c, k_min, s_max, special, rep_max, use_block=True):
    B, gamma = inp.log_q.shape
    D = _dev(inp.D)
    sp = _dev(special) if len(special) else None
    K, Kh, rs = sdd.schedule(_dev(inp.log_q, np.float32), D, signal, eta_b, eta_c, k_min=k_min, s_max=s_max,
                             draft=_dev(inp.draft), block_len=_dev(inp.block_len) if use_block else None,
                             special=sp, rep_max=rep_max)
    torch.cuda.synchronize()
    ref = oracle.schedule(inp.log_q, inp.D, signal, eta_b, eta_c, k_min=k_min, s_max=s_max,
                          block_len=inp.block_len if use_block else None, draft=inp.draft, special=special,
                          rep_max=rep_max)
    got = dict(K=K.cpu().numpy(), K_hat=Kh.cpu().numpy(), reason=rs.cpu().numpy(), D=D.cpu().numpy())
    return got, ref


PARAMS = [(0.90, 0.93, 6, 64, 0), (0.90, 0.90, 6, 64, 3), (0.5, 0.0, 0, 24, 0), (0.0, 0.8, 3, 32, 2),
          (0.95, 0.99, 12, 64, 4)]


@pytest.mark.parametrize("signal", SIGNALS)
@pytest.mark.parametrize("B,gamma", [(64, 32), (200, 32), (1, 1), (130, 7), (70, 64), (5, 0)])
def test_schedule_matches_oracle(sdd, signal, B, gamma):
    inp = W.schedule_inputs(seed=100 + B + gamma, B=B, gamma=gamma, vocab=5000)
    special = inp.draft.reshape(-1)[::37][:5].copy() if gamma else np.array([3], np.int32)
    print(f"schedule signal={signal} B={B} gamma={gamma}", flush=True)
    for eb, ec, kmin, smax, rep in PARAMS:
        for sp in (np.array([], np.int32), special):
            got, ref = _run_both(sdd, inp, signal, eb, ec, kmin, smax, sp, rep)
            for key in ("K", "K_hat", "reason", "D"):
                assert np.array_equal(got[key], ref[key]), (key, eb, ec, kmin, smax, rep, len(sp))
    # the reasons exercised (at the bench shape every guard fires somewhere over the parameter sets)
    if (B, gamma) == (200, 32):
        seen = set()
        for eb, ec, kmin, smax, rep in PARAMS:
            seen |= set(_run_both(sdd, inp, signal, eb, ec, kmin, smax, special, rep)[1]["reason"].tolist())
        assert {oracle.R_SKIP, oracle.R_STALE, oracle.R_SHORT, oracle.R_SHORT_BLOCK} <= seen


def test_schedule_ties_and_invalid_scores(sdd):
    """Scores exactly at fp32 log(eta) pass (>=); NaN and +inf end the prefix; -inf fails every gate."""
    B, gamma = 96, 16
    g = np.random.default_rng(7)
    for eta in (0.9, 0.93, 0.5):
        at = np.float32(math.log(eta))
        lq = np.full((B, gamma), at, np.float32)
        pos = g.integers(0, gamma, size=B)
        kind = g.integers(0, 4, size=B)
        below = np.nextafter(at, np.float32(-np.inf))
        for b in range(B):
            lq[b, pos[b]] = [below, np.nan, np.inf, -np.inf][kind[b]]
        inp = W.ScheduleInputs(lq, np.zeros((B, gamma), np.int32), np.zeros(B, np.int32),
                               np.full(B, gamma, np.int32))
        for signal in SIGNALS:
            for eb, ec in ((eta, eta), (0.0, eta), (eta, 0.0), (0.0, 0.0)):
                got, ref = _run_both(sdd, inp, signal, eb, ec, 0, 1 << 30, np.array([], np.int32), 0)
                for key in ("K", "K_hat", "reason", "D"):
                    assert np.array_equal(got[key], ref[key]), (key, eta, signal, eb, ec)
        # marginal gate: K_hat is exactly the position of the planted value
        got, _ = _run_both(sdd, inp, oracle.SIG_MARGINAL, eta, eta, 0, 1 << 30, np.array([], np.int32), 0)
        assert np.array_equal(got["K_hat"], pos)


def test_schedule_rounds_carry_D_on_device(sdd):
    """50 rounds at the paper's raw setting (eta_b, eta_c) = (0.90, 0.93), K_min 6, S_max 64: D lives on the
    device between calls and must follow the oracle's D every round; D <= S_max + gamma - 1 throughout."""
    B, gamma = 64, 32
    D_dev = _dev(np.zeros(B))
    D_ref = np.zeros(B, np.int32)
    skipped = 0
    for r in range(50):
        inp = W.schedule_inputs(seed=500 + r, B=B, gamma=gamma, vocab=151936, p_short=0.02)
        K, Kh, rs = sdd.schedule(_dev(inp.log_q, np.float32), D_dev, sdd.SIG_RAW, 0.90, 0.93, k_min=6, s_max=64,
                                 draft=_dev(inp.draft), block_len=_dev(inp.block_len))
        ref = oracle.schedule(inp.log_q, D_ref, oracle.SIG_RAW, 0.90, 0.93, k_min=6, s_max=64,
                              block_len=inp.block_len, draft=inp.draft)
        D_ref = ref["D"]
        assert np.array_equal(K.cpu().numpy(), ref["K"]), r
        assert np.array_equal(D_dev.cpu().numpy(), D_ref), r
        assert D_ref.max() <= 64 + gamma - 1
        skipped += int((ref["K"] > 0).sum())
    assert skipped > 0


def test_schedule_from_confidence_kernel(sdd):
    """Raw-confidence chain: sdd_confidence_prefix's log_conf feeds sdd_schedule; the oracle schedules the same
    fp32 log_conf (copied back), and its eta_c = 0 local gate equals the confidence kernel's skip length."""
    B, gamma, V = 24, 32, 151936
    g = np.random.default_rng(3)
    draft = g.integers(0, V, size=(B, gamma), dtype=np.int64).astype(np.int32)
    z = W.drafter_logits(seed=21, draft=draft, rows=gamma, vocab=V, boost=6.0, boost_hi=14.0)
    zt = torch.from_numpy(W.to_bf16_bits(z).view(np.int16)).cuda().view(torch.bfloat16)
    tau = float(np.float32(0.9))  # the confidence kernel takes tau in fp32; give the scheduler the same value
    sk, lc, _ = sdd.confidence_prefix(zt, gamma, tau, log_conf=True)
    D = _dev(np.zeros(B))
    K, Kh, rs = sdd.schedule(lc.contiguous(), D, sdd.SIG_RAW, tau, 0.0)
    torch.cuda.synchronize()
    lq = lc.cpu().numpy()
    ref = oracle.schedule(lq, np.zeros(B, np.int32), oracle.SIG_RAW, tau, 0.0)
    assert np.array_equal(Kh.cpu().numpy(), ref["K_hat"])
    assert np.array_equal(Kh.cpu().numpy(), sk.cpu().numpy())
    for eb, ec in ((0.90, 0.93), (0.8, 0.95)):
        D = _dev(np.zeros(B))
        K, Kh, rs = sdd.schedule(lc.contiguous(), D, sdd.SIG_RAW, eb, ec, k_min=6, s_max=64,
                                 draft=_dev(draft))
        ref = oracle.schedule(lq, np.zeros(B, np.int32), oracle.SIG_RAW, eb, ec, k_min=6, s_max=64, draft=draft)
        assert np.array_equal(K.cpu().numpy(), ref["K"]) and np.array_equal(rs.cpu().numpy(), ref["reason"])


def test_schedule_argument_errors(sdd):
    lq = torch.zeros((4, 8), dtype=torch.float32, device="cuda")
    D = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(sdd.SDDError):
        sdd.schedule(lq, D, 3, 0.9, 0.9)
    with pytest.raises(sdd.SDDError):
        sdd.schedule(lq, D, 0, float("nan"), 0.9)
    with pytest.raises(sdd.SDDError):  # repetition guard needs the drafts
        sdd.schedule(lq, D, 0, 0.9, 0.9, rep_max=2)
    with pytest.raises(sdd.SDDError):
        sdd.schedule(torch.zeros((4, 65), dtype=torch.float32, device="cuda"), D, 0, 0.9, 0.9)
