"""Pins of the oracle's skip scheduler (Sec. 4.1 candidate skip length and guards; Sec. 4.2 confidence
signals and the gate-order inequality; Sec. 4.3 survival equivalence; Appendix "Baselines and Sweep
Settings" guard list) against brute force, closed forms and the properties the paper states."""
import itertools
import math

import numpy as np
import pytest

import oracle

RAW, MARG, COND = oracle.SIG_RAW, oracle.SIG_MARGINAL, oracle.SIG_CONDITIONAL


def _sched(q, signal, eta_b, eta_c, **kw):
    lq = np.log(np.asarray(q, np.float64)).astype(np.float32)
    lq = np.atleast_2d(lq)
    return oracle.schedule(lq, np.zeros(lq.shape[0], np.int32), signal, eta_b, eta_c, **kw)


def _brute_khat(q, signal, eta_b, eta_c):
    """Definition checked prefix by prefix in fp64 with products and powers (no log sums)."""
    best = 0
    for k in range(1, len(q) + 1):
        pre = q[:k]
        B = min(pre)
        if signal == RAW:
            C = math.prod(pre) ** (1.0 / k)
        elif signal == MARG:
            C = B
        else:
            C = math.prod(pre)
        if B >= eta_b and C >= eta_c:
            best = k
    return best


def _near_tie(q, signal, eta_b, eta_c, tol=1e-5):
    for k in range(1, len(q) + 1):
        pre = q[:k]
        vals = [min(pre)]
        if signal == RAW:
            vals.append(math.prod(pre) ** (1.0 / k))
        elif signal == COND:
            vals.append(math.prod(pre))
        for v, e in zip(vals, [eta_b, eta_c]):
            if e > 0 and abs(math.log(v) - math.log(e)) < tol:
                return True
    return False


@pytest.mark.parametrize("signal", [RAW, MARG, COND])
def test_brute_force_tiny(signal):
    rng = np.random.default_rng(10 + signal)
    grid = [0.3, 0.6, 0.85, 0.93, 0.97, 0.995]
    etas = [(0.9, 0.93), (0.8, 0.85), (0.6, 0.5), (0.95, 0.9), (0.0, 0.7), (0.7, 0.0)]
    checked = 0
    for gamma in (1, 2, 3, 4):
        for q in itertools.product(grid, repeat=gamma):
            q = [v * (1 - 1e-3 * rng.random()) for v in q]  # off the threshold grid
            for eb, ec in etas:
                if _near_tie(q, signal, eb, ec):
                    continue
                got = int(_sched(q, signal, eb, ec)["K_hat"][0])
                assert got == _brute_khat(q, signal, eb, ec), (q, signal, eb, ec)
                checked += 1
    assert checked > 1000


def test_gate_order_raw_local_gate_dominates():
    """Eq. (gate order): min q <= geometric mean, so with eta_c <= eta_b the raw two-gate K_hat equals
    the local-only K_hat."""
    rng = np.random.default_rng(1)
    q = np.clip(1 - rng.exponential(0.05, size=(400, 32)), 1e-4, 1)
    lq = np.log(q).astype(np.float32)
    D = np.zeros(400, np.int32)
    for eb, ec in [(0.9, 0.85), (0.95, 0.9), (0.8, 0.5), (0.9, 0.9 - 1e-4)]:
        two = oracle.schedule(lq, D, RAW, eb, ec)["K_hat"]
        local = oracle.schedule(lq, D, RAW, eb, 0.0)["K_hat"]
        assert np.array_equal(two, local)


def test_gate_order_conditional_product_dominates():
    """Eq. (gate order): prod q <= min q, so with eta_c >= eta_b the product gate implies the local gate."""
    rng = np.random.default_rng(2)
    q = np.clip(1 - rng.exponential(0.01, size=(400, 32)), 1e-4, 1)
    lq = np.log(q).astype(np.float32)
    D = np.zeros(400, np.int32)
    for eb, ec in [(0.9, 0.9), (0.8, 0.95), (0.5, 0.99)]:
        two = oracle.schedule(lq, D, COND, eb, ec)["K_hat"]
        prod_only = oracle.schedule(lq, D, COND, 0.0, ec)["K_hat"]
        assert np.array_equal(two, prod_only)


def test_marginal_gates_reduce_to_eta_m_and_to_the_confidence_prefix():
    """Sec. 4.2: for marginal survival both gates equal min a_hat, so they reduce to eta_m = max(eta_b, eta_c),
    and K_hat is the number of positions before the first score below eta_m, for any score sequence."""
    rng = np.random.default_rng(3)
    q = rng.uniform(0.5, 1.0, size=(300, 24))
    lq = np.log(q).astype(np.float32)
    D = np.zeros(300, np.int32)
    for eb, ec in [(0.9, 0.8), (0.7, 0.95), (0.85, 0.85)]:
        em = max(eb, ec)
        a = oracle.schedule(lq, D, MARG, eb, ec)["K_hat"]
        b = oracle.schedule(lq, D, MARG, em, 0.0)["K_hat"]
        c = oracle.schedule(lq, D, MARG, 0.0, em)["K_hat"]
        assert np.array_equal(a, b) and np.array_equal(a, c)
        first_below = np.array([next((j for j in range(24) if not lq[i, j] >= np.float32(math.log(em))), 24)
                                for i in range(300)])
        assert np.array_equal(a, first_below)


def test_survival_equivalence_chain_rule():
    """Eq. (survival equivalence): a_K = prod s_j.  Conditional scores s_j and the marginals a_j they imply give
    the same K_hat (product gate vs running-minimum gate), away from threshold ties."""
    rng = np.random.default_rng(4)
    agree = 0
    for _ in range(300):
        s = np.clip(1 - rng.exponential(0.02, size=32), 1e-3, 1.0)
        a = np.cumprod(s)
        eta = float(rng.uniform(0.5, 0.95))
        if np.min(np.abs(np.log(a) - math.log(eta))) < 1e-4:
            continue
        kc = _sched(s, COND, 0.0, eta)["K_hat"][0]
        km = _sched(a, MARG, 0.0, eta)["K_hat"][0]
        assert kc == km
        agree += 1
    assert agree > 250


def test_constant_hazard_closed_form():
    """Sec. 4.3 example: with conditional failure probability h at every position, a_K = (1-h)^K; multiplying
    the marginals instead gives (1-h)^(K(K+1)/2), which the product gate then cuts much earlier."""
    h, gamma = 0.02, 32
    s = np.full(gamma, 1 - h)
    a = (1 - h) ** np.arange(1, gamma + 1)
    for K0 in (3, 7, 12, 20):
        eta = (1 - h) ** (K0 + 0.5)  # between a_{K0+1} and a_{K0}
        assert _sched(s, COND, 0.0, eta)["K_hat"][0] == K0
        assert _sched(a, MARG, 0.0, eta)["K_hat"][0] == K0
        # wrong aggregation: product of marginals
        wrong = _sched(a, COND, 0.0, eta)["K_hat"][0]
        expect = max(k for k in range(0, gamma + 1) if k * (k + 1) / 2 <= K0 + 0.5)
        assert wrong == expect < K0 or K0 <= 1


def test_invalid_score_stops_the_prefix():
    q = [0.99] * 10
    for j in range(10):
        lq = np.log(np.array(q, np.float64)).astype(np.float32)
        lq[j] = np.nan
        r = oracle.schedule(lq[None], [0], RAW, 0.9, 0.9)
        assert r["K_hat"][0] == j
        lq[j] = np.inf
        assert oracle.schedule(lq[None], [0], RAW, 0.9, 0.9)["K_hat"][0] == j
    # -inf is a valid score (q = 0): it fails the gates for every k >= its position
    lq = np.log(np.array(q, np.float64)).astype(np.float32)
    lq[4] = -np.inf
    assert oracle.schedule(lq[None], [0], RAW, 0.0, 0.0)["K_hat"][0] == 10  # eta = 0 passes everything
    assert oracle.schedule(lq[None], [0], RAW, 0.5, 0.0)["K_hat"][0] == 4


def test_guards_and_staleness_counter():
    """Sec. 4.1 guards and commit rule; Appendix: K_min = 0 still requires K_hat > 0."""
    gamma = 8
    q = np.full((1, gamma), 0.99)
    lq = np.log(q).astype(np.float32)
    draft = np.arange(100, 100 + gamma, dtype=np.int32)[None]
    sch = lambda **kw: oracle.schedule(lq, kw.pop("D", [0]), RAW, 0.9, 0.9, draft=draft, **kw)
    r = sch(k_min=6, s_max=64)
    assert (r["K"][0], r["reason"][0], r["D"][0]) == (8, oracle.R_SKIP, 8)
    r = sch(k_min=6, s_max=64, D=[64])
    assert (r["K"][0], r["reason"][0], r["D"][0]) == (0, oracle.R_STALE, 0)
    r = sch(k_min=9, s_max=64)
    assert (r["K"][0], r["reason"][0], r["D"][0]) == (0, oracle.R_SHORT, 0)
    r = sch(k_min=0, s_max=64, block_len=7)
    assert (r["K"][0], r["reason"][0]) == (0, oracle.R_SHORT_BLOCK)
    r = sch(special=[105], s_max=64)
    assert (r["K"][0], r["reason"][0]) == (0, oracle.R_SPECIAL)
    r = sch(special=[200], s_max=64)  # not in the prefix
    assert r["reason"][0] == oracle.R_SKIP
    d2 = draft.copy()
    d2[0, 3:6] = 7
    r = oracle.schedule(lq, [0], RAW, 0.9, 0.9, draft=d2, rep_max=3)
    assert (r["K"][0], r["reason"][0]) == (0, oracle.R_REPEAT)
    assert oracle.schedule(lq, [0], RAW, 0.9, 0.9, draft=d2, rep_max=4)["reason"][0] == oracle.R_SKIP
    # K_min = 0: a candidate of length 0 is still a strict round
    low = np.log(np.full((1, gamma), 0.5)).astype(np.float32)
    r = oracle.schedule(low, [0], RAW, 0.9, 0.9, k_min=0)
    assert (r["K"][0], r["reason"][0]) == (0, oracle.R_NO_CANDIDATE)


def test_staleness_bound_over_random_rounds():
    """Sec. 4.1: staleness is checked before a skip, so D never exceeds S_max + gamma - 1, and a round with
    D >= S_max is strict."""
    rng = np.random.default_rng(5)
    gamma, s_max = 32, 64
    B = 64
    D = np.zeros(B, np.int32)
    worst = 0
    for _ in range(200):
        q = np.clip(1 - rng.exponential(0.01, size=(B, gamma)), 1e-4, 1)
        lq = np.log(q).astype(np.float32)
        before = D.copy()
        r = oracle.schedule(lq, D, RAW, 0.9, 0.93, k_min=6, s_max=s_max)
        assert np.all(r["K"][before >= s_max] == 0)
        D = r["D"]
        worst = max(worst, int(D.max()))
        assert D.max() <= s_max + gamma - 1
    assert worst > s_max  # the bound is approached, not vacuous


def test_gate_comparisons_are_inclusive():
    """Sec. 4.1: a prefix passes when its score reaches the threshold (>=), decided on fp32 log-scores against
    the fp32 log of the threshold."""
    gamma = 16
    for eta in (0.5, 0.9, 0.93, 0.999):
        at = np.float32(math.log(eta))
        lq = np.full((1, gamma), at, np.float32)
        assert oracle.schedule(lq, [0], MARG, eta, eta)["K_hat"][0] == gamma
        below = np.nextafter(at, np.float32(-np.inf))
        lq[0, 5] = below
        assert oracle.schedule(lq, [0], MARG, eta, eta)["K_hat"][0] == 5
        assert oracle.schedule(lq, [0], MARG, 0.0, eta)["K_hat"][0] == 5
        assert oracle.schedule(lq, [0], COND, eta, 0.0)["K_hat"][0] == 5


def test_block_len_per_sequence():
    """Appendix guard list: a shortened final block refuses the skip for that sequence only."""
    lq = np.log(np.full((3, 8), 0.99)).astype(np.float32)
    r = oracle.schedule(lq, [0, 0, 0], RAW, 0.9, 0.9, block_len=[8, 5, 8])
    assert list(r["reason"]) == [oracle.R_SKIP, oracle.R_SHORT_BLOCK, oracle.R_SKIP]
    assert list(r["K"]) == [8, 0, 8] and list(r["D"]) == [8, 0, 8]


def test_prefix_frequency_construction_monte_carlo():
    """Prop. 1 (construction of its proof, Appendix "Proof"): two score processes with identical positionwise
    joint laws of (q_j, 1{L >= j}) whose local-gate prefixes of length K occur with probabilities
    Pr(L >= K) rho and Pr(L >= K) rho^K.  Monte-Carlo through the scheduler's local gate (K_hat >= K iff
    min_{j<=K} q_j >= tau), each frequency within 5 binomial standard deviations."""
    rng = np.random.default_rng(11)
    n, gamma, K, rho, tau, q_lo, q_hi = 40000, 8, 4, 0.7, 0.8, 0.3, 0.95
    L = np.minimum(rng.geometric(0.15, size=n) - 1, gamma)  # any law with Pr(L >= K) > 0
    Y = (L[:, None] >= np.arange(1, gamma + 1)[None]).astype(np.float64)
    Z = (rng.random((n, 1)) < rho).astype(np.float64)
    Zj = (rng.random((n, gamma)) < rho).astype(np.float64)
    q = q_lo + (q_hi - q_lo) * Y * Z
    q2 = q_lo + (q_hi - q_lo) * Y * Zj
    D = np.zeros(n, np.int32)
    kh = oracle.schedule(np.log(q).astype(np.float32), D, MARG, tau, 0.0)["K_hat"]
    kh2 = oracle.schedule(np.log(q2).astype(np.float32), D, MARG, tau, 0.0)["K_hat"]
    pL = float(np.mean(L >= K))
    for got, p in ((np.mean(kh >= K), pL * rho), (np.mean(kh2 >= K), pL * rho ** K)):
        assert abs(got - p) <= 5 * math.sqrt(p * (1 - p) / n), (got, p)
    # identical positionwise joint law: per position, Pr(q_j = q_hi, Y_j = 1) agree within sampling error
    hi1 = ((q == q_hi) & (Y == 1)).mean(0)
    hi2 = ((q2 == q_hi) & (Y == 1)).mean(0)
    assert np.all(np.abs(hi1 - hi2) <= 5 * np.sqrt(2 * hi1 * (1 - hi1) / n) + 1e-12)
