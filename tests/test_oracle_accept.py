"""Pins of the oracle's acceptance test (CPU only).

Rules: strict greedy and the accepted length L (Sec. 3.1), lenience and top-k
(Appendix "Baselines and Sweep Settings"), the min(1, p/q) ratio test cited in
Sec. 3.1.  Each check is fixed by the paper or by mathematics, not by the
oracle's own code: hand-worked examples, brute force over every draft on tiny
vocabularies, the special cases the paper states (k = 1 and lenience 1 are
strict SDD), and the closed-form acceptance probability of the ratio test.
"""
import itertools
import os

import numpy as np
import pytest
from scipy.special import log_softmax

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "accept_hand_examples.txt")
MODES = {"greedy": oracle.GREEDY, "lenient": oracle.LENIENT, "topk": oracle.TOPK}


def _hand_cases():
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, V, rows, drafts, res = [s.strip() for s in line.split("|")]
        mode, param = head.split()
        p = np.array([[float(x) for x in r.split(",")] for r in rows.split(";")], np.float32)
        yield mode, float(param), int(V), p, [int(x) for x in drafts.split(",")], [int(x) for x in res.split()]


@pytest.mark.parametrize("case", list(_hand_cases()), ids=lambda c: f"{c[0]}-{c[1]}-{c[4]}")
def test_hand_examples(case):
    mode, param, V, p, drafts, (L, nxt) = case
    kw = dict(k=int(param)) if mode == "topk" else dict(lenience=param if mode == "lenient" else 1.0)
    r = oracle.accept(MODES[mode], np.array([drafts]), p[None], **kw)
    assert r["accepted_len"][0] == L and r["next_token"][0] == nxt


def _passes_brute(mode, z, x, k=1, lenience=1.0):
    """Per-position rule via library routines (argsort ranks, max)."""
    if mode == "greedy" or (mode == "lenient" and lenience == 1.0):
        return int(np.argmax(z)) == x  # numpy argmax returns the first maximum
    if mode == "topk":
        order = np.argsort(-z.astype(np.float64), kind="stable")  # stable: lower index first on ties
        return x in order[:k]
    if mode == "lenient":
        return np.float32(z[x] - z.max()) >= np.float32(np.log(lenience))
    raise ValueError(mode)


def _brute_L(mode, p, draft, **kw):
    gamma = len(draft)
    best = 0
    for ell in range(gamma + 1):  # longest prefix whose every position passes
        if all(_passes_brute(mode, p[j], draft[j], **kw) for j in range(ell)):
            best = ell
    return best


@pytest.mark.parametrize("V,gamma", [(2, 3), (3, 2), (4, 2), (5, 1), (3, 4)])
@pytest.mark.parametrize("mode,kw", [("greedy", {}), ("topk", {"k": 2}), ("topk", {"k": 3}),
                                     ("lenient", {"lenience": 0.5}), ("lenient", {"lenience": 1.0})])
def test_brute_force_every_draft(V, gamma, mode, kw):
    g = np.random.default_rng(V * 100 + gamma)
    for trial in range(3):
        # integer-valued logits create ties on purpose
        p = g.integers(-2, 3, size=(gamma + 1, V)).astype(np.float32)
        drafts = np.array(list(itertools.product(range(V), repeat=gamma)), np.int32)
        B = len(drafts)
        P = np.broadcast_to(p, (B, gamma + 1, V)).copy()
        r = oracle.accept(MODES[mode], drafts, P, **kw)
        for b in range(B):
            L = _brute_L(mode, p, drafts[b], **kw)
            assert r["accepted_len"][b] == L, (trial, drafts[b])
            assert r["next_token"][b] == int(np.argmax(p[L]))


def _rand_rows(seed, B, gamma, V, scale=2.0):
    g = np.random.default_rng(seed)
    return (g.standard_normal((B, gamma + 1, V)) * scale).astype(np.float32), \
        g.integers(0, V, size=(B, gamma)).astype(np.int32)


def test_top1_equals_greedy():
    p, d = _rand_rows(1, 64, 6, 7)
    # make drafts hit the argmax often so that L varies
    hit = np.random.default_rng(2).random(d.shape) < 0.7
    d[hit] = p[:, :-1, :].argmax(-1)[hit]
    a = oracle.accept(oracle.GREEDY, d, p)
    b = oracle.accept(oracle.TOPK, d, p, k=1)
    assert (a["accepted_len"] == b["accepted_len"]).all() and (a["next_token"] == b["next_token"]).all()
    assert len(set(a["accepted_len"].tolist())) > 2


def test_lenience_one_is_greedy_with_ties():
    p = np.zeros((1, 3, 4), np.float32)  # all-tie rows
    d = np.array([[0, 1]], np.int32)
    a = oracle.accept(oracle.LENIENT, d, p, lenience=1.0)
    g = oracle.accept(oracle.GREEDY, d, p)
    assert a["accepted_len"][0] == g["accepted_len"][0] == 1  # token 1 is not the lowest-index max


def test_topk_at_least_vocab_accepts_all_and_small_lenience_accepts_all():
    p, d = _rand_rows(3, 8, 5, 6)
    r = oracle.accept(oracle.TOPK, d, p, k=6)
    assert (r["accepted_len"] == 5).all()
    r = oracle.accept(oracle.LENIENT, d, p, lenience=1e-30)
    assert (r["accepted_len"] == 5).all()
    assert (r["next_token"] == p[:, 5, :].argmax(-1)).all()


def test_forced_failure_and_suffix_invariance():
    p, d = _rand_rows(4, 16, 6, 9)
    d[:] = p[:, :-1, :].argmax(-1)  # everything passes
    assert (oracle.accept(oracle.GREEDY, d, p)["accepted_len"] == 6).all()
    for j in range(6):
        d2 = d.copy()
        d2[:, j] = (d2[:, j] + 1) % 9  # no longer the argmax
        r = oracle.accept(oracle.GREEDY, d2, p)
        assert (r["accepted_len"] == j).all()
        # rows after the first failure do not matter
        p2 = p.copy()
        p2[:, j + 1:, :] = np.random.default_rng(j).standard_normal(p2[:, j + 1:, :].shape)
        p2[:, j, :] = p[:, j, :]
        r2 = oracle.accept(oracle.GREEDY, d2, p2)
        assert (r2["accepted_len"] == j).all() and (r2["next_token"] == r["next_token"]).all()


def test_nonfinite_and_out_of_range_fail():
    p, d = _rand_rows(5, 3, 4, 8)
    d[:] = p[:, :-1, :].argmax(-1)
    p[0, 2, 5] = np.nan
    p[1, 1, 0] = np.inf
    d[2, 3] = 8
    r = oracle.accept(oracle.GREEDY, d, p)
    assert r["accepted_len"].tolist() == [2, 1, 3]
    assert r["flags"].tolist() == [1, 1, 2]


def test_ratio_identical_rows_accept_all():
    p, d = _rand_rows(6, 32, 8, 50)
    u = np.random.default_rng(7).random((32, 8)).astype(np.float32)
    r = oracle.accept(oracle.RATIO, d, p, q=p[:, :8, :], u=u)
    assert (r["accepted_len"] == 8).all()


def test_ratio_p_ge_q_accepts_every_u():
    p, d = _rand_rows(8, 16, 4, 20)
    q = p[:, :4, :].copy()
    bi, ji = np.meshgrid(np.arange(16), np.arange(4), indexing="ij")
    q[bi, ji, d] -= 1.5  # lowers q(x) and raises p(x)/q(x) above one
    assert (log_softmax(p[:, :4].astype(np.float64), -1)[bi, ji, d]
            >= log_softmax(q.astype(np.float64), -1)[bi, ji, d]).all()
    for uu in [0.0, 0.5, 1.0 - 2 ** -24]:
        r = oracle.accept(oracle.RATIO, d, p, q=q, u=np.full((16, 4), uu, np.float32))
        assert (r["accepted_len"] == 4).all()


def test_ratio_acceptance_frequency_matches_closed_form():
    # one position, min(1, p/q) in closed form via scipy's log_softmax
    V, n = 6, 10000
    g = np.random.default_rng(9)
    zp = g.standard_normal(V).astype(np.float32)
    zq = g.standard_normal(V).astype(np.float32)
    lp, lq = log_softmax(zp.astype(np.float64)), log_softmax(zq.astype(np.float64))
    for x in range(V):
        prob = min(1.0, np.exp(lp[x] - lq[x]))
        u = (g.integers(0, 1 << 24, size=(n, 1)) * 2.0 ** -24).astype(np.float32)
        P = np.broadcast_to(zp, (n, 2, V)).copy()
        Q = np.broadcast_to(zq, (n, 1, V)).copy()
        r = oracle.accept(oracle.RATIO, np.full((n, 1), x, np.int32), P, q=Q, u=u)
        freq = r["accepted_len"].mean()
        sd = np.sqrt(max(prob * (1 - prob), 1e-12) / n)
        assert abs(freq - prob) <= 3.3 * sd + 1e-12, (x, freq, prob)


def test_ratio_monotone_in_u():
    p, d = _rand_rows(10, 64, 6, 5)
    q = _rand_rows(11, 64, 6, 5)[0][:, :6]
    u = np.random.default_rng(12).random((64, 6)).astype(np.float32) * 0.5
    L1 = oracle.accept(oracle.RATIO, d, p, q=q, u=u)["accepted_len"]
    L2 = oracle.accept(oracle.RATIO, d, p, q=q, u=np.minimum(u * 1.9, 0.999).astype(np.float32))["accepted_len"]
    assert (L2 <= L1).all()


def test_gamma_zero_and_argument_errors():
    p = np.random.default_rng(0).standard_normal((2, 1, 7)).astype(np.float32)
    r = oracle.accept(oracle.GREEDY, np.zeros((2, 0), np.int32), p)
    assert (r["accepted_len"] == 0).all() and (r["next_token"] == p[:, 0].argmax(-1)).all()
    with pytest.raises(ValueError):
        oracle.accept(oracle.TOPK, np.zeros((2, 0), np.int32), p, k=0)
    with pytest.raises(ValueError):
        oracle.accept(oracle.LENIENT, np.zeros((2, 0), np.int32), p, lenience=1.5)
