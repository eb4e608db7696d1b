"""Pins of the oracle's distribution-preserving ratio rule (the min(1, p/q) test that Sec. 3.1 cites, with its
residual draw from norm(max(0, p - q)) after a rejection and the bonus draw from p after a full block).

The rule's defining property: the first emitted token is distributed exactly as the target's p, whatever the
drafter's q.  Checked by Monte-Carlo over draws of the draft from q and of both uniforms, class by class within
5 binomial standard deviations; closed forms for one-hot drafters and identical rows via numpy's inverse CDF
(searchsorted); monotonicity of the draw in its uniform."""
import math

import numpy as np

import oracle

RS = oracle.RATIO_SAMPLE


def _softmax(z):
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max(-1, keepdims=True))
    return e / e.sum(-1, keepdims=True)


def _within(freq, p, n, sig=5.0):
    sd = np.sqrt(np.maximum(p * (1 - p), 1e-12) / n)
    return np.all(np.abs(freq - p) <= sig * sd + 1e-12), np.abs(freq - p) / sd


def test_first_token_follows_target_distribution():
    """x ~ q, accept w.p. min(1, p(x)/q(x)), else draw from norm(max(0, p - q)): the emitted token ~ p."""
    rng = np.random.default_rng(0)
    V, n = 6, 200000
    for trial in range(3):
        zp = rng.normal(0, 1.5, V).astype(np.float32)
        zq = rng.normal(0, 1.5, V).astype(np.float32)
        p, q = _softmax(zp), _softmax(zq)
        x = rng.choice(V, size=n, p=q).astype(np.int32)
        P = np.broadcast_to(np.stack([zp, zp]), (n, 2, V)).copy()  # row 0 decides x, row 1 is the bonus row
        Q = np.broadcast_to(zq, (n, 1, V)).copy()
        u = (rng.integers(0, 1 << 24, size=(n, 2)) * 2.0 ** -24).astype(np.float32)
        r = oracle.accept(RS, x[:, None], P, Q, u, margins=False)
        first = np.where(r["accepted_len"] == 1, x, r["next_token"])
        ok, z = _within(np.bincount(first, minlength=V) / n, p, n)
        assert ok, (trial, z)
        # after an acceptance the bonus token is drawn from p of the bonus row
        acc = r["accepted_len"] == 1
        assert abs(acc.mean() - np.minimum(p, q).sum()) <= 5 * math.sqrt(0.25 / n)
        ok, z = _within(np.bincount(r["next_token"][acc], minlength=V) / acc.sum(), p, int(acc.sum()))
        assert ok, (trial, z)


def test_residual_of_one_hot_drafter_is_target_without_the_draft():
    """q concentrated on x (q(x) = 1 to fp64 precision): max(0, p - q) is p with x removed, so the rejection
    draw is the inverse CDF of that distribution (numpy searchsorted)."""
    rng = np.random.default_rng(1)
    V = 50
    zp = rng.normal(0, 2, V).astype(np.float32)
    x = int(np.argmax(zp))  # the target's favourite, so p(x) < 1 = q(x) and rejections happen
    zq = np.full(V, -1e4, np.float32)
    zq[x] = 0.0
    p = _softmax(zp)
    w = p.copy()
    w[x] = 0.0
    cdf = np.cumsum(w)
    us = (np.arange(1, 400) / 400.0).astype(np.float32)
    n = us.size
    P = np.broadcast_to(np.stack([zp, zp]), (n, 2, V)).copy()
    Q = np.broadcast_to(zq, (n, 1, V)).copy()
    u = np.stack([np.full(n, np.float32(0.999999)), us], 1)  # u_accept near 1: the draft is rejected
    r = oracle.accept(RS, np.full((n, 1), x, np.int32), P, Q, u, margins=False)
    assert np.all(r["accepted_len"] == 0)
    want = np.searchsorted(cdf, us.astype(np.float64) * cdf[-1], side="right")
    clear = r["sample_margin"] > 1e-9
    assert clear.sum() > 0.95 * n
    assert np.array_equal(r["next_token"][clear], want[clear])
    assert not np.any(r["next_token"] == x)


def test_identical_rows_accept_everything_and_bonus_is_inverse_cdf_of_p():
    rng = np.random.default_rng(2)
    B, gamma, V = 300, 4, 40
    z = rng.normal(0, 2, (B, gamma + 1, V)).astype(np.float32)
    draft = rng.integers(0, V, (B, gamma)).astype(np.int32)
    u = rng.random((B, gamma + 1)).astype(np.float32)
    r = oracle.accept(RS, draft, z, z[:, :gamma].copy(), u, margins=False)
    assert np.all(r["accepted_len"] == gamma)
    for b in range(B):
        cdf = np.cumsum(_softmax(z[b, gamma]))
        if r["sample_margin"][b] > 1e-9:
            assert r["next_token"][b] == np.searchsorted(cdf, float(u[b, gamma]) * cdf[-1], side="right")


def test_draw_is_monotone_in_its_uniform_and_ignores_the_accept_uniform_of_later_rows():
    rng = np.random.default_rng(3)
    V, n = 300, 257
    zp = rng.normal(0, 2, (1, 3, V)).astype(np.float32)
    zq = rng.normal(0, 2, (1, 2, V)).astype(np.float32)
    draft = np.array([[int(np.argmin(zp[0, 0] - zq[0, 0])), 0]], np.int32)  # p/q smallest: likely rejected
    us = np.linspace(0, 1, n, endpoint=False, dtype=np.float32)
    u = np.stack([np.full(n, 0.999, np.float32), rng.random(n).astype(np.float32), us], 1)
    P = np.repeat(zp, n, 0)
    Q = np.repeat(zq, n, 0)
    r = oracle.accept(RS, np.repeat(draft, n, 0), P, Q, u, margins=False)
    assert np.all(r["accepted_len"] == 0)
    assert np.all(np.diff(r["next_token"]) >= 0)
    # the draw only takes tokens where p > q
    pz, qz = _softmax(zp[0, 0]), _softmax(zq[0, 0])
    assert np.all(pz[r["next_token"]] > qz[r["next_token"]])


def test_non_finite_row_falls_back_to_argmax():
    V = 16
    zp = np.zeros((1, 2, V), np.float32)
    zp[0, 0, 3] = 5.0
    zp[0, 0, 7] = np.nan
    zq = np.zeros((1, 1, V), np.float32)
    r = oracle.accept(RS, [[3]], zp, zq, np.array([[0.1, 0.5]], np.float32), margins=False)
    assert r["accepted_len"][0] == 0 and r["next_token"][0] == 3 and r["flags"][0] & 1
