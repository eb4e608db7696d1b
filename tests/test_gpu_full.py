"""GPU parity of the full-recompute verifier (sdd_verify_full), the agreement counters
(sdd_audit_accumulate) and a skip-policy loop that audits every skipped round with a shadow verifier call.

sdd_verify_full recomputes every position, so its logits must equal the cached call's on the same context
bit for bit (the kernels do not depend on how rows are batched), and the oracle's no-cache forward within
the logit tolerance (1e-4 x max|z| fp32, 2e-2 bf16).  Agreement counters are integers: bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import argmax_near_tie, row_tol_ok, to_dev_i32

pytestmark = pytest.mark.gpu

MID_BF16 = W.ModelShape(2, 512, 8, 2, 64, 1024, 2048, 1e-6, 1e6, True, "bf16")


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


@pytest.mark.parametrize("shape,n,gamma,ws_rows", [(W.TINY, 72, 8, 64), (W.TINY, 300, 32, 64), (MID_BF16, 140, 16, 64),
                                                  (W.TINY, 9, 0, 64), (W.TINY, 300, 32, 256), (MID_BF16, 240, 16, 256)])
def test_full_recompute_matches_oracle_and_cached_call(S, shape, n, gamma, ws_rows):
    print(f"full recompute {shape.dtype} n={n} gamma={gamma} ws_rows={ws_rows}", flush=True)
    m = S.Model(shape)
    m.init_random(0, 0.02)
    ws = m.workspace(ws_rows)
    toks = W.prompt(n + 3, n, shape.vocab)
    scratch = S.KVCache(m, 1, n + 4)
    lf = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    af = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
    scratch.verify_full(to_dev_i32(toks), gamma, lf, af, ws)
    # the cached call on a cache prefilled with the context
    kv = S.KVCache(m, 1, n + 4)
    kv.prefill(0, to_dev_i32(toks[: n - gamma]), ws)
    lc = torch.empty_like(lf)
    kv.verify(to_dev_i32([0]), to_dev_i32(toks[n - gamma:].reshape(1, gamma)), lc, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(lf, lc)
    # the oracle's full recomputation (no cache)
    om = oracle.Model(shape)
    want = om.forward_full(toks, row0=n - gamma - 1)
    got = lf[0].cpu().numpy()
    tol = 1e-4 if shape.dtype == "f32" else 2e-2
    ok, rel = row_tol_ok(got, want, tol)
    assert ok.all(), rel.max()
    near = argmax_near_tie(want, tol * np.abs(want).max(-1))
    am = af[0].cpu().numpy()
    assert np.all((am == want.argmax(-1)) | near)
    # a second call on the same scratch gives the same result
    lf2 = torch.empty_like(lf)
    scratch.verify_full(to_dev_i32(toks), gamma, lf2, None, ws)
    assert torch.equal(lf, lf2)


def test_full_recompute_argument_errors(S):
    m = S.Model(W.TINY)
    m.init_random(0, 0.02)
    ws = m.workspace(64)
    scratch = S.KVCache(m, 1, 16)
    lf = torch.empty((1, 9, W.TINY.vocab), dtype=torch.float32, device="cuda")
    with pytest.raises(S.SDDError):  # more tokens than the scratch holds
        scratch.verify_full(to_dev_i32(np.arange(20)), 8, lf, None, ws)
    with pytest.raises(S.SDDError):  # fewer tokens than a block
        scratch.verify_full(to_dev_i32(np.arange(5)), 8, lf, None, ws)


def test_audit_counters_match_oracle(S):
    rng = np.random.default_rng(3)
    acc = torch.zeros(4, dtype=torch.int64, device="cuda")
    ref = np.zeros(4, np.int64)
    for _ in range(5):
        B = int(rng.integers(1, 700))
        K = rng.integers(0, 33, B).astype(np.int32)
        K[rng.random(B) < 0.4] = 0
        L = rng.integers(0, 33, B).astype(np.int32)
        S.audit_accumulate(to_dev_i32(K), to_dev_i32(L), acc)
        oracle.audit_accumulate(K, L, ref)
    torch.cuda.synchronize()
    assert acc.cpu().numpy().tolist() == ref.tolist()


def test_policy_loop_with_shadow_audit(S):
    """Decoding with the full-recompute verifier and the two-gate scheduler (raw signal): on a skipped round the
    drafts' prefix of length K is committed unverified and a shadow verifier call (same block, excluded from
    decoding) supplies L for the agreement counters; on a strict round L + 1 tokens are committed.  Every
    round's decision is replayed by the oracle on the GPU's inputs."""
    shape, gamma, rounds, P = W.TINY, 8, 12, 40
    m = S.Model(shape)
    m.init_random(0, 0.02)
    ws = m.workspace(64)
    om = oracle.Model(shape)
    V = shape.vocab
    toks = list(W.prompt(17, P, V))
    max_n = P + rounds * (gamma + 1) + 4
    scratch = S.KVCache(m, 1, max_n)
    g = np.random.default_rng(9)
    D = torch.zeros(1, dtype=torch.int32, device="cuda")
    D_ref = np.zeros(1, np.int32)
    acc = torch.zeros(4, dtype=torch.int64, device="cuda")
    acc_ref = np.zeros(4, np.int64)
    logits = torch.empty((1, gamma + 1, V), dtype=torch.float32, device="cuda")
    am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
    outs = tuple(torch.empty(1, dtype=torch.int32, device="cuda") for _ in range(3))
    n_skip = 0
    for r in range(rounds):
        # drafts: the oracle's greedy continuation with some tokens replaced; drafter logits confident on them
        cont = om.forward_full(np.array(toks, np.int32), row0=len(toks) - 1)[0].argmax()
        drafts = np.full(gamma, cont, np.int32)
        drafts[1:] = g.integers(0, V, gamma - 1)
        z = W.drafter_logits(seed=100 + r, draft=drafts[None], rows=gamma, vocab=V, boost=0.0, boost_hi=6.0)
        sk, lc, _ = S.confidence_prefix(torch.from_numpy(z).cuda(), gamma, 0.5, log_conf=True)
        K, Kh, rs = S.schedule(lc.contiguous(), D, S.SIG_RAW, 0.5, 0.6, k_min=2, s_max=12)
        # verifier call on the block: strict on a strict round, shadow (audit only) on a skipped one
        seq = np.array(toks + list(drafts), np.int32)
        scratch.verify_full(to_dev_i32(seq), gamma, logits, am, ws)
        L, nxt, _ = S.accept(to_dev_i32(drafts[None]), logits, S.GREEDY, out=outs)
        S.audit_accumulate(K, L, acc)
        torch.cuda.synchronize()
        k, l, t = int(K.item()), int(L.item()), int(nxt.item())
        # oracle replay of the round on the same drafts and drafter scores
        want = om.forward_full(seq, row0=len(seq) - gamma - 1)
        ref_acc = oracle.accept(oracle.GREEDY, drafts[None], want[None].astype(np.float32), margins=True)
        near = (ref_acc["dec_margin"][0] < 1e-4 * np.abs(want).max()).any()
        assert near or (l, t) == (int(ref_acc["accepted_len"][0]), int(ref_acc["next_token"][0]))
        ref_s = oracle.schedule(lc.cpu().numpy(), D_ref, oracle.SIG_RAW, 0.5, 0.6, k_min=2, s_max=12)
        assert int(ref_s["K"][0]) == k
        D_ref = ref_s["D"]
        oracle.audit_accumulate([k], [l], acc_ref)
        if k > 0:
            toks += list(drafts[:k])
            n_skip += 1
        else:
            toks += list(drafts[:l]) + [t]
    assert acc.cpu().numpy().tolist() == acc_ref.tolist()
    st, fp = oracle.agreement(acc_ref)
    print(f"rounds {rounds}, skipped {n_skip}, StrictToken {st:.3f}, FullPrefix {fp:.3f}", flush=True)
    assert n_skip > 0 and n_skip < rounds
