"""GPU parity of sdd_accept and sdd_confidence_prefix against the CPU oracle.

Full size: logits [16, 33, 151936] bf16 (the acceptance workload), every
mode; integer outputs must be bit-exact (greedy, top-k and lenience decide by
comparisons of identical inputs), the ratio test and the confidence decisions
bit-exact except at oracle near-ties (margin below 1e-4 / 1e-5), which are
counted.  Edge cases: gamma = 0, a single sequence, vocabularies that are not
a multiple of the vector width, fp32 logits, non-finite values, draft tokens
out of range, repeated calls (bit-stable).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sdd():
    from paper_2608_14787_amd import sdd as S
    assert S.device_ok(), "needs a gfx950 device"
    return S


def _bf16(bits, dev="cuda"):
    return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)


@pytest.fixture(scope="module", params=["literal", "rowmax"])
def full(request):
    return request.param, W.accept_inputs(seed=11, variant=request.param)


CASES = [("greedy", 0, 1, 1.0), ("topk", 2, 1, 1.0), ("topk", 2, 4, 1.0), ("topk", 2, 16, 1.0),
         ("lenient", 3, 1, 0.3), ("lenient", 3, 1, 1.0), ("ratio", 1, 1, 1.0)]


@pytest.mark.parametrize("name,mode,k,len_", CASES, ids=[f"{c[0]}-{c[2]}-{c[3]}" for c in CASES])
def test_accept_full_size(sdd, full, name, mode, k, len_):
    variant, inp = full
    print(f"accept {variant} {name} k={k} l={len_}", flush=True)
    B, R, V = inp.target_bits.shape
    p = _bf16(inp.target_bits)
    q = _bf16(inp.drafter_bits)
    d = torch.from_numpy(inp.draft).cuda()
    u = torch.from_numpy(inp.u).cuda()
    L, nxt, fl = sdd.accept(d, p, mode, q=q if mode == 1 else None, uniforms=u if mode == 1 else None,
                            k=k, lenience=len_)
    L2, nxt2, _ = sdd.accept(d, p, mode, q=q if mode == 1 else None, uniforms=u if mode == 1 else None,
                             k=k, lenience=len_)
    torch.cuda.synchronize()
    assert torch.equal(L, L2) and torch.equal(nxt, nxt2)  # bit-stable
    ref = oracle.accept(mode, inp.draft, inp.target, q=inp.drafter[:, :R - 1] if mode == 1 else None,
                        u=inp.u if mode == 1 else None, k=k, lenience=len_, margins=(mode == 1))
    Lg, ng = L.cpu().numpy(), nxt.cpu().numpy()
    if mode == 1:
        # exclude sequences whose decisions up to the first failure include an oracle near-tie
        dm = ref["dec_margin"]
        near = np.array([(dm[b, :min(ref["accepted_len"][b] + 1, R - 1)] < 1e-4).any() for b in range(B)])
        print(f"ratio near-tie exclusions: {near.sum()} of {B}")
        assert (Lg[~near] == ref["accepted_len"][~near]).all()
        assert (ng[~near] == ref["next_token"][~near]).all()
        assert near.sum() <= 2
    else:
        assert (Lg == ref["accepted_len"]).all(), (Lg, ref["accepted_len"])
        assert (ng == ref["next_token"]).all()
    assert (fl.cpu().numpy() == ref["flags"]).all()
    if variant == "rowmax" and mode in (0, 2):
        assert len(set(Lg.tolist())) > 3  # the workload exercises varied accepted lengths


@pytest.mark.parametrize("V", [7, 1001, 4096, 20000])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_accept_small_shapes(sdd, V, dtype):
    g = np.random.default_rng(V)
    B, gamma = 5, 6
    z = (g.standard_normal((B, gamma + 1, V)) * 3).astype(np.float32)
    z[:, :, :3] = np.round(z[:, :, :3])  # ties
    draft = z[:, :gamma].argmax(-1).astype(np.int32)
    flip = g.random((B, gamma)) < 0.2
    draft[flip] = g.integers(0, V, size=int(flip.sum()))
    if dtype == "bf16":
        bits = W.to_bf16_bits(z)
        zt, zv = _bf16(bits), W.bf16_bits_to_f32(bits)
    else:
        zt, zv = torch.from_numpy(z).cuda(), z
    qz = (g.standard_normal((B, gamma + 1, V))).astype(np.float32)
    qt = torch.from_numpy(qz).cuda().to(zt.dtype)
    qv = qt.float().cpu().numpy()
    u = W.uniforms(3, (B, gamma))
    for mode, k, ln in [(0, 1, 1.0), (2, 2, 1.0), (3, 1, 0.5), (1, 1, 1.0)]:
        L, nxt, fl = sdd.accept(torch.from_numpy(draft).cuda(), zt, mode, q=qt, uniforms=torch.from_numpy(u).cuda(),
                                k=k, lenience=ln)
        ref = oracle.accept(mode, draft, zv, q=qv[:, :gamma], u=u, k=k, lenience=ln)
        ok = np.ones(B, bool)
        if mode == 1:
            dm = ref["dec_margin"]
            ok = np.array([not (dm[b, :min(ref["accepted_len"][b] + 1, gamma)] < 1e-4).any() for b in range(B)])
        assert (L.cpu().numpy()[ok] == ref["accepted_len"][ok]).all(), mode
        assert (nxt.cpu().numpy()[ok] == ref["next_token"][ok]).all(), mode


def test_accept_edge_cases(sdd):
    g = np.random.default_rng(5)
    V = 512
    z = g.standard_normal((4, 5, V)).astype(np.float32)
    d = z[:, :4].argmax(-1).astype(np.int32)
    z[0, 2, 9] = np.nan
    z[1, 1, 3] = np.inf
    z[3, 4, 0] = -np.inf
    d[2, 3] = V + 5  # out of range
    L, nxt, fl = sdd.accept(torch.from_numpy(d).cuda(), torch.from_numpy(z).cuda(), 0)
    ref = oracle.accept(0, d, z)
    assert L.cpu().tolist() == ref["accepted_len"].tolist() == [2, 1, 3, 4]
    assert nxt.cpu().tolist() == ref["next_token"].tolist()
    assert fl.cpu().tolist() == ref["flags"].tolist()
    # gamma = 0: only the bonus row
    z0 = g.standard_normal((3, 1, V)).astype(np.float32)
    L, nxt, _ = sdd.accept(torch.zeros((3, 0), dtype=torch.int32, device="cuda"), torch.from_numpy(z0).cuda(), 0)
    assert L.cpu().tolist() == [0, 0, 0] and nxt.cpu().tolist() == z0[:, 0].argmax(-1).tolist()
    with pytest.raises(sdd.SDDError):
        sdd.accept(torch.from_numpy(d).cuda(), torch.from_numpy(z).cuda(), 2, k=0)
    with pytest.raises(sdd.SDDError):
        sdd.accept(torch.from_numpy(d).cuda(), torch.from_numpy(z).cuda(), 3, lenience=0.0)


@pytest.mark.parametrize("variant", ["literal", "boosted"])
def test_confidence_full_size(sdd, variant):
    B, gamma, V = 16, 32, 151936
    draft = W.rng(21).integers(0, V, size=(B, gamma)).astype(np.int32)
    if variant == "literal":
        z = W.drafter_logits(22, draft, gamma + 1, V, scale=4.0, boost=0.0)
    else:
        z = W.drafter_logits(22, draft, gamma + 1, V, scale=4.0, boost=0.0, boost_hi=30.0)
    bits = W.to_bf16_bits(z)
    zt = _bf16(bits)
    zv = W.bf16_bits_to_f32(bits)
    for tau in [0.3, 0.5, 0.7, 0.9]:
        sk, lc, lp = sdd.confidence_prefix(zt, gamma, tau, draft=torch.from_numpy(draft).cuda(), log_conf=True)
        ref = oracle.confidence_prefix(zv, gamma, tau, draft=draft)
        lcg = lc.cpu().numpy()
        np.testing.assert_allclose(lcg, ref["log_conf"], atol=2e-5, rtol=0)
        np.testing.assert_allclose(lp.cpu().numpy(), ref["log_p_draft"], atol=5e-5, rtol=0)
        near = np.array([(np.abs(ref["log_conf"][b, :min(ref["skip_len"][b] + 1, gamma)] - np.log(tau)) < 1e-5).any()
                         for b in range(B)])
        assert (sk.cpu().numpy()[~near] == ref["skip_len"][~near]).all(), tau
        if variant == "boosted" and tau == 0.5:
            assert len(set(ref["skip_len"].tolist())) > 2


def test_confidence_edges(sdd):
    V = 1000
    z = np.zeros((2, 3, V), np.float32)
    z[1, :, 4] = 10.0
    sk, lc, _ = sdd.confidence_prefix(torch.from_numpy(z).cuda(), 3, 0.5, log_conf=True)
    np.testing.assert_allclose(lc.cpu().numpy()[0], -np.log(V), atol=1e-5)
    assert sk.cpu().tolist() == [0, 3]
    assert sdd.confidence_prefix(torch.from_numpy(z).cuda(), 3, 0.5 / V).cpu().tolist() == [3, 3]
    assert sdd.confidence_prefix(torch.from_numpy(z).cuda(), 0, 0.5).cpu().tolist() == [0, 0]
    z[1, 1, 7] = np.nan
    assert sdd.confidence_prefix(torch.from_numpy(z).cuda(), 3, 0.5 / V).cpu().tolist() == [3, 1]
    with pytest.raises(sdd.SDDError):
        sdd.confidence_prefix(torch.from_numpy(z).cuda(), 3, float("nan"))
