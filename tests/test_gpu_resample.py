"""GPU parity of sdd_accept's distribution-preserving ratio mode (RATIO_SAMPLE) against the CPU oracle.

The acceptance decisions are the ratio test's (compared as for RATIO: bit-exact away from oracle near-ties);
the drawn token is an inverse-CDF pick whose fp32 CDF (GPU) and fp64 CDF (oracle) differ by rounding, so it
must equal the oracle's wherever u * W lies farther than 1e-5 W from the edges of the oracle's interval, and
everywhere it must be a valid pick of the fp64 CDF within that tolerance.  Shapes: the full acceptance
workload (bf16 [16, 33, 151936]) with drafter rows close to the target's so that rejections are frequent;
fp32 rows with vocabularies that take the scalar and 16-byte paths and more than one chunk (20000, 300000);
a tiny vocabulary run checks the rule's defining property on the GPU itself: the first emitted token follows
the target distribution.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module")
def sdd():
    from paper_2608_14787_amd import sdd as S
    assert S.device_ok(), "needs a gfx950 device"
    return S


def _softmax64(z):
    z = np.asarray(z, np.float64)
    e = np.exp(z - z.max())
    return e / e.sum()


def _valid_pick(zp, zq, u, v):
    """v is a valid inverse-CDF pick of the fp64 residual (or p) distribution at u, within TOL of the total."""
    p = _softmax64(zp)
    w = p if zq is None else np.maximum(0.0, p - _softmax64(zq))
    if not w.sum() > 0:
        w = p
    c = np.cumsum(w)
    t = u * c[-1]
    before = c[v - 1] if v > 0 else 0.0
    return w[v] > 0 and before <= t + TOL * c[-1] and c[v] >= t - TOL * c[-1]


def _check(sdd, draft, U, p_np, q_np, dev_p, dev_q):
    B, R, V = p_np.shape
    gamma = R - 1
    L, nxt, fl = sdd.accept(torch.from_numpy(draft).cuda(), dev_p, sdd.RATIO_SAMPLE, q=dev_q,
                            uniforms=torch.from_numpy(U).cuda())
    torch.cuda.synchronize()
    L, nxt = L.cpu().numpy(), nxt.cpu().numpy()
    ref = oracle.accept(oracle.RATIO_SAMPLE, draft, p_np, q_np, U)
    near = np.array([(ref["dec_margin"][b, :gamma] < 1e-4).any() if gamma else False for b in range(B)])
    same_L = L == ref["accepted_len"]
    assert np.all(same_L | near), np.nonzero(~(same_L | near))
    n_exact = n_tie = 0
    n_diff = int((nxt != ref["next_token"])[same_L].sum())
    for b in np.nonzero(same_L)[0]:
        if ref["sample_margin"][b] > TOL:
            assert nxt[b] == ref["next_token"][b], (b, int(L[b]), ref["sample_margin"][b])
            n_exact += 1
        else:
            n_tie += 1
        Lb = int(L[b])
        if np.isfinite(ref["sample_margin"][b]):
            zq = q_np[b, Lb] if Lb < gamma else None
            assert _valid_pick(p_np[b, Lb], zq, float(U[b, gamma]), int(nxt[b])), b
    print(f"draws: {n_exact} outside the tolerance band (equal), {n_tie} inside, {n_diff} differ", flush=True)
    return L, nxt, n_exact, n_tie


def test_resample_full_size_bf16(sdd):
    inp = W.accept_inputs(seed=31)
    B, R, V = inp.target_bits.shape
    gamma = R - 1
    g = np.random.default_rng(5)
    # drafter rows = target rows + N(0, 0.7^2) noise: p/q near 1, so rejections are frequent
    t32 = inp.target
    q32 = t32[:, :gamma] + g.normal(0, 0.7, size=(B, gamma, V)).astype(np.float32)
    q_bits = W.to_bf16_bits(q32)
    q_np = W.bf16_bits_to_f32(q_bits)
    U = W.uniforms(77, (B, gamma + 1))
    dev_p = torch.from_numpy(inp.target_bits.view(np.int16)).cuda().view(torch.bfloat16)
    dev_q = torch.from_numpy(q_bits.view(np.int16)).cuda().view(torch.bfloat16)
    print("resample full size bf16", flush=True)
    L, nxt, n_exact, n_tie = _check(sdd, inp.draft, U, t32, q_np, dev_p, dev_q)
    assert (L < gamma).sum() >= B // 2  # the residual draw is exercised
    assert n_exact >= B - 1
    # bit-stable on a repeated call
    L2, nxt2, _ = sdd.accept(torch.from_numpy(inp.draft).cuda(), dev_p, sdd.RATIO_SAMPLE, q=dev_q,
                             uniforms=torch.from_numpy(U).cuda())
    assert np.array_equal(L2.cpu().numpy(), L) and np.array_equal(nxt2.cpu().numpy(), nxt)


@pytest.mark.parametrize("V", [7, 1000, 20000, 300000])
def test_resample_fp32_shapes(sdd, V):
    B, gamma = 16, 3
    g = np.random.default_rng(V)
    p = g.normal(0, 2, size=(B, gamma + 1, V)).astype(np.float32)
    q = (p[:, :gamma] + g.normal(0, 0.8, size=(B, gamma, V))).astype(np.float32)
    draft = np.argmax(q, axis=2).astype(np.int32)
    U = W.uniforms(V + 1, (B, gamma + 1))
    U[:, :gamma] = np.float32(0.999)  # mostly rejections
    U[0, :gamma] = 0.0  # sequence 0: everything accepted, bonus draw from p_gamma
    print(f"resample fp32 V={V}", flush=True)
    L, nxt, n_exact, n_tie = _check(sdd, draft, U, p, q, torch.from_numpy(p).cuda(),
                                    torch.from_numpy(q).cuda())
    assert L[0] == gamma
    # a token's interval is about W / V wide: at small V most draws lie outside the tolerance band
    if V <= 20000:
        assert n_exact >= B // 2


def test_resample_gamma0_and_edges(sdd):
    V = 4096
    g = np.random.default_rng(9)
    p = g.normal(0, 2, size=(3, 1, V)).astype(np.float32)
    U = np.array([[0.0], [0.5], [1.0 - 2 ** -24]], np.float32)
    L, nxt, fl = sdd.accept(torch.zeros((3, 0), dtype=torch.int32, device="cuda"), torch.from_numpy(p).cuda(),
                            sdd.RATIO_SAMPLE, uniforms=torch.from_numpy(U).cuda())
    torch.cuda.synchronize()
    ref = oracle.accept(oracle.RATIO_SAMPLE, np.zeros((3, 0), np.int32), p, None, U)
    assert np.array_equal(L.cpu().numpy(), [0, 0, 0])
    for b in range(3):
        assert _valid_pick(p[b, 0], None, float(U[b, 0]), int(nxt.cpu().numpy()[b]))
    assert nxt.cpu().numpy()[0] == ref["next_token"][0] == 0 or ref["sample_margin"][0] <= TOL
    # a non-finite row L keeps the argmax
    p2 = g.normal(0, 1, size=(1, 2, V)).astype(np.float32)
    p2[0, 0, 5] = np.nan
    p2[0, 0, 9] = 50.0
    q2 = g.normal(0, 1, size=(1, 1, V)).astype(np.float32)
    L, nxt, fl = sdd.accept(torch.tensor([[9]], dtype=torch.int32, device="cuda"), torch.from_numpy(p2).cuda(),
                            sdd.RATIO_SAMPLE, q=torch.from_numpy(q2).cuda(),
                            uniforms=torch.tensor([[0.1, 0.3]], device="cuda"))
    torch.cuda.synchronize()
    assert L.item() == 0 and nxt.item() == 9 and fl.item() & 1
    with pytest.raises(sdd.SDDError):  # the draw needs uniforms
        sdd.accept(torch.zeros((1, 0), dtype=torch.int32, device="cuda"), torch.from_numpy(p[:1]).cuda(),
                   sdd.RATIO_SAMPLE)


def test_resample_first_token_follows_target_on_gpu(sdd):
    """The rule's defining property on the GPU path alone: with x ~ q, the first emitted token ~ p."""
    V, n = 6, 16384
    g = np.random.default_rng(12)
    zp = g.normal(0, 1.5, V).astype(np.float32)
    zq = g.normal(0, 1.5, V).astype(np.float32)
    p, q = _softmax64(zp), _softmax64(zq)
    x = g.choice(V, size=n, p=q).astype(np.int32)
    P = torch.from_numpy(np.broadcast_to(np.stack([zp, zp]), (n, 2, V)).copy()).cuda()
    Q = torch.from_numpy(np.broadcast_to(zq, (n, 1, V)).copy()).cuda()
    U = torch.from_numpy(W.uniforms(13, (n, 2))).cuda()
    L, nxt, _ = sdd.accept(torch.from_numpy(x[:, None]).cuda(), P, sdd.RATIO_SAMPLE, q=Q, uniforms=U)
    torch.cuda.synchronize()
    first = np.where(L.cpu().numpy() == 1, x, nxt.cpu().numpy())
    freq = np.bincount(first, minlength=V) / n
    sd = np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(freq - p) <= 5 * sd), (freq, p)
