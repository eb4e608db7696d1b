"""Pins of the oracle's target decoder (CPU only).

The paper names its verifier but prints no architecture, so the decoder is
pinned by (a) agreement of its two independent routes -- full recomputation
with no cache, the paper's measured verifier (Appendix "Evaluation and
Throughput"), and the cached block verify; (b) closed forms (one-token
sequences, zeroed residual branches); (c) a composition of
torch.nn.functional library ops in float64 at the tiny shape.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import workloads as W

SMALL = W.ModelShape(2, 64, 4, 2, 16, 96, 200, 1e-6, 1e4, True, "f32")
SMALL_BF16 = W.ModelShape(2, 64, 8, 2, 16, 96, 200, 1e-6, 1e6, False, "bf16")


def _weights(shape, seed=0, sigma=0.02):
    out = {}
    bf16 = shape.dtype == "bf16"
    for kind in [oracle.EMBED, oracle.LM_HEAD]:
        r, c = oracle.tensor_shape(shape, kind)
        out[kind] = oracle.weight_values(seed, oracle.tensor_id(kind), 0, r * c, sigma, bf16).reshape(r, c)
    for l in range(shape.n_layers):
        for kind in [oracle.WQ, oracle.WK, oracle.WV, oracle.WO, oracle.WGATE, oracle.WUP, oracle.WDOWN]:
            r, c = oracle.tensor_shape(shape, kind)
            out[(kind, l)] = oracle.weight_values(seed, oracle.tensor_id(kind, l), 0, r * c, sigma,
                                                  bf16).reshape(r, c)
    return out


def _rope_torch(x, pos, theta):
    # x [n, heads, hd]; rotate-half with inv_freq theta^(-2i/hd)
    hd = x.shape[-1]
    inv = theta ** (-torch.arange(0, hd // 2, dtype=torch.float64) * 2 / hd)
    ang = pos[:, None].double() * inv[None, :]
    cos = torch.cat([ang.cos(), ang.cos()], -1)[:, None, :]
    sin = torch.cat([ang.sin(), ang.sin()], -1)[:, None, :]
    x1, x2 = x[..., : hd // 2], x[..., hd // 2:]
    return x * cos + torch.cat([-x2, x1], -1) * sin


def _bf16_f64(a: torch.Tensor) -> torch.Tensor:
    """Nearest BF16 value of each float64 (ties to even), by bit arithmetic on the binary64 encoding:
    keep 7 of the 52 fraction bits, round the dropped 45 half to even."""
    u = a.contiguous().numpy().view(np.uint64)
    drop = np.uint64(45)
    lsb = (u >> drop) & np.uint64(1)
    r = (u + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    return torch.from_numpy(r.view(np.float64).copy())


def _torch_reference(shape, w, tokens, gains=None, bf16_operands=False):
    """Decoder as a composition of torch.nn.functional ops, float64 on the CPU.

    gains: optional dict of RMSNorm gains keyed like w ((kind, layer) or FINAL_NORM); missing ones are 1.
    bf16_operands: the activations entering each matrix product are rounded to BF16 (x * g of each
    projection, whose row scale 1/rms(x) then multiplies the product; q, k, v; attention output; FFN
    hidden state)."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    d, hd, hq, hk = shape.d_model, shape.head_dim, shape.n_q_heads, shape.n_kv_heads
    n = len(tokens)
    gains = gains or {}
    g = lambda key, size: t(gains[key]) if key in gains else torch.ones(size, dtype=torch.float64)
    b = _bf16_f64 if bf16_operands else (lambda a: a)

    def norm_linear(x, gain, *mats):
        if not bf16_operands:
            h = F.rms_norm(x, (x.shape[-1],), gain, eps=shape.rms_eps)
            return [F.linear(h, W) for W in mats]
        r = torch.rsqrt((x * x).mean(-1, keepdim=True) + shape.rms_eps)
        h = _bf16_f64(x * gain)
        return [F.linear(h, W) * r for W in mats]

    x = F.embedding(torch.from_numpy(np.asarray(tokens, np.int64)), t(w[oracle.EMBED]))
    pos = torch.arange(n)
    for l in range(shape.n_layers):
        q, k, v = norm_linear(x, g((oracle.ATTN_NORM, l), d), t(w[(oracle.WQ, l)]), t(w[(oracle.WK, l)]),
                              t(w[(oracle.WV, l)]))
        q, k, v = q.view(n, hq, hd), k.view(n, hk, hd), v.view(n, hk, hd)
        if shape.qk_norm:
            q = F.rms_norm(q, (hd,), g((oracle.Q_NORM, l), hd), eps=shape.rms_eps)
            k = F.rms_norm(k, (hd,), g((oracle.K_NORM, l), hd), eps=shape.rms_eps)
        q, k = _rope_torch(q, pos, shape.rope_theta), _rope_torch(k, pos, shape.rope_theta)
        q, k, v = b(q), b(k), b(v)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True, enable_gqa=True)
        x = x + F.linear(b(o.transpose(0, 1).reshape(n, hq * hd)), t(w[(oracle.WO, l)]))
        gt, up = norm_linear(x, g((oracle.FFN_NORM, l), d), t(w[(oracle.WGATE, l)]), t(w[(oracle.WUP, l)]))
        x = x + F.linear(b(F.silu(gt) * up), t(w[(oracle.WDOWN, l)]))
    return norm_linear(x, g(oracle.FINAL_NORM, d), t(w[oracle.LM_HEAD]))[0].numpy()


_GAIN_KIND = {"final": oracle.FINAL_NORM, "attn": oracle.ATTN_NORM, "ffn": oracle.FFN_NORM,
              "q": oracle.Q_NORM, "k": oracle.K_NORM}


def random_gains(shape, seed):
    """workloads.norm_gains keyed like _weights: (kind, layer), or FINAL_NORM."""
    out = {}
    for (name, layer), v in W.norm_gains(seed, shape).items():
        kind = _GAIN_KIND[name]
        out[kind if kind == oracle.FINAL_NORM else (kind, layer)] = v
    return out


def _set_gains(m, gains):
    for key, v in gains.items():
        kind, layer = key if isinstance(key, tuple) else (key, 0)
        m.set_tensor(kind, layer, v)


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["qknorm-f32", "gqa4-bf16"])
def test_matches_torch_functional_composition(shape):
    toks = W.prompt(1, 13, shape.vocab)
    m = oracle.Model(shape)
    got = m.forward_full(toks)
    want = _torch_reference(shape, _weights(shape), toks)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-10 * np.abs(want).max())


def test_tiny_shape_matches_torch_functional():
    shape = W.TINY
    toks = W.prompt(2, 20, shape.vocab)
    m = oracle.Model(shape)
    want = _torch_reference(shape, _weights(shape), toks)
    np.testing.assert_allclose(m.forward_full(toks, 10), want[10:], rtol=0, atol=1e-10 * np.abs(want).max())


@pytest.mark.parametrize("shape", [SMALL, W.TINY], ids=["small", "tiny"])
def test_cached_verify_equals_full_recompute(shape):
    m = oracle.Model(shape)
    toks = W.prompt(3, 30, shape.vocab)
    kv = oracle.KV(m, 64)
    kv.prefill(toks[:20])  # caches 0..18, pending = toks[19]
    assert kv.len == 19 and kv.pending == toks[19]
    drafts = toks[20:26]
    got = kv.verify(drafts)  # rows at positions 19..25
    want = m.forward_full(toks[:26], 19)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-11 * np.abs(want).max())
    # gamma = 0 is a decode step: the last row of the full recompute
    got0 = kv.verify([])
    np.testing.assert_allclose(got0, want[:1], rtol=0, atol=1e-11 * np.abs(want).max())


def test_commit_then_decode_equals_fresh_prefill():
    shape = SMALL
    m = oracle.Model(shape)
    toks = W.prompt(4, 40, shape.vocab)
    kv = oracle.KV(m, 64)
    kv.prefill(toks[:10])
    drafts = toks[10:17]
    kv.verify(drafts)
    L, nxt = 3, int(toks[30])
    kv.commit(L, nxt)  # keeps [pending, d0, d1, d2] = toks[9:13], pending = nxt
    assert kv.len == 13 and kv.pending == nxt
    a = kv.verify(toks[31:33])
    seq = np.concatenate([toks[:13], [nxt], toks[31:33]]).astype(np.int32)
    kv2 = oracle.KV(m, 64)
    kv2.prefill(seq[:14])
    b = kv2.verify(seq[14:])
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-11 * np.abs(b).max())
    np.testing.assert_allclose(a, m.forward_full(seq, 13), rtol=0, atol=1e-11 * np.abs(b).max())


def test_single_token_closed_form():
    # one position: attention returns v itself; RoPE at position 0 is the identity
    shape = SMALL_BF16.with_layers(1)
    m = oracle.Model(shape)
    w = _weights(shape)
    tok = 5
    x = w[oracle.EMBED][tok].astype(np.float64)
    rms = lambda a: a / np.sqrt((a * a).mean() + shape.rms_eps)
    h = rms(x)
    v = w[(oracle.WV, 0)].astype(np.float64) @ h
    grp = shape.n_q_heads // shape.n_kv_heads
    o = np.concatenate([v.reshape(shape.n_kv_heads, -1)[hh // grp] for hh in range(shape.n_q_heads)])
    x = x + w[(oracle.WO, 0)].astype(np.float64) @ o
    h = rms(x)
    g = w[(oracle.WGATE, 0)].astype(np.float64) @ h
    u = w[(oracle.WUP, 0)].astype(np.float64) @ h
    x = x + w[(oracle.WDOWN, 0)].astype(np.float64) @ (g / (1 + np.exp(-g)) * u)
    want = w[oracle.LM_HEAD].astype(np.float64) @ rms(x)
    np.testing.assert_allclose(m.forward_full([tok])[0], want, rtol=0, atol=1e-12)
    # K cached at position 0 is the un-rotated projection
    kv = oracle.KV(m, 4)
    kv.prefill([tok, 1])
    k0, v0 = kv.read(0, 0)
    np.testing.assert_allclose(k0, w[(oracle.WK, 0)].astype(np.float64) @ rms(w[oracle.EMBED][tok].astype(np.float64)), atol=1e-12)


def test_zeroed_branches_give_embedding_logits():
    shape = SMALL
    m = oracle.Model(shape)
    w = _weights(shape)
    for l in range(shape.n_layers):
        m.set_tensor(oracle.WO, l, np.zeros(oracle.tensor_shape(shape, oracle.WO), np.float32))
        m.set_tensor(oracle.WDOWN, l, np.zeros(oracle.tensor_shape(shape, oracle.WDOWN), np.float32))
    toks = W.prompt(5, 9, shape.vocab)
    e = w[oracle.EMBED][toks].astype(np.float64)
    h = e / np.sqrt((e * e).mean(-1, keepdims=True) + shape.rms_eps)
    want = h @ w[oracle.LM_HEAD].astype(np.float64).T
    np.testing.assert_allclose(m.forward_full(toks), want, rtol=0, atol=1e-12)


def test_capacity_and_bad_tokens():
    m = oracle.Model(SMALL)
    kv = oracle.KV(m, 8)
    kv.prefill([1, 2, 3])
    with pytest.raises(ValueError):
        kv.verify([1, 2, 3, 4, 5, 6])  # 2 + 7 rows > 8
    with pytest.raises(ValueError):
        kv.verify([SMALL.vocab])


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["qknorm-f32", "gqa4-bf16"])
def test_nonunit_norm_gains_match_torch(shape):
    """Every RMSNorm gain (attention, FFN, final, and q/k with QK-norm) applied where the decoder applies it:
    random gains per tensor and layer, against torch's rms_norm with the same weights."""
    gains = random_gains(shape, 17)
    m = oracle.Model(shape)
    _set_gains(m, gains)
    toks = W.prompt(18, 15, shape.vocab)
    want = _torch_reference(shape, _weights(shape), toks, gains)
    np.testing.assert_allclose(m.forward_full(toks), want, rtol=0, atol=1e-10 * np.abs(want).max())
    # a gain moved to another layer or norm changes the logits (the check above sees misplaced gains)
    swapped = dict(gains)
    swapped[(oracle.ATTN_NORM, 0)], swapped[(oracle.FFN_NORM, 0)] = gains[(oracle.FFN_NORM, 0)], gains[(oracle.ATTN_NORM, 0)]
    other = _torch_reference(shape, _weights(shape), toks, swapped)
    assert np.abs(other - want).max() > 1e-6 * np.abs(want).max()
    # the cached route agrees
    kv = oracle.KV(m, 32)
    kv.prefill(toks[:9])
    np.testing.assert_allclose(kv.verify(toks[9:15]), want[8:15], rtol=0, atol=1e-10 * np.abs(want).max())


def test_long_sequence_matches_torch_functional():
    """Attention over a few hundred positions (the loops whose order was interchanged to read V by rows)."""
    shape = SMALL.with_layers(1)
    toks = W.prompt(19, 300, shape.vocab)
    m = oracle.Model(shape)
    want = _torch_reference(shape, _weights(shape), toks)
    np.testing.assert_allclose(m.forward_full(toks, 250), want[250:], rtol=0, atol=1e-10 * np.abs(want).max())
    kv = oracle.KV(m, 320)
    kv.prefill(toks[:280])
    np.testing.assert_allclose(kv.verify(toks[280:300]), want[279:300], rtol=0, atol=1e-10 * np.abs(want).max())


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16, W.TINY], ids=["small", "small-bf16", "tiny"])
def test_streamed_model_equals_materialized(shape):
    """Layer streaming generates each layer's weights when the forward reaches it: the same values, so both
    routes give bit-identical logits to the materialized model."""
    m = oracle.Model(shape)
    ms = oracle.Model(shape, streamed=True)
    toks = W.prompt(20, 24, shape.vocab)
    a = m.forward_full(toks, 10)
    b = ms.forward_full(toks, 10)
    assert np.array_equal(a, b)
    kv, kvs = oracle.KV(m, 32), oracle.KV(ms, 32)
    kv.prefill(toks[:12])
    kvs.prefill(toks[:12])
    assert np.array_equal(kv.verify(toks[12:20]), kvs.verify(toks[12:20]))
    # a second forward regenerates the layers (nothing was kept from the first); the layer-by-layer steps
    # compute the same
    seen = []
    assert np.array_equal(ms.forward_full(toks, 10, progress=seen.append), a)
    assert seen == list(range(shape.n_layers))
    with pytest.raises(ValueError):
        ms.set_tensor(oracle.WO, 0, np.zeros(oracle.tensor_shape(shape, oracle.WO), np.float32))


@pytest.mark.parametrize("shape", [SMALL, SMALL_BF16], ids=["qknorm-f32", "gqa4-bf16"])
def test_bf16_operand_mode_matches_torch(shape):
    """BF16-operand mode (the verifier as a BF16 model): against torch.nn.functional with the same
    activations rounded by bit arithmetic on float64 (an implementation independent of the oracle's
    frexp / nearbyint rounding), with non-unit gains; the cached route agrees with full recompute."""
    gains = random_gains(shape, 21)
    m = oracle.Model(shape, bf16_operands=True)
    _set_gains(m, gains)
    toks = W.prompt(22, 15, shape.vocab)
    want = _torch_reference(shape, _weights(shape), toks, gains, bf16_operands=True)
    np.testing.assert_allclose(m.forward_full(toks), want, rtol=0, atol=1e-10 * np.abs(want).max())
    kv = oracle.KV(m, 32)
    kv.prefill(toks[:9])
    np.testing.assert_allclose(kv.verify(toks[9:15]), want[8:15], rtol=0, atol=1e-10 * np.abs(want).max())
    # the mode changes the logits by about the BF16 rounding scale, and turning it off restores exactness
    exact = _torch_reference(shape, _weights(shape), toks, gains)
    rel = np.abs(want - exact).max() / np.abs(exact).max()
    assert 1e-5 < rel < 5e-2, rel
    m0 = oracle.Model(shape)
    _set_gains(m0, gains)
    np.testing.assert_allclose(m0.forward_full(toks), exact, rtol=0, atol=1e-10 * np.abs(exact).max())


def test_bf16_rounding_of_the_bit_method_matches_fp32_rounding():
    """The test's float64 -> BF16 rounding agrees with workloads' fp32 -> BF16 bit rounding on values that
    are exactly representable in fp32 (so no double rounding is involved), ties included."""
    rg = W.rng(23)
    a = (rg.standard_normal(100000) * 10.0 ** rg.integers(-6, 6, 100000)).astype(np.float32)
    ties = ((W.bf16_bits_to_f32(W.to_bf16_bits(a)).view(np.uint32) | np.uint32(0x8000)).view(np.float32))
    a = np.concatenate([a, ties])
    want = W.bf16_bits_to_f32(W.to_bf16_bits(a)).astype(np.float64)
    got = _bf16_f64(torch.from_numpy(a.astype(np.float64))).numpy()
    assert np.array_equal(got, want)
