"""GPU parity of the verify path (sdd_kv_prefill, sdd_verify_block, sdd_kv_commit) against the oracle.

Logits must agree per row within max|dz| <= tol * max|z_oracle| (tol 1e-4 for fp32 models,
2e-2 for bf16); argmax and accepted lengths must be bit-exact except at positions whose oracle
margin is below that absolute tolerance (counted and printed).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import argmax_near_tie, row_tol_ok, to_dev_i32, untile

pytestmark = pytest.mark.gpu

MID_BF16 = W.ModelShape(2, 512, 8, 2, 64, 1024, 2048, 1e-6, 1e6, True, "bf16")
MID_GQA128 = W.ModelShape(2, 256, 8, 2, 128, 512, 1024, 1e-6, 1e6, False, "bf16")
# 400 column groups of LM head over 256 workgroups: stream-K with unequal (cost-balanced) shares
WIDE_VOCAB = W.ModelShape(2, 256, 8, 2, 128, 512, 51200, 1e-6, 1e6, False, "bf16")


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


def _tol(shape):
    return 1e-4 if shape.dtype == "f32" else 2e-2


def _gpu_model(S, shape, seed=0):
    m = S.Model(shape)
    m.init_random(seed, 0.02)
    return m


def test_weight_generator_bit_identical(S):
    shape = W.TINY
    m = _gpu_model(S, shape)
    torch.cuda.synchronize()
    buf = m.buf.cpu().numpy()
    V, d = shape.vocab, shape.d_model
    emb = buf[: V * d * 4].view(np.float32).reshape(V, d)
    want = oracle.weight_values(0, oracle.tensor_id(oracle.EMBED), 0, V * d, 0.02, False).reshape(V, d)
    assert np.array_equal(emb, want)
    lm = untile(buf, m.matrix_layout(1), V, d, "f32")
    want = oracle.weight_values(0, oracle.tensor_id(oracle.LM_HEAD), 0, V * d, 0.02, False).reshape(V, d)
    assert np.array_equal(lm, want)
    # bf16 generator on a small shape
    m2 = _gpu_model(S, MID_BF16)
    torch.cuda.synchronize()
    b2 = m2.buf.cpu().numpy()
    V, d = MID_BF16.vocab, MID_BF16.d_model
    emb = W.bf16_bits_to_f32(b2[: V * d * 2].view(np.uint16)).reshape(V, d)
    want = oracle.weight_values(0, oracle.tensor_id(oracle.EMBED), 0, V * d, 0.02, True).reshape(V, d)
    assert np.array_equal(emb, want)
    lm = untile(b2, m2.matrix_layout(1), V, d, "bf16")
    want = oracle.weight_values(0, oracle.tensor_id(oracle.LM_HEAD), 0, V * d, 0.02, True).reshape(V, d)
    assert np.array_equal(lm, want)
    # an LM head stored in cost-balanced stream-K order (unequal shares)
    m3 = _gpu_model(S, WIDE_VOCAB)
    torch.cuda.synchronize()
    lay = m3.matrix_layout(1)
    assert lay["c"] > 0 and lay["G"] > lay["n_wg"]
    b3 = m3.buf.cpu().numpy()
    V, d = WIDE_VOCAB.vocab, WIDE_VOCAB.d_model
    lm = untile(b3, lay, V, d, "bf16")
    want = oracle.weight_values(0, oracle.tensor_id(oracle.LM_HEAD), 0, V * d, 0.02, True).reshape(V, d)
    assert np.array_equal(lm, want)


def _run_case(S, shape, prompt_len, gamma, seed, n_rounds=1, max_len=None, ws_rows=64):
    """Prefill + verify rounds on the GPU and the oracle's cached route; returns per-round results."""
    print(f"case {shape} prompt={prompt_len} gamma={gamma} seed={seed} ws_rows={ws_rows}", flush=True)
    m = _gpu_model(S, shape)
    max_len = max_len or prompt_len + n_rounds * (gamma + 1) + 8
    kv = S.KVCache(m, 1, max_len)
    ws = m.workspace(max(ws_rows, gamma + 1))
    om = oracle.Model(shape)
    okv = oracle.KV(om, max_len)
    toks = W.prompt(seed, prompt_len, shape.vocab)
    kv.prefill(0, to_dev_i32(toks), ws)
    okv.prefill(toks)
    ln, pd, err = kv.state()
    assert ln[0] == prompt_len - 1 and pd[0] == toks[-1] and err == 0
    out = []
    for r in range(n_rounds):
        drafts = W.prompt(seed * 100 + r, gamma, shape.vocab)
        logits = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
        am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
        kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), logits, am, ws)
        want = okv.verify(drafts)
        got = logits[0].cpu().numpy()
        ok, rel = row_tol_ok(got, want, _tol(shape))
        print(f"round {r}: max rel err {rel.max():.2e}", flush=True)
        assert ok.all(), rel
        print(f"  bf16/f32 logits vs oracle: max rel {rel.max():.2e}, median {np.median(rel):.2e}", flush=True)
        tol_abs = _tol(shape) * np.abs(want).max(-1)
        near = argmax_near_tie(want, tol_abs)
        amg = am[0].cpu().numpy()
        assert (amg[~near] == want.argmax(-1)[~near]).all()
        assert (amg == got.argmax(-1)).all() or near.any()
        # greedy accept on the GPU logits, commit, mirror on the oracle with the same decision
        L, nxt, _ = S.accept(to_dev_i32(drafts.reshape(1, gamma)), logits, S.GREEDY)
        kv.commit(to_dev_i32([0]), L, nxt)
        Lh, nh = int(L.item()), int(nxt.item())
        ref = oracle.accept(oracle.GREEDY, drafts.reshape(1, gamma), want[None].astype(np.float32))
        if not near[: Lh + 1].any():
            assert Lh == ref["accepted_len"][0] and nh == ref["next_token"][0]
        okv.commit(Lh, nh)  # teacher-forced on the GPU's decision
        out.append((got, want, Lh))
    ln, pd, err = kv.state()
    assert ln[0] == okv.len and pd[0] == okv.pending and err == 0
    return out


def test_tiny_fp32_prefill_verify_commit(S):
    _run_case(S, W.TINY, W.TINY_PROMPT, W.GAMMA_TINY, seed=1, n_rounds=3)


@pytest.mark.parametrize("shape", [MID_BF16, MID_GQA128, WIDE_VOCAB], ids=["hd64-qknorm", "hd128-gqa4", "wide-vocab"])
def test_small_bf16(S, shape):
    _run_case(S, shape, 40, 32, seed=2, n_rounds=2)


def test_gamma_zero_and_long_prefill_chunks(S):
    # prompt longer than one prefill chunk, gamma = 0 decode step
    _run_case(S, MID_GQA128, 300, 0, seed=3, n_rounds=2)


@pytest.mark.parametrize("shape,prompt_len", [(MID_GQA128, 400), (MID_BF16, 101), (W.TINY, 200)],
                         ids=["hd128-chunks-256+143", "hd64-qknorm-chunk-100", "tiny-f32-chunk-199"])
def test_many_row_prefill_chunks(S, shape, prompt_len):
    """Prefill chunks of more than 64 rows (workspace for 256) run the 128-row-tile GEMM: full and ragged
    tiles, one and two tiles per chunk; the cache it writes must give the oracle's verify logits."""
    _run_case(S, shape, prompt_len, 16, seed=4, n_rounds=2, ws_rows=256)


def test_tiny_config_full_pipeline(S):
    """Configuration-1 workload: drafts = oracle greedy tokens w.p. 0.8; all acceptance modes and the
    confidence prefix on GPU logits vs oracle logits."""
    shape = W.TINY
    m = _gpu_model(S, shape)
    om = oracle.Model(shape)
    toks = W.prompt(7, W.TINY_PROMPT, shape.vocab)
    g = W.GAMMA_TINY
    # oracle greedy continuation of the prompt
    cont = []
    seq = list(toks)
    for _ in range(g):
        z = om.forward_full(np.array(seq, np.int32), len(seq) - 1)[0]
        cont.append(int(z.argmax()))
        seq.append(cont[-1])
    drafts = W.corrupt(np.array(cont, np.int32), 8, 0.8, shape.vocab)
    kv = S.KVCache(m, 1, 128)
    ws = m.workspace(64)
    kv.prefill(0, to_dev_i32(toks), ws)
    logits = torch.empty((1, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, g)), logits, None, ws)
    want = om.forward_full(np.concatenate([toks, drafts]).astype(np.int32), len(toks) - 1)
    got = logits[0].cpu().numpy()
    assert row_tol_ok(got, want, 1e-4)[0].all()
    dl = W.drafter_logits(9, drafts.reshape(1, g), g + 1, shape.vocab, scale=3.0, boost=6.0)
    u = W.uniforms(10, (1, g))
    tol = 1e-4 * np.abs(want).max()
    for mode, k, ln in [(0, 1, 1.0), (2, 1, 1.0), (2, 5, 1.0), (3, 1, 0.5), (1, 1, 1.0)]:
        L, nxt, _ = S.accept(to_dev_i32(drafts.reshape(1, g)), logits, mode,
                             q=torch.from_numpy(dl).cuda(), uniforms=torch.from_numpy(u).cuda(), k=k, lenience=ln)
        ref = oracle.accept(mode, drafts.reshape(1, g), want[None].astype(np.float32), q=dl[:, :g], u=u, k=k,
                            lenience=ln)
        dm = ref["dec_margin"][0]
        gap = ref["argmax_gap"][0]
        Lr = ref["accepted_len"][0]
        near = (dm[: min(Lr + 1, g)] < tol).any() or gap[Lr] < tol
        print(f"mode {mode} k={k}: L gpu {int(L.item())} oracle {Lr} near-tie={near}")
        if not near:
            assert int(L.item()) == Lr and int(nxt.item()) == ref["next_token"][0]
    for tau in [0.5, 0.7, 0.9]:
        sk = S.confidence_prefix(torch.from_numpy(dl).cuda(), g, tau)
        ref = oracle.confidence_prefix(dl, g, tau)
        assert int(sk.item()) == ref["skip_len"][0]


def test_batched_ragged_verify(S):
    shape = MID_BF16
    m = _gpu_model(S, shape)
    om = oracle.Model(shape)
    lens = [20, 45, 33]
    gamma = 12
    kv = S.KVCache(m, 4, 128)
    ws = m.workspace(64)
    okvs = []
    for s, n in enumerate(lens):
        t = W.prompt(40 + s, n, shape.vocab)
        kv.prefill(s + 1, to_dev_i32(t), ws)  # slots 1..3
        o = oracle.KV(om, 128)
        o.prefill(t)
        okvs.append(o)
    drafts = W.prompt(50, 3 * gamma, shape.vocab).reshape(3, gamma)
    logits = torch.empty((3, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    am = torch.empty((3, gamma + 1), dtype=torch.int32, device="cuda")
    kv.verify(to_dev_i32([1, 2, 3]), to_dev_i32(drafts), logits, am, ws)
    got = logits.cpu().numpy()
    for s in range(3):
        want = okvs[s].verify(drafts[s])
        ok, rel = row_tol_ok(got[s], want, 2e-2)
        assert ok.all(), (s, rel.max())


def test_capacity_refusal_and_determinism(S):
    shape = MID_GQA128
    m = _gpu_model(S, shape)
    kv = S.KVCache(m, 1, 50)
    ws = m.workspace(64)
    kv.prefill(0, to_dev_i32(W.prompt(3, 30, shape.vocab)), ws)
    d = to_dev_i32(W.prompt(4, 8, shape.vocab).reshape(1, 8))
    l1 = torch.empty((1, 9, shape.vocab), dtype=torch.float32, device="cuda")
    l2 = torch.empty_like(l1)
    kv.verify(to_dev_i32([0]), d, l1, None, ws)
    kv.verify(to_dev_i32([0]), d, l2, None, ws)
    assert torch.equal(l1, l2)  # bit-stable
    # 29 cached + 33 rows > 50: refused on the device, outputs untouched
    d32 = to_dev_i32(W.prompt(5, 32, shape.vocab).reshape(1, 32))
    l3 = torch.full((1, 33, shape.vocab), 7.0, dtype=torch.float32, device="cuda")
    kv.verify(to_dev_i32([0]), d32, l3, None, ws)
    _, _, err = kv.state()
    assert err & 1
    assert (l3 == 7.0).all()


@pytest.mark.parametrize("shape", [MID_BF16, MID_GQA128, W.TINY], ids=["hd64-qknorm", "hd128-gqa4", "tiny-f32"])
def test_block_verify_equals_sequential_decode(S, shape):
    """Row j of a gamma-row verify must equal a decode step at the same position after committing
    drafts 1..j one at a time (same cache contents, same arithmetic up to summation order)."""
    m = _gpu_model(S, shape)
    gamma, P = 12, 30
    kv = S.KVCache(m, 2, 64)
    ws = m.workspace(64)
    toks = to_dev_i32(W.prompt(11, P, shape.vocab))
    kv.prefill(0, toks, ws)
    kv.prefill(1, toks, ws)
    drafts = W.prompt(12, gamma, shape.vocab)
    lb = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), lb, None, ws)
    l1 = torch.empty((1, 1, shape.vocab), dtype=torch.float32, device="cuda")
    one, zero = to_dev_i32([1]), to_dev_i32([0])
    worst = 0.0
    for j in range(gamma + 1):
        kv.verify(one, torch.empty((1, 0), dtype=torch.int32, device="cuda"), l1, None, ws)
        a, b = lb[0, j].cpu().numpy(), l1[0, 0].cpu().numpy()
        rel = np.abs(a - b).max() / np.abs(a).max()
        worst = max(worst, rel)
        if j < gamma:
            kv.commit(one, zero, to_dev_i32([drafts[j]]))
    print(f"{shape.dtype} verify-vs-decode max rel diff {worst:.2e}")
    assert worst == 0.0, worst  # a row's arithmetic does not depend on the other rows of its block
