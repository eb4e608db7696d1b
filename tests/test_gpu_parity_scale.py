"""GPU parity against the oracle at the workloads' real depths, cache lengths and batch sizes.

* Full depth: the 64-layer Qwen3-32B shape, the 28-layer 7B shape and the first 16 layers of the 32B
  shape (random N(0, 0.02)-like weights, unit gains) verify a gamma = 32 block after a 16-token prompt;
  the oracle runs the same model with layer streaming (its fp32 copy of the 32B weights would need
  131 GB), exactly and as a BF16 forward, and the GPU's deviation from the exact logits is bounded by
  the 2e-2 logit-scale tolerance or, where BF16 rounding itself exceeds it, by 1.5 times the BF16
  forward's own deviation (the bar at depth, below).  A narrow 64-layer model does the same cheaply.
* Long caches: verify blocks whose attention spans ~600 to 4129 positions (the Qwen3-32B workloads'
  1024-1552-position caches and the batched workload's U[256, 4096] prompts plus a 33-row block), on a
  2-layer GQA model and on a model with the Qwen3-32B attention configuration (64 query / 8 KV heads of
  128, QK-norm, theta 1e6) at a narrow width: the attention kernel depends on the heads and positions,
  not on d_model, so this is its full-size case.
* Non-unit RMSNorm gains (attention, FFN, final, q and k) loaded through sdd_model_load_tensor on both
  the verify rows and prefill chunks of more than 64 rows.
* Batched verification of more than 64 rows: 3 x 33 and 8 x 33 rows of ragged sequences, and the
  batched workload at a narrow width: 8 sequences with prompt lengths drawn from U[256, 4096], a skip
  mask from the confidence prefix at tau = 0.7 with K_min = 6 (drafter logits boosted at the draft token
  so that some sequences skip), and one verify call over the sequences that do not.

Bar: per row max |z_gpu - z_oracle| <= 2e-2 * max |z_oracle|; argmax bit-exact except where the
oracle's top-2 gap is below that tolerance (counted and printed); accepted lengths, lengths and pending
tokens after commit equal.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import argmax_near_tie, load_gains, oracle_gains, row_tol_ok, to_dev_i32

pytestmark = pytest.mark.gpu

TOL = 2e-2
MID_BF16 = W.ModelShape(2, 512, 8, 2, 64, 1024, 2048, 1e-6, 1e6, True, "bf16")
MID_GQA128 = W.ModelShape(2, 256, 8, 2, 128, 512, 1024, 1e-6, 1e6, False, "bf16")
# the Qwen3-32B attention configuration at a narrow width
HEADS32B = W.ModelShape(1, 512, 64, 8, 128, 512, 2048, 1e-6, 1e6, True, "bf16")


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


def _check_rows(got, want, tag):
    """Logits within tolerance; argmax equal outside near-ties.  Returns (max rel err, near-tie count)."""
    ok, rel = row_tol_ok(got, want, TOL)
    near = argmax_near_tie(want, TOL * np.abs(want).max(-1))
    ag, aw = got.argmax(-1), want.argmax(-1)
    print(f"  {tag}: logits max rel {rel.max():.3e} median {np.median(rel):.3e}; "
          f"argmax near-ties excluded {int(near.sum())} of {len(near)}", flush=True)
    assert ok.all(), (tag, rel.max())
    assert (ag[~near] == aw[~near]).all(), tag
    return rel.max(), int(near.sum())


def _gpu_model(S, shape, gains=None):
    m = S.Model(shape)
    m.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    if gains:
        load_gains(m, gains)
    return m


# ---------------------------------------------------------------------------------------------
# full depth


# The bar at depth.  The 2e-2 bound is a BF16-agreement bar, and BF16 rounding of the activations is
# what limits agreement: a BF16 forward of these random-weight models (the oracle in its BF16-operand
# mode: every activation entering a matrix product rounded to BF16, every sum exact) deviates from the
# exact forward by about 2e-2 of the logit scale at 16 layers of the Qwen3-32B shape and 3.4e-2 at 64,
# growing as sqrt(depth) (5.8e-3 at one layer).  Two BF16 forwards that round differently anywhere
# (fp32 against fp64 sums, the online softmax's probabilities) stop rounding alike and drift apart by
# the same amount, so at depth the GPU is bounded by the BF16 forward's own deviation: per row,
# max |z_gpu - z_exact| <= max(2e-2, 1.5 * max |z_bf16 - z_exact| / max |z_exact|) * max |z_exact|.
DEPTH_FACTOR = 1.5


@pytest.mark.parametrize("shape", [W.QWEN32B, W.QWEN7B, W.QWEN32B.with_layers(16), MID_BF16.with_layers(64)],
                         ids=["qwen32b-64layers", "qwen7b-28layers", "qwen32b-16layers", "narrow-64layers"])
def test_full_depth_verify_vs_streamed_oracle(S, shape):
    P, gamma = 16, 32
    print(f"full depth {shape}", flush=True)
    toks = W.prompt(61, P, shape.vocab)
    drafts = W.prompt(62, gamma, shape.vocab)
    m = _gpu_model(S, shape)
    kv = S.KVCache(m, 1, P + gamma + 8)
    ws = m.workspace(64)
    kv.prefill(0, to_dev_i32(toks), ws)
    logits = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), logits, am, ws)
    got = logits[0].cpu().numpy()
    amg = am[0].cpu().numpy()
    del kv, ws, m, logits
    torch.cuda.empty_cache()
    # the oracle: full recomputation over prompt + drafts (the paper's cache-free verifier), layer streamed,
    # exact and as a BF16 forward
    wants = {}
    for bf16 in (False, True):
        t0 = time.time()
        om = oracle.Model(shape, W.WEIGHT_SEED, W.WEIGHT_SIGMA, streamed=True, bf16_operands=bf16)

        def progress(layer):
            if layer % 16 == 15 or layer == shape.n_layers - 1:
                print(f"  oracle ({'bf16 operands' if bf16 else 'exact'}) layer {layer + 1}/{shape.n_layers} "
                      f"({time.time() - t0:.0f} s)", flush=True)

        wants[bf16] = om.forward_full(np.concatenate([toks, drafts]), P - 1, progress=progress)
        del om
    want = wants[False]
    scale = np.abs(want).max(-1)
    err_gpu = np.abs(got - want).max(-1) / scale
    err_bf16 = np.abs(wants[True] - want).max(-1) / scale
    bound = np.maximum(TOL, DEPTH_FACTOR * err_bf16)
    print(f"  {shape.n_layers} layers: GPU vs exact max rel {err_gpu.max():.3e} median {np.median(err_gpu):.3e}; "
          f"BF16 forward vs exact max {err_bf16.max():.3e} median {np.median(err_bf16):.3e}; "
          f"worst ratio {(err_gpu / err_bf16).max():.2f}", flush=True)
    assert (err_gpu <= bound).all(), (err_gpu / bound).max()
    near = argmax_near_tie(want, bound * scale)
    print(f"  argmax near-ties excluded {int(near.sum())} of {gamma + 1}", flush=True)
    assert (amg[~near] == want.argmax(-1)[~near]).all()
    assert (got.argmax(-1)[~near] == want.argmax(-1)[~near]).all()
    # greedy acceptance on both sides agrees outside near-ties
    L, _, _ = S.accept(to_dev_i32(drafts.reshape(1, gamma)), torch.from_numpy(got[None]).cuda(), S.GREEDY)
    ref = oracle.accept(oracle.GREEDY, drafts.reshape(1, gamma), want[None].astype(np.float32), margins=False)
    Lr = int(ref["accepted_len"][0])
    if not near[: Lr + 1].any():
        assert int(L.item()) == Lr


# ---------------------------------------------------------------------------------------------
# long caches


def _long_case(S, shape, P, gamma=32, rounds=1, gains=None, seed=70):
    print(f"long cache {shape} prompt {P} rounds {rounds}", flush=True)
    max_len = P + rounds * (gamma + 1) + 8
    m = _gpu_model(S, shape, gains)
    kv = S.KVCache(m, 1, max_len)
    ws = m.workspace(256)
    om = oracle.Model(shape)
    if gains:
        oracle_gains(om, gains)
    okv = oracle.KV(om, max_len)
    toks = W.prompt(seed, P, shape.vocab)
    kv.prefill(0, to_dev_i32(toks), ws)
    t0 = time.time()
    okv.prefill(toks)
    print(f"  oracle prefill {time.time() - t0:.1f} s", flush=True)
    for r in range(rounds):
        drafts = W.prompt(seed * 10 + r, gamma, shape.vocab)
        logits = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
        am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
        kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), logits, am, ws)
        want = okv.verify(drafts)
        got = logits[0].cpu().numpy()
        _check_rows(got, want, f"round {r}, positions {okv.len}..{okv.len + gamma}")
        near = argmax_near_tie(want, TOL * np.abs(want).max(-1))
        assert (am[0].cpu().numpy()[~near] == want.argmax(-1)[~near]).all()
        # teacher-forced commit: the oracle's greedy decision on both sides
        ref = oracle.accept(oracle.GREEDY, drafts.reshape(1, gamma), want[None].astype(np.float32), margins=False)
        L, nxt = int(ref["accepted_len"][0]), int(ref["next_token"][0])
        kv.commit(to_dev_i32([0]), to_dev_i32([L]), to_dev_i32([nxt]))
        okv.commit(L, nxt)
    ln, pd, err = kv.state()
    assert ln[0] == okv.len and pd[0] == okv.pending and err == 0


@pytest.mark.parametrize("P", [600, 1100, 1552, 4097], ids=["kv633", "kv1133", "kv1585", "kv4129"])
def test_long_cache_gqa(S, P):
    _long_case(S, MID_GQA128, P)


@pytest.mark.parametrize("P", [1100, 4097], ids=["kv1133", "kv4129"])
def test_long_cache_qwen32b_heads(S, P):
    _long_case(S, HEADS32B, P)


def test_qwen32b_heads_rounds_after_1024_prompt(S):
    """Three committed rounds after a 1024-token prompt (the headline workload's cache growth)."""
    _long_case(S, HEADS32B, 1024, rounds=3, seed=71)


# ---------------------------------------------------------------------------------------------
# non-unit gains


@pytest.mark.parametrize("shape", [MID_BF16, MID_GQA128], ids=["hd64-qknorm", "hd128-gqa4"])
def test_nonunit_gains(S, shape):
    """Random gains for every norm; a 150-token prompt runs a 150-row prefill chunk (many-row GEMMs)."""
    _long_case(S, shape, 150, rounds=2, gains=W.norm_gains(80, shape), seed=72)


def test_nonunit_gains_qwen32b_heads(S):
    _long_case(S, HEADS32B, 300, rounds=1, gains=W.norm_gains(81, HEADS32B), seed=73)


# ---------------------------------------------------------------------------------------------
# batched verification of more than 64 rows


def _batched(S, shape, lens, gamma, seed, skip_tau=None, k_min=6, max_len=None):
    n = len(lens)
    max_len = max_len or int(max(lens)) + gamma + 8
    print(f"batched {shape} lens {list(map(int, lens))} gamma {gamma}", flush=True)
    m = _gpu_model(S, shape)
    kv = S.KVCache(m, n, max_len)
    ws = m.workspace(max(256, n * (gamma + 1)))
    om = oracle.Model(shape)
    okvs = []
    t0 = time.time()
    for s, ln in enumerate(lens):
        t = W.prompt(seed + s, int(ln), shape.vocab)
        kv.prefill(s, to_dev_i32(t), ws)
        o = oracle.KV(om, max_len)
        o.prefill(t)
        okvs.append(o)
    print(f"  oracle prefills {time.time() - t0:.1f} s", flush=True)
    drafts = W.prompt(seed + 100, n * gamma, shape.vocab).reshape(n, gamma)
    active = np.arange(n)
    if skip_tau is not None:
        # skip mask: confidence prefix of the drafter rows at tau; a sequence skips when skip_len >= K_min
        dl = W.drafter_logits(seed + 200, drafts, gamma + 1, shape.vocab, scale=3.0, boost=1.0, boost_hi=9.0)
        sk = S.confidence_prefix(torch.from_numpy(dl).cuda(), gamma, skip_tau).cpu().numpy()
        ref = oracle.confidence_prefix(dl, gamma, skip_tau)["skip_len"]
        assert np.array_equal(sk, ref)
        active = np.nonzero(sk < k_min)[0]
        print(f"  skip_len {sk.tolist()}: {n - len(active)} skipped, B_eff {len(active)}", flush=True)
        assert 0 < len(active) < n, "the workload should both skip and verify"
    ids = to_dev_i32(active)
    logits = torch.empty((len(active), gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    am = torch.empty((len(active), gamma + 1), dtype=torch.int32, device="cuda")
    kv.verify(ids, to_dev_i32(drafts[active]), logits, am, ws)
    got = logits.cpu().numpy()
    amg = am.cpu().numpy()
    Ls, nxts, nears = [], [], []
    for i, s in enumerate(active):
        want = okvs[s].verify(drafts[s])
        _check_rows(got[i], want, f"seq {s} (len {okvs[s].len})")
        near = argmax_near_tie(want, TOL * np.abs(want).max(-1))
        assert (amg[i][~near] == want.argmax(-1)[~near]).all()
        ref = oracle.accept(oracle.GREEDY, drafts[s].reshape(1, gamma), want[None].astype(np.float32), margins=False)
        Ls.append(int(ref["accepted_len"][0]))
        nxts.append(int(ref["next_token"][0]))
        nears.append(near)
    # acceptance on the GPU logits agrees with the oracle's outside near-ties
    Lg, _, _ = S.accept(to_dev_i32(drafts[active]), logits, S.GREEDY)
    Lg = Lg.cpu().numpy()
    for i in range(len(active)):
        if not nears[i][: Ls[i] + 1].any():
            assert Lg[i] == Ls[i], i
    # teacher-forced commit of the oracle's decisions
    kv.commit(ids, to_dev_i32(Ls), to_dev_i32(nxts))
    for i, s in enumerate(active):
        okvs[s].commit(Ls[i], nxts[i])
    ln, pd, err = kv.state()
    assert err == 0
    for s in range(n):
        assert ln[s] == okvs[s].len and pd[s] == okvs[s].pending, s  # skipped sequences unchanged
    return Lg, np.array(Ls)


@pytest.mark.parametrize("n", [3, 8], ids=["3x33-rows", "8x33-rows"])
def test_batched_verify_over_64_rows(S, n):
    lens = W.rng(90 + n).integers(20, 100, size=n)
    _batched(S, MID_BF16, lens, 32, seed=91 + n)


def test_batched_verify_full_width(S):
    """Three sequences (99 rows) through one full-width Qwen3-32B layer and the real LM head: gate/up and the
    LM head run the column-group-pair kernel at their real sizes (400 groups, one pair per workgroup; 1187
    groups, an odd count, so the last pair holds one group, stream-K over the workgroup budget), qkv, o_proj
    and down the many-row kernel on their stored split plans."""
    lens = W.rng(97).integers(16, 48, size=3)
    _batched(S, W.QWEN32B.with_layers(1), lens, 32, seed=98)


def test_batched_ragged_long_with_skip_mask(S):
    """The batched workload at a narrow width: 8 prompts of U[256, 4096] tokens, skip mask at tau 0.7 and
    K_min 6, one verify call over the remaining sequences (variable effective batch)."""
    lens = W.batch8_lengths(5)
    _batched(S, MID_GQA128, lens, 32, seed=95, skip_tau=0.7)
