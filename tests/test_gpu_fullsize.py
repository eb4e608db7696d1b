"""Parity at the full Qwen3-32B / Qwen2.5-7B widths, in the launch configuration the benchmark times.

* 1-layer models of the exact widths (d 5120 / 3584, 64/8 and 28/4 heads x 128, FFN 25600 / 18944,
  V 151936 / 152064) against the oracle: logits within 2e-2 of the logit scale, argmax bit-exact
  outside near-ties.  Every kernel of a layer runs at its real shape; depth does not change them.
* 256- and 149-row prefill chunks at the 32B width (the many-row GEMM launches) against the oracle.
* The full 64-layer 32B model: block verification equals sequential decode steps bit for bit (a
  property that holds at any size: a row's arithmetic does not depend on how rows are batched), and
  repeated calls are bit-identical.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import argmax_near_tie, row_tol_ok, to_dev_i32

pytestmark = pytest.mark.gpu


_ORACLE_MODELS = {}


def _oracle_model(shape):
    """One oracle model per shape for the whole module (building one at full width takes ~15 s)."""
    if shape not in _ORACLE_MODELS:
        _ORACLE_MODELS[shape] = oracle.Model(shape, W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    return _ORACLE_MODELS[shape]


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


@pytest.mark.parametrize("shape", [W.QWEN32B.with_layers(1), W.QWEN7B.with_layers(1)], ids=["qwen32b-1layer", "qwen7b-1layer"])
def test_one_layer_full_width_vs_oracle(S, shape):
    print(f"full-width 1-layer parity {shape}", flush=True)
    m = S.Model(shape)
    m.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    P, gamma = 24, 32
    kv = S.KVCache(m, 1, P + 2 * (gamma + 1) + 8)
    ws = m.workspace(64)
    toks = W.prompt(31, P, shape.vocab)
    kv.prefill(0, to_dev_i32(toks), ws)
    om = _oracle_model(shape)
    okv = oracle.KV(om, P + 2 * (gamma + 1) + 8)
    okv.prefill(toks)
    for r in range(2):
        drafts = W.prompt(32 + r, gamma, shape.vocab)
        logits = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
        am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
        kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), logits, am, ws)
        want = okv.verify(drafts)
        got = logits[0].cpu().numpy()
        ok, rel = row_tol_ok(got, want, 2e-2)
        print(f"  round {r}: logits max rel {rel.max():.2e} median {np.median(rel):.2e}", flush=True)
        assert ok.all()
        near = argmax_near_tie(want, 2e-2 * np.abs(want).max(-1))
        amg = am[0].cpu().numpy()
        print(f"  argmax near-ties excluded: {near.sum()} of {gamma + 1}")
        assert (amg[~near] == want.argmax(-1)[~near]).all()
        # commit the oracle's greedy decision on both sides (teacher forcing)
        ref = oracle.accept(oracle.GREEDY, drafts.reshape(1, gamma), want[None].astype(np.float32), margins=False)
        L, nxt = int(ref["accepted_len"][0]), int(ref["next_token"][0])
        kv.commit(to_dev_i32([0]), to_dev_i32([L]), to_dev_i32([nxt]))
        okv.commit(L, nxt)


@pytest.mark.parametrize("P", [300, 150], ids=["chunks-256+43", "chunk-149"])
def test_one_layer_full_width_long_prefill_vs_oracle(S, P):
    """Prefill chunks of 256 and 149 rows at the full 32B width (workspace for 256-row chunks): every GEMM
    runs all its 64-row tiles in one launch (4 full tiles; 2 full tiles and a ragged one); the verify logits
    on the cache they wrote must match the oracle's."""
    shape = W.QWEN32B.with_layers(1)
    print(f"full-width 1-layer long prefill P={P}", flush=True)
    m = S.Model(shape)
    m.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    gamma = 16
    kv = S.KVCache(m, 1, P + gamma + 8)
    ws = m.workspace(256)
    toks = W.prompt(35, P, shape.vocab)
    kv.prefill(0, to_dev_i32(toks), ws)
    om = _oracle_model(shape)
    okv = oracle.KV(om, P + gamma + 8)
    okv.prefill(toks)
    drafts = W.prompt(36, gamma, shape.vocab)
    logits = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), logits, am, ws)
    want = okv.verify(drafts)
    got = logits[0].cpu().numpy()
    ok, rel = row_tol_ok(got, want, 2e-2)
    print(f"  logits max rel {rel.max():.2e} median {np.median(rel):.2e}", flush=True)
    assert ok.all()
    near = argmax_near_tie(want, 2e-2 * np.abs(want).max(-1))
    amg = am[0].cpu().numpy()
    assert (amg[~near] == want.argmax(-1)[~near]).all()


def test_qwen32b_verify_equals_decode_and_is_bit_stable(S):
    shape = W.QWEN32B
    m = S.Model(shape)
    m.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    P, gamma = 1024, 32
    kv = S.KVCache(m, 2, P + 2 * (gamma + 1) + 8)
    ws = m.workspace(256)
    toks = to_dev_i32(W.prompt(1, P, shape.vocab))
    kv.prefill(0, toks, ws)
    kv.prefill(1, toks, ws)
    drafts = W.prompt(41, gamma, shape.vocab)
    lb = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    lb2 = torch.empty_like(lb)
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), lb, None, ws)
    kv.verify(to_dev_i32([0]), to_dev_i32(drafts.reshape(1, gamma)), lb2, None, ws)
    assert torch.equal(lb, lb2)
    l1 = torch.empty((1, 1, shape.vocab), dtype=torch.float32, device="cuda")
    one, zero = to_dev_i32([1]), to_dev_i32([0])
    nodraft = torch.empty((1, 0), dtype=torch.int32, device="cuda")
    worst, flips = 0.0, 0
    for j in range(gamma + 1):
        kv.verify(one, nodraft, l1, None, ws)
        a, b = lb[0, j].cpu().numpy(), l1[0, 0].cpu().numpy()
        rel = np.abs(a - b).max() / np.abs(a).max()
        worst = max(worst, rel)
        flips += int(a.argmax() != b.argmax())
        if j < gamma:
            kv.commit(one, zero, to_dev_i32([drafts[j]]))
    print(f"qwen32b verify-vs-decode max rel diff {worst:.2e}, argmax flips {flips}", flush=True)
    assert worst == 0.0 and flips == 0  # rows do not depend on how they are batched
