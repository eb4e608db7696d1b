#!/usr/bin/env python3
"""Benchmark of the verify hot path on one MI355X.

One step = one pass of the whole hot path over one block: the pre-call
confidence prefix on the drafter's logits and the skip decision (two-gate
scheduler, raw signal; the drafter logits are unconfident noise, so every
round is strict and the verifier runs), the gamma = 32 block verification
(causal decoder forward of gamma + 1 rows against the KV cache, fp32 logits),
the acceptance test and the commit.  Default workload: the Qwen3-32B-shaped
target (64 layers, d 5120, 64/8 heads x 128, QK-norm, FFN 25600, V 151936,
bf16, random weights) with a 1024-token prompt, 16 rounds of gamma = 32
(each round appends the accepted tokens).  Drafts follow the target's own
greedy continuation (precomputed, untimed) with 20% of the tokens replaced,
so accepted lengths vary as in speculative decoding.

Prints one JSON line (see the contract in the repository docs).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as W  # noqa: E402

METRIC = "verify-call ms & tokens verified/s at γ=32, Qwen3-32B shape; % HBM peak"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
TAU = 0.7
# skip scheduler at the paper's main raw-confidence setting: (eta_b, eta_c) = (0.90, 0.93), K_min 6, S_max 64
ETA_B, ETA_C, K_MIN, S_MAX = 0.90, 0.93, 6, 64


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gateup_gemm_qwen32b_hbm_traffic.txt")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_14787_amd", "csrc", f)
                  for f in ("decoder.hip", "gemm.h", "sdd_internal.h", "model.h")]


def measured_traffic():
    """HBM bytes per launch of the gate/up kernel at 33 rows from the committed rocprofv3 counter summary,
    or None when the kernel sources have changed since the counters were taken."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        parts = line.split()
        if len(parts) == 3 and parts[0] == "traffic_bytes_per_launch":
            vals[parts[1]] = float(parts[2])
        elif len(parts) == 2 and parts[0] == "kernel_source_sha256":
            vals["sha256"] = parts[1]
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    if vals.get("sha256") != h.hexdigest():
        return None
    return vals.get("gateup_33rows")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=16)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="qwen32b", choices=["qwen32b", "qwen7b", "tiny"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-next-rows", action="store_true", help="skip the timing of the scheduler, residual draw and "
                                                               "survival predictor workloads")
    p.add_argument("--drafts", default="greedy", choices=["greedy", "random"])
    p.add_argument("--all-kernels", action="store_true", help="report every kernel class (extra pass)")
    p.add_argument("--leg", default=None, choices=["batch8", "qwen7b"],
                   help="only run one next_rows leg on the Qwen3-32B-shaped model (profiling) and print its JSON")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain 1 GiB device copy: the reference kernel whose rocprofv3 FETCH_SIZE / "
                        "WRITE_SIZE readings scale the verify kernels' counters to bytes")
    return p.parse_args()


def log(msg):
    print(msg, file=sys.stderr, flush=True)


SHAPES = {"qwen32b": (W.QWEN32B, W.QWEN32B_PROMPT, W.GAMMA),
          "qwen7b": (W.QWEN7B, W.QWEN7B_PROMPT, W.GAMMA),
          "tiny": (W.TINY, W.TINY_PROMPT, W.GAMMA_TINY)}


def layer_params(s: W.ModelShape) -> int:
    d, hd = s.d_model, s.head_dim
    return d * (s.n_q_heads + 2 * s.n_kv_heads) * hd + s.n_q_heads * hd * d + 3 * d * s.d_ff


def cpu_baseline(shape: W.ModelShape, gamma: int, P: int) -> dict:
    """The oracle on this host: gamma-row verify calls through 1 layer + LM head against a cache of the bench's
    prompt length (attention over the cache included), scaled to all layers."""
    import oracle

    s1 = shape.with_layers(1)
    log("cpu baseline: building 1-layer oracle model")
    m = oracle.Model(s1, W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    kv = oracle.KV(m, P + gamma + 8)
    t0 = time.perf_counter()
    kv.prefill(W.prompt(1, P, shape.vocab))
    log(f"cpu baseline: oracle prefill of {P} tokens through 1 layer in {time.perf_counter() - t0:.1f} s (untimed)")
    drafts = W.prompt(102, gamma, shape.vocab)
    n_calls = 6  # about 10 s of CPU work on the 16-thread host share
    t0 = time.perf_counter()
    for _ in range(n_calls):
        kv.verify(drafts)
    t = (time.perf_counter() - t0) / n_calls
    lp, lm = layer_params(shape), shape.vocab * shape.d_model
    scale = (shape.n_layers * lp + lm) / (lp + lm)
    call_s = t * scale
    return {"value": gamma / call_s, "unit": "drafted tokens verified/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": (f"{n_calls} gamma={gamma} verify calls ({gamma + 1} rows) through 1 of {shape.n_layers} layers "
                       f"plus the LM head, {P - 1}-token cache, fp64 oracle: {t:.2f} s per call, scaled by the MAC ratio "
                       f"{scale:.1f} to {call_s:.1f} s per full call")}


def next_rows(sdd, torch, reps: int = 20) -> dict:
    """Timing of the rows beyond the verify call, each on its own workload (the workloads follow the input
    recipes of the parity tests).  Each figure is the average over `reps` back-to-back calls captured in one
    HIP graph (so that host launch overhead does not separate them), replayed between two events."""
    out = {}

    def timed(fn):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(reps):
                fn(i)
        graph.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3  # us per call

    dev = "cuda"
    # residual draw (RATIO_SAMPLE) vs plain RATIO on the acceptance workload [16, 33, 151936] bf16;
    # four input sets (1.3 GB) rotate so that the 256 MB Infinity Cache does not serve the reads
    B, gamma, V = 16, 32, 151936
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    sets = []
    for _ in range(4):
        p = (torch.randn((B, gamma + 1, V), generator=g, device=dev) * 4).to(torch.bfloat16)
        q = (p[:, :gamma].float() + torch.randn((B, gamma, V), generator=g, device=dev) * 0.7).to(torch.bfloat16)
        sets.append((p, q.contiguous()))
    draft = torch.randint(0, V, (B, gamma), generator=g, device=dev, dtype=torch.int32)
    u = torch.rand((B, gamma + 1), generator=g, device=dev)
    ws = sdd.rowstats_workspace(B, gamma, V)
    outs = tuple(torch.empty(B, dtype=torch.int32, device=dev) for _ in range(3))
    row_bytes = V * 2
    modes = (("greedy", sdd.GREEDY, 1, 1.0), ("topk4", sdd.TOPK, 4, 1.0), ("topk16", sdd.TOPK, 16, 1.0),
             ("lenience0.3", sdd.LENIENT, 1, 0.3), ("ratio", sdd.RATIO, 1, 1.0),
             ("ratio_sample", sdd.RATIO_SAMPLE, 1, 1.0))
    for name, mode, k, lam in modes:
        us = timed(lambda i: sdd.accept(draft, sets[i % 4][0], mode, q=sets[i % 4][1], uniforms=u, k=k,
                                        lenience=lam, ws=ws, out=outs))
        L = outs[0].cpu().numpy()
        # bytes: target rows up to the first rejection and the drafter rows they compare (the kernel reads every
        # row: one pass over [B][33][V] target + [B][32][V] drafter), plus the draw's row L of p and q
        nbytes = B * (gamma + 1) * row_bytes + (B * gamma * row_bytes if mode in (sdd.RATIO, sdd.RATIO_SAMPLE) else 0)
        if mode == sdd.RATIO_SAMPLE:
            nbytes += int(sum(2 * row_bytes if l < gamma else row_bytes for l in L))
        out[f"accept_{name}"] = {"workload": f"accept-{B}x{gamma + 1}x{V}-bf16", "us": us, "bytes": nbytes,
                                 "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_hbm": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}
    # confidence prefix over the drafter rows (the same [16, 33, V] bf16 sets: gamma rows per sequence read)
    sk = torch.empty(B, dtype=torch.int32, device=dev)
    us = timed(lambda i: sdd.confidence_prefix(sets[i % 4][0], gamma, TAU, ws=ws, out=sk))
    nbytes = B * gamma * row_bytes
    out["confidence"] = {"workload": f"confidence-{B}x{gamma}x{V}-bf16-tau{TAU}", "us": us, "bytes": nbytes,
                         "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_hbm": nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}
    del sets
    # survival predictor, 32 positions of the paper's shape
    x = W.survival_inputs(seed=1, n=32)
    mlp = sdd.SurvivalMLP(x.mu, x.sigma, x.W1, x.b1, x.W2, x.b2, x.W3, x.b3, x.w4, x.b4, d_hid=x.hidden_bits.shape[1])
    hid = torch.from_numpy(x.hidden_bits.view(np.int16)).to(dev).view(torch.bfloat16)
    sc = torch.from_numpy(x.scalars).to(dev)
    mws = mlp.workspace(32)
    ls = torch.empty(32, dtype=torch.float32, device=dev)
    us = timed(lambda i: mlp(hid, sc, ws=mws, out=ls))
    H, d_in = x.W1.shape
    mbytes = 4 * (H * d_in + 2 * H * H + 4 * H + 2 * d_in) + 32 * (x.hidden_bits.shape[1] * 2 + x.scalars.shape[1] * 4)
    out["survival_mlp"] = {"workload": f"32x{d_in}->{H}->{H}->{H}->1", "us": us, "launches_per_call": 1,
                           "bytes": mbytes, "GB/s": mbytes / (us * 1e-6) / 1e9, "bound": "latency",
                           "mfma_flops": 2 * 32 * (H * d_in + 2 * H * H + H)}
    # skip scheduler, 64 sequences x 32 positions
    si = W.schedule_inputs(seed=3)
    lq = torch.from_numpy(si.log_q).to(dev)
    dr = torch.from_numpy(si.draft).to(dev)
    D = torch.from_numpy(si.D).to(dev)
    so = tuple(torch.empty(64, dtype=torch.int32, device=dev) for _ in range(3))
    us = timed(lambda i: sdd.schedule(lq, D, sdd.SIG_RAW, ETA_B, ETA_C, k_min=K_MIN, s_max=S_MAX, draft=dr, out=so))
    out["schedule"] = {"workload": "64x32 raw signal", "us": us, "bound": "latency"}
    return out


def full_recompute(sdd, torch, model, shape: W.ModelShape, P: int, gamma: int, ws, reps: int = 2) -> dict:
    """The verifier the paper measures: a forward over the whole sequence (P context tokens + gamma drafts) with
    no verifier cache, on the verify workload's model; MFMA-bound (prefill-shaped)."""
    n = P + gamma
    scratch = sdd.KVCache(model, 1, n + 8)
    toks = torch.from_numpy(np.concatenate([W.prompt(1, P, shape.vocab), W.prompt(41, gamma, shape.vocab)])).cuda()
    lg = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
    scratch.verify_full(toks, gamma, lg, None, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        scratch.verify_full(toks, gamma, lg, None, ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    d, L, hd = shape.d_model, shape.n_layers, shape.head_dim
    flops = 2.0 * n * layer_params(shape) * L + 2.0 * (gamma + 1) * shape.vocab * d
    flops += L * shape.n_q_heads * hd * 2.0 * 2.0 * (n * (n + 1) / 2)  # causal QK^T and PV
    del scratch
    return {"workload": f"{n} tokens ({P} context + {gamma} drafts), no verifier cache", "ms_per_call": ms,
            "flops": flops, "TFLOP/s": flops / (ms * 1e-3) / 1e12, "bound": "mfma",
            "frac_mfma_bf16": flops / (ms * 1e-3) / 2.5e15}


def batch8(sdd, torch, model, shape: W.ModelShape, gamma: int, reps: int = 6) -> dict:
    """Batched verification: 8 sequences of the verify workload's model with prompts of U[256, 4096] tokens
    (seeded), a skip mask from the confidence prefix of each sequence's drafter logits at tau = 0.7 with
    K_min = 6, then one verify call over the sequences that are not skipped (B_eff of them, M = 33 B_eff rows),
    greedy acceptance and the commit.  Drafter logits 3 N(0, 1) as stated (no sequence skips: B_eff = 8), and a
    variant boosting the draft token to the row maximum + U[3, 12] so that some sequences skip."""
    dev = "cuda"
    V, d, L = shape.vocab, shape.d_model, shape.n_layers
    lens = W.batch8_lengths(5)
    n = len(lens)
    max_len = int(lens.max()) + (reps + 2) * (gamma + 1) + 8
    kv = sdd.KVCache(model, n, max_len)
    ws = model.workspace(n * (gamma + 1))
    t0 = time.perf_counter()
    for s, ln in enumerate(lens):
        kv.prefill(s, torch.from_numpy(W.prompt(200 + s, int(ln), V)).to(dev), ws)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t0
    log(f"batch8: prefill of {int(lens.sum())} tokens in {prefill_s:.2f} s")
    drafts_np = W.prompt(300, n * gamma, V).reshape(n, gamma)
    drafts = torch.from_numpy(drafts_np).to(dev)
    conf_ws = sdd.rowstats_workspace(n, gamma, V)
    skbuf = torch.empty(n, dtype=torch.int32, device=dev)
    out = {"workload": f"8 sequences, prompts {lens.tolist()} (U[256, 4096]), gamma {gamma}, tau {TAU}, K_min {K_MIN}",
           "prefill_s": prefill_s, "prefill_tokens_per_s": float(lens.sum()) / prefill_s}
    hd, hq, hkv = shape.head_dim, shape.n_q_heads, shape.n_kv_heads
    for variant, boost in (("literal", None), ("boosted", (3.0, 12.0))):
        if boost is None:
            dl = W.drafter_logits(301, drafts_np, gamma + 1, V, scale=3.0, boost=0.0)
        else:
            dl = W.drafter_logits(301, drafts_np, gamma + 1, V, scale=3.0, boost=boost[0], boost_hi=boost[1])
        dlt = torch.from_numpy(W.to_bf16_bits(dl).view(np.int16)).to(dev).view(torch.bfloat16)
        del dl
        sk = sdd.confidence_prefix(dlt, gamma, TAU, ws=conf_ws, out=skbuf)
        active = (sk < K_MIN).nonzero().flatten().to(torch.int32).contiguous()
        B = int(active.numel())
        d_act = drafts[active.long()].contiguous()
        logits = torch.empty((B, gamma + 1, V), dtype=torch.float32, device=dev)
        am = torch.empty((B, gamma + 1), dtype=torch.int32, device=dev)
        acc_ws = sdd.rowstats_workspace(B, gamma, V)
        outs = tuple(torch.empty(B, dtype=torch.int32, device=dev) for _ in range(3))
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]

        def step(i=None):
            sdd.confidence_prefix(dlt, gamma, TAU, ws=conf_ws, out=skbuf)
            if i is not None:
                ev[i][0].record()
            kv.verify(active, d_act, logits, am, ws)
            if i is not None:
                ev[i][1].record()
            Lacc, nxt, _ = sdd.accept(d_act, logits, sdd.GREEDY, ws=acc_ws, out=outs)
            kv.commit(active, Lacc, nxt)

        step()
        torch.cuda.synchronize()
        lens_before = kv.state()[0]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            step(i)
        e1.record()
        torch.cuda.synchronize()
        round_ms = e0.elapsed_time(e1) / reps
        verify_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
        M = B * (gamma + 1)
        act = active.cpu().numpy()
        ctx = float(np.mean(lens_before[act])) + reps / 2.0  # mean cache length over the timed rounds
        weight_bytes = (L * layer_params(shape) + V * d) * 2
        kv_bytes = B * ctx * L * 2 * hkv * hd * 2
        nbytes = weight_bytes + kv_bytes + M * V * 4
        flops = 2.0 * M * (L * layer_params(shape) + V * d) + L * hq * hd * 4.0 * M * ctx
        out[variant] = {"B_eff": B, "rows": M, "skip_len": sk.cpu().numpy().tolist(), "ms_per_round": round_ms,
                        "verify_ms": verify_ms, "verify_calls_per_s": 1e3 / verify_ms,
                        "sequence_blocks_verified_per_s": B * 1e3 / verify_ms,
                        "drafted_tokens_verified_per_s": B * gamma * 1e3 / verify_ms,
                        "bytes": nbytes, "flops": flops,
                        "frac_hbm": nbytes / (verify_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                        "frac_mfma_bf16": flops / (verify_ms * 1e-3) / 2.5e15,
                        "floor_ms_hbm": nbytes / (HBM_PEAK_GBS * 1e9) * 1e3, "floor_ms_mfma": flops / 2.5e15 * 1e3}
        log(f"batch8 {variant}: B_eff {B}, verify {verify_ms:.2f} ms, round {round_ms:.2f} ms")
        del dlt, logits
    del kv, ws
    torch.cuda.empty_cache()
    return out


def qwen7b_leg(sdd, torch, rounds: int = 8, warmup: int = 2) -> dict:
    """The Qwen2.5-7B-shaped verifier (28 layers, d 3584, 28/4 heads x 128, FFN 18944, V 152064, bf16, random
    weights) with a 512-token prompt at gamma = 32: per round the confidence prefix on the drafter's logits, the
    verify call, greedy acceptance and the commit (random drafts: about one token committed per round)."""
    dev = "cuda"
    shape, P, gamma = W.QWEN7B, W.QWEN7B_PROMPT, W.GAMMA
    V, d, L = shape.vocab, shape.d_model, shape.n_layers
    model = sdd.Model(shape)
    model.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    kv = sdd.KVCache(model, 1, P + (rounds + warmup) * (gamma + 1) + 8)
    ws = model.workspace(256)
    kv.prefill(0, torch.from_numpy(W.prompt(1, P, V)).to(dev), ws)
    seq0 = torch.zeros(1, dtype=torch.int32, device=dev)
    drafts = torch.from_numpy(W.prompt(41, (rounds + warmup) * gamma, V).reshape(rounds + warmup, gamma)).to(dev)
    dl = torch.from_numpy(W.to_bf16_bits(W.rng(8).standard_normal((1, gamma + 1, V), dtype=np.float32) *
                                         np.float32(3.0)).view(np.int16)).to(dev).view(torch.bfloat16)
    logits = torch.empty((1, gamma + 1, V), dtype=torch.float32, device=dev)
    am = torch.empty((1, gamma + 1), dtype=torch.int32, device=dev)
    acc_ws = sdd.rowstats_workspace(1, gamma, V)
    conf_ws = sdd.rowstats_workspace(1, gamma, V)
    outs = tuple(torch.empty(1, dtype=torch.int32, device=dev) for _ in range(3))
    sk = torch.empty(1, dtype=torch.int32, device=dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(rounds)]

    def step(r, i=None):
        sdd.confidence_prefix(dl, gamma, TAU, ws=conf_ws, out=sk)
        if i is not None:
            ev[i][0].record()
        kv.verify(seq0, drafts[r:r + 1], logits, am, ws)
        if i is not None:
            ev[i][1].record()
        Lacc, nxt, _ = sdd.accept(drafts[r:r + 1], logits, sdd.GREEDY, ws=acc_ws, out=outs)
        kv.commit(seq0, Lacc, nxt)

    for r in range(warmup):
        step(r)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(rounds):
        step(warmup + i, i)
    e1.record()
    torch.cuda.synchronize()
    round_ms = e0.elapsed_time(e1) / rounds
    verify_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    ctx = float(kv.state()[0][0]) - rounds / 2.0
    nbytes = (L * layer_params(shape) + V * d) * 2 + ctx * L * 2 * shape.n_kv_heads * shape.head_dim * 2 + \
        (gamma + 1) * V * 4
    del kv, ws, model
    torch.cuda.empty_cache()
    return {"workload": f"qwen7b-verify-gamma{gamma}, prompt {P}, batch 1", "ms_per_round": round_ms,
            "verify_ms": verify_ms, "verify_calls_per_s": 1e3 / verify_ms,
            "drafted_tokens_verified_per_s": gamma * 1e3 / verify_ms, "bytes": nbytes,
            "frac_hbm": nbytes / (verify_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "floor_ms_hbm": nbytes / (HBM_PEAK_GBS * 1e9) * 1e3}


def main():
    a = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if a.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (no collectives); "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_14787_amd import sdd
    if not os.path.exists(sdd.LIB_PATH):
        raise SystemExit("libsdd.so is not built: run `python __graft_entry__.py` first")
    torch.cuda.set_device(0)
    assert sdd.device_ok(), "needs a gfx950 GPU"
    if a.copy_calibration:
        n = 1 << 30
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}))
        return

    if a.leg == "qwen7b":
        print(json.dumps({"qwen7b_verify": qwen7b_leg(sdd, torch)}), flush=True)
        return
    shape, P, gamma = SHAPES[a.workload]
    V = shape.vocab
    rounds = a.warmup + a.steps
    log(f"workload {a.workload}: {shape}")
    t0 = time.perf_counter()
    model = sdd.Model(shape)
    model.init_random(W.WEIGHT_SEED, W.WEIGHT_SIGMA)
    torch.cuda.synchronize()
    log(f"weights {model.weight_bytes / 1e9:.2f} GB generated in {time.perf_counter() - t0:.2f} s")
    if a.leg == "batch8":
        print(json.dumps({"batch8": batch8(sdd, torch, model, shape, gamma)}), flush=True)
        return

    # committed tokens per round average about 5 at a 20% replacement rate; past the end of the
    # continuation, drafts repeat its last token and are rejected
    n_cont = rounds * 12 + gamma if a.drafts == "greedy" else 0
    max_len = P + rounds * (gamma + 1) + n_cont + gamma + 8
    kv = sdd.KVCache(model, 2, max_len)
    ws = model.workspace(256)
    prompt = torch.from_numpy(W.prompt(1, P, V)).cuda()
    t0 = time.perf_counter()
    kv.prefill(0, prompt, ws)
    torch.cuda.synchronize()
    log(f"prefill {P} tokens: {time.perf_counter() - t0:.2f} s")

    # greedy continuation of the prompt (untimed): decode steps on slot 1
    one = torch.tensor([1], dtype=torch.int32, device="cuda")
    zero = torch.zeros(1, dtype=torch.int32, device="cuda")
    cont = torch.zeros(max(n_cont, 1), dtype=torch.int32, device="cuda")
    if n_cont:
        kv.prefill(1, prompt, ws)
        lg1 = torch.empty((1, 1, V), dtype=torch.float32, device="cuda")
        am1 = torch.empty((1, 1), dtype=torch.int32, device="cuda")
        nodraft = torch.empty((1, 0), dtype=torch.int32, device="cuda")
        t0 = time.perf_counter()
        for i in range(n_cont):
            kv.verify(one, nodraft, lg1, am1, ws)
            cont[i] = am1[0, 0]
            kv.commit(one, zero, am1[0])
        torch.cuda.synchronize()
        log(f"greedy continuation of {n_cont} tokens: {time.perf_counter() - t0:.2f} s")

    # per-round draft corruption (20% replaced) and drafter logits for the confidence prefix
    g = W.rng(7)
    mask = torch.from_numpy(g.random((rounds, gamma)) < (0.2 if n_cont else 1.0)).cuda()
    repl = torch.from_numpy(g.integers(0, V, size=(rounds, gamma)).astype(np.int32)).cuda()
    dl_bits = W.to_bf16_bits(W.rng(8).standard_normal((rounds, gamma + 1, V), dtype=np.float32) * np.float32(3.0))
    drafter = torch.from_numpy(dl_bits.view(np.int16)).cuda().view(torch.bfloat16).view(rounds, 1, gamma + 1, V)

    len_ptr = kv.device_len_ptr()
    kv_len = torch.as_strided(kv.buf, (4,), (1,), (len_ptr - kv.buf.data_ptr())).view(torch.int32)
    ar = torch.arange(gamma, dtype=torch.int32, device="cuda")
    seq0 = torch.zeros(1, dtype=torch.int32, device="cuda")
    drafts = torch.empty((1, gamma), dtype=torch.int32, device="cuda")
    logits = torch.empty((1, gamma + 1, V), dtype=torch.float32, device="cuda")
    am = torch.empty((1, gamma + 1), dtype=torch.int32, device="cuda")
    acc_ws = sdd.rowstats_workspace(1, gamma, V)
    conf_ws = sdd.rowstats_workspace(1, gamma, V)
    outs = tuple(torch.empty(1, dtype=torch.int32, device="cuda") for _ in range(3))
    skip = torch.empty(1, dtype=torch.int32, device="cuda")
    log_conf = torch.empty((1, gamma), dtype=torch.float32, device="cuda")
    stale = torch.zeros(1, dtype=torch.int32, device="cuda")
    sched_out = tuple(torch.empty(1, dtype=torch.int32, device="cuda") for _ in range(3))
    skips = torch.zeros(rounds, dtype=torch.int32, device="cuda")
    accepted = torch.zeros(rounds, dtype=torch.int32, device="cuda")

    def step(r):
        # drafter stand-in: the next gamma continuation tokens after the cache, 20% replaced
        idx = (kv_len[0] + 1 - P + ar).clamp_(0, max(n_cont - 1, 0)).long()
        torch.where(mask[r], repl[r], cont[idx], out=drafts[0])
        sdd.confidence_prefix(drafter[r], gamma, TAU, ws=conf_ws, out=skip, log_conf=log_conf)
        K, _, _ = sdd.schedule(log_conf, stale, sdd.SIG_RAW, ETA_B, ETA_C, k_min=K_MIN, s_max=S_MAX,
                               draft=drafts, out=sched_out)
        skips[r] = K[0]
        kv.verify(seq0, drafts, logits, am, ws)
        L, nxt, _ = sdd.accept(drafts, logits, sdd.GREEDY, ws=acc_ws, out=outs)
        kv.commit(seq0, L, nxt)
        accepted[r] = L[0]

    for r in range(a.warmup):
        step(r)
    torch.cuda.synchronize()
    dom = sdd.PROF_GEMM_GATEUP
    # every 8th launch of the dominant kernel is bracketed by events (an event pair adds a few
    # microseconds of stream time; sampling keeps the timed steps close to untimed ones)
    sdd.profile_start(dom, 64 * a.steps * 4 + 16, every=8)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for r in range(a.warmup, rounds):
        step(r)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / a.steps
    n_dom, tot_dom, mn_dom, mx_dom = sdd.profile_read(dom)
    sdd.profile_stop()
    acc_l = accepted[a.warmup:].cpu().numpy()
    assert int(skips.sum()) == 0, "a round was scheduled as a skip: the step would not call the verifier"
    final_len = int(kv.state()[0][0])
    log(f"timed {a.steps} steps: {ms:.3f} ms/step (wall {wall * 1e3 / a.steps:.3f}), "
        f"accepted lengths {acc_l.tolist()}, final len {final_len}")

    # algorithmic bytes
    d, dff = shape.d_model, shape.d_ff
    es = 2 if shape.dtype == "bf16" else 4
    R = gamma + 1
    gu_bytes = 2 * dff * d * es + R * d * es + R * dff * es  # weights + input rows + output rows
    dom_ms = tot_dom / max(n_dom, 1)
    achieved = gu_bytes / (dom_ms * 1e-3) / 1e9
    weights_streamed = shape.n_layers * layer_params(shape) * es + V * d * es
    kv_bytes = shape.n_layers * 2 * shape.n_kv_heads * shape.head_dim * es * (final_len - acc_l.mean() / 2)
    call_bytes = weights_streamed + kv_bytes + R * V * 4
    result = {
        "metric": METRIC,
        "value": gamma * 1e3 / ms,
        "unit": "drafted tokens verified/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup,
        "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": f"{a.workload}-verify-gamma{gamma}", "layers": shape.n_layers,
                   "d_model": d, "heads": f"{shape.n_q_heads}/{shape.n_kv_heads}x{shape.head_dim}",
                   "d_ff": dff, "vocab": V, "prompt": P, "gamma": gamma, "batch": 1,
                   "rounds": a.steps, "drafts": a.drafts, "tau": TAU,
                   "scheduler": {"signal": "raw", "eta_b": ETA_B, "eta_c": ETA_C, "k_min": K_MIN, "s_max": S_MAX}},
        "verify_calls_per_s": 1e3 / ms,
        "accepted_tokens_per_s": float((acc_l + 1).sum()) * 1e3 / (ms * a.steps),
        "call_hbm_frac": call_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "call_bytes": call_bytes,
        "roofline": {"bound": "hbm", "kernel": "gemm_ws_kernel gate/up (SwiGLU epilogue)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": measured_traffic() if a.workload == "qwen32b" else None,
                     "traffic_source": os.path.relpath(TRAFFIC_FILE, ROOT), "bytes_per_launch": gu_bytes, "launches": n_dom,
                     "avg_ms": dom_ms, "min_ms": mn_dom, "max_ms": mx_dom},
    }
    if a.all_kernels:
        sdd.profile_start(0x3FF, 4096)
        step(rounds - 1)
        torch.cuda.synchronize()
        names = {"embed": 1, "qkv": 2, "attention": 4, "o_proj": 8, "gate_up": 16, "down": 32, "lm_head": 64,
                 "accept": 128, "confidence": 256, "schedule": 512}
        result["kernels_ms_per_step"] = {k: sdd.profile_read(v)[1] for k, v in names.items()}
        sdd.profile_stop()
    if not a.no_next_rows:
        del drafter
        torch.cuda.empty_cache()
        result["next_rows"] = next_rows(sdd, torch)
        if a.workload != "tiny":
            result["next_rows"]["full_recompute_verify"] = full_recompute(sdd, torch, model, shape, P, gamma, ws)
            result["next_rows"]["batch8"] = batch8(sdd, torch, model, shape, gamma)
        if a.workload == "qwen32b":
            result["next_rows"]["qwen7b_verify"] = qwen7b_leg(sdd, torch)
    if not a.no_cpu_baseline:
        del model, kv, ws
        torch.cuda.empty_cache()
        result["cpu_baseline"] = cpu_baseline(shape, gamma, P)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
