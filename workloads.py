"""Seeded synthetic workloads shared by the tests and the benchmark.

Holds the model shapes of the measured configurations and numpy generators
for their inputs (prompts, drafts, logits, uniforms).  Contains none of the
method's arithmetic: both the GPU path and the CPU oracle receive what these
functions return.  (Model weights are produced by each side's own
implementation of one published counter-based generator, SplitMix64.)

Workload recipes (the paper's benchmark, HumanEval with DiffuCoder-7B and
Qwen3-32B at gamma = 32, Sec. 5.1, is stood in for by uniform-token prompts of
code-prompt length and random-weight decoders of the named shapes):
  tiny     2-layer fp32 decoder, d 256, 4/2 heads x 64, FFN 688, V 4096, 64-token prompt, gamma 8
  accept   logits [16, 33, 151936] bf16 ~ 4 N(0,1); target +8 at the draft token w.p. 0.85
  qwen7b   28 layers, d 3584, 28/4 heads x 128, FFN 18944, V 152064, 512-token prompt
  qwen32b  64 layers, d 5120, 64/8 heads x 128, QK-norm, FFN 25600, V 151936, 1024-token prompt
  batch8   qwen32b shape, 8 sequences with KV lengths U[256, 4096]
  schedule log scores [64, 32] from log(1 - e), e ~ Exp(lam), lam log-uniform per sequence
  survival 32 positions x (3584 bf16 hidden + 19 scalar features), MLP 3603 -> 256 -> 256 -> 256 -> 1
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 1e6
    qk_norm: bool = False
    dtype: str = "bf16"  # "f32" or "bf16"

    def with_layers(self, n: int) -> "ModelShape":
        return replace(self, n_layers=n)

    def weight_count(self) -> int:
        d, hd = self.d_model, self.head_dim
        per_layer = (d * (self.n_q_heads + 2 * self.n_kv_heads) * hd + self.n_q_heads * hd * d
                     + 3 * d * self.d_ff)
        return self.n_layers * per_layer + 2 * self.vocab * d


TINY = ModelShape(2, 256, 4, 2, 64, 688, 4096, 1e-6, 1e4, False, "f32")
QWEN7B = ModelShape(28, 3584, 28, 4, 128, 18944, 152064, 1e-6, 1e6, False, "bf16")
QWEN32B = ModelShape(64, 5120, 64, 8, 128, 25600, 151936, 1e-6, 1e6, True, "bf16")
WEIGHT_SEED = 0
WEIGHT_SIGMA = 0.02

TINY_PROMPT, QWEN7B_PROMPT, QWEN32B_PROMPT = 64, 512, 1024
GAMMA_TINY, GAMMA = 8, 32


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def prompt(seed: int, n: int, vocab: int) -> np.ndarray:
    """Uniform tokens in [0, vocab)."""
    return rng(seed).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


def corrupt(tokens: np.ndarray, seed: int, keep: float, vocab: int) -> np.ndarray:
    """Each token kept with probability `keep`, else replaced by a uniform token."""
    g = rng(seed)
    t = np.asarray(tokens, np.int32).copy()
    repl = g.random(t.shape) >= keep
    t[repl] = g.integers(0, vocab, size=int(repl.sum()), dtype=np.int64)
    return t


def uniforms(seed: int, shape) -> np.ndarray:
    """fp32 uniforms in [0, 1) on a 2^-24 grid (exact in fp32)."""
    return (rng(seed).integers(0, 1 << 24, size=shape, dtype=np.int64) * 2.0 ** -24).astype(np.float32)


def drafter_logits(seed: int, draft: np.ndarray, rows: int, vocab: int, scale: float = 3.0,
                   boost: float = 6.0, boost_hi: float | None = None) -> np.ndarray:
    """Drafter logits [B, rows, V] = scale * N(0,1); +boost at the draft token of rows j < gamma.

    With boost_hi set, the boost is drawn U[boost, boost_hi] relative to the row maximum instead
    (variant whose confidences span (0, 1))."""
    draft = np.asarray(draft, np.int32)
    B, gamma = draft.shape
    g = rng(seed)
    z = (g.standard_normal((B, rows, vocab), dtype=np.float32) * np.float32(scale))
    bi, ji = np.meshgrid(np.arange(B), np.arange(gamma), indexing="ij")
    if boost_hi is None:
        z[bi, ji, draft] += np.float32(boost)
    else:
        extra = g.uniform(boost, boost_hi, size=(B, gamma)).astype(np.float32)
        z[bi, ji, draft] = z[:, :gamma, :].max(axis=2) + extra
    return z


@dataclass
class AcceptInputs:
    draft: np.ndarray         # int32 [B, gamma]
    target_bits: np.ndarray   # uint16 bf16 [B, gamma+1, V]
    drafter_bits: np.ndarray  # uint16 bf16 [B, gamma+1, V]
    u: np.ndarray             # fp32 [B, gamma]

    @property
    def target(self) -> np.ndarray:
        return bf16_bits_to_f32(self.target_bits)

    @property
    def drafter(self) -> np.ndarray:
        return bf16_bits_to_f32(self.drafter_bits)


def accept_inputs(seed: int, B: int = 16, gamma: int = 32, vocab: int = 151936,
                  scale: float = 4.0, boost: float = 8.0, p_boost: float = 0.85,
                  variant: str = "literal") -> AcceptInputs:
    """Acceptance/confidence workload: bf16 logits [B, gamma+1, V] ~ scale * N(0,1).

    literal: target +boost at draft token j w.p. p_boost (as the workload states).
    rowmax:  target logit at draft token set to rowmax + boost w.p. p_boost, so that accepted
             prefixes have geometric lengths (variant reported separately)."""
    g = rng(seed)
    draft = g.integers(0, vocab, size=(B, gamma), dtype=np.int64).astype(np.int32)
    t = g.standard_normal((B, gamma + 1, vocab), dtype=np.float32) * np.float32(scale)
    hit = g.random((B, gamma)) < p_boost
    bi, ji = np.nonzero(hit)
    if variant == "literal":
        t[bi, ji, draft[bi, ji]] += np.float32(boost)
    elif variant == "rowmax":
        t[bi, ji, draft[bi, ji]] = t[bi, ji, :].max(axis=1) + np.float32(boost)
    else:
        raise ValueError(variant)
    d = g.standard_normal((B, gamma + 1, vocab), dtype=np.float32) * np.float32(scale)
    u = uniforms(seed + 1, (B, gamma))
    return AcceptInputs(draft, to_bf16_bits(t), to_bf16_bits(d), u)


def norm_gains(seed: int, shape: ModelShape, spread: float = 0.25) -> dict:
    """Non-unit RMSNorm gains 1 + spread * N(0,1) (fp32) for every norm of the shape, keyed
    ("final", 0), ("attn", layer), ("ffn", layer) and, with QK-norm, ("q", layer), ("k", layer)."""
    g = rng(seed)
    gn = lambda n: (1.0 + spread * g.standard_normal(n)).astype(np.float32)
    out = {("final", 0): gn(shape.d_model)}
    for l in range(shape.n_layers):
        out[("attn", l)] = gn(shape.d_model)
        out[("ffn", l)] = gn(shape.d_model)
        if shape.qk_norm:
            out[("q", l)] = gn(shape.head_dim)
            out[("k", l)] = gn(shape.head_dim)
    return out


def batch8_lengths(seed: int, n: int = 8, lo: int = 256, hi: int = 4096) -> np.ndarray:
    """Ragged prompt lengths U[lo, hi]."""
    return rng(seed).integers(lo, hi + 1, size=n, dtype=np.int64).astype(np.int32)


@dataclass
class ScheduleInputs:
    log_q: np.ndarray      # fp32 [B, gamma] log position scores
    draft: np.ndarray      # int32 [B, gamma]
    D: np.ndarray          # int32 [B] unverified tokens since the last verifier call
    block_len: np.ndarray  # int32 [B] (gamma, or shorter for a truncated final block)


def schedule_inputs(seed: int, B: int = 64, gamma: int = 32, vocab: int = 151936,
                    p_short: float = 0.1, p_repeat: float = 0.2, d_max: int = 80) -> ScheduleInputs:
    """Skip-scheduler workload: per-position failure probability e ~ Exp(mean lam) clipped to 0.999,
    with lam log-uniform in [1e-3, 0.3] per sequence (confident and unsure sequences in one batch),
    log score = log(1 - e) in fp32; drafts uniform tokens with a run of one repeated token inserted
    w.p. p_repeat; D uniform in [0, d_max]; a shortened block (length U[1, gamma-1]) w.p. p_short."""
    g = rng(seed)
    lam = np.exp(g.uniform(np.log(1e-3), np.log(0.3), size=(B, 1)))
    e = np.minimum(g.exponential(1.0, size=(B, gamma)) * lam, 0.999)
    log_q = np.log1p(-e).astype(np.float32)
    draft = g.integers(0, vocab, size=(B, gamma), dtype=np.int64).astype(np.int32)
    if gamma >= 2:
        for b in np.nonzero(g.random(B) < p_repeat)[0]:
            n = int(g.integers(2, min(gamma, 6) + 1))
            s = int(g.integers(0, gamma - n + 1))
            draft[b, s:s + n] = draft[b, s]
    D = g.integers(0, d_max + 1, size=B, dtype=np.int64).astype(np.int32)
    block_len = np.full(B, gamma, np.int32)
    if gamma >= 2:
        short = g.random(B) < p_short
        block_len[short] = g.integers(1, gamma, size=int(short.sum()), dtype=np.int64)
    return ScheduleInputs(log_q, draft, D, block_len)


@dataclass
class SurvivalInputs:
    hidden_bits: np.ndarray  # uint16 bf16 [n, d_hid]: the drafter's LM-head input per draft position
    scalars: np.ndarray      # fp32 [n, n_sc]
    mu: np.ndarray           # fp32 [d_in] normalization mean
    sigma: np.ndarray        # fp32 [d_in] normalization scale (> 0)
    W1: np.ndarray           # fp32 [H, d_in]
    b1: np.ndarray
    W2: np.ndarray           # fp32 [H, H]
    b2: np.ndarray
    W3: np.ndarray           # fp32 [H, H]
    b3: np.ndarray
    w4: np.ndarray           # fp32 [1, H]
    b4: float


def survival_inputs(seed: int, n: int = 32, d_hid: int = 3584, n_sc: int = 19, H: int = 256) -> SurvivalInputs:
    """Survival-predictor workload (Appendix "Predictor Details" shape: 3584 + 19 -> 256 -> 256 -> 256 -> 1).

    Hidden states bf16 N(0, 1.5^2); the 19 scalars in the ranges of the listed features (reveal step,
    rank, parallelism, late flag, top-1 probability and its log, entropy and its negative, margin, top-5
    mass, step-0 values and changes, block position, generated length, segment position, two dataset
    flags); normalization statistics from a separate draw of the same distribution (dataset flags: mean
    the constant, scale 1); weights U(-1/sqrt(fan_in), 1/sqrt(fan_in)) as a freshly initialized Linear."""
    g = rng(seed)
    hidden = to_bf16_bits((g.standard_normal((n, d_hid)) * 1.5).astype(np.float32))

    def feats(m):
        p1 = g.uniform(0.05, 1.0, m)
        ent = g.uniform(0.0, 3.0, m)
        p1_0 = g.uniform(0.05, 1.0, m)
        ent0 = g.uniform(0.0, 3.0, m)
        cols = [g.integers(0, 2, m), g.uniform(0, 1, m), g.integers(1, 33, m), g.integers(0, 2, m), p1, np.log(p1),
                ent, -ent, g.uniform(0, 1, m) * p1, np.minimum(1.0, p1 + g.uniform(0, 0.5, m)), p1_0, -ent0,
                p1 - p1_0, ent0 - ent, g.integers(0, 32, m), g.integers(0, 513, m), g.uniform(0, 1, m),
                np.ones(m), np.zeros(m)]
        return np.stack(cols, 1)[:, :n_sc].astype(np.float32)

    scalars = feats(n)
    ref = feats(4096)
    mu = np.concatenate([np.zeros(d_hid), ref.mean(0)]).astype(np.float32)
    sd = ref.std(0)
    sigma = np.concatenate([np.full(d_hid, 1.5), np.where(sd > 1e-6, sd, 1.0)]).astype(np.float32)
    d_in = d_hid + n_sc

    def lin(o, i):
        bound = 1.0 / np.sqrt(i)
        return (g.uniform(-bound, bound, (o, i)).astype(np.float32), g.uniform(-bound, bound, o).astype(np.float32))

    W1, b1 = lin(H, d_in)
    W2, b2 = lin(H, H)
    W3, b3 = lin(H, H)
    w4, b4 = lin(1, H)
    return SurvivalInputs(hidden, scalars, mu, sigma, W1, b1, W2, b2, W3, b3, w4, float(b4[0]))
