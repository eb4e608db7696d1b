"""CPU oracle for verifier-skipped speculative diffusion decoding.

TEST INFRASTRUCTURE ONLY.  Only tests/, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The GPU product
path (``paper_2608_14787_amd``) never imports it and shares no code with it.

A ctypes wrapper over ``libsdd_oracle.so`` (plain C, fp64; see sdd_oracle.c for
the passages each function follows).
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

GREEDY, RATIO, TOPK, LENIENT, RATIO_SAMPLE = 0, 1, 2, 3, 4
(EMBED, LM_HEAD, FINAL_NORM, WQ, WK, WV, WO, WGATE, WUP, WDOWN,
 ATTN_NORM, FFN_NORM, Q_NORM, K_NORM) = range(14)

_lib = None


class _Cfg(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("d_model", C.c_int), ("n_q_heads", C.c_int),
                ("n_kv_heads", C.c_int), ("head_dim", C.c_int), ("d_ff", C.c_int),
                ("vocab", C.c_int), ("rms_eps", C.c_double), ("rope_theta", C.c_double),
                ("qk_norm", C.c_int), ("bf16_weights", C.c_int), ("bf16_operands", C.c_int)]


def lib():
    """Loads the oracle library, compiling it first if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        P = C.c_void_p
        L.orc_splitmix64.restype = C.c_uint64
        L.orc_splitmix64.argtypes = [C.c_uint64]
        L.orc_weight_values.argtypes = [C.c_uint64, C.c_int, C.c_uint64, C.c_uint64, C.c_double, C.c_int, P]
        L.orc_tensor_id.argtypes = [C.c_int, C.c_int]
        L.orc_model_create.restype = P
        L.orc_model_create.argtypes = [C.POINTER(_Cfg), C.c_uint64, C.c_double]
        L.orc_model_free.argtypes = [P]
        L.orc_model_create_streamed.restype = P
        L.orc_model_create_streamed.argtypes = [C.POINTER(_Cfg), C.c_uint64, C.c_double]
        L.orc_model_set_tensor.argtypes = [P, C.c_int, C.c_int, P]
        L.orc_forward_full.argtypes = [P, P, C.c_int, C.c_int, P]
        L.orc_embed.argtypes = [P, P, C.c_int, P]
        L.orc_layer_full.argtypes = [P, C.c_int, C.c_int, P]
        L.orc_final_logits.argtypes = [P, P, C.c_int, P]
        L.orc_forward_full_hidden.argtypes = [P, P, C.c_int, C.c_int, P]
        L.orc_kv_create.restype = P
        L.orc_kv_create.argtypes = [P, C.c_int]
        L.orc_kv_free.argtypes = [P]
        L.orc_kv_len.argtypes = [P]
        L.orc_kv_pending.argtypes = [P]
        L.orc_kv_read.argtypes = [P, C.c_int, C.c_int, P, P]
        L.orc_kv_prefill.argtypes = [P, P, C.c_int]
        L.orc_verify.argtypes = [P, P, C.c_int, P]
        L.orc_commit.argtypes = [P, C.c_int, C.c_int]
        L.orc_accept.argtypes = [C.c_int, P, P, P, C.c_size_t, P, C.c_int, C.c_int, C.c_int,
                                 C.c_int, C.c_double, P, P, P, P, P, P]
        L.orc_confidence_prefix.argtypes = [P, C.c_size_t, C.c_int, C.c_int, C.c_int, C.c_double,
                                            P, P, P, P]
        L.orc_schedule.argtypes = [P, P, C.c_int, C.c_int, C.c_int, C.c_double, C.c_double, C.c_int, C.c_int,
                                   P, P, C.c_int, C.c_int, P, P, P, P]
        L.orc_survival_mlp.argtypes = [P, P, C.c_int, C.c_int, C.c_int, C.c_int, P, P, P, P, P, P, P, P, P,
                                       C.c_float, P, P]
        L.orc_audit_accumulate.argtypes = [P, P, C.c_int, P]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def num_threads() -> int:
    return lib().orc_num_threads()


def splitmix64(x: int) -> int:
    return lib().orc_splitmix64(x)


def tensor_id(kind: int, layer: int = 0) -> int:
    return lib().orc_tensor_id(kind, layer)


def weight_values(seed: int, tid: int, start: int, count: int, sigma: float, bf16: bool) -> np.ndarray:
    out = np.empty(count, np.float32)
    lib().orc_weight_values(seed, tid, start, count, sigma, int(bf16), _p(out))
    return out


def tensor_shape(shape, kind: int):
    d, hq, hk = shape.d_model, shape.n_q_heads * shape.head_dim, shape.n_kv_heads * shape.head_dim
    return {EMBED: (shape.vocab, d), LM_HEAD: (shape.vocab, d), FINAL_NORM: (1, d),
            ATTN_NORM: (1, d), FFN_NORM: (1, d), Q_NORM: (1, shape.head_dim),
            K_NORM: (1, shape.head_dim), WQ: (hq, d), WK: (hk, d), WV: (hk, d), WO: (d, hq),
            WGATE: (shape.d_ff, d), WUP: (shape.d_ff, d), WDOWN: (d, shape.d_ff)}[kind]


class Model:
    """The target decoder with synthetic weights (seed, sigma) held in host memory.

    streamed=True holds only the embedding, LM head and final norm and generates each layer's
    weights when a forward reaches it (same values; for shapes whose fp32 copy exceeds host memory).
    bf16_operands=True: every activation entering a matrix product is rounded to BF16 (the verifier
    as a BF16 model); otherwise everything is exact fp64."""

    def __init__(self, shape, seed: int = 0, sigma: float = 0.02, streamed: bool = False,
                 bf16_operands: bool = False):
        self.shape = shape
        self.streamed = streamed
        c = _Cfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                 shape.head_dim, shape.d_ff, shape.vocab, shape.rms_eps, shape.rope_theta,
                 int(shape.qk_norm), int(shape.dtype == "bf16"), int(bf16_operands))
        create = lib().orc_model_create_streamed if streamed else lib().orc_model_create
        self._h = create(C.byref(c), seed, sigma)
        if not self._h:
            raise MemoryError("oracle model creation failed")

    def __del__(self):
        if getattr(self, "_h", None):
            lib().orc_model_free(self._h)
            self._h = None

    def set_tensor(self, kind: int, layer: int, values: np.ndarray):
        v = np.ascontiguousarray(values, np.float32)
        assert v.size == int(np.prod(tensor_shape(self.shape, kind)))
        if lib().orc_model_set_tensor(self._h, kind, layer, _p(v)) != 0:
            raise ValueError("bad tensor")

    def forward_full(self, tokens, row0: int = 0, progress=None) -> np.ndarray:
        """Logits of rows [row0, n) from full recomputation (no cache).

        progress: optional callable(layer) called after each layer (the forward then runs layer by layer
        through orc_embed / orc_layer_full / orc_final_logits: the same computation)."""
        t = np.ascontiguousarray(tokens, np.int32)
        out = np.empty((len(t) - row0, self.shape.vocab), np.float64)
        if progress is None:
            if lib().orc_forward_full(self._h, _p(t), len(t), row0, _p(out)) != 0:
                raise ValueError("forward_full failed")
            return out
        x = np.empty((len(t), self.shape.d_model), np.float64)
        if lib().orc_embed(self._h, _p(t), len(t), _p(x)) != 0:
            raise ValueError("forward_full failed")
        for layer in range(self.shape.n_layers):
            if lib().orc_layer_full(self._h, layer, len(t), _p(x)) != 0:
                raise ValueError(f"layer {layer} failed")
            progress(layer)
        xr = np.ascontiguousarray(x[row0:])
        if lib().orc_final_logits(self._h, _p(xr), len(t) - row0, _p(out)) != 0:
            raise ValueError("forward_full failed")
        return out

    def hidden_full(self, tokens, row0: int = 0) -> np.ndarray:
        t = np.ascontiguousarray(tokens, np.int32)
        out = np.empty((len(t) - row0, self.shape.d_model), np.float64)
        if lib().orc_forward_full_hidden(self._h, _p(t), len(t), row0, _p(out)) != 0:
            raise ValueError("forward_full failed")
        return out


class KV:
    """One sequence's cache in the cached route."""

    def __init__(self, model: Model, max_len: int):
        self.model = model
        self._h = lib().orc_kv_create(model._h, max_len)
        if not self._h:
            raise MemoryError("oracle kv creation failed")

    def __del__(self):
        if getattr(self, "_h", None):
            lib().orc_kv_free(self._h)
            self._h = None

    @property
    def len(self) -> int:
        return lib().orc_kv_len(self._h)

    @property
    def pending(self) -> int:
        return lib().orc_kv_pending(self._h)

    def read(self, layer: int, pos: int):
        s = self.model.shape
        k = np.empty(s.n_kv_heads * s.head_dim, np.float64)
        v = np.empty_like(k)
        if lib().orc_kv_read(self._h, layer, pos, _p(k), _p(v)) != 0:
            raise IndexError("kv read out of range")
        return k, v

    def prefill(self, tokens):
        t = np.ascontiguousarray(tokens, np.int32)
        if lib().orc_kv_prefill(self._h, _p(t), len(t)) != 0:
            raise ValueError("prefill failed")

    def verify(self, drafts) -> np.ndarray:
        d = np.ascontiguousarray(drafts, np.int32)
        out = np.empty((len(d) + 1, self.model.shape.vocab), np.float64)
        rc = lib().orc_verify(self._h, _p(d) if len(d) else None, len(d), _p(out))
        if rc != 0:
            raise ValueError(f"verify failed ({rc})")
        return out

    def commit(self, accepted_len: int, next_token: int):
        if lib().orc_commit(self._h, int(accepted_len), int(next_token)) != 0:
            raise ValueError("commit failed")


def accept(mode: int, draft, p, q=None, u=None, k: int = 1, lenience: float = 1.0,
           margins: bool = True):
    """Acceptance test over target rows p [B, gamma+1, V] (fp32 values).

    Returns dict(accepted_len, next_token, dec_margin, argmax_gap, flags, sample_margin).
    q: drafter rows [B, >=gamma, V] (ratio modes), u: uniforms [B, gamma] (RATIO) or
    [B, gamma+1] (RATIO_SAMPLE: column gamma draws the next token)."""
    p = np.ascontiguousarray(p, np.float32)
    B, R, V = p.shape
    gamma = R - 1
    draft = np.ascontiguousarray(np.asarray(draft, np.int32).reshape(B, gamma))
    qs = 0
    if q is not None:
        q = np.ascontiguousarray(q, np.float32)
        qs = q.shape[1] * V
    if u is not None:
        u = np.ascontiguousarray(u, np.float32).reshape(B, gamma + (mode == RATIO_SAMPLE))
    L = np.empty(B, np.int32)
    nxt = np.empty(B, np.int32)
    fl = np.empty(B, np.int32)
    dm = np.empty((B, max(gamma, 1)), np.float64) if margins else None
    gap = np.empty((B, gamma + 1), np.float64) if margins else None
    sm = np.empty(B, np.float64)
    rc = lib().orc_accept(mode, _p(draft), _p(p), _p(q), qs, _p(u), B, gamma, V, int(k),
                          float(lenience), _p(L), _p(nxt), _p(dm), _p(gap), _p(fl), _p(sm))
    if rc != 0:
        raise ValueError("invalid accept arguments")
    return dict(accepted_len=L, next_token=nxt, dec_margin=None if dm is None else dm[:, :gamma],
                argmax_gap=gap, flags=fl, sample_margin=sm)


def confidence_prefix(logits, gamma: int, tau: float, draft=None):
    """skip_len [B] and log_conf [B, gamma] from drafter rows logits [B, >=gamma, V]."""
    z = np.ascontiguousarray(logits, np.float32)
    B, R, V = z.shape
    sk = np.empty(B, np.int32)
    lc = np.empty((B, max(gamma, 1)), np.float64)
    lp = None
    if draft is not None:
        draft = np.ascontiguousarray(np.asarray(draft, np.int32).reshape(B, gamma))
        lp = np.empty((B, max(gamma, 1)), np.float64)
    rc = lib().orc_confidence_prefix(_p(z), R * V, B, gamma, V, float(tau), _p(sk), _p(lc),
                                     _p(draft), _p(lp))
    if rc != 0:
        raise ValueError("invalid confidence arguments")
    out = dict(skip_len=sk, log_conf=lc[:, :gamma])
    if lp is not None:
        out["log_p_draft"] = lp[:, :gamma]
    return out


# skip scheduler (Sec. 4.1 - 4.2)
SIG_RAW, SIG_MARGINAL, SIG_CONDITIONAL = 0, 1, 2
R_SKIP, R_STALE, R_NO_CANDIDATE, R_SHORT, R_SHORT_BLOCK, R_SPECIAL, R_REPEAT = range(7)


def schedule(log_q, D, signal: int, eta_b: float, eta_c: float, k_min: int = 0, s_max: int = 1 << 30,
             block_len=None, draft=None, special=(), rep_max: int = 0):
    """Two-gate skip decision per sequence.  log_q [B, gamma] fp32 position log-scores; D [B] unverified
    tokens since the last verifier call (returned updated).  Returns dict K, K_hat, reason, D."""
    lq = np.ascontiguousarray(log_q, np.float32)
    B, gamma = lq.shape
    d = np.ascontiguousarray(np.asarray(D, np.int32).reshape(B)).copy()
    K = np.empty(B, np.int32)
    Kh = np.empty(B, np.int32)
    rs = np.empty(B, np.int32)
    dr = None if draft is None else np.ascontiguousarray(np.asarray(draft, np.int32).reshape(B, gamma))
    sp = np.ascontiguousarray(np.asarray(special, np.int32).reshape(-1)) if len(special) else None
    bl = None if block_len is None else np.ascontiguousarray(np.broadcast_to(np.asarray(block_len, np.int32), (B,)))
    rc = lib().orc_schedule(_p(lq), _p(dr), B, gamma, int(signal), float(eta_b), float(eta_c), int(k_min),
                            int(s_max), _p(bl), _p(sp),
                            0 if sp is None else sp.size, int(rep_max), _p(d), _p(K), _p(Kh), _p(rs))
    if rc != 0:
        raise ValueError("invalid schedule arguments")
    return dict(K=K, K_hat=Kh, reason=rs, D=d)


def survival_mlp(hidden_bits, scalars, mu, sigma, W1, b1, W2, b2, W3, b3, w4, b4):
    """Survival predictor: hidden_bits uint16 bf16 [n, d_hid], scalars fp32 [n, n_sc], normalization
    mu/sigma [d_in], Linear weights [out][in] fp32.  Returns (log_score, logit) fp64 [n]."""
    h = np.ascontiguousarray(hidden_bits, np.uint16)
    n, d_hid = h.shape
    sc = np.ascontiguousarray(scalars, np.float32).reshape(n, -1)
    n_sc = sc.shape[1]
    H = np.asarray(b1).shape[0]
    f = lambda a: np.ascontiguousarray(a, np.float32)
    ls = np.empty(max(n, 1), np.float64)
    lg = np.empty(max(n, 1), np.float64)
    rc = lib().orc_survival_mlp(_p(h), _p(sc) if n_sc else None, n, d_hid, n_sc, H, _p(f(mu)), _p(f(sigma)),
                                _p(f(W1)), _p(f(b1)), _p(f(W2)), _p(f(b2)), _p(f(W3)), _p(f(b3)), _p(f(w4)),
                                float(b4), _p(ls), _p(lg))
    if rc != 0:
        raise ValueError("invalid survival_mlp arguments")
    return ls[:n], lg[:n]


def audit_accumulate(K, L, acc=None):
    """Adds the rounds with K > 0 to acc = int64 [4] (|A|, sum K, sum min(K, L), count K <= L); returns acc."""
    k = np.ascontiguousarray(np.asarray(K, np.int32).reshape(-1))
    l = np.ascontiguousarray(np.asarray(L, np.int32).reshape(-1))
    a = np.zeros(4, np.int64) if acc is None else acc
    if lib().orc_audit_accumulate(_p(k), _p(l), k.size, _p(a)) != 0:
        raise ValueError("invalid audit arguments")
    return a


def agreement(acc):
    """(StrictToken, FullPrefix) from accumulated counters; 1.0 when no round skipped (Strict SDD)."""
    n, sk, smin, full = (int(x) for x in acc)
    return (smin / sk if sk else 1.0), (full / n if n else 1.0)
