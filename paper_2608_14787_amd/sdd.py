"""Thin ctypes binding of libsdd (include/sdd.h): argument marshalling only.

Every step of the hot path runs in the HIP kernels of libsdd.so.  torch is
used for device memory and streams.  There is no fallback: if the library is
missing or no gfx950 GPU is present, calls raise.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsdd.so")

OK, EINVAL, ENOMEM, EHIP, ECAPACITY, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
F32, BF16 = 0, 1
GREEDY, RATIO, TOPK, LENIENT, RATIO_SAMPLE = 0, 1, 2, 3, 4
(T_EMBED, T_LM_HEAD, T_FINAL_NORM, T_WQ, T_WK, T_WV, T_WO, T_WGATE, T_WUP, T_WDOWN,
 T_ATTN_NORM, T_FFN_NORM, T_Q_NORM, T_K_NORM) = range(14)


class SDDError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sdd error {code}: {msg}")
        self.code = code


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("d_model", C.c_int), ("n_q_heads", C.c_int),
                ("n_kv_heads", C.c_int), ("head_dim", C.c_int), ("d_ff", C.c_int),
                ("vocab", C.c_int), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("qk_norm", C.c_int), ("dtype", C.c_int)]

    @staticmethod
    def from_shape(s) -> "ModelConfig":
        return ModelConfig(s.n_layers, s.d_model, s.n_q_heads, s.n_kv_heads, s.head_dim, s.d_ff,
                           s.vocab, s.rms_eps, s.rope_theta, int(s.qk_norm),
                           BF16 if s.dtype == "bf16" else F32)


_lib = None
P, I, SZ, F = C.c_void_p, C.c_int, C.c_size_t, C.c_float
_SIGS = {
    "sdd_status_string": (C.c_char_p, [I]),
    "sdd_last_error": (C.c_char_p, []),
    "sdd_device_ok": (I, []),
    "sdd_weights_bytes": (I, [P, P]),
    "sdd_model_create": (I, [P, P, SZ, P]),
    "sdd_model_destroy": (I, [P]),
    "sdd_model_init_random": (I, [P, C.c_uint64, F, P]),
    "sdd_model_load_tensor": (I, [P, I, I, P, P]),
    "sdd_model_matrix_layout": (I, [P, I, I, P, P, P, P, P, P, P]),
    "sdd_kv_bytes": (I, [P, I, I, P]),
    "sdd_kv_create": (I, [P, I, I, P, SZ, P, P]),
    "sdd_kv_destroy": (I, [P]),
    "sdd_kv_state": (I, [P, P, P, P, P]),
    "sdd_kv_device_state": (I, [P, P, P]),
    "sdd_workspace_bytes": (I, [P, I, P]),
    "sdd_workspace_init": (I, [P, SZ, P]),
    "sdd_kv_prefill": (I, [P, P, I, P, I, P, SZ, P]),
    "sdd_verify_block": (I, [P, P, P, I, P, I, P, P, P, SZ, P]),
    "sdd_kv_commit": (I, [P, P, I, P, P, P]),
    "sdd_rowstats_workspace_bytes": (I, [I, I, I, P]),
    "sdd_accept": (I, [P, P, I, P, I, SZ, P, I, I, I, I, I, F, P, P, P, P, SZ, P]),
    "sdd_accept_noalloc": (I, [P, P, I, P, I, SZ, P, I, I, I, I, I, F, P, P, P, P]),
    "sdd_confidence_prefix": (I, [P, I, SZ, I, I, I, F, P, P, P, P, P, SZ, P]),
    "sdd_schedule": (I, [P, P, P, I, I, I, C.c_double, C.c_double, I, I, P, I, I, P, P, P, P, P]),
    "sdd_verify_full": (I, [P, P, P, I, I, P, P, P, SZ, P]),
    "sdd_audit_accumulate": (I, [P, P, I, P, P]),
    "sdd_survival_workspace_bytes": (I, [P, I, P]),
    "sdd_survival_mlp": (I, [P, P, P, I, P, P, P, SZ, P]),
    "sdd_profile_start": (I, [C.c_uint, I, I]),
    "sdd_profile_read": (I, [C.c_uint, P, P, P, P]),
    "sdd_profile_stop": (I, []),
}

PROF_EMBED, PROF_GEMM_QKV, PROF_ATTN, PROF_GEMM_O = 1, 2, 4, 8
PROF_GEMM_GATEUP, PROF_GEMM_DOWN, PROF_GEMM_LM, PROF_ACCEPT, PROF_CONF = 16, 32, 64, 128, 256
PROF_SCHED, PROF_MLP = 512, 1024
SIG_RAW, SIG_MARGINAL, SIG_CONDITIONAL = 0, 1, 2
(SKIP_OK, SKIP_STALE, SKIP_NO_CANDIDATE, SKIP_SHORT, SKIP_SHORT_BLOCK, SKIP_SPECIAL,
 SKIP_REPEAT) = range(7)


def lib() -> C.CDLL:
    """Loads libsdd.so (built by paper_2608_14787_amd.build); raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run paper_2608_14787_amd.build.build()")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            fn = getattr(L, name, None)
            if fn is None:  # reported by the export test; calls to it fail loudly
                continue
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(rc: int):
    if rc != OK:
        raise SDDError(rc, lib().sdd_last_error().decode())


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _i32(t, name: str, allow_none: bool = False):
    """An int32 contiguous device tensor (the C ABI reads int32 arrays with no strides)."""
    if t is None:
        _need(allow_none, f"{name} is required")
        return
    _need(t.dtype == torch.int32, f"{name} must be int32, got {t.dtype}")
    _need(t.is_contiguous(), f"{name} must be contiguous")


def _rows(t, name: str):
    """Logit rows the C ABI addresses as base + b * stride(0) + j * V: unit element stride, rows V apart."""
    _need(t.dim() == 3, f"{name} must be [B, rows, V]")
    _need(t.stride(2) == 1 and t.stride(1) == t.shape[2], f"{name}: rows must be contiguous and V elements apart")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def device_ok() -> bool:
    return bool(lib().sdd_device_ok())


def _size_out(fn, *args) -> int:
    out = C.c_size_t(0)
    _check(fn(*args, C.byref(out)))
    return out.value


def workspace_init(ws: torch.Tensor, stream=None):
    _check(lib().sdd_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def rowstats_workspace(B: int, gamma: int, V: int, device="cuda") -> torch.Tensor:
    n = _size_out(lib().sdd_rowstats_workspace_bytes, B, gamma, V)
    ws = torch.empty(n, dtype=torch.uint8, device=device)
    workspace_init(ws)
    return ws


def accept(draft: torch.Tensor, p: torch.Tensor, mode: int, *, q: torch.Tensor | None = None,
           uniforms: torch.Tensor | None = None, k: int = 1, lenience: float = 1.0,
           ws: torch.Tensor | None = None, out=None, stream=None):
    """sdd_accept: returns (accepted_len, next_token, flags) int32 device tensors [B]."""
    B, R, V = p.shape
    gamma = R - 1
    if ws is None:
        ws = rowstats_workspace(B, gamma, V, p.device)
    if out is None:
        out = tuple(torch.empty(B, dtype=torch.int32, device=p.device) for _ in range(3))
    L, nxt, fl = out
    _need(p.is_contiguous(), "p must be contiguous [B, gamma+1, V]")
    _i32(draft, "draft", allow_none=gamma == 0)
    for t, nm in ((L, "accepted_len"), (nxt, "next_token"), (fl, "flags")):
        _i32(t, nm, allow_none=nm == "flags")
    if uniforms is not None:
        _need(uniforms.dtype == torch.float32 and uniforms.is_contiguous(), "uniforms must be contiguous fp32")
    qd, qs = F32, 0
    if q is not None:
        _rows(q, "q")
        qd, qs = _dtype_code(q), q.stride(0)
    _check(lib().sdd_accept(_ptr(draft), _ptr(p), _dtype_code(p), _ptr(q), qd, qs, _ptr(uniforms),
                            B, gamma, V, mode, k, lenience, _ptr(L), _ptr(nxt), _ptr(fl), _ptr(ws),
                            ws.numel(), _stream(stream)))
    return L, nxt, fl


def confidence_prefix(logits: torch.Tensor, gamma: int, tau: float, *, draft=None,
                      log_conf=False, ws: torch.Tensor | None = None, out=None, stream=None):
    """sdd_confidence_prefix over drafter rows logits[B, >=gamma, V].

    log_conf: False, True (allocate) or a contiguous fp32 [B, gamma] tensor to write into.
    Returns skip_len int32 [B] (and log_conf, log_p_draft fp32 [B, gamma] when requested)."""
    B, R, V = logits.shape
    _rows(logits, "logits")
    _i32(draft, "draft", allow_none=True)
    if ws is None:
        ws = rowstats_workspace(B, gamma, V, logits.device)
    sk = out if out is not None else torch.empty(B, dtype=torch.int32, device=logits.device)
    if isinstance(log_conf, torch.Tensor):
        assert log_conf.dtype == torch.float32 and log_conf.is_contiguous() and log_conf.numel() >= B * gamma
        lc = log_conf
    else:
        lc = torch.empty((B, max(gamma, 1)), dtype=torch.float32, device=logits.device) if log_conf else None
    lp = torch.empty((B, max(gamma, 1)), dtype=torch.float32, device=logits.device) if draft is not None else None
    _check(lib().sdd_confidence_prefix(_ptr(logits), _dtype_code(logits), logits.stride(0), B, gamma,
                                       V, tau, _ptr(sk), _ptr(lc), _ptr(draft), _ptr(lp), _ptr(ws),
                                       ws.numel(), _stream(stream)))
    if lc is None and draft is None:
        return sk
    return sk, (lc[:, :gamma] if lc is not None else None), (lp[:, :gamma] if lp is not None else None)


def schedule(log_q: torch.Tensor, D: torch.Tensor, signal: int, eta_b: float, eta_c: float, *,
             k_min: int = 0, s_max: int = 1 << 30, draft=None, block_len=None, special=None,
             rep_max: int = 0, out=None, stream=None):
    """sdd_schedule: two-gate skip decision for log_q fp32 [B, gamma]; D int32 [B] is updated in place.

    Returns (K, K_hat, reason), int32 [B] each."""
    B, gamma = log_q.shape
    dev = log_q.device
    if out is None:
        out = tuple(torch.empty(B, dtype=torch.int32, device=dev) for _ in range(3))
    K, Kh, rs = out
    n_special = 0 if special is None else special.numel()
    _check(lib().sdd_schedule(_ptr(log_q), _ptr(draft), _ptr(block_len), B, gamma, signal, float(eta_b),
                              float(eta_c), k_min, s_max, _ptr(special), n_special, rep_max, _ptr(D),
                              _ptr(K), _ptr(Kh), _ptr(rs), _stream(stream)))
    return K, Kh, rs


class MlpDesc(C.Structure):
    _fields_ = [("d_hid", C.c_int), ("n_sc", C.c_int), ("H", C.c_int), ("mu", P), ("sigma", P), ("W1", P),
                ("b1", P), ("W2", P), ("b2", P), ("W3", P), ("b3", P), ("w4", P), ("b4", C.c_float)]


class SurvivalMLP:
    """Survival-predictor weights as device fp32 tensors (torch-owned) and their sdd_mlp descriptor."""

    def __init__(self, mu, sigma, W1, b1, W2, b2, W3, b3, w4, b4: float, d_hid: int, device="cuda"):
        t = lambda a: torch.as_tensor(a, dtype=torch.float32).contiguous().to(device)
        self.tensors = [t(x) for x in (mu, sigma, W1, b1, W2, b2, W3, b3, w4)]
        H = self.tensors[3].numel()
        d_in = self.tensors[0].numel()
        self.desc = MlpDesc(d_hid, d_in - d_hid, H, *[C.c_void_p(x.data_ptr()) for x in self.tensors], float(b4))
        self.device = device

    def workspace(self, n: int) -> torch.Tensor:
        out = C.c_size_t()
        _check(lib().sdd_survival_workspace_bytes(C.byref(self.desc), n, C.byref(out)))
        ws = torch.empty(max(int(out.value), 256), dtype=torch.uint8, device=self.device)
        workspace_init(ws)
        return ws

    def __call__(self, hidden: torch.Tensor, scalars: torch.Tensor | None, *, ws=None, out=None, logit=None,
                 stream=None) -> torch.Tensor:
        """log sigmoid scores fp32 [n] for hidden bf16 [n, d_hid] and scalars fp32 [n, n_sc]."""
        n = hidden.shape[0]
        if ws is None:
            ws = self.workspace(n)
        ls = out if out is not None else torch.empty(n, dtype=torch.float32, device=hidden.device)
        _check(lib().sdd_survival_mlp(C.byref(self.desc), _ptr(hidden), _ptr(scalars), n, _ptr(ls), _ptr(logit),
                                      _ptr(ws), ws.numel(), _stream(stream)))
        return ls


def audit_accumulate(K: torch.Tensor, L: torch.Tensor, acc: torch.Tensor, stream=None):
    """sdd_audit_accumulate into acc (int64 [4] device, zero it once)."""
    _check(lib().sdd_audit_accumulate(_ptr(K), _ptr(L), K.numel(), _ptr(acc), _stream(stream)))


def profile_start(class_mask: int, max_launches: int = 65536, every: int = 1):
    """Brackets every `every`-th launch of the given kernel classes with HIP events until profile_stop()."""
    _check(lib().sdd_profile_start(class_mask, max_launches, every))


def profile_read(cls: int):
    """(launches, total_ms, min_ms, max_ms) over the recorded launches of the classes in cls."""
    n, tot, mn, mx = C.c_int(), C.c_double(), C.c_double(), C.c_double()
    _check(lib().sdd_profile_read(cls, C.byref(n), C.byref(tot), C.byref(mn), C.byref(mx)))
    return n.value, tot.value, mn.value, mx.value


def profile_stop():
    _check(lib().sdd_profile_stop())


# ---- decoder ------------------------------------------------------------------------------


class Model:
    """Target decoder weights in a torch-owned device buffer, in libsdd's tiled layout."""

    def __init__(self, shape, device="cuda"):
        self.shape = shape
        self.cfg = ModelConfig.from_shape(shape)
        n = _size_out(lib().sdd_weights_bytes, C.byref(self.cfg))
        self.buf = torch.empty(n, dtype=torch.uint8, device=device)
        h = C.c_void_p()
        _check(lib().sdd_model_create(C.byref(self.cfg), _ptr(self.buf), n, C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.sdd_model_destroy(self.handle)
            self.handle = None

    @property
    def weight_bytes(self) -> int:
        return self.buf.numel()

    def init_random(self, seed: int = 0, sigma: float = 0.02, stream=None):
        _check(lib().sdd_model_init_random(self.handle, seed, sigma, _stream(stream)))

    def load_tensor(self, kind: int, layer: int, t: torch.Tensor, stream=None):
        _check(lib().sdd_model_load_tensor(self.handle, kind, layer, _ptr(t.contiguous()), _stream(stream)))

    def matrix_layout(self, kind: int, layer: int = 0) -> dict:
        """sdd_model_matrix_layout: where and in which order a tiled matrix is stored."""
        off, nb = C.c_size_t(), C.c_size_t()
        kt, g, ng, nwg, c = C.c_int(), C.c_int(), C.c_int(), C.c_int(), C.c_int()
        _check(lib().sdd_model_matrix_layout(self.handle, kind, layer, C.byref(off), C.byref(nb), C.byref(kt),
                                             C.byref(g), C.byref(ng), C.byref(nwg), C.byref(c)))
        return {"offset": off.value, "bytes": nb.value, "KT": kt.value, "G": g.value, "ng": ng.value,
                "n_wg": nwg.value, "c": c.value}

    def workspace(self, max_rows: int) -> torch.Tensor:
        n = _size_out(lib().sdd_workspace_bytes, self.handle, max_rows)
        ws = torch.empty(n, dtype=torch.uint8, device=self.buf.device)
        workspace_init(ws)
        return ws


class KVCache:
    def __init__(self, model: Model, max_batch: int, max_len: int, stream=None):
        self.model, self.max_batch, self.max_len = model, max_batch, max_len
        n = _size_out(lib().sdd_kv_bytes, C.byref(model.cfg), max_batch, max_len)
        self.buf = torch.empty(n, dtype=torch.uint8, device=model.buf.device)
        h = C.c_void_p()
        _check(lib().sdd_kv_create(model.handle, max_batch, max_len, _ptr(self.buf), n, _stream(stream),
                                   C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.sdd_kv_destroy(self.handle)
            self.handle = None

    def state(self, stream=None):
        """(len [max_batch], pending [max_batch], error_bits) read synchronously."""
        import numpy as np
        ln = np.zeros(self.max_batch, np.int32)
        pd = np.zeros(self.max_batch, np.int32)
        eb = np.zeros(1, np.int32)
        _check(lib().sdd_kv_state(self.handle, ln.ctypes.data_as(C.c_void_p), pd.ctypes.data_as(C.c_void_p),
                                  eb.ctypes.data_as(C.c_void_p), _stream(stream)))
        return ln, pd, int(eb[0])

    def device_len_ptr(self) -> int:
        """Device address of the int32[max_batch] length array."""
        p = C.c_void_p()
        _check(lib().sdd_kv_device_state(self.handle, C.byref(p), None))
        return p.value

    def prefill(self, seq: int, tokens: torch.Tensor, ws: torch.Tensor, stream=None):
        _i32(tokens, "tokens")
        _check(lib().sdd_kv_prefill(self.model.handle, self.handle, seq, _ptr(tokens), tokens.numel(),
                                    _ptr(ws), ws.numel(), _stream(stream)))

    def verify(self, seq_ids: torch.Tensor, drafts: torch.Tensor, logits: torch.Tensor,
               argmax: torch.Tensor | None, ws: torch.Tensor, stream=None):
        n_seq, gamma = drafts.shape
        _i32(seq_ids, "seq_ids")
        _i32(drafts, "drafts")
        _i32(argmax, "argmax", allow_none=True)
        _need(logits.dtype == torch.float32 and logits.is_contiguous(), "logits must be contiguous fp32")
        _need(logits.numel() >= n_seq * (gamma + 1) * self.model.shape.vocab, "logits too small")
        _check(lib().sdd_verify_block(self.model.handle, self.handle, _ptr(seq_ids), n_seq,
                                      _ptr(drafts) if gamma else None, gamma, _ptr(logits), _ptr(argmax),
                                      _ptr(ws), ws.numel(), _stream(stream)))

    def verify_full(self, tokens: torch.Tensor, gamma: int, logits: torch.Tensor, argmax: torch.Tensor | None,
                    ws: torch.Tensor, stream=None):
        """sdd_verify_full: this cache is the scratch (slot 0 overwritten); tokens int32 [n] = context + drafts."""
        _i32(tokens, "tokens")
        _i32(argmax, "argmax", allow_none=True)
        _need(logits.dtype == torch.float32 and logits.is_contiguous(), "logits must be contiguous fp32")
        _check(lib().sdd_verify_full(self.model.handle, self.handle, _ptr(tokens), tokens.numel(), gamma, _ptr(logits),
                                     _ptr(argmax), _ptr(ws), ws.numel(), _stream(stream)))

    def commit(self, seq_ids: torch.Tensor, accepted_len: torch.Tensor, next_token: torch.Tensor, stream=None):
        for t, nm in ((seq_ids, "seq_ids"), (accepted_len, "accepted_len"), (next_token, "next_token")):
            _i32(t, nm)
        _check(lib().sdd_kv_commit(self.handle, _ptr(seq_ids), seq_ids.numel(), _ptr(accepted_len),
                                   _ptr(next_token), _stream(stream)))
