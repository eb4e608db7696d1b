"""The C-ABI library loads and exports every function include/sdd.h declares; host-side argument
checks return the documented status codes without touching a GPU."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from gpu_helpers import share_starts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "sdd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sdd_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    if not os.path.exists(sdd.LIB_PATH):
        from paper_2608_14787_amd import build
        build.build()
    return sdd


def test_every_declared_symbol_is_exported(S):
    names = _declared()
    assert len(names) >= 18
    lib = C.CDLL(S.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_host_side_argument_errors(S):
    L = S.lib()
    assert L.sdd_status_string(S.EINVAL).decode() == "invalid argument"
    out = C.c_size_t()
    assert L.sdd_rowstats_workspace_bytes(0, 4, 10, C.byref(out)) == S.EINVAL
    assert L.sdd_rowstats_workspace_bytes(2, 65, 10, C.byref(out)) == S.EINVAL
    assert L.sdd_rowstats_workspace_bytes(2, 4, 10, C.byref(out)) == S.OK and out.value > 0
    cfg = S.ModelConfig(2, 256, 4, 2, 64, 688, 4096, 1e-6, 1e4, 0, S.F32)
    assert L.sdd_weights_bytes(C.byref(cfg), C.byref(out)) == S.OK
    # 14.2 MB of fp32 weights for the tiny decoder, plus alignment and at most n_wg padding slots (of <= 8 KiB)
    # per tiled matrix (9 of them)
    total = out.value
    assert 14.0e6 < total < 14.6e6 + 9 * 256 * 8192
    # the tiled matrices' documented layouts (host-only queries on a model over an unused, aligned address)
    h = C.c_void_p()
    assert L.sdd_model_create(C.byref(cfg), C.c_void_p(1 << 20), total, C.byref(h)) == S.OK
    off, nb = C.c_size_t(), C.c_size_t()
    kt, g, ng, nwg, sc = C.c_int(), C.c_int(), C.c_int(), C.c_int(), C.c_int()
    d, hd, V, dff = 256, 64, 4096, 688
    spans = []
    for kind, layer, rows, cols in [(1, 0, V, d)] + [(k, l, r, c) for l in range(2) for k, r, c in
                                                      ((3, 4 * hd + 2 * 2 * hd, d), (6, d, 4 * hd),
                                                       (7, 2 * dff, d), (9, d, dff))]:
        assert L.sdd_model_matrix_layout(h, kind, layer, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g),
                                         C.byref(ng), C.byref(nwg), C.byref(sc)) == S.OK
        U = g.value * kt.value
        assert g.value * ng.value * 16 >= rows and kt.value * 16 >= cols
        # at most 256 groups: equal shares (or equal k-ranges of every group)
        assert sc.value == 0 and 1 <= nwg.value <= U and nb.value == -(-U // nwg.value) * nwg.value * ng.value * 1024
        spans.append((off.value, off.value + nb.value))
    spans.sort()
    assert all(a1 <= b0 for (_, a1), (b0, _) in zip(spans, spans[1:])) and spans[-1][1] <= total
    assert L.sdd_model_matrix_layout(h, 2, 0, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g), C.byref(ng),
                                     C.byref(nwg), C.byref(sc)) == S.EINVAL
    assert L.sdd_model_matrix_layout(h, 3, 2, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g), C.byref(ng),
                                     C.byref(nwg), C.byref(sc)) == S.EINVAL
    assert L.sdd_model_matrix_layout(h, 3, 0, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g), C.byref(ng),
                                     C.byref(nwg), None) == S.EINVAL
    assert L.sdd_model_destroy(h) == S.OK
    # a 51200-token vocabulary gives the LM head 400 column groups of 8 tiles: stream-K over the 256-CU count
    # the library plans for, with cost-balanced shares (every share non-empty and contiguous; the matrix holds
    # n_wg times the longest share; a share entering one more group holds fewer units)
    wide = S.ModelConfig(2, 256, 4, 2, 64, 688, 51200, 1e-6, 1e4, 0, S.F32)
    assert L.sdd_weights_bytes(C.byref(wide), C.byref(out)) == S.OK
    h = C.c_void_p()
    assert L.sdd_model_create(C.byref(wide), C.c_void_p(1 << 20), out.value, C.byref(h)) == S.OK
    assert L.sdd_model_matrix_layout(h, 1, 0, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g), C.byref(ng),
                                     C.byref(nwg), C.byref(sc)) == S.OK
    KT, G, n, c = kt.value, g.value, nwg.value, sc.value
    assert G * ng.value * 16 == 51200 and G > n and c > 0
    st = share_starts(KT, G, c, n)
    shares = np.diff(st)
    assert st[0] == 0 and st[-1] == G * KT and shares.min() >= 1
    assert nb.value == shares.max() * n * ng.value * 1024
    segs = (st[1:] - 1) // KT - st[:-1] // KT + 1
    cost = shares + c * (segs - 1)
    assert cost.max() - cost.min() <= c + 1 and shares.max() > shares.min()
    assert L.sdd_model_destroy(h) == S.OK
    bad = S.ModelConfig(2, 256, 4, 2, 96, 688, 4096, 1e-6, 1e4, 0, S.F32)
    assert L.sdd_weights_bytes(C.byref(bad), C.byref(out)) == S.EUNSUPPORTED
    bad = S.ModelConfig(2, 256, 5, 2, 64, 688, 4096, 1e-6, 1e4, 0, S.F32)
    assert L.sdd_weights_bytes(C.byref(bad), C.byref(out)) == S.EINVAL
    # KV cache: the position stride is max_len rounded up to 64, so 1..64 positions size alike
    kv1, kv64, kv65 = C.c_size_t(), C.c_size_t(), C.c_size_t()
    assert L.sdd_kv_bytes(C.byref(cfg), 1, 1, C.byref(kv1)) == S.OK
    assert L.sdd_kv_bytes(C.byref(cfg), 1, 64, C.byref(kv64)) == S.OK
    assert L.sdd_kv_bytes(C.byref(cfg), 1, 65, C.byref(kv65)) == S.OK
    rope = lambda n: -(-n * 64 * 4 // 256) * 256  # [max_len][head_dim] fp32 (cos, sin) table
    per_layer64 = 1 * 2 * 64 * 64 * 4  # [batch][kv heads][64 positions][head_dim] fp32, for K and for V
    assert kv64.value - kv1.value == rope(64) - rope(1)
    assert kv65.value - kv64.value == rope(65) - rope(64) + 2 * 2 * per_layer64
    # profiling: the sampling interval must be positive
    assert L.sdd_profile_start(1, 16, 0) == S.EINVAL
    # accept: NULL required pointers, bad mode parameters, bad shapes
    P = C.c_void_p(16)
    args = lambda **kw: [kw.get("draft", P), kw.get("p", P), S.BF16, None, S.BF16, 0, None, kw.get("B", 2),
                         kw.get("gamma", 4), 100, kw.get("mode", S.GREEDY), kw.get("k", 1), kw.get("len", 1.0),
                         P, P, None, P, 1 << 20, None]
    assert L.sdd_accept(*args(p=None)) == S.EINVAL
    assert L.sdd_accept(*args(B=0)) == S.EINVAL
    assert L.sdd_accept(*args(gamma=65)) == S.EINVAL
    assert L.sdd_accept(*args(mode=S.TOPK, k=0)) == S.EINVAL
    assert L.sdd_accept(*args(mode=S.LENIENT, len=1.5)) == S.EINVAL
    assert L.sdd_accept(*args(mode=S.RATIO)) == S.EINVAL  # ratio needs q and uniforms
    assert L.sdd_confidence_prefix(P, S.BF16, 400, 2, 4, 100, float("nan"), P, None, None, None, P, 1 << 20, None) == S.EINVAL
    assert L.sdd_confidence_prefix(P, S.BF16, 10, 2, 4, 100, 0.5, P, None, None, None, P, 1 << 20, None) == S.EINVAL

    def sched(lq=P, draft=None, B=4, gamma=8, signal=S.SIG_RAW, eb=0.9, ec=0.93, special=None, n_special=0,
              rep_max=0, D=P, K=P):
        return L.sdd_schedule(lq, draft, None, B, gamma, signal, eb, ec, 6, 64, special, n_special, rep_max, D, K,
                              None, None, None)
    assert sched(lq=None) == S.EINVAL
    assert sched(D=None) == S.EINVAL and sched(K=None) == S.EINVAL
    assert sched(B=0) == S.EINVAL and sched(gamma=65) == S.EINVAL and sched(gamma=-1) == S.EINVAL
    assert sched(signal=3) == S.EINVAL and sched(signal=-1) == S.EINVAL
    assert sched(eb=float("nan")) == S.EINVAL and sched(ec=float("nan")) == S.EINVAL
    assert sched(special=P, n_special=257, draft=P) == S.EINVAL
    assert sched(special=None, n_special=1, draft=P) == S.EINVAL
    assert sched(special=P, n_special=1, draft=None) == S.EINVAL  # the special-token guard reads drafts
    assert sched(rep_max=2, draft=None) == S.EINVAL


@pytest.mark.parametrize("which", ["QWEN32B", "QWEN7B"])
def test_streaming_plans_of_the_real_shapes(S, which):
    """Host-only layout queries of the Qwen-shaped models (weights over an unused address): every
    stream-K plan (more column groups than workgroups) balances its shares by cost (c > 0, every share
    non-empty, costs within c + 1 of each other); every plan with fewer groups than workgroups splits
    each group into equal k-ranges (c = 0); each matrix's extent is n_wg times its longest share."""
    import workloads as W
    shape = getattr(W, which)
    L = S.lib()
    cfg = S.ModelConfig.from_shape(shape)
    out = C.c_size_t()
    assert L.sdd_weights_bytes(C.byref(cfg), C.byref(out)) == S.OK
    h = C.c_void_p()
    assert L.sdd_model_create(C.byref(cfg), C.c_void_p(1 << 20), out.value, C.byref(h)) == S.OK
    off, nb = C.c_size_t(), C.c_size_t()
    kt, g, ng, nwg, sc = C.c_int(), C.c_int(), C.c_int(), C.c_int(), C.c_int()
    seen = set()
    for kind, layer in [(S.T_LM_HEAD, 0), (S.T_WQ, 0), (S.T_WO, 0), (S.T_WGATE, 0), (S.T_WDOWN, shape.n_layers - 1)]:
        assert L.sdd_model_matrix_layout(h, kind, layer, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g),
                                         C.byref(ng), C.byref(nwg), C.byref(sc)) == S.OK
        KT, G, n, c = kt.value, g.value, nwg.value, sc.value
        st = share_starts(KT, G, c, n)
        shares = np.diff(st)
        assert st[0] == 0 and st[-1] == G * KT and shares.min() >= 1
        assert nb.value == shares.max() * n * ng.value * 1024
        if G > n:
            assert c > 0
            segs = (st[1:] - 1) // KT - st[:-1] // KT + 1
            cost = shares + c * (segs - 1)
            assert cost.max() - cost.min() <= c + 1, (kind, cost.min(), cost.max())
        else:
            split = n // G
            assert c == 0 and n % G == 0 and np.isin(shares, [KT // split, -(-KT // split)]).all()
            # one segment per workgroup: a share never crosses a group boundary
            assert ((st[1:] - 1) // KT == st[:-1] // KT).all()
        seen.add("streamk" if G > n else "split")
    assert seen == {"streamk", "split"}
    assert L.sdd_model_destroy(h) == S.OK


@pytest.mark.parametrize("which", ["QWEN32B", "QWEN7B"])
def test_pair_partition_reads_every_stored_tile(S, which):
    """Host-only: the many-row kernel for the wide matrices (gate/up, LM head) covers pairs of adjacent
    8-tile column groups, P = ceil(G / 2) pairs as P x KT units split evenly over P x min(n_wg / P, KT)
    workgroups (or stream-K over n_wg when P >= n_wg), and finds each weight tile where the matrix's own
    plan stores it by following the storing workgroup as k rises.  Replayed here against the documented
    storage formula (slot (u - start(w)) n_wg + w of unit u = g KT + k, owner w): every tile of the matrix
    is read exactly once, from its stored slot, and every pair's contributors are contiguous workgroups."""
    import workloads as W
    shape = getattr(W, which)
    L = S.lib()
    cfg = S.ModelConfig.from_shape(shape)
    out = C.c_size_t()
    assert L.sdd_weights_bytes(C.byref(cfg), C.byref(out)) == S.OK
    h = C.c_void_p()
    assert L.sdd_model_create(C.byref(cfg), C.c_void_p(1 << 20), out.value, C.byref(h)) == S.OK
    off, nb = C.c_size_t(), C.c_size_t()
    kt, g, ng, nwg, sc = C.c_int(), C.c_int(), C.c_int(), C.c_int(), C.c_int()
    for kind in (S.T_WGATE, S.T_LM_HEAD):
        assert L.sdd_model_matrix_layout(h, kind, 0, C.byref(off), C.byref(nb), C.byref(kt), C.byref(g), C.byref(ng),
                                         C.byref(nwg), C.byref(sc)) == S.OK
        KT, G, n, c = kt.value, g.value, nwg.value, sc.value
        assert ng.value == 8
        st = share_starts(KT, G, c, n)  # storage plan
        P = (G + 1) // 2
        NP = n if P >= n else P * min(n // P, KT)
        pst = np.arange(NP + 1, dtype=np.int64) * (P * KT) // NP  # pair partition, equal shares
        assert (np.diff(pst) >= 1).all()
        seen = np.zeros(G * KT, np.int32)

        def owner(u):
            return int(np.searchsorted(st, u, side="right")) - 1

        for w in range(NP):
            u = int(pst[w])
            while u < pst[w + 1]:
                p = u // KT
                kb = u - p * KT
                ke = min(KT, kb + int(pst[w + 1]) - u)
                for gg in (2 * p, 2 * p + 1):
                    if gg >= G:
                        continue
                    o = owner(gg * KT + kb)  # tracker: owner of the segment's first k-step, then advance
                    kend = int(st[o + 1]) - gg * KT
                    base = (gg * KT - int(st[o])) * n + o
                    for k in range(kb, ke):
                        while k >= kend:
                            o += 1
                            kend = int(st[o + 1]) - gg * KT
                            base = (gg * KT - int(st[o])) * n + o
                        uu = gg * KT + k
                        ref = (uu - int(st[owner(uu)])) * n + owner(uu)
                        assert base + k * n == ref
                        assert 0 <= ref * 8 * 1024 < nb.value
                        seen[uu] += 1
                if not (kb == 0 and ke == KT):  # a split pair: its contributors are w's neighbours
                    wf = int(np.searchsorted(pst, p * KT, side="right")) - 1
                    wl = int(np.searchsorted(pst, (p + 1) * KT - 1, side="right")) - 1
                    assert wf <= w <= wl
                u += ke - kb
        assert (seen == 1).all(), kind
    assert L.sdd_model_destroy(h) == S.OK
