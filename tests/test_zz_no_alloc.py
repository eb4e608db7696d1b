"""sdd_accept_noalloc (acceptance with the library's own per-GPU scratch, for callers that cannot allocate)
against sdd_accept with a caller workspace: identical integer outputs, bit for bit, on consecutive calls
whose second input is smaller than the first, and a clear refusal of shapes beyond the scratch size."""
import ctypes as C

import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


def _noalloc(S, draft, p, mode, q=None, u=None, k=1, lenience=1.0):
    B, R, V = p.shape
    gamma = R - 1
    out = [torch.full((B,), -7, dtype=torch.int32, device="cuda") for _ in range(3)]
    qd, qs = (S._dtype_code(q), q.stride(0)) if q is not None else (S.F32, 0)
    rc = S.lib().sdd_accept_noalloc(S._ptr(draft), S._ptr(p), S._dtype_code(p), S._ptr(q), qd, qs, S._ptr(u), B,
                                    gamma, V, mode, k, C.c_float(lenience), S._ptr(out[0]), S._ptr(out[1]),
                                    S._ptr(out[2]), S._stream(None))
    return rc, out


def _with_ws(S, draft, p, mode, q=None, u=None, k=1, lenience=1.0):
    L, nxt, fl = S.accept(draft, p, mode, q=q, uniforms=u, k=k, lenience=lenience)
    return [L, nxt, fl]


def _same(a, b):
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y), (x, y)


def test_noalloc_accept_matches_workspace_accept(S):
    # call 1: the [16, 33, 151936] bf16 workload, ratio test (target and drafter rows)
    x = W.accept_inputs(31, variant="rowmax")
    p = torch.from_numpy(x.target_bits.view(np.int16)).cuda().view(torch.bfloat16)
    q = torch.from_numpy(x.drafter_bits.view(np.int16)).cuda().view(torch.bfloat16)
    draft = torch.from_numpy(x.draft).cuda()
    u = torch.from_numpy(x.u).cuda()
    print("call 1: B=16 gamma=32 V=151936 bf16 ratio", flush=True)
    rc, got = _noalloc(S, draft, p, S.RATIO, q=q, u=u)
    assert rc == 0, S.lib().sdd_last_error()
    _same(got, _with_ws(S, draft, p, S.RATIO, q=q, u=u))
    print(f"  accepted {got[0].cpu().numpy().tolist()}", flush=True)
    # call 2: a smaller input (fp32, B=3, gamma=5, V=4096), top-k
    g = W.rng(32)
    p2 = torch.from_numpy((g.standard_normal((3, 6, 4096)) * 2).astype(np.float32)).cuda()
    d2 = p2[:, :5].argmax(-1).to(torch.int32).contiguous()
    d2[1, 2] = 7
    print("call 2: B=3 gamma=5 V=4096 fp32 top-4", flush=True)
    rc, got2 = _noalloc(S, d2, p2, S.TOPK, k=4)
    assert rc == 0, S.lib().sdd_last_error()
    _same(got2, _with_ws(S, d2, p2, S.TOPK, k=4))
    assert got2[0].cpu().numpy().tolist()[1] >= 2
    # call 3: greedy on the first input again (the scratch keeps the last call's contents)
    print("call 3: B=16 gamma=32 greedy", flush=True)
    rc, got3 = _noalloc(S, draft, p, S.GREEDY)
    assert rc == 0
    _same(got3, _with_ws(S, draft, p, S.GREEDY))


def test_noalloc_refuses_shapes_beyond_its_scratch(S):
    p = torch.zeros((200, 65, 64), dtype=torch.float32, device="cuda")
    d = torch.zeros((200, 64), dtype=torch.int32, device="cuda")
    rc, _ = _noalloc(S, d, p, S.GREEDY)
    assert rc == S.ECAPACITY
    assert b"scratch" in S.lib().sdd_last_error()
