"""GPU check of sdd_model_load_tensor: loading every tensor row-major (the fused q/k/v parts, the gate/up
pairs interleaved per 16-row tile, the k-step-major tiling, the row-major embedding, the fp32 norm gains)
must reproduce, byte for byte, the weight buffer that sdd_model_init_random writes from the same
generator values; and a model loaded that way must give the same verify logits.

The row-major values come from the oracle's copy of the counter-based generator (CPU), so the loader is
checked against an independent source of the same numbers.  Integer and byte work: bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_helpers import to_dev_i32

pytestmark = pytest.mark.gpu

MID_BF16 = W.ModelShape(2, 512, 8, 2, 64, 1024, 2048, 1e-6, 1e6, True, "bf16")
MID_GQA128 = W.ModelShape(2, 256, 8, 2, 128, 512, 1024, 1e-6, 1e6, False, "bf16")

# tensor kinds of include/sdd.h
T_EMBED, T_LM_HEAD, T_FINAL_NORM, T_WQ, T_WK, T_WV, T_WO, T_WGATE, T_WUP, T_WDOWN = range(10)
T_ATTN_NORM, T_FFN_NORM, T_Q_NORM, T_K_NORM = range(10, 14)
MATRICES = (T_WQ, T_WK, T_WV, T_WO, T_WGATE, T_WUP, T_WDOWN)
GAINS = (T_ATTN_NORM, T_FFN_NORM, T_Q_NORM, T_K_NORM)


@pytest.fixture(scope="module")
def S():
    from paper_2608_14787_amd import sdd
    assert sdd.device_ok(), "needs a gfx950 device"
    return sdd


def _rowmajor(shape, kind, layer, seed, sigma):
    rows, cols = oracle.tensor_shape(shape, kind)
    bf16 = shape.dtype == "bf16"
    v = oracle.weight_values(seed, oracle.tensor_id(kind, layer), 0, rows * cols, sigma, bf16).reshape(rows, cols)
    t = torch.from_numpy(v).cuda()
    return t.to(torch.bfloat16) if bf16 else t


@pytest.mark.parametrize("shape", [MID_BF16, MID_GQA128, W.TINY], ids=["hd64-qknorm", "hd128-gqa4", "tiny-f32"])
def test_load_tensor_reproduces_init_random(S, shape):
    seed, sigma = 7, 0.02
    print(f"load_tensor vs init_random {shape}", flush=True)
    ref = S.Model(shape)
    ref.buf.zero_()  # alignment gaps between tensors are written by neither path
    ref.init_random(seed, sigma)
    m = S.Model(shape)
    m.buf.zero_()
    m.load_tensor(T_EMBED, 0, _rowmajor(shape, T_EMBED, 0, seed, sigma))
    m.load_tensor(T_LM_HEAD, 0, _rowmajor(shape, T_LM_HEAD, 0, seed, sigma))
    m.load_tensor(T_FINAL_NORM, 0, torch.ones(shape.d_model, dtype=torch.float32, device="cuda"))
    for layer in range(shape.n_layers):
        for kind in MATRICES:
            m.load_tensor(kind, layer, _rowmajor(shape, kind, layer, seed, sigma))
        for kind in GAINS:
            n = oracle.tensor_shape(shape, kind)[1]
            m.load_tensor(kind, layer, torch.ones(n, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    diff = (m.buf != ref.buf).nonzero()
    assert diff.numel() == 0, f"{diff.numel()} bytes differ, first at {int(diff[0])}"
    # and the loaded model computes the same verify logits
    gamma, P = 8, 20
    toks = to_dev_i32(W.prompt(3, P, shape.vocab))
    drafts = to_dev_i32(W.prompt(4, gamma, shape.vocab).reshape(1, gamma))
    out = []
    for model in (ref, m):
        kv = S.KVCache(model, 1, P + gamma + 4)
        ws = model.workspace(64)
        kv.prefill(0, toks, ws)
        lg = torch.empty((1, gamma + 1, shape.vocab), dtype=torch.float32, device="cuda")
        kv.verify(to_dev_i32([0]), drafts, lg, None, ws)
        out.append(lg)
    torch.cuda.synchronize()
    assert torch.equal(out[0], out[1])


def test_load_tensor_rejects_bad_kind_and_layer(S):
    m = S.Model(W.TINY)
    t = torch.zeros((W.TINY.d_model,), dtype=torch.float32, device="cuda")
    with pytest.raises(S.SDDError):
        m.load_tensor(99, 0, t)
    with pytest.raises(S.SDDError):
        m.load_tensor(T_ATTN_NORM, W.TINY.n_layers, t)
