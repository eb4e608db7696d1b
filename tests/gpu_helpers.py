"""Helpers shared by the GPU tests (no method arithmetic)."""
import numpy as np
import torch

import workloads as W


def untile(buf: np.ndarray, rows: int, cols: int, dtype: str) -> np.ndarray:
    """Decodes libsdd's documented tiled weight layout back to a row-major [rows][cols] matrix.

    Tiles of 16 rows x ktile columns (ktile 32 for bf16, 16 for fp32), 1 KiB each; tile (nt, kt) at
    index kt * NT + nt (k-step major, NT = ceil(rows / 16)); lane l of a tile holds row l%16 and
    EPL = 16/sizeof(elem) columns from (l//16)*EPL."""
    es = 2 if dtype == "bf16" else 4
    epl = 16 // es
    kt = 4 * epl
    NT, KT = -(-rows // 16), -(-cols // kt)
    if dtype == "bf16":
        vals = W.bf16_bits_to_f32(buf[: NT * KT * 1024].view(np.uint16))
    else:
        vals = buf[: NT * KT * 1024].view(np.float32)
    a = vals.reshape(KT, NT, 4, 16, epl).transpose(1, 3, 0, 2, 4).reshape(NT * 16, KT * kt)
    return a[:rows, :cols]


def to_dev_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def row_tol_ok(got: np.ndarray, want: np.ndarray, rel: float):
    """Per-row max |got - want| <= rel * max |want| (the logit-scale tolerance)."""
    err = np.abs(got - want).max(-1)
    scale = np.abs(want).max(-1)
    return err <= rel * scale, err / scale


def argmax_near_tie(z: np.ndarray, tol: np.ndarray) -> np.ndarray:
    """True where the top-2 gap of a row is below tol (an argmax that rounding may flip)."""
    s = np.sort(z, axis=-1)
    return (s[..., -1] - s[..., -2]) < tol


# tensor kinds of include/sdd.h for the norm gains (the oracle numbers them alike)
_GAIN_KIND = {"final": 2, "attn": 10, "ffn": 11, "q": 12, "k": 13}


def load_gains(model, gains: dict):
    """Loads workloads.norm_gains into a GPU model (sdd_model_load_tensor)."""
    for (name, layer), v in gains.items():
        model.load_tensor(_GAIN_KIND[name], layer, torch.from_numpy(np.ascontiguousarray(v, np.float32)).cuda())


def oracle_gains(om, gains: dict):
    """The same gains into an oracle model (orc_model_set_tensor)."""
    for (name, layer), v in gains.items():
        om.set_tensor(_GAIN_KIND[name], layer, v)
