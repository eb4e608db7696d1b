"""Helpers shared by the GPU tests (no method arithmetic)."""
import numpy as np
import torch

import workloads as W


def share_starts(KT: int, G: int, c: int, nwg: int) -> np.ndarray:
    """start(w) for w = 0..n_wg of the documented stream-K plan (sdd_model_matrix_layout): each column group
    counts as KT + c units, the virtual range is split into n_wg equal parts, and a virtual position x maps to
    unit g*KT + max(0, o - c) with g = x // (KT + c), o = x % (KT + c)."""
    L = KT + c
    x = np.arange(nwg + 1, dtype=np.int64) * (G * L) // nwg
    return x // L * KT + np.maximum(0, x % L - c)


def untile(buf: np.ndarray, layout: dict, rows: int, cols: int, dtype: str) -> np.ndarray:
    """Decodes libsdd's documented tiled weight layout (sdd_model_matrix_layout) back to a row-major
    [rows][cols] matrix.

    Tiles of 16 rows x kt columns (kt 32 for bf16, 16 for fp32), 1 KiB each; lane l of a tile holds row l%16
    and 16/elem columns from (l//16)*16/elem.  Unit (g, k) = the ng row tiles of column group g at k-step k;
    workgroup w of n_wg owns units [start(w), start(w+1)) of U = G*KT (u = g*KT + k; share_starts), and its
    i-th unit sits at slot i*n_wg + w; tile j of a unit at byte offset + (slot*ng + j)*1024."""
    es = 2 if dtype == "bf16" else 4
    epl = 16 // es
    kt = 4 * epl
    KT, G, ng, nwg = layout["KT"], layout["G"], layout["ng"], layout["n_wg"]
    U = G * KT
    st = share_starts(KT, G, layout["c"], nwg)
    u = np.arange(U, dtype=np.int64)
    w = np.searchsorted(st[1:], u, side="right")  # owner of unit u
    slot = (u - st[w]) * nwg + w
    raw = buf[layout["offset"]: layout["offset"] + layout["bytes"]]
    if dtype == "bf16":
        vals = W.bf16_bits_to_f32(raw.view(np.uint16))
    else:
        vals = raw.view(np.float32)
    tiles = vals.reshape(-1, ng, 4, 16, epl)[slot]            # [U = (g, k)][ng][lane group][row][epl]
    a = tiles.reshape(G, KT, ng, 4, 16, epl).transpose(0, 2, 4, 1, 3, 5).reshape(G * ng * 16, KT * kt)
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
