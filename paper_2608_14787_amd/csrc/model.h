// Device data layout of the target decoder, the KV cache and the per-call
// workspace (internal to libsdd).
#pragma once

#include "sdd_internal.h"

// Weight matrices ([out][in] = [N][K]) are stored as 1 KiB tiles of 16 rows x
// KT columns (KT = 32 for bf16, 16 for fp32).  Inside a tile, lane l of a wave
// reads 16 contiguous bytes holding row (l % 16) and the EPL = 16/sizeof(T)
// consecutive columns starting at (l / 16) * EPL: exactly one MFMA A-operand
// fragment per lane, so a wave streams a tile with one coalesced 16-byte load
// per lane.  Tiles are stored k-step by k-step: tile (nt, kt) sits at index
// kt * NT + nt (NT = N / 16 row tiles), so one k-step of a column group (NG
// consecutive row tiles, NG in {8, 4, 2} per matrix) is NG KiB of contiguous
// memory and one k-step of the whole matrix is one contiguous run.  Q, K and V projections are fused into one
// matrix (rows [Wq; Wk; Wv]); gate and up projections are fused and
// interleaved per 16-row tile (tile 2t = gate rows 16t.., tile 2t+1 = up rows
// 16t..), so that one column group holds matching gate/up outputs.
struct sdd_model {
  sdd_model_config cfg;
  char* base;
  size_t bytes;
  int es;    // element size of weights/activations: 2 (bf16) or 4 (fp32)
  int ktile; // columns per tile
  int n_cu;  // compute units of the device
  size_t off_embed, off_lm, off_final_norm;
  int ng_qkv, ng_o, ng_gu, ng_down, ng_lm;  // row tiles per column group
  struct Layer {
    size_t qkv, o, gu, down, attn_norm, ffn_norm, q_norm, k_norm;
  };
  Layer* layers;
};

struct sdd_kv {
  sdd_model* m;
  int max_batch, max_len;
  int ld;            // position stride of the caches: max_len rounded up to 64 (128-byte V^T rows)
  char* base;
  size_t bytes;
  int32_t* len;      // [max_batch]
  int32_t* pending;  // [max_batch]
  int32_t* err;      // sticky error bits
  float* rope;       // [max_len][head_dim/2][2] (cos, sin)
  char* k;           // [layers][max_batch][n_kv_heads][ld][head_dim]
  char* v;           // [layers][max_batch][n_kv_heads][head_dim][ld] (transposed)
  size_t layer_stride;  // bytes per layer of k (and of v)
};

namespace sdd {
inline int kv_ld(int max_len) { return (max_len + 63) / 64 * 64; }
}  // namespace sdd

namespace sdd {

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Row tiles per column group: the largest of 8, 4, 2 (at most max_ng) dividing
// the tile count (even for the gate/up interleave, which pairs tiles).
inline int pick_ng(int64_t ntiles, bool pairs, int max_ng = 8) {
  for (int ng : {8, 4, 2})
    if (ng <= max_ng && ntiles % ng == 0 && (!pairs || ng % 2 == 0)) return ng;
  return pairs ? 2 : 1;
}

// tiled matrix bytes
inline size_t tiled_bytes(int64_t N, int64_t K, int ktile) {
  return (size_t)ceil_div(N, 16) * (size_t)ceil_div(K, ktile) * 1024;
}

struct RowInfo {
  int seq;    // KV slot
  int pos;    // absolute position
  int valid;  // 0: refused (capacity), rows of that block are skipped
  int pad;
};

// Per-call workspace carve-up for up to max_rows rows.
struct WsLayout {
  size_t rowinfo, x, xa, ss_part, q, ao, ffh, part, cnt, amax, total;
  int mp;         // padded rows
  int max_groups; // column groups of the widest GEMM
  int n_wg;       // GEMM workgroups
};

WsLayout ws_layout(const sdd_model* m, int max_rows);

}  // namespace sdd
