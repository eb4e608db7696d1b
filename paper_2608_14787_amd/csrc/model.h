// Device data layout of the target decoder, the KV cache and the per-call
// workspace (internal to libsdd).
#pragma once

#include <algorithm>

#include "sdd_internal.h"

// Weight matrices ([out][in] = [N][K]) are stored as 1 KiB tiles of 16 rows x
// KT columns (KT = 32 for bf16, 16 for fp32).  Inside a tile, lane l of a wave
// reads 16 contiguous bytes holding row (l % 16) and the EPL = 16/sizeof(T)
// consecutive columns starting at (l / 16) * EPL: exactly one MFMA A-operand
// fragment per lane, so a wave streams a tile with one coalesced 16-byte load
// per lane.  A column group is NG consecutive row tiles (NG in {8, 4, 2} per
// matrix); one k-step of a group (NG tiles, NG KiB) is the GEMM's unit of work.
// The units (g, kt) of a matrix are split over the n_wg workgroups of its
// streaming plan (MatPlan: workgroup w owns the units u = g * KT + kt in
// [w U / n_wg, (w + 1) U / n_wg), U = G * KT), and the matrix is stored in the
// order the plan streams it: the i-th unit of workgroup w at slot i * n_wg + w.
// A workgroup's units are then n_wg slots apart, and since all workgroups
// stream at about the same rate, the whole launch reads one narrow window of
// memory at a time (measured: the gate/up launch 7-10% faster than with every
// k-step of the matrix contiguous, when workgroups start at unrelated k-steps).
// Q, K and V projections are fused into one matrix (rows [Wq; Wk; Wv]); gate
// and up projections are fused and interleaved per 16-row tile (tile 2t = gate
// rows 16t.., tile 2t+1 = up rows 16t..), so that one column group holds
// matching gate/up outputs.
namespace sdd {

// A split group costs one tail (partial publish, last-arriver reduction,
// epilogue); splitting every group into equal k-ranges pays when the longer
// share streams for less than this.
constexpr double kTailStreamBytes = 224.0 * 1024;
// Stream-K shares are balanced by cost rather than by units: every segment
// (one column group's part of a share) beyond the first costs a workgroup a
// cross-wave reduction and a partial publish or an epilogue, about as long as
// streaming this many bytes (measured: gate/up workgroups whose share touches
// three groups ended their stream ~4 us after those touching two).
constexpr int kSegmentCostBytes = 96 * 1024;

// Streaming plan of one weight matrix: KT k-steps of G column groups of ng row
// tiles over n_wg workgroups.  With more groups than CUs, stream-K: each group
// counts as KT + c units, the c leading ones virtual (the cost of entering one
// more group), the virtual range V = G (KT + c) is split into n_wg equal shares
// and mapped back onto the real units, so that a share touching one more group
// holds c fewer real units.  With at most one group per CU, equal shares would
// leave about a third of the workgroups straddling two groups, each paying a
// second tail; then every group is split into s = n_cu / G equal k-ranges over
// G x s workgroups (one segment each, c = 0) when the longer share costs less
// stream time than one tail.  S is the longest share (units).
struct MatPlan {
  int KT, G, ng, n_wg, c, S;
};

// First unit of workgroup w's share (unit u = g * KT + kt), from the virtual
// position x = w V / n_wg: its group x / (KT + c), its offset past the group's
// c virtual units.  32-bit: V * n_wg < 2^31 is checked on the host.  c = 0:
// the equal shares [w U / n_wg, (w + 1) U / n_wg) of U = G * KT units.
__host__ __device__ inline uint32_t unit_start(uint32_t w, uint32_t KT, uint32_t G, uint32_t c, uint32_t n) {
  if (c == 0) return w * (G * KT) / n;  // (one division: this runs before a launch's first loads)
  const uint32_t L = KT + c, x = w * (G * L) / n, g = x / L, o = x - g * L;
  return g * KT + (o > c ? o - c : 0);
}
// The workgroup whose share holds unit u: the one whose virtual range holds u's
// virtual position g (KT + c) + c + kt.
__host__ __device__ inline int unit_owner(uint32_t u, uint32_t KT, uint32_t G, uint32_t c, uint32_t n) {
  const uint32_t V = G * (KT + c), x = c ? u + (u / KT + 1) * c : u;
  return (int)(((x + 1) * n + V - 1) / V) - 1;
}

inline MatPlan plan_matrix(int64_t N, int64_t K, int ktile, int ng, int n_cu) {
  MatPlan p;
  p.KT = (int)ceil_div(K, ktile);
  p.ng = ng;
  p.G = (int)(ceil_div(N, 16) / ng);
  p.c = 0;
  const int64_t U = (int64_t)p.G * p.KT;
  p.n_wg = (int)std::min<int64_t>(U, n_cu);
  if (p.G <= n_cu) {
    const int s = std::min(n_cu / p.G, p.KT);
    const double extra_units = (double)p.KT / s - (double)U / p.n_wg;
    if (extra_units * ng * 1024 < kTailStreamBytes) p.n_wg = p.G * s;
  }
  auto shares = [&](int c, int& lo, int& hi) {
    lo = p.KT, hi = 0;
    for (int w = 0; w < p.n_wg; ++w) {
      const int n = (int)(unit_start(w + 1, p.KT, p.G, c, p.n_wg) - unit_start(w, p.KT, p.G, c, p.n_wg));
      lo = std::min(lo, n), hi = std::max(hi, n);
    }
  };
  int lo, hi;
  if (p.n_wg < p.G && (int64_t)p.G * (p.KT + kSegmentCostBytes / (ng * 1024)) * p.n_wg < (int64_t(1) << 31)) {
    // cost-balanced shares where no share is left without a real unit
    p.c = kSegmentCostBytes / (ng * 1024);
    shares(p.c, lo, hi);
    if (lo < 1) p.c = 0;
  }
  shares(p.c, lo, hi);
  p.S = hi;
  return p;
}

// slots of the stored matrix: the longest share times n_wg (shorter shares leave empty slots at the end)
__host__ __device__ inline int64_t plan_slots(const MatPlan& p) { return (int64_t)p.S * p.n_wg; }
inline size_t plan_bytes(const MatPlan& p) { return (size_t)plan_slots(p) * p.ng * 1024; }

// slot of unit (g, kt)
__host__ __device__ inline int64_t plan_slot(const MatPlan& p, int g, int kt) {
  const uint32_t u = (uint32_t)g * p.KT + kt;
  const int w = unit_owner(u, p.KT, p.G, p.c, p.n_wg);
  return (int64_t)(u - unit_start(w, p.KT, p.G, p.c, p.n_wg)) * p.n_wg + w;
}

}  // namespace sdd

struct sdd_model {
  sdd_model_config cfg;
  char* base;
  size_t bytes;
  int es;    // element size of weights/activations: 2 (bf16) or 4 (fp32)
  int ktile; // columns per tile
  int n_cu;  // compute units of the device
  size_t off_embed, off_lm, off_final_norm;
  int ng_qkv, ng_o, ng_gu, ng_down, ng_lm;  // row tiles per column group
  sdd::MatPlan plan_qkv, plan_o, plan_gu, plan_down, plan_lm;  // streaming plans (and storage order)
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
