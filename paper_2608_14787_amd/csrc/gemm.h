// GEMM building blocks shared by the 33-row stream-K kernel (decoder.hip) and
// the many-row kernel (rows.hip): launch arguments, the fragment-major K/V
// cache indexing, and the fused epilogues that run on a [rows][C] output tile.
#pragma once

#include <algorithm>
#include <type_traits>
#include <cmath>

#include "model.h"

namespace sdd {

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };

constexpr int kGemmThreads = 256;
constexpr int kXcds = 8;  // XCDs of the MI355X (32 CUs each); workgroups go to them round-robin by linear id
constexpr int kMaxPassRows = 64;  // rows per GEMM pass (TB <= 4 row tiles of 16)
// Arrival counters of split column groups sit one 128-byte line apart: the groups of a launch finish
// together, and device-scope atomics on one line serialize.
constexpr int kCntStride = 32;

struct GemmArgs {
  const char* W;  // tiled weights
  int KT;         // k-tiles per row strip
  int G;          // column groups
  int N;          // valid output columns
  const char* X;  // activations, row-major [rows][ldx], element type T
  int ldx;
  int m0, M;      // rows of this pass
  int mp;         // padded row stride of per-row scratch
  int n_wg;
  int segc;       // virtual units per column group of the plan (cost-balanced shares; 0: equal)
  int share;      // longest share (units): the stored matrix holds share x n_wg slots
  float* part;    // partial tiles [n_wg][2][M][NG*16]
  int32_t* err;   // the KV cache's sticky error word (bit3: a workgroup's internal hand-off gave up)
  int* cnt;       // arrival counter per column group (group g at cnt[g * kCntStride])
  const RowInfo* rows;
  // RMSNorm of the input rows: r_m = 1/sqrt(sum_g ss_in[g][m] / d_in + eps),
  // from per-column-group sums of squares written by the producer (NULL: none)
  const float* ss_in;
  int ss_groups, d_in;
  float eps;
  // EPI_QKV
  char* q_out;
  int hq, hkv, hd, qk_norm;
  const float* qn;
  const float* kn;
  const float* rope;
  int kv_ld;  // position stride of the K / V^T caches
  char* kc;
  char* vc;
  // EPI_RESID
  float* x;
  char* xa;
  int d;
  const float* g_next;
  float* ss_part;  // sums of squares of this GEMM's output rows per column group
  // EPI_SWIGLU
  char* ffh;
  int dff;
  // EPI_LOGITS
  float* logits;
  int V;
  float* amax_v;
  int* amax_i;
  // the forward's next GEMM (NULL: none), whose first k-steps a workgroup that
  // only contributed a partial loads into L2 before it ends
  const char* Wn;
  int KTn, Gn, ngn, nwg_n, cn;
};

template <typename T>
__device__ inline void mma_tile(const uint4& a, const uint4& b, f32x4& acc) {
  if constexpr (sizeof(T) == 2) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc, 0,
                                                  0, 0);
  } else {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, a.x), __builtin_bit_cast(float, b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, a.y), __builtin_bit_cast(float, b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, a.z), __builtin_bit_cast(float, b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__builtin_bit_cast(float, a.w), __builtin_bit_cast(float, b.w), acc, 0, 0, 0);
  }
}

// bf16 K / V caches, fragment-major.  Per (sequence, KV head) a cache holds ld positions (a multiple of
// 64) as 32-position steps of 32 x HD elements.  A step is the list of 1 KB blocks that one attention step
// loads, one block per 16-byte-per-lane load, lane-major (lane l holds elements 8 l .. 8 l + 7), so every
// load reads whole cache lines:
//   K block b * HD/32 + kk, lane 16 g + rho: K[32 s + kv_row(rho, b)][32 kk + 8 g + e],  e = 0..7
//   V block db,             lane 16 g + rho: V[32 s + 8 g + e][16 db + rho],             e = 0..7
// kv_row(rho, b) is the position that K sub-tile b feeds to MFMA row rho; it leaves the scores of lane
// group g on positions 8 g .. 8 g + 7 of the step, the positions of that lane's V block entries.
__device__ inline int kv_row(int rho, int b) { return 8 * (rho / 4) + 4 * b + rho % 4; }
__device__ inline int64_t kfrag_index(int p, int d, int HD) {
  const int i = p % 32, rho = 4 * (i / 8) + i % 4, b = (i / 4) % 2;
  return (int64_t)(p / 32) * 32 * HD + (b * (HD / 32) + d / 32) * 512 + (16 * ((d % 32) / 8) + rho) * 8 + d % 8;
}
__device__ inline int64_t vfrag_index(int p, int d, int HD) {
  const int i = p % 32;
  return (int64_t)(p / 32) * 32 * HD + (d / 16) * 512 + (16 * (i / 8) + d % 16) * 8 + i % 8;
}

template <typename T>
__device__ inline void store_t(char* base, int64_t idx, float v) {
  reinterpret_cast<T*>(base)[idx] = Elem<T>::from_f32(v);
}

// Stream-K bookkeeping (unit_start, unit_owner: model.h) is 32-bit unsigned
// arithmetic: 64-bit division is a long software sequence on this GPU.

// Loads into L2 the k-steps st0 .. st0 + NS - 1 that workgroup w of a GEMM launch
// (weights Wn stored in the order of their plan: workgroup w's i-th unit of
// ngn tiles at slot i * nwg + w) streams, wave `wave` (0..3) the k-steps that
// wave streams (local units wave + 4 st, st0 <= st < st0 + NS).  Called from a
// workgroup on XCD w mod 8: workgroups are dispatched to the XCDs round-robin,
// so the lines land in the L2 that serves them.  Plain (cached) loads whose
// values are consumed by an empty asm statement.
template <int NS = 3>
__device__ inline void prefetch_gemm_start(const char* Wn, int KTn, int Gn, int cn, int ngn, int nwg, int w_,
                                           int wave, int lane, int st0 = 0) {
  const uint32_t n = (uint32_t)nwg, w = (uint32_t)w_;
  const int nloc = (int)(unit_start(w + 1, KTn, Gn, cn, n) - unit_start(w, KTn, Gn, cn, n));
  const int nk = nloc > wave ? (nloc - wave + 3) / 4 : 0;  // this wave's units
  if (nk <= st0) return;
  const uint4* base = reinterpret_cast<const uint4*>(Wn) + (int64_t)w * ngn * kWave + lane;
  uint4 v[NS][8];  // unconditional loads (unit clamped to the wave's last, tile to the group's last)
#pragma unroll
  for (int st = 0; st < NS; ++st) {
    const int64_t i = wave + 4 * min(st0 + st, nk - 1);
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) v[st][nt] = base[(i * nwg * ngn + min(nt, ngn - 1)) * kWave];
  }
  uint32_t x = 0;
#pragma unroll
  for (int st = 0; st < NS; ++st)
#pragma unroll
    for (int nt = 0; nt < 8; ++nt) x ^= v[st][nt].x ^ v[st][nt].w;
  asm volatile("" ::"v"(x));
}

// the same for the workgroup of the same index of the forward's next GEMM
__device__ inline void prefetch_next(const GemmArgs& a, int wave, int lane) {
  prefetch_gemm_start(a.Wn, a.KTn, a.Gn, a.cn, a.ngn, a.nwg_n, blockIdx.x, wave, lane);
}

// Epilogues run on the final [rows][C] tile of one column group (LDS, row
// stride C + 4), on 4 waves (wave index taken mod 4, so that the two halves of
// an 8-wave workgroup can run two chunks of a tile at once).  Each wave owns
// rows wave, wave + 4, ... (R / 4 of them, the
// padded ones included: their results are computed and not stored), so the
// rows' work is straight-line code that the compiler interleaves.  A row's
// reductions run over its columns lane, lane + 64 and then across the wave,
// in an order that does not depend on the number of rows, so a row's result
// is the same whatever block it is verified in (floating-point contraction is
// off here, so that the compiler cannot fuse a row's operations differently in
// instantiations for different row counts).  Every global load a wave needs is
// issued before any of them is used.
// Sum over the n lanes of each aligned group of n (n in 1, 2, 4, 8, 16) by DPP row permutations, the same
// butterfly in every lane (the wave must be fully active).
template <int N>
__device__ inline float group_sum(float v) {
  if constexpr (N >= 2) v += dpp_f<kDppXor1>(v);
  if constexpr (N >= 4) v += dpp_f<kDppXor2>(v);
  if constexpr (N >= 8) v += dpp_f<kDppHalfMirror>(v);
  if constexpr (N >= 16) v += dpp_f<kDppMirror>(v);
  return v;
}

// The Q / K epilogue works on 8 consecutive dimensions per lane: LPR = C / 8
// lanes hold a row, RPI = 64 / LPR rows per pass, NIT passes over the wave's
// R / 4 rows (row wave + 4 j, j = it * RPI + lane / LPR).
template <int NG, int R>
struct QkvShape {
  static constexpr int C = NG * 16, RPW = R / 4, LPR = C / 8, RPI = kWave / LPR, NIT = (RPW + RPI - 1) / RPI;
};
// Global inputs of the Q / K epilogue of column group g (head g): the QK-norm
// gains of the lane's 8 dimensions and, for each pass, the RoPE (cos, sin) of
// those dimensions at its row's position (table [pos][C/2] of float2; dimension
// d uses entry d mod C/2), all loaded before any is used.
template <int NG, int R>
struct QkvPre {
  f32x4 gn[2];
  f32x4 cs[QkvShape<NG, R>::NIT][4];  // (cos, sin) pairs of dimensions d0 .. d0 + 7
};
template <int NG, int R>
__device__ inline void qkv_pre_load(const GemmArgs& a, int g, const RowInfo* ri_s, QkvPre<NG, R>& p) {
  using S = QkvShape<NG, R>;
  constexpr int C = S::C;
  if constexpr (C == 64 || C == 128) {
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x / kWave) & 3), lane = threadIdx.x % kWave;
    const int rsub = lane / S::LPR, d0 = 8 * (lane % S::LPR);
    const bool is_q = g < a.hq;
    p.gn[0] = p.gn[1] = f32x4{1.f, 1.f, 1.f, 1.f};
    if (g >= a.hq + a.hkv) return;  // V head: no inputs
    if (a.qk_norm) {
      const float* gp = (is_q ? a.qn : a.kn) + d0;
      p.gn[0] = *reinterpret_cast<const f32x4*>(gp);
      p.gn[1] = *reinterpret_cast<const f32x4*>(gp + 4);
    }
#pragma unroll
    for (int it = 0; it < S::NIT; ++it) {
      const int mm = wave + 4 * min(it * S::RPI + rsub, S::RPW - 1);
      const RowInfo ri = ri_s[mm < a.M ? mm : 0];
      const f32x4* t = reinterpret_cast<const f32x4*>(a.rope + ((size_t)(ri.valid ? ri.pos : 0) * (C / 2) + d0 % (C / 2)) * 2);
#pragma unroll
      for (int k = 0; k < 4; ++k) p.cs[it][k] = t[k];
    }
  }
}

template <typename T, int NG, int R>
__device__ void epilogue_qkv(const GemmArgs& a, const float* tile, int g, const float* rsl, const RowInfo* ri_s) {
  // no contraction: every instantiation (row count) must round each row alike
#pragma clang fp contract(off)
  constexpr int C = NG * 16;  // == head_dim
  constexpr int CP = C + 4, RPW = R / 4;
  if constexpr (C == 64 || C == 128) {
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x / kWave) & 3), lane = threadIdx.x % kWave;
    const int h = g;
    const bool is_q = h < a.hq, is_k = !is_q && h < a.hq + a.hkv;
    if (!is_q && !is_k) {
      // V head: lane = row, so that consecutive positions of a cached
      // dimension are written together (adjacent in both cache layouts)
      const int mm = lane;
      const bool ok = mm < a.M && ri_s[mm < a.M ? mm : 0].valid;
      const RowInfo ri = ri_s[mm < a.M ? mm : 0];
      const float r = rsl[mm < a.M ? mm : 0];
      const int64_t head = (int64_t)ri.seq * a.hkv + (h - a.hq - a.hkv);
      constexpr int DPW = C / 4;  // dimensions per wave
#pragma unroll 8
      for (int dd = 0; dd < DPW; ++dd) {
        const int dim = wave * DPW + dd;
        const float y = tile[(mm < R ? mm : 0) * CP + dim] * r;
        if (ok) {
          if constexpr (sizeof(T) == 2)
            store_t<T>(a.vc, head * a.kv_ld * C + vfrag_index(ri.pos, dim, C), y);
          else
            store_t<T>(a.vc, (head * C + dim) * a.kv_ld + ri.pos, y);  // fp32: V^T rows
        }
      }
      return;
    }
    using S = QkvShape<NG, R>;
    QkvPre<NG, R> pp;
    qkv_pre_load<NG, R>(a, g, ri_s, pp);
    const int rsub = lane / S::LPR, d0 = 8 * (lane % S::LPR);
    const bool lo = d0 < C / 2;  // the rotation pairs dimension d with d + C/2
#pragma unroll
    for (int it = 0; it < S::NIT; ++it) {
      const int j = it * S::RPI + rsub, mm = wave + 4 * j;
      const int mt = wave + 4 * min(j, RPW - 1);  // tile row (a valid one for the last pass's spare lanes)
      const float r = rsl[mt < a.M ? mt : 0];
      const f32x4 t0 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + d0]);
      const f32x4 t1 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + d0 + 4]);
      float y[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y[e] = t0[e] * r;
        y[4 + e] = t1[e] * r;
      }
      if (a.qk_norm) {
        float ss = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += y[e] * y[e];
        ss = group_sum<S::LPR>(ss);
        const float inv = 1.f / sqrtf(ss / (float)C + a.eps);
#pragma unroll
        for (int e = 0; e < 8; ++e) y[e] *= inv * (e < 4 ? pp.gn[0][e] : pp.gn[1][e - 4]);
      }
      // the partner dimensions (d +- C/2) sit LPR / 2 lanes away in the row's lane group
      float o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if constexpr (C == 128)
          o[e] = dpp_f<kDppRor8>(y[e]);
        else
          o[e] = __shfl_xor(y[e], S::LPR / 2);
      }
      float z[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = pp.cs[it][e / 2][2 * (e % 2)], sn = pp.cs[it][e / 2][2 * (e % 2) + 1];
        z[e] = lo ? y[e] * c - o[e] * sn : y[e] * c + o[e] * sn;
      }
      if (j < RPW && mm < a.M && ri_s[mm].valid) {
        const RowInfo ri = ri_s[mm];
        int64_t off;  // element offset of the lane's 8 dimensions (16-byte aligned, contiguous)
        char* base;
        if (is_q) {
          base = a.q_out;
          off = ((int64_t)(a.m0 + mm) * a.hq + h) * C + d0;
        } else if constexpr (sizeof(T) == 2) {
          base = a.kc;
          off = ((int64_t)ri.seq * a.hkv + (h - a.hq)) * a.kv_ld * C + kfrag_index(ri.pos, d0, C);
        } else {
          base = a.kc;
          off = (((int64_t)ri.seq * a.hkv + (h - a.hq)) * a.kv_ld + ri.pos) * C + d0;  // fp32: [pos][hd]
        }
        if constexpr (sizeof(T) == 2) {
          *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(base) + off) =
              make_uint4(pack_bf16x2(z[0], z[1]), pack_bf16x2(z[2], z[3]), pack_bf16x2(z[4], z[5]), pack_bf16x2(z[6], z[7]));
        } else {
          float* dst = reinterpret_cast<float*>(base) + off;
          *reinterpret_cast<f32x4*>(dst) = f32x4{z[0], z[1], z[2], z[3]};
          *reinterpret_cast<f32x4*>(dst + 4) = f32x4{z[4], z[5], z[6], z[7]};
        }
      }
    }
  }
}


// Residual epilogue, 8 consecutive columns per lane: LPR = C / 8 lanes hold a row (16-byte loads and
// stores), RPI = 64 / LPR rows per pass; a row's sum of squares adds the lane's 8 squares in column order,
// then the LPR lanes by a fixed butterfly.
template <typename T, int NG, int R>
__device__ void epilogue_resid(const GemmArgs& a, const float* tile, int g) {
  // no contraction: every instantiation (row count) must round each row alike
#pragma clang fp contract(off)
  constexpr int C = NG * 16, CP = C + 4, RPW = R / 4;
  constexpr int LPR = C / 8, RPI = kWave / LPR, NIT = (RPW + RPI - 1) / RPI;
  const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x / kWave) & 3), lane = threadIdx.x % kWave;
  const int rsub = lane / LPR, c0 = 8 * (lane % LPR);
  const int64_t n0 = (int64_t)g * C + c0;
  const f32x4 gv0 = *reinterpret_cast<const f32x4*>(a.g_next + n0), gv1 = *reinterpret_cast<const f32x4*>(a.g_next + n0 + 4);
  // every pass's residual loads first (padded rows read row 0)
  f32x4 xa0[NIT], xa1[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = it * RPI + rsub, mm = wave + 4 * j;
    const int mc = (j < RPW && mm < a.M) ? mm : 0;
    const float* xr = a.x + (int64_t)(a.m0 + mc) * a.d + n0;
    xa0[it] = *reinterpret_cast<const f32x4*>(xr);
    xa1[it] = *reinterpret_cast<const f32x4*>(xr + 4);
  }
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = it * RPI + rsub, mm = wave + 4 * j;
    const int mt = wave + 4 * min(j, RPW - 1);  // tile row (a valid one for the last pass's spare lanes)
    const f32x4 t0 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + c0]);
    const f32x4 t1 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + c0 + 4]);
    float xv[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xv[e] = xa0[it][e] + t0[e];
      xv[4 + e] = xa1[it][e] + t1[e];
    }
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += xv[e] * xv[e];
    ss = group_sum<LPR>(ss);
    if (j < RPW && mm < a.M) {
      const int m = a.m0 + mm;
      float* xr = a.x + (int64_t)m * a.d + n0;
      *reinterpret_cast<f32x4*>(xr) = f32x4{xv[0], xv[1], xv[2], xv[3]};
      *reinterpret_cast<f32x4*>(xr + 4) = f32x4{xv[4], xv[5], xv[6], xv[7]};
      float y[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        y[e] = xv[e] * gv0[e];
        y[4 + e] = xv[4 + e] * gv1[e];
      }
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.xa) + (int64_t)m * a.d + n0) =
            make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]), pack_bf16x2(y[6], y[7]));
      } else {
        float* ar = reinterpret_cast<float*>(a.xa) + (int64_t)m * a.d + n0;
        *reinterpret_cast<f32x4*>(ar) = f32x4{y[0], y[1], y[2], y[3]};
        *reinterpret_cast<f32x4*>(ar + 4) = f32x4{y[4], y[5], y[6], y[7]};
      }
      if (lane % LPR == 0) a.ss_part[(int64_t)g * a.mp + m] = ss;
    }
  }
}

// SwiGLU epilogue: the group's C columns are P = NG / 2 pairs of 16 gate and 16 up columns, i.e. P * 16
// hidden outputs per row; a lane computes 8 consecutive ones (LPR = NG lanes per row, RPI = 64 / LPR rows
// per pass) and stores them with one 16-byte store.
template <typename T, int NG, int R>
__device__ void epilogue_swiglu(const GemmArgs& a, const float* tile, int g, const float* rsl) {
  // no contraction: every instantiation (row count) must round each row alike
#pragma clang fp contract(off)
  constexpr int C = NG * 16, CP = C + 4, P = NG / 2, RPW = R / 4;
  constexpr int LPR = P * 2, RPI = kWave / LPR, NIT = (RPW + RPI - 1) / RPI;
  static_assert(NG % 2 == 0, "gate/up groups hold whole pairs");
  const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x / kWave) & 3), lane = threadIdx.x % kWave;
  const int rsub = lane / LPR, h0 = 8 * (lane % LPR);      // first hidden column of the lane
  const int cg = (h0 / 16) * 32 + h0 % 16, cu = cg + 16;  // its gate and up tile columns
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = it * RPI + rsub, mm = wave + 4 * j;
    const int mt = wave + 4 * min(j, RPW - 1);
    const float r = rsl[mt];
    const f32x4 g0 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + cg]);
    const f32x4 g1 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + cg + 4]);
    const f32x4 u0 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + cu]);
    const f32x4 u1 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + cu + 4]);
    float hv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float gt = (e < 4 ? g0[e] : g1[e - 4]) * r;
      const float up = (e < 4 ? u0[e] : u1[e - 4]) * r;
      hv[e] = gt / (1.f + expf(-gt)) * up;
    }
    if (j < RPW && mm < a.M) {
      const int64_t off = (int64_t)(a.m0 + mm) * a.dff + (int64_t)g * P * 16 + h0;
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.ffh) + off) =
            make_uint4(pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3]), pack_bf16x2(hv[4], hv[5]),
                       pack_bf16x2(hv[6], hv[7]));
      } else {
        float* hr = reinterpret_cast<float*>(a.ffh) + off;
        *reinterpret_cast<f32x4*>(hr) = f32x4{hv[0], hv[1], hv[2], hv[3]};
        *reinterpret_cast<f32x4*>(hr + 4) = f32x4{hv[4], hv[5], hv[6], hv[7]};
      }
    }
  }
}

__device__ inline bool arg_better(float v2, int i2, float v1, int i1) {
  if (i2 < 0 || v2 != v2) return false;
  if (i1 < 0) return true;
  return v2 > v1 || (v2 == v1 && i2 < i1);
}

// Best (value, lowest index) over the n lanes of each aligned group of n (n in 1, 2, 4, 8, 16), left in
// every lane of the group; the combine is associative and commutative, so the butterfly's order is free.
template <int N>
__device__ inline void group_argmax(float& bv, int& bi) {
  auto step = [&](auto ctrl) {
    constexpr int CTRL = decltype(ctrl)::value;
    const float v2 = dpp_f<CTRL>(bv);
    const int i2 = dpp_i<CTRL>(bi);
    if (arg_better(v2, i2, bv, bi)) {
      bv = v2;
      bi = i2;
    }
  };
  if constexpr (N >= 2) step(std::integral_constant<int, kDppXor1>{});
  if constexpr (N >= 4) step(std::integral_constant<int, kDppXor2>{});
  if constexpr (N >= 8) step(std::integral_constant<int, kDppHalfMirror>{});
  if constexpr (N >= 16) step(std::integral_constant<int, kDppMirror>{});
}

// LM-head epilogue: fp32 logits of the valid rows and each row's best (value, index) over the group's
// columns below V.  A lane takes 8 consecutive columns (LPR = C / 8 lanes per row, RPI = 64 / LPR rows per
// pass): 16-byte stores where V keeps rows 16-byte aligned and the 8 columns are all below V.
template <int NG, int R>
__device__ void epilogue_logits(const GemmArgs& a, const float* tile, int g, const float* rsl, const RowInfo* ri_s) {
  // no contraction: every instantiation (row count) must round each row alike
#pragma clang fp contract(off)
  constexpr int C = NG * 16, CP = C + 4, RPW = R / 4;
  constexpr int LPR = C / 8, RPI = kWave / LPR, NIT = (RPW + RPI - 1) / RPI;
  static_assert(LPR <= 16, "a row's lanes must lie in one DPP row");
  const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x / kWave) & 3), lane = threadIdx.x % kWave;
  const int rsub = lane / LPR, c0 = 8 * (lane % LPR), n0 = g * C + c0;
  const bool vec = (a.V & 3) == 0 && n0 + 8 <= a.V;
  float bv[NIT];
  int bi[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int j = it * RPI + rsub, mm = wave + 4 * j;
    const int mt = wave + 4 * min(j, RPW - 1);
    const float r = rsl[mt < a.M ? mt : 0];
    const f32x4 t0 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + c0]);
    const f32x4 t1 = *reinterpret_cast<const f32x4*>(&tile[mt * CP + c0 + 4]);
    float v[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = t0[e] * r;
      v[4 + e] = t1[e] * r;
    }
    bv[it] = -INFINITY;
    bi[it] = -1;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (n0 + e < a.V && arg_better(v[e], n0 + e, bv[it], bi[it])) {
        bv[it] = v[e];
        bi[it] = n0 + e;
      }
    if (j < RPW && mm < a.M && ri_s[mm].valid) {
      float* lr = a.logits + (int64_t)(a.m0 + mm) * a.V + n0;
      if (vec) {
        *reinterpret_cast<f32x4*>(lr) = f32x4{v[0], v[1], v[2], v[3]};
        *reinterpret_cast<f32x4*>(lr + 4) = f32x4{v[4], v[5], v[6], v[7]};
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (n0 + e < a.V) lr[e] = v[e];
      }
    }
    group_argmax<LPR>(bv[it], bi[it]);
  }
  // one lane per row, so the rows' candidates take two store instructions, not
  // two per row: with the next segment's loads in flight, a wave's outstanding
  // memory operations would otherwise exceed the 63 the counter holds, and
  // issue would stall until those loads land
  float av = 0.f;
  int ai = -1;
#pragma unroll
  for (int it = 0; it < NIT; ++it)
#pragma unroll
    for (int q = 0; q < RPI; ++q) {
      const int j = it * RPI + q;
      if (j < RPW) {
        const float v2 = lane_f(bv[it], q * LPR);
        const int i2 = __builtin_amdgcn_readlane(bi[it], q * LPR);
        if (lane == j) {
          av = v2;
          ai = i2;
        }
      }
    }
  const int mm = wave + 4 * lane;
  if (lane < RPW && mm < a.M) {
    a.amax_v[(int64_t)g * a.mp + a.m0 + mm] = av;
    a.amax_i[(int64_t)g * a.mp + a.m0 + mm] = ai;
  }
}

// Many-row GEMM (rows.hip): bf16 weights, column groups of 8 or 4 tiles, up to
// kRowsMaxRows rows [a.m0, a.m0 + a.M) per launch of nblocks workgroups (the
// stream-K partition of a.G x a.KT units); fused epilogue `epi`.  Partial
// tiles need kRowsPartBytes per workgroup in a.part.  Returns SDD_OK or
// SDD_EUNSUPPORTED (other group widths, too many rows).
constexpr int kRowsMaxTBW = 5;     // row tiles per computing wave
constexpr int kRowsMaxRows = 288;  // rows per launch: the final tile of 288 x 132 fp32 fits the 160 KB of LDS
constexpr size_t kRowsPartBytes = (size_t)2 * 2 * kRowsMaxTBW * 8 * 4 * 64 * 16;  // 2 slots x a pair of 8-tile groups
int launch_gemm_rows(int ng, int epi, const GemmArgs& a, int nblocks, hipStream_t st);

}  // namespace sdd
