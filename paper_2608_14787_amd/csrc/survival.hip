// Survival predictor inference (Appendix "Predictor Details"; its sigmoid output is the marginal or
// conditional survival score of Sec. 4.2): per draft position x = [h, s] (the drafter's LM-head input and
// the scalar features), normalized as (x - mu) / sigma, then d_in -> H -> H -> H -> 1 with GELU (erf form)
// after each hidden layer; the output is log sigmoid(z), the log position score the skip scheduler reads.
//
// One launch; every contraction on fp32 MFMA (v_mfma_f32_16x16x4_f32, weights as the A operand so a wave's
// accumulators hold 16 output columns x 16 positions).  The grid holds three sets of workgroups, in id order:
//   layer 1:    (16-column tile, k-split, 64-row tile) per workgroup; the input slice is normalized while it is
//               staged into LDS; partial tiles are published with device-coherent 16-byte stores and the last
//               arriving split of a tile adds them in split order, adds the bias, applies GELU, writes its h1
//               tile and counts it done for its row tile;
//   layer 2:    (16-column tile, 64-row tile) per workgroup over K = H, bias + GELU, once every h1 tile of its
//               row tile is done; counts its h2 tile done;
//   layer 3(+4): the same from h2, then each tile's share of w4 . h3; the last tile of a row tile adds the
//               shares in tile order, adds b4 and writes log sigmoid(z).
// A workgroup of layers 2 and 3 waits for its inputs by polling a counter (bounded; past the bound the scores
// come out NaN, and stay so).  Workgroups are dispatched in id order, so every workgroup it waits for was
// dispatched before it: the wait never holds a compute unit that those need.  Hidden activations move
// through device-coherent stores and loads.  The k-order of every sum is fixed, so results are
// bit-reproducible.
#include "sdd_internal.h"

namespace sdd {
namespace {

constexpr int kMlpThreads = 256;
constexpr int kRowTile = 64;   // positions per workgroup (4 waves x 16)
constexpr int kKc = 128;       // k-chunk staged in LDS by layer 1
constexpr int kMaxH = 256;
constexpr int kCntLine = 32;  // ints per 128-byte line

struct MlpArgs {
  const uint16_t* hidden;  // [n][d_hid] bf16
  const float* scalars;    // [n][n_sc]
  const float *mu, *sigma, *W1, *b1, *W2, *b2, *W3, *b3, *w4;
  float b4;
  int n, d_hid, n_sc, d_in, H;
  int S, kc_split;  // layer-1 k-splits and k per split (a multiple of kKc)
  float* part;      // layer-1 partial tiles [rt][ct][S][64][16]
  float* h1;        // [rt*64][H]
  float* h2;
  float* zpart;     // [rt][ct][64]
  // counters one 128-byte line apart (index x at [x * kCntLine]): the workgroups that count on them, and
  // those polling them, do so at about the same time, and device-scope atomics on one line serialize
  int* cnt1;        // [rt][ct]
  int* cnt3;        // [rt]
  int* done1;       // [rt]: h1 tiles written
  int* done2;       // [rt]: h2 tiles written
  int* err;         // sticky: a wait ran past its bound
  float* log_score;
  float* logit;
};

#pragma clang fp contract(off)
__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }
__device__ inline float log_sigmoid(float z) { return z >= 0.f ? -log1pf(__expf(-z)) : z - log1pf(__expf(z)); }
// h . w over 4 consecutive columns, added left to right
__device__ inline float dot4(const float* h, const float* w) { return ((h[0] * w[0] + h[1] * w[1]) + h[2] * w[2]) + h[3] * w[3]; }
#pragma clang fp contract(on)

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) { return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0); }

constexpr int kSpinMax = 1 << 17;  // polls of a wait (each after a short sleep): tens of milliseconds

// Thread 0 polls *cnt until it reaches `target` (device-coherent loads), within a bound; true (in every
// thread) when it did.
__device__ bool wait_count(const int* cnt, int target, int* s_flag) {
  if (threadIdx.x == 0) {
    int ok = 0;
    for (int it = 0; it < kSpinMax; ++it) {
      if (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target) {
        ok = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(4);
    }
    *s_flag = ok;
  }
  __syncthreads();
  return *s_flag != 0;
}

// Counts one tile done (after this workgroup's coherent stores have completed).
__device__ void count_done(int* cnt) {
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ void layer1_body(const MlpArgs& a, int bid, float* smem, int* s_flag) {
  float (*sW)[kKc + 1] = reinterpret_cast<float (*)[kKc + 1]>(smem);
  float (*sX)[kKc + 1] = reinterpret_cast<float (*)[kKc + 1]>(smem + 16 * (kKc + 1));
  const int CT = a.H / 16;
  const int ct = bid % CT, s = (bid / CT) % a.S, rt = bid / (CT * a.S);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int c0 = ct * 16, r0 = rt * kRowTile;
  const int kb = s * a.kc_split, ke = min(a.d_in, kb + a.kc_split);
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = kb; k0 < ke; k0 += kKc) {
    // stage W1[c0..c0+16)[k0..k0+kKc) and the normalized inputs of 64 rows (zeros past d_in and n).
    // Thread t always takes column k = k0 + t % kKc, rows (or weight columns) t / kKc + 2 u: every load of
    // the chunk is issued before any is used.
    const int kl = tid % kKc, k = k0 + kl, rsub = tid / kKc;
    const bool kin = k < ke;
    float wv[16 / 2], xv[kRowTile / 2];
#pragma unroll
    for (int u = 0; u < 8; ++u) wv[u] = kin ? a.W1[(int64_t)(c0 + rsub + 2 * u) * a.d_in + k] : 0.f;
    const bool hid = k < a.d_hid;
#pragma unroll
    for (int u = 0; u < kRowTile / 2; ++u) {
      const int row = r0 + rsub + 2 * u;
      float raw = 0.f;
      if (kin && row < a.n)
        raw = hid ? bf16_to_f32(a.hidden[(int64_t)row * a.d_hid + k]) : a.scalars[(int64_t)row * a.n_sc + (k - a.d_hid)];
      xv[u] = raw;
    }
    const float mu = kin ? a.mu[k] : 0.f, sg = kin ? a.sigma[k] : 1.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) sW[rsub + 2 * u][kl] = wv[u];
#pragma unroll
    for (int u = 0; u < kRowTile / 2; ++u) {
      const int row = r0 + rsub + 2 * u;
      sX[rsub + 2 * u][kl] = (kin && row < a.n) ? (xv[u] - mu) / sg : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kKc; kk += 4)
      acc = mfma4(sW[lane % 16][kk + lane / 16], sX[wave * 16 + lane % 16][kk + lane / 16], acc);
    __syncthreads();
  }
  // acc[t]: column c0 + 4 (lane / 16) + t, row r0 + 16 wave + lane % 16
  const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7fffffff, kBufferRsrcWord3);
  const int tile = rt * CT + ct;
  const int row_l = wave * 16 + lane % 16, col4 = 4 * (lane / 16);
  const int off = (((tile * a.S + s) * kRowTile + row_l) * 16 + col4) * 4;  // bytes (< 2^31: checked on the host)
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc), prs, off, 0, kCoherentCpol);
  if (!arrive_last(&a.cnt1[tile * kCntLine], a.S, s_flag)) return;
  // last split of this tile: sum the splits in order, bias, GELU
  // (eight splits' loads in flight at a time, added in split order)
  f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < a.S; s0 += 8) {
    f32x4 pv[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int ss = min(s0 + q, a.S - 1);
      pv[q] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            prs, (((tile * a.S + ss) * kRowTile + row_l) * 16 + col4) * 4, 0, kCoherentCpol));
    }
#pragma unroll
    for (int q = 0; q < 8; ++q)
      if (s0 + q < a.S) sum += pv[q];
  }
  const int row = r0 + row_l;
  f32x4 hv;
#pragma unroll
  for (int t = 0; t < 4; ++t) hv[t] = gelu_erf(sum[t] + a.b1[c0 + col4 + t]);
  const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(a.h1, 0, 0x7fffffff, kBufferRsrcWord3);
  if (row < a.n)
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, hv), hrs, (row * a.H + c0 + col4) * 4, 0,
                                           kCoherentCpol);
  count_done(&a.done1[rt * kCntLine]);
}

template <bool LAST>
__device__ void dense_body(const MlpArgs& a, int bid, const float* hin, const float* W, const float* b, float* hout,
                           float* smem, int* s_flag) {
  float (*sW)[kMaxH + 1] = reinterpret_cast<float (*)[kMaxH + 1]>(smem);
  float (*sX)[kMaxH + 1] = reinterpret_cast<float (*)[kMaxH + 1]>(smem + 16 * (kMaxH + 1));
  const int CT = a.H / 16;
  const int ct = bid % CT, rt = bid / CT;
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int c0 = ct * 16, r0 = rt * kRowTile, H = a.H;
  // stage the weight slice [16][H] and the input rows [64][H] with 16-byte loads, all issued before use
  // (H is a multiple of 16: a row is H / 4 float4s)
  const int H4 = H / 4;
  f32x4 wv[kMaxH / 64], xv[kMaxH / 4];
#pragma unroll
  for (int u = 0; u < kMaxH / 64; ++u) {
    const int i = tid + kMlpThreads * u;
    wv[u] = i < 16 * H4 ? *reinterpret_cast<const f32x4*>(W + (int64_t)(c0 + i / H4) * H + 4 * (i % H4)) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // the input rows were written by other workgroups of this launch: device-coherent loads
  const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(hin), 0, 0x7fffffff,
                                                                       kBufferRsrcWord3);
#pragma unroll
  for (int u = 0; u < kMaxH / 4; ++u) {
    const int i = tid + kMlpThreads * u, r = i / H4;
    xv[u] = (i < kRowTile * H4 && r0 + r < a.n)
                ? __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                irs, ((r0 + r) * H + 4 * (i % H4)) * 4, 0, kCoherentCpol))
                : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int u = 0; u < kMaxH / 64; ++u) {
    const int i = tid + kMlpThreads * u;
    if (i < 16 * H4)
#pragma unroll
      for (int e = 0; e < 4; ++e) sW[i / H4][4 * (i % H4) + e] = wv[u][e];
  }
#pragma unroll
  for (int u = 0; u < kMaxH / 4; ++u) {
    const int i = tid + kMlpThreads * u;
    if (i < kRowTile * H4)
#pragma unroll
      for (int e = 0; e < 4; ++e) sX[i / H4][4 * (i % H4) + e] = xv[u][e];
  }
  __syncthreads();
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int kk = 0; kk < H; kk += 4) acc = mfma4(sW[lane % 16][kk + lane / 16], sX[wave * 16 + lane % 16][kk + lane / 16], acc);
  const int row_l = wave * 16 + lane % 16, col4 = 4 * (lane / 16), row = r0 + row_l;
  float hv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) hv[t] = gelu_erf(acc[t] + b[c0 + col4 + t]);
  if constexpr (!LAST) {
    const __amdgpu_buffer_rsrc_t ors = __builtin_amdgcn_make_buffer_rsrc(hout, 0, 0x7fffffff, kBufferRsrcWord3);
    if (row < a.n)
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, (f32x4){hv[0], hv[1], hv[2], hv[3]}), ors,
                                             (row * H + c0 + col4) * 4, 0, kCoherentCpol);
    count_done(&a.done2[rt * kCntLine]);
  } else {
    // this tile's share of w4 . h3 for the row: the lane's 4 columns in order, then the 4 lane groups in order
    const float zs = dot4(hv, a.w4 + c0 + col4);
    const float z1 = __shfl(zs, lane % 16 + 16), z2 = __shfl(zs, lane % 16 + 32), z3 = __shfl(zs, lane % 16 + 48);
    const float tz = ((zs + z1) + z2) + z3;  // lanes 0..15: rows 16 wave + lane
    const __amdgpu_buffer_rsrc_t zrs = __builtin_amdgcn_make_buffer_rsrc(a.zpart, 0, 0x7fffffff, kBufferRsrcWord3);
    if (lane < 16)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, tz), zrs, ((rt * CT + ct) * kRowTile + row_l) * 4,
                                            0, kCoherentCpol);
    if (!arrive_last(&a.cnt3[rt * kCntLine], CT, s_flag)) return;
    // every wait of this row tile has ended: its counters go back to zero for the next call
    if (tid == 0) {
      __hip_atomic_store(&a.done1[rt * kCntLine], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.done2[rt * kCntLine], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const bool bad = __hip_atomic_load(a.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
    if (tid < kRowTile && r0 + tid < a.n) {
      // every tile's share loaded at once (CT <= 16), added in tile order
      float zt[kMaxH / 16];
#pragma unroll
      for (int t = 0; t < kMaxH / 16; ++t)
        zt[t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                              zrs, ((rt * CT + min(t, CT - 1)) * kRowTile + tid) * 4, 0, kCoherentCpol));
      float z = 0.f;
#pragma unroll
      for (int t = 0; t < kMaxH / 16; ++t)
        if (t < CT) z += zt[t];
      z += a.b4;
      if (bad) z = __builtin_nanf("");
      a.log_score[r0 + tid] = log_sigmoid(z);
      if (a.logit) a.logit[r0 + tid] = z;
    }
  }
}

__global__ void __launch_bounds__(kMlpThreads) survival_kernel(MlpArgs a) {
  __shared__ __attribute__((aligned(16))) float smem[(16 + kRowTile) * (kMaxH + 1)];
  __shared__ int s_flag;
  const int CT = a.H / 16, RT = (a.n + kRowTile - 1) / kRowTile;
  const int n1 = RT * CT * a.S, n2 = RT * CT;
  const int bid = blockIdx.x;
  if (bid < n1) {
    layer1_body(a, bid, smem, &s_flag);
  } else if (bid < n1 + n2) {
    const int b2 = bid - n1;
    if (!wait_count(&a.done1[(b2 / CT) * kCntLine], CT, &s_flag) && threadIdx.x == 0) atomicOr(a.err, 1);
    dense_body<false>(a, b2, a.h1, a.W2, a.b2, a.h2, smem, &s_flag);
  } else {
    const int b3 = bid - n1 - n2;
    if (!wait_count(&a.done2[(b3 / CT) * kCntLine], CT, &s_flag) && threadIdx.x == 0) atomicOr(a.err, 1);
    dense_body<true>(a, b3, a.h2, a.W3, a.b3, nullptr, smem, &s_flag);
  }
}

struct MlpWs {
  size_t part, h1, h2, zpart, cnt1, cnt3, done, total;
};

MlpWs mlp_ws(int n, int H, int S) {
  const int RT = (int)ceil_div(n > 0 ? n : 1, kRowTile), CT = H / 16;
  MlpWs w{};
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o += (bytes + 255) / 256 * 256;
    return at;
  };
  w.cnt1 = take((size_t)RT * CT * kCntLine * sizeof(int));
  w.cnt3 = take((size_t)RT * kCntLine * sizeof(int));
  w.done = take((size_t)(2 * RT + 1) * kCntLine * sizeof(int));  // done1 [RT], done2 [RT], the sticky error word
  w.part = take((size_t)RT * CT * S * kRowTile * 16 * sizeof(float));
  w.h1 = take((size_t)RT * kRowTile * H * sizeof(float));
  w.h2 = take((size_t)RT * kRowTile * H * sizeof(float));
  w.zpart = take((size_t)RT * CT * kRowTile * sizeof(float));
  w.total = o;
  return w;
}

// k-splits of layer 1: about 256 workgroups in all, each split a whole number of LDS chunks
void layer1_splits(int n, int H, int d_in, int& S, int& kc_split) {
  const int RT = (int)ceil_div(n > 0 ? n : 1, kRowTile), CT = H / 16;
  int want = std::max(1, 256 / (RT * CT));
  kc_split = (int)ceil_div(ceil_div(d_in, want), kKc) * kKc;
  S = (int)ceil_div(d_in, kc_split);
}

int check_mlp(const sdd_mlp* m) {
  SDD_REQUIRE(m != nullptr, "NULL predictor");
  SDD_REQUIRE(m->d_hid >= 0 && m->n_sc >= 0 && m->d_hid + m->n_sc > 0, "bad input width %d + %d", m->d_hid, m->n_sc);
  SDD_REQUIRE(m->H >= 16 && m->H <= kMaxH && m->H % 16 == 0, "hidden width %d: a multiple of 16 in [16, %d]", m->H, kMaxH);
  SDD_REQUIRE(m->mu && m->sigma && m->W1 && m->b1 && m->W2 && m->b2 && m->W3 && m->b3 && m->w4, "NULL predictor tensor");
  return SDD_OK;
}

}  // namespace
}  // namespace sdd

using namespace sdd;

extern "C" int sdd_survival_workspace_bytes(const sdd_mlp* m, int n, size_t* bytes) {
  int rc = check_mlp(m);
  if (rc) return rc;
  SDD_REQUIRE(bytes != nullptr && n >= 0, "bad arguments");
  int S, kc;
  layer1_splits(n, m->H, m->d_hid + m->n_sc, S, kc);
  *bytes = mlp_ws(n, m->H, S).total;
  return SDD_OK;
}

extern "C" int sdd_survival_mlp(const sdd_mlp* m, const uint16_t* hidden, const float* scalars, int n,
                                float* log_score, float* logit, void* ws, size_t ws_bytes, sdd_stream_t stream) {
  int rc = check_mlp(m);
  if (rc) return rc;
  SDD_REQUIRE(n >= 0, "n = %d", n);
  if (n == 0) return SDD_OK;
  SDD_REQUIRE(log_score && (m->d_hid == 0 || hidden) && (m->n_sc == 0 || scalars), "NULL input or output");
  MlpArgs a{};
  a.hidden = hidden;
  a.scalars = scalars;
  a.mu = m->mu;
  a.sigma = m->sigma;
  a.W1 = m->W1;
  a.b1 = m->b1;
  a.W2 = m->W2;
  a.b2 = m->b2;
  a.W3 = m->W3;
  a.b3 = m->b3;
  a.w4 = m->w4;
  a.b4 = m->b4;
  a.n = n;
  a.d_hid = m->d_hid;
  a.n_sc = m->n_sc;
  a.d_in = m->d_hid + m->n_sc;
  a.H = m->H;
  layer1_splits(n, a.H, a.d_in, a.S, a.kc_split);
  const MlpWs L = mlp_ws(n, a.H, a.S);
  SDD_REQUIRE(ws != nullptr && ws_bytes >= L.total, "predictor workspace needs %zu bytes, got %zu", L.total, ws_bytes);
  SDD_REQUIRE((uintptr_t)ws % 256 == 0, "workspace must be 256-byte aligned");
  const int RT = (int)ceil_div(n, kRowTile), CT = a.H / 16;
  if ((int64_t)RT * CT * a.S * kRowTile * 16 * 4 >= (int64_t(1) << 31))
    return fail(SDD_EUNSUPPORTED, "%d positions exceed the 32-bit partial offsets", n);
  char* w = reinterpret_cast<char*>(ws);
  a.part = reinterpret_cast<float*>(w + L.part);
  a.h1 = reinterpret_cast<float*>(w + L.h1);
  a.h2 = reinterpret_cast<float*>(w + L.h2);
  a.zpart = reinterpret_cast<float*>(w + L.zpart);
  a.cnt1 = reinterpret_cast<int*>(w + L.cnt1);
  a.cnt3 = reinterpret_cast<int*>(w + L.cnt3);
  a.done1 = reinterpret_cast<int*>(w + L.done);
  a.done2 = a.done1 + (size_t)RT * kCntLine;
  a.err = a.done2 + (size_t)RT * kCntLine;
  a.log_score = log_score;
  a.logit = logit;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if ((int64_t)RT * kRowTile * a.H * 4 >= (int64_t(1) << 31))
    return fail(SDD_EUNSUPPORTED, "%d positions exceed the 32-bit activation offsets", n);
  prof_begin(PROF_MLP, st);
  hipLaunchKernelGGL(survival_kernel, dim3(RT * CT * (a.S + 2)), dim3(kMlpThreads), 0, st, a);
  prof_end(PROF_MLP, st);
  return check_launch("survival_kernel");
}
