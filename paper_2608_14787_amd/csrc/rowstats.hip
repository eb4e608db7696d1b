// Vocab-wide row reductions for the acceptance test and the confidence
// prefix (gfx950).
//
// Acceptance (Sec. 3.1; lenience equation and top-k rule in Appendix
// "Baselines and Sweep Settings"): for every target row j < gamma decide
// whether draft j passes; L = first failure; next token = argmax of row L,
// or, in the distribution-preserving ratio mode (the min(1, p/q) rule that
// Sec. 3.1 cites), a draw from norm(max(0, p_L - q_L)) after a rejection and
// from p_gamma after a full block (second kernel, resample_kernel).
// Confidence (Sec. 4.1 local gate, Sec. 4.2 raw confidence): q_j = max softmax
// of drafter row j; skip length = first j with q_j < tau.
//
// Both are HBM-bound streams over [B][rows][V] logits.  Each row is split into
// C equal chunks; one 256-thread workgroup streams its chunk with 16-byte
// loads, four in flight per thread and row (one pass over HBM), keeping running
// max / first-argmax / online sum-exp / rank counts in registers, reduces them
// across the wave with shuffles and across the four waves through LDS, and
// writes one record.  The last workgroup of a
// sequence to finish (arrival counter) combines that sequence's records in a
// fixed order, so results are bit-reproducible, and takes the decisions; it
// resets the counter so the workspace can be reused.
#include <mutex>

#include "sdd_internal.h"

namespace sdd {

namespace {

constexpr int kThreads = 256;
// per-sequence arrival counters one 128-byte line apart: a sequence's workgroups all arrive within a few
// microseconds, and device-scope atomics on one line serialize
constexpr int kSeqCntStride = 32;
constexpr int kRecBatch = 512;  // chunk records staged in LDS at a time by the finishing workgroup (16 KB)

struct RowRec {
  float m;    // row max over the chunk (NaN ignored)
  int arg;    // first index of the max (-1 if the chunk held only NaN)
  float s;    // sum over finite values of exp(z - m)
  int cnt;    // top-k rank count: z > z_x, or z == z_x at a lower index
  float qm;   // drafter row max (ratio mode)
  float qs;   // drafter row sum exp (ratio mode)
  int flags;  // bit0: non-finite value in the target chunk; bit2: in the drafter chunk
  int pad;
};

// Row-L statistics that the acceptance pass hands to the residual draw.
struct SeqRec {
  int L;
  int bad;  // row L of p (or of q, L < gamma) holds a non-finite value: no draw, next = argmax
  float m, s, qm, qs;
  int pad[2];
};

// Per-chunk weight totals of the residual draw: residual max(0, p - q), and p alone (fallback when the
// residual total is not positive).
struct ResRec {
  float r, p;
};

struct Job {
  const void* p;  // rows to reduce
  size_t p_seq_stride, p_row_stride;
  const void* q;  // drafter rows (ratio)
  size_t q_seq_stride;
  const int32_t* draft;
  const float* u;
  int B, gamma, V, rows, C, chunk;
  int mode, k;
  int sample;     // ratio mode with the residual draw
  int u_stride;   // uniforms per sequence: gamma, or gamma + 1 with the draw
  int C2, seg;    // residual draw: chunks per row, elements per thread (C2 = ceil(V / (256 seg)))
  SeqRec* seqs;
  ResRec* rrecs;
  int* counters2;
  float log_len;  // fp32 log(lenience)
  float log_tau;  // fp32 log(tau)
  RowRec* recs;
  int* counters;
  int32_t* out_len;
  int32_t* out_next;
  int32_t* out_flags;
  float* out_log_conf;
  float* out_log_pdraft;
};

enum Kind { kAccept = 0, kConfidence = 1 };

__device__ inline bool better(float m2, int a2, float m1, int a1) {
  if (a2 < 0) return false;
  if (a1 < 0) return true;
  return m2 > m1 || (m2 == m1 && a2 < a1);
}

__device__ inline float exp_shift(float z, float m) {  // exp(z - m) for finite z, m
  return __expf(z - m);
}

// Block-wide combine of (m, arg, s) and an int count; result valid in thread 0.
struct BlockRed {
  float m[kThreads / kWave];
  int a[kThreads / kWave];
  float s[kThreads / kWave];
  int c[kThreads / kWave];
  int f[kThreads / kWave];
};

// Combines (m2, a2, s2, c2, f2) into (m, a, s, cnt, fl): max with the first argmax, sums relative to the
// larger max (finite maxima only), counts, flags.  Commutative, so both lanes of a butterfly agree.
template <bool kSum>
__device__ __attribute__((always_inline)) inline void stat_combine(float& m, int& a, float& s, int& cnt, int& fl, float m2,
                                                                   int a2, float s2, int c2, int f2) {
  if (kSum) {
    const float mm = fmaxf(m, m2);
    const float sa = (s > 0.f) ? s * __expf(m - mm) : 0.f;
    const float sb = (s2 > 0.f) ? s2 * __expf(m2 - mm) : 0.f;
    s = sa + sb;
  }
  const bool bt = better(m2, a2, m, a);
  m = bt ? m2 : m;
  a = bt ? a2 : a;
  cnt += c2;
  fl |= f2;
}

template <int CTRL, bool kSum>
__device__ __attribute__((always_inline)) inline void stat_dpp_step(float& m, int& a, float& s, int& cnt, int& fl) {
  const float m2 = dpp_f<CTRL>(m), s2 = kSum ? dpp_f<CTRL>(s) : 0.f;
  const int a2 = dpp_i<CTRL>(a), c2 = dpp_i<CTRL>(cnt), f2 = dpp_i<CTRL>(fl);
  stat_combine<kSum>(m, a, s, cnt, fl, m2, a2, s2, c2, f2);
}

template <bool kSum>
__device__ __attribute__((always_inline)) void block_reduce(float& m, int& a, float& s, int& cnt, int& fl, BlockRed* red) {
  // wave level: DPP within rows of 16 (pairs, quads, eights, sixteens), then the four rows in order
  stat_dpp_step<kDppXor1, kSum>(m, a, s, cnt, fl);
  stat_dpp_step<kDppXor2, kSum>(m, a, s, cnt, fl);
  stat_dpp_step<kDppHalfMirror, kSum>(m, a, s, cnt, fl);
  stat_dpp_step<kDppMirror, kSum>(m, a, s, cnt, fl);
  {
    float wm = lane_f(m, 0), ws = lane_f(s, 0);
    int wa = __builtin_amdgcn_readlane(a, 0), wc = __builtin_amdgcn_readlane(cnt, 0), wf = __builtin_amdgcn_readlane(fl, 0);
#pragma unroll
    for (int r = 16; r < kWave; r += 16)
      stat_combine<kSum>(wm, wa, ws, wc, wf, lane_f(m, r), __builtin_amdgcn_readlane(a, r), lane_f(s, r),
                         __builtin_amdgcn_readlane(cnt, r), __builtin_amdgcn_readlane(fl, r));
    m = wm;
    a = wa;
    s = ws;
    cnt = wc;
    fl = wf;
  }
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (lane == 0) {
    red->m[w] = m;
    red->a[w] = a;
    red->s[w] = s;
    red->c[w] = cnt;
    red->f[w] = fl;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = red->m[0];
    int A = red->a[0];
    int Cn = red->c[0], F = red->f[0];
    for (int i = 1; i < kThreads / kWave; ++i) {
      if (better(red->m[i], red->a[i], M, A)) {
        M = red->m[i];
        A = red->a[i];
      }
      Cn += red->c[i];
      F |= red->f[i];
    }
    float S = 0.f;
    if (kSum) {
      float mx = -INFINITY;
      for (int i = 0; i < kThreads / kWave; ++i)
        if (red->s[i] > 0.f) mx = fmaxf(mx, red->m[i]);
      for (int i = 0; i < kThreads / kWave; ++i)
        if (red->s[i] > 0.f) S += red->s[i] * __expf(red->m[i] - mx);
      // express relative to the chunk max M (== mx whenever finite values exist)
      if (S > 0.f && mx != M) S *= __expf(mx - M);
    }
    m = M;
    a = A;
    s = S;
    cnt = Cn;
    fl = F;
  }
}

template <typename T, int VEC>
__device__ inline void unpack(const uint4& r, float* v) {
  if constexpr (VEC > 1) {
    unpack16(r, v, T());
  } else {
    v[0] = __builtin_bit_cast(float, r.x);
  }
}

// One vector of a row: a 16-byte streaming load, or one element (rows that are not 16-byte aligned).
template <typename T, int VEC>
__device__ inline uint4 load_vec(const T* row, int e) {
  if constexpr (VEC > 1) {
    return load_nt16(row + e);
  } else {
    uint4 r;
    r.x = __builtin_bit_cast(uint32_t, Elem<T>::to_f32(row[e]));
    return r;
  }
}

// Running statistics of the elements a thread has seen, in increasing index order: max and first index of
// the max over non-NaN values (m, a); sum over finite values of exp(z - mf), mf their max (online: the sum
// is rescaled when mf grows); rank count against (zx, x); non-finite flag.
struct ThreadStats {
  float m, mf, s;
  int a, cnt, fl;
};

__device__ inline ThreadStats stats_init() { return ThreadStats{-INFINITY, -INFINITY, 0.f, -1, 0, 0}; }

template <int VEC, bool kSum, bool kCount, bool kIdx = true>
__device__ __attribute__((always_inline)) inline void stats_update(ThreadStats& st, const float* v, bool valid, int e0,
                                                                   float zx, int x) {
  // branch-free per element (selects; an invalid vector changes nothing), so the streaming loop has no
  // divergent blocks and its loads stay in flight; two wave-uniform branches skip work no lane needs.  The max and first argmax are
  // taken per vector: vx = the vector's max over non-NaN values (fmaxf skips NaN); it replaces the running
  // max when greater (or when none is held yet), at the vector's first element equal to it -- the same
  // result as visiting the elements one by one in index order.  kIdx = false (drafter rows, whose argmax is
  // never used) records index 0 instead of searching.
  float vm = -INFINITY;  // max over finite values (reference of the sum)
  float vx = -INFINITY;  // max over non-NaN values (comparisons with NaN are false)
  float zf[VEC];         // the finite values of a valid vector, -inf elsewhere (exp(-inf - m) adds exactly 0)
  bool nonfin = false, has = false, tie = false;
  int gt = 0;
#pragma unroll
  for (int t = 0; t < VEC; ++t) {
    const float z = v[t];
    const bool fin = __builtin_isfinite(z);
    nonfin |= !fin;
    has |= !__builtin_isnan(z);
    zf[t] = (valid && fin) ? z : -INFINITY;
    vm = fmaxf(vm, zf[t]);
    vx = z > vx ? z : vx;
    if (kCount) {
      gt += z > zx ? 1 : 0;
      tie |= z == zx;
    }
  }
  if (kCount) {
    // rank count: values above the draft token's, plus equal values at a lower index; the index test runs
    // only for vectors where some lane holds an equal value (wave-uniform branch, rare for real logits)
    st.cnt += valid ? gt : 0;
    if (__builtin_amdgcn_ballot_w64(valid && tie)) {
#pragma unroll
      for (int t = 0; t < VEC; ++t) st.cnt += (valid && v[t] == zx && e0 + t < x) ? 1 : 0;
    }
  }
  st.fl |= (valid && nonfin) ? 1 : 0;
  const bool take = valid && has && (st.a < 0 || vx > st.m);
  int idx = 0;
  if (kIdx) {
    // the first index of the vector's max, searched only for vectors where some lane takes a new max
    // (wave-uniform branch: after a row's first vectors a new running max is rare)
    if (__builtin_amdgcn_ballot_w64(take)) {
#pragma unroll
      for (int t = VEC - 1; t >= 0; --t) idx = v[t] == vx ? t : idx;
    }
  }
  st.m = take ? vx : st.m;
  st.a = take ? e0 + idx : st.a;
  if (kSum) {
    const float mn = fmaxf(st.mf, vm);  // -inf while no finite value has been seen
    float add = 0.f;  // (mn = -inf: no finite value yet, the sum is left unchanged below)
#pragma unroll
    for (int t = 0; t < VEC; ++t) add += exp_shift(zf[t], mn);
    const float scale = st.mf > -INFINITY ? exp_shift(st.mf, mn) : 0.f;
    st.s = mn > -INFINITY ? st.s * scale + add : st.s;
    st.mf = mn;
  }
}

// Streams this thread's vectors of [base, base + n) of a row (and of the drafter row) with kDepth to
// 2 kDepth 16-byte loads of each in flight, updating the running statistics.  Vector i of the thread starts
// at element base + (i * kThreads + threadIdx.x) * VEC.  The loads are unconditional (a vector past the
// thread's last one reads zero without a memory access, or, for rows that are not 16-byte aligned, re-reads
// the last one, and its values are not used) and the trip count is uniform over the workgroup, so the
// compiler can wait for exactly the older group.
template <typename T, typename TQ, int VEC, bool kSum, bool kCount, bool kQ>
__device__ __attribute__((always_inline)) inline void stream_stats(const T* row, const TQ* qrow, int base, int n, float zx,
                                                                   int x, ThreadStats& st, ThreadStats& qst) {
  constexpr int kDepth = kQ ? 2 : 4;  // two rows streamed in the ratio mode: fewer registers, more workgroups
  const int nvec = n / VEC;  // n is a multiple of VEC (VEC > 1 only when V is); n > 0
  // trip count uniform over the workgroup; a thread's vectors past its last one re-read that one (valid = 0)
  const int nvt = nvec > (int)threadIdx.x ? (nvec - (int)threadIdx.x + kThreads - 1) / kThreads : 0;
  const int nvmax = (nvec + kThreads - 1) / kThreads;
  const int last = max(nvt - 1, 0);
  const int tofs = nvt > 0 ? (int)threadIdx.x : 0;  // a thread with no vector reads the chunk's first one
  auto elem = [&](int i) { return base + (min(i, last) * kThreads + tofs) * VEC; };
  const bool hq = kQ && qrow != nullptr;
  // 16-byte vectors through buffer descriptors over the chunk: a vector past the thread's last one lies past
  // the descriptor's range, so its load returns zero without a memory access (no clamped re-reads)
  const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(row + base), 0, n * (int)sizeof(T),
                                                                       kBufferRsrcWord3);
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<TQ*>(hq ? qrow + base : reinterpret_cast<const TQ*>(row)), 0, hq ? n * (int)sizeof(TQ) : 0, kBufferRsrcWord3);
  // two register buffers of kDepth vectors: the next group's loads are issued (and kept ahead of the
  // arithmetic by a scheduling barrier) before the current group is consumed
  uint4 pa[kDepth], pb[kDepth], qa[kQ ? kDepth : 1], qb[kQ ? kDepth : 1];
  auto load_group = [&](int i, uint4* pv, uint4* qv) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      if constexpr (VEC > 1) {
        const int off = ((i + d) * kThreads + (int)threadIdx.x) * 16;
        pv[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(prs, off, 0, kNtCpol));
        if (kQ) qv[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(qrs, off, 0, kNtCpol));
      } else {
        pv[d] = load_vec<T, VEC>(row, elem(i + d));
        if (kQ) qv[d] = hq ? load_vec<TQ, VEC>(qrow, elem(i + d)) : uint4{0, 0, 0, 0};
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto use_group = [&](int i, const uint4* pv, const uint4* qv) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      float v[VEC], w[VEC];
      unpack<T, VEC>(pv[d], v);
      if (kQ) unpack<TQ, VEC>(qv[d], w);
      const int e = base + ((i + d) * kThreads + (int)threadIdx.x) * VEC;
      const bool valid = i + d < nvt;
      stats_update<VEC, kSum, kCount>(st, v, valid, e, zx, x);
      if (kQ) stats_update<VEC, true, false, false>(qst, w, valid && hq, e, 0.f, -1);
    }
  };
  load_group(0, pa, qa);
  for (int i = 0; i < nvmax; i += 2 * kDepth) {
    load_group(i + kDepth, pb, qb);
    use_group(i, pa, qa);
    if (i + kDepth >= nvmax) break;
    load_group(i + 2 * kDepth, pa, qa);
    use_group(i + kDepth, pb, qb);
  }
  // the block reduction takes the sum relative to m: they differ only when the row holds +inf (flagged)
  if (st.m != st.mf) st.s = 0.f;
  if (kQ && qst.m != qst.mf) qst.s = 0.f;
}

// Combined statistics of one row.
struct RowStats {
  float m, s, qm, qs;
  int arg, cnt, flags;
};

// One thread folds the C chunk records of its row (staged in LDS) in chunk order: the max and first argmax,
// the sums rescaled to the running max, counts and flags.  A fixed order, so results are bit-reproducible.
__device__ __attribute__((always_inline)) inline RowStats fold_row(const RowRec* rp, int C) {
  float M = -INFINITY, S = 0.f, QM = -INFINITY, QS = 0.f;
  int A = -1, cnt = 0, fl = 0;
  for (int c = 0; c < C; ++c) {
    const RowRec r = rp[c];
    if (better(r.m, r.arg, M, A)) {
      // rescale the running sum to the new max (sums are kept relative to the max of finite values)
      if (r.s > 0.f) S = (S > 0.f ? S * __expf(M - r.m) : 0.f) + r.s;
      M = r.m;
      A = r.arg;
    } else if (r.s > 0.f) {
      S += r.s * __expf(r.m - M);
    }
    if (r.qs > 0.f) {
      const float qn = fmaxf(QM, r.qm);
      QS = (QS > 0.f ? QS * __expf(QM - qn) : 0.f) + r.qs * __expf(r.qm - qn);
      QM = qn;
    }
    cnt += r.cnt;
    fl |= r.flags;
  }
  RowStats o;
  o.m = M;
  o.arg = A;
  o.s = S;
  o.cnt = cnt;
  o.flags = fl;
  o.qm = QM;
  o.qs = QS;
  return o;
}

template <typename T, typename TQ, int VEC, int KIND, bool kSum, bool kCount, bool kQ>
__global__ void __launch_bounds__(kThreads) rowstats_kernel(Job job) {
  __shared__ BlockRed red;
  __shared__ int s_last;
  __shared__ int s_pass[72];
  __shared__ int s_arg[72];
  __shared__ int s_flag[72];
  __shared__ int s_bad[72];
  __shared__ float s_st[72][4];
  __shared__ int s_x[72];
  __shared__ float s_zp[72], s_zq[72], s_u[72];
  __shared__ RowRec s_rec[kRecBatch];

  const int c = blockIdx.x % job.C;
  const int rowid = blockIdx.x / job.C;  // b * rows + j
  const int b = rowid / job.rows, j = rowid % job.rows;
  const int base = c * job.chunk;
  const int n = min(job.chunk, job.V - base);

  const T* row = reinterpret_cast<const T*>(job.p) + (size_t)b * job.p_seq_stride + (size_t)j * job.p_row_stride;
  // the draft token and its value are needed in the stream only by the rank count (top-k)
  int x = -1;
  float zx = 0.f;
  if (kCount && job.draft != nullptr && j < job.gamma) {
    x = job.draft[(size_t)b * job.gamma + j];
    if (x >= 0 && x < job.V) zx = Elem<T>::to_f32(row[x]);
  }

  const bool has_q = kQ && j < job.gamma;
  const TQ* qrow = has_q ? reinterpret_cast<const TQ*>(job.q) + (size_t)b * job.q_seq_stride + (size_t)j * job.V : nullptr;
  ThreadStats st = stats_init(), qst = stats_init();
  stream_stats<T, TQ, VEC, kSum, kCount, kQ>(row, qrow, base, n, zx, x, st, qst);

  float m = st.m, s = st.s;
  int a = st.a, cnt = st.cnt, fl = st.fl;
  block_reduce<kSum>(m, a, s, cnt, fl, &red);
  RowRec rec;
  rec.m = m;
  rec.arg = a;
  rec.s = s;
  rec.cnt = cnt;
  rec.flags = fl;
  rec.qm = -INFINITY;
  rec.qs = 0.f;
  rec.pad = 0;
  if (kQ) {
    __syncthreads();
    float qm = qst.m, qs = qst.s;
    int qa = qst.a, qc = 0, qf = qst.fl;
    block_reduce<true>(qm, qa, qs, qc, qf, &red);
    rec.qm = qm;
    rec.qs = qs;
    rec.flags |= qf ? 4 : 0;
  }

  if (threadIdx.x == 0) {
    RowRec* dst = &job.recs[blockIdx.x];
    st_coherent(&dst->m, rec.m);
    st_coherent(&dst->arg, rec.arg);
    st_coherent(&dst->s, rec.s);
    st_coherent(&dst->cnt, rec.cnt);
    st_coherent(&dst->qm, rec.qm);
    st_coherent(&dst->qs, rec.qs);
    st_coherent(&dst->flags, rec.flags);
  }
  if (!arrive_last(&job.counters[b * kSeqCntStride], job.rows * job.C, &s_last)) return;

  // ---- last workgroup of sequence b: combine and decide ----
  // (1) every row's decision inputs at once (thread t: row t): draft token, uniform, and the target and
  //     drafter values at the draft token (these two wait only for the token)
  const int tid = threadIdx.x;
  const bool need_z = KIND == kAccept ? (job.mode != SDD_GREEDY && job.mode != SDD_TOPK) : job.out_log_pdraft != nullptr;
  if (tid < job.rows) {
    int xx = -1;
    float zp = 0.f, zq = 0.f, uu = 1.f;
    if (tid < job.gamma && job.draft) {
      xx = job.draft[(size_t)b * job.gamma + tid];
      if (KIND == kAccept && kQ) uu = job.u[(size_t)b * job.u_stride + tid];
      if (xx >= 0 && xx < job.V && need_z) {
        zp = Elem<T>::to_f32(reinterpret_cast<const T*>(job.p)[(size_t)b * job.p_seq_stride + (size_t)tid * job.p_row_stride + xx]);
        if (KIND == kAccept && kQ)
          zq = Elem<TQ>::to_f32(reinterpret_cast<const TQ*>(job.q)[(size_t)b * job.q_seq_stride + (size_t)tid * job.V + xx]);
      }
    }
    s_x[tid] = xx;
    s_zp[tid] = zp;
    s_zq[tid] = zq;
    s_u[tid] = uu;
  }
  // (2) chunk records staged into LDS in batches of whole rows (16-byte device-coherent loads, all in
  //     flight together), then one thread per row folds its records and decides
  const RowRec* recs = job.recs + (size_t)b * job.rows * job.C;
  const __amdgpu_buffer_rsrc_t rrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<RowRec*>(recs), 0, 0x7fffffff, kBufferRsrcWord3);
  const int rows_per_batch = kRecBatch / job.C;  // >= 1: C <= 64 < kRecBatch
  for (int r0 = 0; r0 < job.rows; r0 += rows_per_batch) {
    const int r1 = min(job.rows, r0 + rows_per_batch);
    const int nrec = (r1 - r0) * job.C;
    __syncthreads();  // the previous batch's readers are done
    for (int h = tid; h < 2 * nrec; h += kThreads) {
      const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rrs, (r0 * job.C) * (int)sizeof(RowRec) + 16 * h, 0, kCoherentCpol);
      reinterpret_cast<u32x4*>(s_rec)[h] = v;
    }
    __syncthreads();
    const int t = r0 + tid;
    if (t < r1) {
      const RowStats st = fold_row(s_rec + tid * job.C, job.C);
      const bool bad = (st.flags & 1) != 0;
      s_arg[t] = st.arg < 0 ? 0 : st.arg;
      s_flag[t] = bad ? 1 : 0;
      if (KIND == kAccept && job.sample) {
        s_bad[t] = bad || (kQ && (st.flags & 4)) ? 1 : 0;
        s_st[t][0] = st.m;
        s_st[t][1] = st.s;
        s_st[t][2] = st.qm;
        s_st[t][3] = st.qs;
      }
      const int xx = s_x[t];
      if (KIND == kAccept) {
        int pass = 0;
        if (t < job.gamma) {
          if (xx < 0 || xx >= job.V) {
            pass = 0;
            s_flag[t] |= 2;
          } else if (bad || (kQ && (st.flags & 4))) {
            pass = 0;
            s_flag[t] |= 1;
          } else {
            const float z = s_zp[t];
            if (job.mode == SDD_GREEDY) {
              pass = st.arg == xx;
            } else if (job.mode == SDD_TOPK) {
              pass = st.cnt < job.k;
            } else if (job.mode == SDD_LENIENT) {
              const float diff = z - st.m;
              pass = diff >= job.log_len;
            } else {  // SDD_RATIO: log u < (z - LSE_p) - (zq - LSE_q)
              const float lp = z - (st.m + logf(st.s));
              const float lq = s_zq[t] - (st.qm + logf(st.qs));
              const float uu = s_u[t];
              const float lu = uu > 0.f ? logf(uu) : -INFINITY;
              pass = lu < lp - lq;
            }
          }
        }
        s_pass[t] = pass;
      } else {
        const float lc = bad ? __builtin_nanf("") : -logf(st.s);
        s_pass[t] = (lc >= job.log_tau) ? 1 : 0;
        if (job.out_log_conf) job.out_log_conf[(size_t)b * job.gamma + t] = lc;
        if (job.out_log_pdraft && job.draft) {
          float lp = __builtin_nanf("");
          if (!bad && xx >= 0 && xx < job.V) lp = s_zp[t] - st.m - logf(st.s);
          job.out_log_pdraft[(size_t)b * job.gamma + t] = lp;
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (KIND == kAccept) {
      int L = job.gamma, fl = 0;
      for (int jj = 0; jj < job.gamma; ++jj) {
        fl |= s_flag[jj] & 2;
        if (!s_pass[jj]) {
          fl |= s_flag[jj];
          L = jj;
          break;
        }
      }
      fl |= s_flag[L] & 1;
      job.out_len[b] = L;
      job.out_next[b] = s_arg[L];
      if (job.out_flags) job.out_flags[b] = fl;
      if (job.sample) {
        SeqRec r;
        r.L = L;
        r.bad = s_bad[L];
        r.m = s_st[L][0];
        r.s = s_st[L][1];
        r.qm = s_st[L][2];
        r.qs = s_st[L][3];
        r.pad[0] = r.pad[1] = 0;
        job.seqs[b] = r;  // read by the next launch on the stream
      }
    } else {
      int K = job.gamma;
      for (int jj = 0; jj < job.gamma; ++jj)
        if (!s_pass[jj]) {
          K = jj;
          break;
        }
      job.out_len[b] = K;
    }
  }
}

// ---- residual draw of the distribution-preserving ratio rule ---------------
//
// After the acceptance pass has fixed L and the statistics of row L, the next
// token is drawn by inverse CDF in vocabulary order: weights w(v) = max(0,
// p(v) - q(v)) (p alone at the bonus row), target t = u W with W the total,
// draw = the first v whose running weight exceeds t.  The CDF is defined by
// one fixed summation tree: each thread sums its own contiguous segment of
// `seg` elements in index order; a wave sums 4 consecutive thread sums and
// takes an inclusive scan over its 64 lanes (one chunk); the last workgroup
// scans the chunk totals over lanes.  The search re-walks the same tree from
// the top (chunk, lane, thread, element) with the same arithmetic, so every
// partial sum it compares is bit-identical to the one that defined the total.
// If rounding leaves t at or beyond a level's total, the last positive weight
// of that level is taken.
#pragma clang fp contract(off)
template <typename T, int VEC>
__device__ inline void load_vals(const T* ptr, float* v) {
  static_assert(VEC == 1 || VEC * sizeof(T) == 16, "one element or one 16-byte load");
  if constexpr (VEC > 1) {
    unpack16(load16(ptr), v, T());
  } else {
    v[0] = Elem<T>::to_f32(*ptr);
  }
}

struct DrawRow {
  const void* p;
  const void* q;  // nullptr: weights are p alone
  float m, inv_s, qm, inv_qs;
  int use_p;  // residual total not positive: draw from p
};

template <typename T>
__device__ inline float draw_weight(const DrawRow& d, float zp, float zq) {
  const float pv = __expf(zp - d.m) * d.inv_s;
  if (d.use_p || d.q == nullptr) return pv;
  const float diff = pv - __expf(zq - d.qm) * d.inv_qs;
  return diff > 0.f ? diff : 0.f;
}

// Sum of the weights of elements [lo, hi) in index order (both the residual and p alone).
template <typename T, int VEC>
__device__ inline void segment_sums(const DrawRow& d, int lo, int hi, float& wr, float& wp) {
  const T* pr = reinterpret_cast<const T*>(d.p);
  const T* qr = reinterpret_cast<const T*>(d.q);
  wr = 0.f;
  wp = 0.f;
  for (int e = lo; e < hi; e += VEC) {
    float zp[VEC], zq[VEC];
    load_vals<T, VEC>(pr + e, zp);
    if (qr) load_vals<T, VEC>(qr + e, zq);
#pragma unroll
    for (int t = 0; t < VEC; ++t) {
      const float pv = __expf(zp[t] - d.m) * d.inv_s;
      float r = pv;
      if (qr) {
        const float diff = pv - __expf(zq[t] - d.qm) * d.inv_qs;
        r = diff > 0.f ? diff : 0.f;
      }
      wr += r;
      wp += pv;
    }
  }
}

// First element of [lo, hi) whose running weight exceeds t (same order and arithmetic as segment_sums);
// the last positive one if none does.
template <typename T, int VEC>
__device__ inline int segment_find(const DrawRow& d, int lo, int hi, float t) {
  const T* pr = reinterpret_cast<const T*>(d.p);
  const T* qr = reinterpret_cast<const T*>(d.q);
  float c = 0.f;
  int last = lo;
  for (int e = lo; e < hi; e += VEC) {
    float zp[VEC], zq[VEC];
    load_vals<T, VEC>(pr + e, zp);
    if (qr && !d.use_p) load_vals<T, VEC>(qr + e, zq);
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const float w = draw_weight<T>(d, zp[k], (qr && !d.use_p) ? zq[k] : 0.f);
      if (w > 0.f) {
        if (c + w > t) return e + k;
        last = e + k;
      }
      c += w;
    }
  }
  return last;
}

// Wave 0: lane l combines thread sums 4l..4l+3 in order, then an inclusive scan over the lanes.
__device__ inline float lane_sum4(const float* w, int lane) {
  return ((w[4 * lane] + w[4 * lane + 1]) + w[4 * lane + 2]) + w[4 * lane + 3];
}
__device__ inline float wave_incl_scan(float v, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const float y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  return v;
}
// Index of the first lane whose inclusive sum exceeds t and the remainder of t past the lanes before it;
// with none, the last lane of positive weight and t = +inf (take the last positive weight below).
__device__ inline int lane_select(float incl, float w, float t, int lane, float& t_rest) {
  const uint64_t hit = __ballot(incl > t);
  const float excl = __shfl_up(incl, 1);
  if (hit) {
    const int l = __builtin_ctzll(hit);
    const float e = __shfl(excl, l);
    t_rest = l == 0 ? t : t - e;
    return l;
  }
  const uint64_t pos = __ballot(w > 0.f);
  t_rest = INFINITY;
  return pos ? 63 - __builtin_clzll(pos) : 0;
}

template <typename T, int VEC>
__global__ void __launch_bounds__(kThreads) resample_kernel(Job job) {
  __shared__ float s_wr[kThreads], s_wp[kThreads];
  __shared__ int s_last, s_sel;
  __shared__ float s_t;
  const int c = blockIdx.x % job.C2, b = blockIdx.x / job.C2;
  const SeqRec r = job.seqs[b];
  if (r.bad) return;  // every workgroup of b returns: nobody arrives, next stays the argmax
  DrawRow d;
  d.p = reinterpret_cast<const T*>(job.p) + (size_t)b * job.p_seq_stride + (size_t)r.L * job.p_row_stride;
  d.q = r.L < job.gamma ? reinterpret_cast<const T*>(job.q) + (size_t)b * job.q_seq_stride + (size_t)r.L * job.V
                        : nullptr;
  d.m = r.m;
  d.inv_s = 1.f / r.s;
  d.qm = r.qm;
  d.inv_qs = d.q ? 1.f / r.qs : 0.f;
  d.use_p = 0;
  const int tid = threadIdx.x, lane = tid % kWave;
  const int chunk2 = kThreads * job.seg;

  {  // this chunk's totals
    const int lo = min(job.V, c * chunk2 + tid * job.seg), hi = min(job.V, lo + job.seg);
    float wr, wp;
    segment_sums<T, VEC>(d, lo, hi, wr, wp);
    s_wr[tid] = wr;
    s_wp[tid] = wp;
    __syncthreads();
    if (tid < kWave) {
      const float tr = __shfl(wave_incl_scan(lane_sum4(s_wr, lane), lane), kWave - 1);
      const float tp = __shfl(wave_incl_scan(lane_sum4(s_wp, lane), lane), kWave - 1);
      if (tid == 0) {
        st_coherent(&job.rrecs[(size_t)b * 64 + c].r, tr);
        st_coherent(&job.rrecs[(size_t)b * 64 + c].p, tp);
      }
    }
  }
  if (!arrive_last(&job.counters2[b * kSeqCntStride], job.C2, &s_last)) return;

  // ---- last workgroup of sequence b: select the chunk, then the lane, thread and element ----
  if (tid < kWave) {
    const bool have = lane < job.C2;
    const float wr = have ? ld_coherent(&job.rrecs[(size_t)b * 64 + lane].r) : 0.f;
    const float wp = have ? ld_coherent(&job.rrecs[(size_t)b * 64 + lane].p) : 0.f;
    const float ir = wave_incl_scan(wr, lane), ip = wave_incl_scan(wp, lane);
    const float R = __shfl(ir, kWave - 1);
    const int use_p = !(R > 0.f);
    const float W = use_p ? __shfl(ip, kWave - 1) : R;
    const float t = job.u[(size_t)b * job.u_stride + job.gamma] * W;
    float t_rest;
    const int cs = lane_select(use_p ? ip : ir, use_p ? wp : wr, t, lane, t_rest);
    if (tid == 0) {
      s_sel = cs | (use_p << 16);
      s_t = t_rest;
    }
  }
  __syncthreads();
  const int cs = s_sel & 0xffff;
  d.use_p = s_sel >> 16;
  float t = s_t;
  const int lo = min(job.V, cs * chunk2 + tid * job.seg), hi = min(job.V, lo + job.seg);
  {
    float wr, wp;
    segment_sums<T, VEC>(d, lo, hi, wr, wp);
    s_wr[tid] = d.use_p ? wp : wr;
  }
  __syncthreads();
  if (tid < kWave) {
    const float ls = lane_sum4(s_wr, lane);
    float t_rest;
    const int l = lane_select(wave_incl_scan(ls, lane), ls, t, lane, t_rest);
    if (tid == 0) {
      // the thread within lane l's four, in the lane sum's order
      int pick = -1, lastpos = 4 * l;
      float run = 0.f, t_thr = INFINITY;
      for (int i = 0; i < 4; ++i) {
        const float w = s_wr[4 * l + i];
        if (w > 0.f) {
          if (pick < 0 && run + w > t_rest) {
            pick = 4 * l + i;
            t_thr = t_rest - run;
          }
          lastpos = 4 * l + i;
        }
        run += w;
      }
      s_sel = pick >= 0 ? pick : lastpos;
      s_t = pick >= 0 ? t_thr : INFINITY;
    }
  }
  __syncthreads();
  if (tid == s_sel) job.out_next[b] = segment_find<T, VEC>(d, lo, hi, s_t);
}
#pragma clang fp contract(on)

__global__ void fill_i32_kernel(int32_t* p, int n, int v) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

int choose_vec(const void* p, size_t seq_stride, size_t row_stride, int V, int esize, const void* q,
               size_t q_seq_stride) {
  const int vec = 16 / esize;
  auto al = [&](const void* ptr, size_t s1, size_t s2) {
    return ptr == nullptr ||
           (((uintptr_t)ptr % 16) == 0 && (s1 * esize) % 16 == 0 && (s2 * esize) % 16 == 0);
  };
  if (V % vec == 0 && al(p, seq_stride, row_stride) && al(q, q_seq_stride, (size_t)V)) return vec;
  return 1;
}

// Chunks per row: as many workgroups as can be resident at once (one round: a second, partly empty
// round would cost a whole workgroup's time), no chunk under 8192 elements, at most 64 (one finishing
// thread folds a row's records).  resident <= 2048 (8 workgroups on each of 256 CUs) bounds the workspace.
int chunks_for(int nrows, int V, int resident = 2048) {
  int c = resident / (nrows > 0 ? nrows : 1);
  c = min(c, (int)ceil_div(V, 8192));
  c = min(c, 64);
  return max(1, c);
}

size_t counters_region(int B) { return ((size_t)B * kSeqCntStride * sizeof(int) + 255) / 256 * 256; }
// Residual draw records: per sequence the row-L statistics and up to 64 chunk totals.
size_t draw_region(int B) { return (size_t)B * (sizeof(SeqRec) + 64 * sizeof(ResRec)); }

// Workspace: [acceptance counters][draw counters][SeqRec x B][ResRec x B x 64][RowRec records]
size_t rowstats_ws(int B, int rows, int V) {
  size_t best = 0;
  {
    // rows x chunks <= max(rows, 2048) for any row count (chunks_for gives 1 or at most 2048 / rows), so the
    // same bound serves the gamma confidence rows and the gamma + 1 acceptance rows
    const size_t nrec = std::max<size_t>((size_t)B * rows, 2048);
    best = nrec * sizeof(RowRec);
  }
  return 2 * counters_region(B) + draw_region(B) + best;
}

// Elements per thread of the residual draw: at least 16, and few enough chunks (<= 64) for one wave.
int draw_seg(int V) {
  const int need = (int)ceil_div(ceil_div(V, 64), kThreads);
  return need <= 16 ? 16 : (int)ceil_div(need, 16) * 16;
}

template <typename T>
int launch_draw(Job& job, int vec, hipStream_t st) {
  const int blocks = job.B * job.C2;
  constexpr int kVec = 16 / sizeof(T);  // one 16-byte load (choose_vec returns this or 1)
  prof_begin(PROF_ACCEPT, st);
  if (vec == kVec)
    hipLaunchKernelGGL((resample_kernel<T, kVec>), dim3(blocks), dim3(kThreads), 0, st, job);
  else
    hipLaunchKernelGGL((resample_kernel<T, 1>), dim3(blocks), dim3(kThreads), 0, st, job);
  prof_end(PROF_ACCEPT, st);
  return check_launch("resample_kernel");
}

// Resident workgroups of one kernel instantiation on the whole device (occupancy x compute units), queried
// once per instantiation.
template <typename T, typename TQ, int VEC, int KIND, bool kSum, bool kCount, bool kQ>
int resident_wgs() {
  static int cached = 0;
  if (cached == 0) {
    int occ = 0, cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, rowstats_kernel<T, TQ, VEC, KIND, kSum, kCount, kQ>, kThreads,
                                                     0) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || occ < 1 || cus < 1)
      return 2048;
    cached = occ * cus;
  }
  return cached;
}

// Arrivals on one sequence's counter (rows x chunks) at most: they serialize on its line, and past a few
// hundred they cost more than the extra chunks gain (one sequence of 33 rows: 18 chunks per row 21 us, 8
// chunks 13 us)
constexpr int kMaxSeqArrivals = 256;

// Chunks per row for this kernel's occupancy; never more than the workspace was sized for.
inline void fit_chunks(Job& job, int vec, int resident) {
  const int nrows = job.B * job.rows;
  const int c = std::min({job.C, chunks_for(nrows, job.V, std::min(resident, 2048)),
                          std::max(1, kMaxSeqArrivals / std::max(1, job.rows))});
  job.chunk = (int)ceil_div(ceil_div(job.V, c), vec) * vec;
  job.C = (int)ceil_div(job.V, job.chunk);
}

template <int KIND, bool kSum, bool kCount, bool kQ, typename T, typename TQ>
int launch_t(Job& job, int vec, hipStream_t st) {
  constexpr int kVec = 16 / sizeof(T);
  fit_chunks(job, vec, vec == kVec ? resident_wgs<T, TQ, kVec, KIND, kSum, kCount, kQ>()
                                    : resident_wgs<T, TQ, 1, KIND, kSum, kCount, kQ>());
  const int blocks = job.B * job.rows * job.C;
  const unsigned prof = KIND == kAccept ? PROF_ACCEPT : PROF_CONF;
  prof_begin(prof, st);
  if (vec == kVec)
    hipLaunchKernelGGL((rowstats_kernel<T, TQ, kVec, KIND, kSum, kCount, kQ>), dim3(blocks), dim3(kThreads), 0, st, job);
  else
    hipLaunchKernelGGL((rowstats_kernel<T, TQ, 1, KIND, kSum, kCount, kQ>), dim3(blocks), dim3(kThreads), 0, st, job);
  prof_end(prof, st);
  return check_launch("rowstats_kernel");
}

}  // namespace
}  // namespace sdd

using namespace sdd;

extern "C" int sdd_rowstats_workspace_bytes(int B, int gamma, int V, size_t* bytes) {
  SDD_REQUIRE(bytes != nullptr, "bytes is NULL");
  SDD_REQUIRE(B > 0 && gamma >= 0 && gamma <= 64 && V > 0, "bad shape B=%d gamma=%d V=%d", B, gamma, V);
  *bytes = rowstats_ws(B, gamma + 1, V);
  return SDD_OK;
}

static int setup_ws(Job& job, void* ws, size_t ws_bytes, int vec) {
  job.C = chunks_for(job.B * job.rows, job.V);  // the workspace bound; launch_t fits it to the kernel
  job.chunk = (int)ceil_div(ceil_div(job.V, job.C), vec) * vec;
  job.C = (int)ceil_div(job.V, job.chunk);
  if (job.C > 64) return fail(SDD_EUNSUPPORTED, "vocabulary of %d needs %d chunks per row (at most 64)", job.V, job.C);
  size_t need = rowstats_ws(job.B, job.rows, job.V);
  if (ws == nullptr || ws_bytes < need)
    return fail(SDD_ENOMEM, "rowstats workspace needs %zu bytes, got %zu", need, ws_bytes);
  if ((uintptr_t)ws % 16) return fail(SDD_EINVAL, "workspace must be 16-byte aligned");
  char* w = reinterpret_cast<char*>(ws);
  job.counters = reinterpret_cast<int*>(w);
  job.counters2 = reinterpret_cast<int*>(w + counters_region(job.B));
  job.seqs = reinterpret_cast<SeqRec*>(w + 2 * counters_region(job.B));
  job.rrecs = reinterpret_cast<ResRec*>(w + 2 * counters_region(job.B) + (size_t)job.B * sizeof(SeqRec));
  job.recs = reinterpret_cast<RowRec*>(w + 2 * counters_region(job.B) + draw_region(job.B));
  return SDD_OK;
}

extern "C" int sdd_accept(const int32_t* draft, const void* p_logits, int p_dtype, const void* q_logits,
                          int q_dtype, size_t q_seq_stride, const float* uniforms, int B, int gamma, int V,
                          int mode, int k, float lenience, int32_t* accepted_len, int32_t* next_token,
                          int32_t* flags, void* ws, size_t ws_bytes, sdd_stream_t stream) {
  SDD_REQUIRE(p_logits && accepted_len && next_token, "NULL required pointer");
  SDD_REQUIRE(B > 0 && gamma >= 0 && gamma <= 64 && V > 0, "bad shape B=%d gamma=%d V=%d", B, gamma, V);
  SDD_REQUIRE(gamma == 0 || draft, "draft is NULL");
  SDD_REQUIRE(mode >= SDD_GREEDY && mode <= SDD_RATIO_SAMPLE, "bad mode %d", mode);
  SDD_REQUIRE(mode != SDD_TOPK || k >= 1, "top-k needs k >= 1 (k=%d)", k);
  SDD_REQUIRE(mode != SDD_LENIENT || (lenience > 0.f && lenience <= 1.f), "lenience must be in (0,1]");
  SDD_REQUIRE(p_dtype == SDD_F32 || p_dtype == SDD_BF16, "bad p dtype");
  const bool sample = mode == SDD_RATIO_SAMPLE;
  if (sample) SDD_REQUIRE(uniforms, "the residual draw needs uniforms [B][gamma+1]");
  const bool ratio = (mode == SDD_RATIO || sample) && gamma > 0;
  if (ratio) {
    SDD_REQUIRE(q_logits && uniforms, "ratio mode needs drafter logits and uniforms");
    SDD_REQUIRE(q_dtype == p_dtype, "ratio mode needs drafter and target logits of one dtype");
    SDD_REQUIRE(q_seq_stride >= (size_t)gamma * V, "q_seq_stride too small");
  }
  Job job{};
  job.p = p_logits;
  job.p_row_stride = (size_t)V;
  job.p_seq_stride = (size_t)(gamma + 1) * V;
  job.q = ratio ? q_logits : nullptr;
  job.q_seq_stride = q_seq_stride;
  job.draft = gamma > 0 ? draft : nullptr;
  job.u = uniforms;
  job.B = B;
  job.gamma = gamma;
  job.V = V;
  job.rows = gamma + 1;
  job.mode = (mode == SDD_LENIENT && lenience == 1.f) ? SDD_GREEDY : sample ? SDD_RATIO : mode;
  job.sample = sample ? 1 : 0;
  job.u_stride = sample ? gamma + 1 : gamma;
  job.seg = draw_seg(V);
  job.C2 = (int)ceil_div(V, (int64_t)kThreads * job.seg);
  if (job.C2 > 64) return fail(SDD_EUNSUPPORTED, "vocabulary of %d needs %d draw chunks (at most 64)", V, job.C2);
  job.k = k;
  job.log_len = (float)std::log((double)lenience);
  job.out_len = accepted_len;
  job.out_next = next_token;
  job.out_flags = flags;
  const int es = p_dtype == SDD_F32 ? 4 : 2;
  const int vec = choose_vec(p_logits, job.p_seq_stride, job.p_row_stride, V, es, job.q, q_seq_stride);
  int rc = setup_ws(job, ws, ws_bytes, vec);
  if (rc) return rc;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const bool bf = p_dtype == SDD_BF16;
  if (sample) {  // acceptance pass (ratio test, every row's statistics), then the draw from row L
    rc = bf ? launch_t<kAccept, true, false, true, uint16_t, uint16_t>(job, vec, st)
            : launch_t<kAccept, true, false, true, float, float>(job, vec, st);
    if (rc) return rc;
    return bf ? launch_draw<uint16_t>(job, vec, st) : launch_draw<float>(job, vec, st);
  }
  switch (job.mode) {
    case SDD_GREEDY:
    case SDD_LENIENT:
      return bf ? launch_t<kAccept, false, false, false, uint16_t, uint16_t>(job, vec, st)
                : launch_t<kAccept, false, false, false, float, float>(job, vec, st);
    case SDD_TOPK:
      return bf ? launch_t<kAccept, false, true, false, uint16_t, uint16_t>(job, vec, st)
                : launch_t<kAccept, false, true, false, float, float>(job, vec, st);
    default:
      if (!ratio)  // gamma == 0: only the bonus row's argmax is needed
        return bf ? launch_t<kAccept, false, false, false, uint16_t, uint16_t>(job, vec, st)
                  : launch_t<kAccept, false, false, false, float, float>(job, vec, st);
      return bf ? launch_t<kAccept, true, false, true, uint16_t, uint16_t>(job, vec, st)
                : launch_t<kAccept, true, false, true, float, float>(job, vec, st);
  }
}

// ---------------------------------------------------------------------------
// sdd_accept_noalloc: the acceptance test for callers that cannot allocate device memory.  Its workspace
// is this file-scope array (one copy per GPU, held until the process ends).  In host code `scratch` names a
// host-side stand-in, never the device memory: every host use goes through the per-device address that
// hipGetSymbolAddress returns.
constexpr size_t kNoallocScratchBytes = 256 * 1024;
static __device__ __align__(256) char scratch[kNoallocScratchBytes];

namespace {
__global__ void zero_scratch_kernel(uint32_t* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0u;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device (nullptr: not set up)

// The current device's scratch address; set up once per device (address lookup, and a kernel that zeroes the
// arrival counters on `st`; every call leaves them zero again).
int scratch_for_current_device(hipStream_t st, void** out) {
  int dev = 0;
  SDD_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(SDD_EUNSUPPORTED, "device %d beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    SDD_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(SDD_EHIP, "hipGetSymbolAddress returned no address for the scratch array");
    // a kernel, not hipMemsetAsync: the first call may sit inside a captured graph
    const int n = (int)(kNoallocScratchBytes / 4);
    hipLaunchKernelGGL(zero_scratch_kernel, dim3(64), dim3(256), 0, st, reinterpret_cast<uint32_t*>(ptr), n);
    int rc = check_launch("zero_scratch_kernel");
    if (rc) return rc;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return SDD_OK;
}
}  // namespace

extern "C" int sdd_accept_noalloc(const int32_t* draft, const void* p_logits, int p_dtype, const void* q_logits,
                                  int q_dtype, size_t q_seq_stride, const float* uniforms, int B, int gamma, int V,
                                  int mode, int k, float lenience, int32_t* accepted_len, int32_t* next_token,
                                  int32_t* flags, sdd_stream_t stream) {
  SDD_REQUIRE(B > 0 && gamma >= 0 && gamma <= 64 && V > 0, "bad shape B=%d gamma=%d V=%d", B, gamma, V);
  const size_t need = rowstats_ws(B, gamma + 1, V);
  if (need > kNoallocScratchBytes)
    return fail(SDD_ECAPACITY, "B=%d, gamma=%d needs %zu bytes of scratch; sdd_accept_noalloc holds %zu (use sdd_accept)",
                B, gamma, need, kNoallocScratchBytes);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  void* ws = nullptr;
  int rc = scratch_for_current_device(st, &ws);
  if (rc) return rc;
  return sdd_accept(draft, p_logits, p_dtype, q_logits, q_dtype, q_seq_stride, uniforms, B, gamma, V, mode, k, lenience,
                    accepted_len, next_token, flags, ws, kNoallocScratchBytes, stream);
}

extern "C" int sdd_confidence_prefix(const void* logits, int dtype, size_t seq_stride, int B, int gamma,
                                     int V, float tau, int32_t* skip_len, float* log_conf,
                                     const int32_t* draft, float* log_p_draft, void* ws, size_t ws_bytes,
                                     sdd_stream_t stream) {
  SDD_REQUIRE(logits && skip_len, "NULL required pointer");
  SDD_REQUIRE(B > 0 && gamma >= 0 && gamma <= 64 && V > 0, "bad shape B=%d gamma=%d V=%d", B, gamma, V);
  SDD_REQUIRE(!__builtin_isnan(tau), "tau is NaN");
  SDD_REQUIRE(dtype == SDD_F32 || dtype == SDD_BF16, "bad dtype");
  SDD_REQUIRE(seq_stride >= (size_t)gamma * V, "seq_stride too small");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (gamma == 0) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3((B + 255) / 256), dim3(256), 0, st, skip_len, B, 0);
    return check_launch("fill_i32_kernel");
  }
  Job job{};
  job.p = logits;
  job.p_row_stride = (size_t)V;
  job.p_seq_stride = seq_stride;
  job.draft = draft;
  job.B = B;
  job.gamma = gamma;
  job.V = V;
  job.rows = gamma;
  job.log_tau = tau > 0.f ? (float)std::log((double)tau) : -INFINITY;
  job.out_len = skip_len;
  job.out_log_conf = log_conf;
  job.out_log_pdraft = draft ? log_p_draft : nullptr;
  const int es = dtype == SDD_F32 ? 4 : 2;
  const int vec = choose_vec(logits, seq_stride, (size_t)V, V, es, nullptr, 0);
  int rc = setup_ws(job, ws, ws_bytes, vec);
  if (rc) return rc;
  return dtype == SDD_BF16 ? launch_t<kConfidence, true, false, false, uint16_t, uint16_t>(job, vec, st)
                           : launch_t<kConfidence, true, false, false, float, float>(job, vec, st);
}
