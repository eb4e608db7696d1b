// Block verification forward pass of the target decoder on gfx950.
//
// One verify call (Sec. 3.1: the target scores a drafted block and accepts a
// prefix) runs the gamma drafts plus one bonus position of every sequence
// through the decoder against its KV cache.  At gamma + 1 = 33 rows each
// projection is a skinny, weight-streaming contraction, so the call is bound
// by reading the weights from HBM once.
//
// Kernels of one call:
//   embed        gathers token rows, the residual stream x (fp32), the GEMM
//                input xa = T(x * g) and the RMSNorm row scale r
//   per layer:   gemm<QKV>   fused q/k/v projection; epilogue: row scale, per-head
//                            QK RMSNorm, rotate-half RoPE, K/V append to the cache
//                attention   causal GQA attention of the block rows over the cache
//                gemm<RESID> output projection + residual; epilogue also writes the
//                            next GEMM input and the next RMSNorm row scale
//                gemm<SWIGLU> fused gate/up projection; epilogue silu(gate) * up
//                gemm<RESID> down projection + residual
//   gemm<LOGITS> final norm (row scale) + LM head, fp32 logits and row argmax
//
// The GEMMs are stream-K over (column group, k-tile) units: every workgroup
// gets an equal contiguous share of the weight bytes, whatever the matrix
// shape, so all compute units stream the same amount.  A column group whose
// K-range is split between workgroups is reduced by its last-arriving
// contributor, which sums the partials in a fixed order (deterministic).
#include <algorithm>
#include <type_traits>
#include <cmath>
#include <new>

#include "gemm.h"

namespace sdd {

// Row argmax over the per-column-group maxima of the LM head: one workgroup per
// row; max value, lowest index among equal maxima (NaN never wins).
__global__ void __launch_bounds__(256) row_argmax_kernel(const float* amax_v, const int* amax_i, int G, int mp,
                                                        const RowInfo* rows, int32_t* out) {
  __shared__ float sv[256];
  __shared__ int si[256];
  const int m = blockIdx.x, t = threadIdx.x;
  float bv = -INFINITY;
  int bi = -1;
  for (int g = t; g < G; g += 256) {
    const float v = amax_v[(int64_t)g * mp + m];
    const int i = amax_i[(int64_t)g * mp + m];
    if (arg_better(v, i, bv, bi)) {
      bv = v;
      bi = i;
    }
  }
  sv[t] = bv;
  si[t] = bi;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (t < o && arg_better(sv[t + o], si[t + o], sv[t], si[t])) {
      sv[t] = sv[t + o];
      si[t] = si[t + o];
    }
    __syncthreads();
  }
  if (t == 0 && rows[m].valid) out[m] = si[0] < 0 ? 0 : si[0];
}

template <typename T, int TB, int NG, int EPI>
__global__ void __launch_bounds__(kGemmThreads, 1) gemm_kernel(GemmArgs a) {
  constexpr int C = NG * 16;       // output columns of a column group
  constexpr int CP = C + 4;        // LDS row stride of the output tile (16-byte row writes hit distinct banks)
  constexpr int R = TB * 16;       // padded rows of this pass
  constexpr int NACC = NG * TB;    // 16x16 accumulator tiles per wave
  constexpr int IPW = (NACC + 3) / 4;
  constexpr int EPL = 16 / sizeof(T);
  constexpr int KTILE = 4 * EPL;
  constexpr int EPT4 = (R * C / 4 + kGemmThreads - 1) / kGemmThreads;  // tile float4s per thread (cross-workgroup reduction)
  // each wave's accumulators; after the cross-wave sum the same memory holds the output tile [R][CP]
  __shared__ f32x4 red[4][NACC][kWave];
  __shared__ RowInfo s_ri[kMaxPassRows];
  __shared__ float s_rs[kMaxPassRows];
  __shared__ float s_part4[4][kMaxPassRows];
  __shared__ int s_flag;
  float* tile = reinterpret_cast<float*>(&red[0][0][0]);
  static_assert(4 * NACC * kWave * 4 >= R * CP, "tile must fit the reduction buffer");
  touch_kernargs<GemmArgs>();

  const int w = blockIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const uint32_t KT = (uint32_t)a.KT, G = (uint32_t)a.G, SC = (uint32_t)a.segc;
  const uint32_t u0 = unit_start(w, KT, G, SC, a.n_wg), u1 = unit_start(w + 1, KT, G, SC, a.n_wg);
  const int g_first = (int)(u0 / KT);
  const uint4* W = reinterpret_cast<const uint4*>(a.W);
  const int MC = a.M * C;
  // activation fragments by buffer loads: descriptor in scalars, the lane's byte offset in one 32-bit register,
  // the k-step as a scalar offset, so that no address registers are recomputed in the stream (a recomputed
  // address register can alias an in-flight load's destination and force a full wait)
  // The descriptor's range ends at the pass's last row: fragments of the padded rows (33 rows pad to 48) are
  // out of range, read as zero without a memory access (a row's offset is at least row x ldx elements and
  // below (row + 1) x ldx, so every real row is in range and every padded one is not)
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(a.X), 0, (a.m0 + a.M) * a.ldx * (int)sizeof(T), kBufferRsrcWord3);
  const int xlane = ((a.m0 + lane % 16) * a.ldx + (lane / 16) * EPL) * (int)sizeof(T);  // < 2^31: checked on the host
  const int xrow16 = 16 * a.ldx * (int)sizeof(T);
  // the whole matrix, stored in the order of this launch's plan: the i-th unit (NG tiles) of workgroup w at
  // slot i * n_wg + w, so a workgroup's consecutive units are n_wg slots apart
  const uint32_t slot_bytes = (uint32_t)NG * kWave * 16, wstride = (uint32_t)a.n_wg * slot_bytes;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(W), 0, (int)(a.share * wstride), kBufferRsrcWord3);
  const uint32_t kstep4w = 4u * wstride;    // bytes between a wave's consecutive k-steps
  const uint32_t kstep4x = 4u * KTILE * (uint32_t)sizeof(T);
  const int wlane = lane * 16;

  // a descriptor with no range: every load through it returns zero without a memory access
  const __amdgpu_buffer_rsrc_t nrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(W), 0, 0, kBufferRsrcWord3);

  // Local k-step kt of this wave in its segment: the NG contiguous 1 KiB
  // weight tiles of its column group and the TB activation fragments, all
  // buffer loads (descriptors in scalars, the lane's offset in one register,
  // the k-step as a scalar offset: recomputed address registers could alias an
  // in-flight load's destination and force a wait for every load).  The loads
  // are unconditional, so that the compiler can wait for exactly the oldest
  // stage; a k-step past the wave's range (the stream's last stages) selects
  // the empty descriptor and so costs no memory traffic (its offset is not
  // used, and unsigned arithmetic keeps it defined).
  auto load = [&](uint32_t wo, uint32_t xo, int kt, int kz, uint4* wa, uint4* xb) {
    const bool in = kt < kz;
    const __amdgpu_buffer_rsrc_t wd = in ? wrs : nrs, xd = in ? xrs : nrs;
#pragma unroll
    for (int nt = 0; nt < NG; ++nt)
      wa[nt] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                             wd, wlane, (int)(wo + (uint32_t)kt * kstep4w + (uint32_t)nt * kWave * 16), kNtCpol));
#pragma unroll
    for (int tb = 0; tb < TB; ++tb)
      xb[tb] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xd, xlane + tb * xrow16,
                                                                                 (int)(xo + (uint32_t)kt * kstep4x), 0));
    // keep the next stages' loads ahead of this stage's MFMAs
    __builtin_amdgcn_sched_barrier(0);
  };
  // A segment is this workgroup's part of one column group: k-tiles [kb, ke);
  // wave w streams k-tiles kb + w, kb + w + 4, ... (kz of them), so that at any
  // time the four waves read adjacent k-steps and, the matrix being stored
  // k-step by k-step, the launch reads few long runs of memory.  wo and xo are
  // the byte offsets of the wave's first k-step in the weights and in an
  // activation row.
  struct Seg {
    int g, kb, ke, ka, kz;
    uint32_t wo, xo;
  };
  auto make_seg = [&](uint32_t u) {
    Seg s;
    s.g = (int)(u / KT);
    s.kb = (int)(u - (uint32_t)s.g * KT);
    s.ke = (int)std::min<uint32_t>(KT, s.kb + (u1 - u));
    const int S = s.ke - s.kb;
    s.ka = 0;
    s.kz = __builtin_amdgcn_readfirstlane(S > wave ? (S - wave + 3) / 4 : 0);
    const uint32_t k0 = (uint32_t)(s.kb + wave);
    s.wo = __builtin_amdgcn_readfirstlane((u - u0 + (uint32_t)wave) * wstride + (uint32_t)w * slot_bytes);
    s.xo = __builtin_amdgcn_readfirstlane(k0 * KTILE * (uint32_t)sizeof(T));
    return s;
  };
  // Row info and RMSNorm row scales of this pass, used only by the epilogues.
  // The scales come from the producer's per-group sums of squares: four
  // threads per row take every fourth group (in group order), then the four
  // partial sums are added in a fixed order.  Where registers allow (kPreSS
  // groups per thread), the loads go out with the first weight loads and are
  // summed after the first segment's stream, so that the stream does not wait
  // for them; groups beyond kPreSS are loaded when summed.
  // (the gate/up GEMM reads the o_proj's narrower groups: more of them)
  constexpr int kPreSS = (EPI == EPI_RESID || TB > 3) ? 0 : EPI == EPI_SWIGLU ? 20 : 12;
  float pre_ss[kPreSS > 0 ? kPreSS : 1];
  int4 pre_ri = {0, 0, 0, 0};  // RowInfo as one 16-byte load
  static_assert(sizeof(RowInfo) == sizeof(int4), "RowInfo is loaded as one int4");
  auto prologue_issue = [&]() {
    if constexpr (EPI == EPI_QKV || EPI == EPI_LOGITS) {
      if ((int)threadIdx.x < a.M) pre_ri = reinterpret_cast<const int4*>(a.rows)[a.m0 + threadIdx.x];
    }
    if constexpr (kPreSS > 0) {
      const int ng_in = a.ss_in ? a.ss_groups : 0;
      if (ng_in > 0) {
        // unconditional loads (rows past M read row 0, groups past ng_in the last group): one batch in flight
        const int row = threadIdx.x % kMaxPassRows, q4 = threadIdx.x / kMaxPassRows;
        const int64_t rr = a.m0 + (row < a.M ? row : 0);
#pragma unroll
        for (int j = 0; j < kPreSS; ++j) pre_ss[j] = a.ss_in[(int64_t)min(q4 + 4 * j, ng_in - 1) * a.mp + rr];
      }
    }
  };
  auto prologue_finish = [&]() {
    if constexpr (EPI == EPI_QKV || EPI == EPI_LOGITS) {
      if ((int)threadIdx.x < a.M) s_ri[threadIdx.x] = RowInfo{pre_ri.x, pre_ri.y, pre_ri.z, pre_ri.w};
    }
    if constexpr (EPI != EPI_RESID) {
      const int ng_in = a.ss_in ? a.ss_groups : 0;
      const int row = threadIdx.x % kMaxPassRows, q4 = threadIdx.x / kMaxPassRows;
      float ssum = 0.f;
      if (row < a.M) {
#pragma unroll
        for (int j = 0; j < kPreSS; ++j)
          if (q4 + 4 * j < ng_in) ssum += pre_ss[j];
        for (int g0 = q4 + 4 * kPreSS; g0 < ng_in; g0 += 64) {
          float v[16];
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int gg = g0 + 4 * j;
            v[j] = gg < ng_in ? a.ss_in[(int64_t)gg * a.mp + a.m0 + row] : 0.f;
          }
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (g0 + 4 * j < ng_in) ssum += v[j];
        }
      }
      s_part4[q4][row] = ssum;
      __syncthreads();
      if ((int)threadIdx.x < a.M) {
        const int t = threadIdx.x;
        const float tot = (s_part4[0][t] + s_part4[1][t]) + (s_part4[2][t] + s_part4[3][t]);
        s_rs[t] = ng_in ? 1.f / sqrtf(tot / (float)a.d_in + a.eps) : 1.f;
      }
    }
  };
  auto prologue = [&]() {
    prologue_issue();
    if constexpr (kPreSS == 0) prologue_finish();
  };

  // Epilogues that read nothing from global memory let the next segment's first loads go out before them,
  // so that their stores do not stall the next stream (loads and stores complete in order).
  constexpr bool kEarly = EPI == EPI_SWIGLU || EPI == EPI_LOGITS;
  uint4 wa0[NG], wa1[NG], wa2[NG], wa3[NG], xb0[TB], xb1[TB], xb2[TB], xb3[TB];
  auto issue = [&](const Seg& sg) {  // the first three stages (a wave with an empty range loads nothing)
    load(sg.wo, sg.xo, 0, sg.kz, wa0, xb0);
    load(sg.wo, sg.xo, 1, sg.kz, wa1, xb1);
    load(sg.wo, sg.xo, 2, sg.kz, wa2, xb2);
  };
  uint32_t u = u0;
  Seg s = make_seg(u);  // carried across segments: uniform values only
  if constexpr (kEarly) {
    issue(s);
    prologue();  // the prologue's loads queue behind the first weight loads
  }
  for (bool first = true;; first = false) {
    const uint32_t wo = s.wo, xo = s.xo;
    // ---- stream this segment: four register stages, three in flight ----
    if constexpr (!kEarly) {
      issue(s);
      if (first) prologue();
    }
    f32x4 acc[NACC];
#pragma unroll
    for (int i = 0; i < NACC; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    auto mma = [&](const uint4* wa, const uint4* xb) {
#pragma unroll
      for (int nt = 0; nt < NG; ++nt)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) mma_tile<T>(wa[nt], xb[tb], acc[nt * TB + tb]);
    };
    int kt = s.ka;
    if (kt < s.kz) {
      for (; kt + 4 <= s.kz; kt += 4) {
        load(wo, xo, kt + 3, s.kz, wa3, xb3);
        mma(wa0, xb0);
        load(wo, xo, kt + 4, s.kz, wa0, xb0);
        mma(wa1, xb1);
        load(wo, xo, kt + 5, s.kz, wa1, xb1);
        mma(wa2, xb2);
        load(wo, xo, kt + 6, s.kz, wa2, xb2);
        mma(wa3, xb3);
      }
      // 0..3 k-tiles left, already loaded in stages 0..2
      const int left = s.kz - kt;
      if (left > 0) mma(wa0, xb0);
      if (left > 1) mma(wa1, xb1);
      if (left > 2) mma(wa2, xb2);
    }
    if constexpr (kPreSS > 0)
      if (first) prologue_finish();
    const int g = s.g;
    const bool full = s.kb == 0 && s.ke == a.KT;
    const int which = g == g_first ? 0 : 1;
    u += s.ke - s.kb;
    const bool more = u < u1;
    // Epilogues that read nothing from global memory: the next segment's first
    // three stages go out now, so that they stream while this segment is
    // reduced, published and (by its last arriver) finished.  Every older load
    // has landed (the segment's stages were consumed; the clamped reloads past
    // its end touch no memory): waiting for them first, on every path, tells
    // the compiler so.  Otherwise a register that one of them last wrote makes
    // it wait for every load, the next segment's too, before it is reused.
    Seg sn = s;
    if constexpr (kEarly) __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    if (more) {
      sn = make_seg(u);
      if constexpr (kEarly) issue(sn);
    }

    // ---- sum the four waves, (w0 + w2) + (w1 + w3) per element ----
    __syncthreads();  // the previous tile's readers are done
#pragma unroll
    for (int i = 0; i < NACC; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    f32x4 rs[IPW];
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int i = wave + 4 * j;
      if (i < NACC) rs[j] = (red[0][i][lane] + red[2][i][lane]) + (red[1][i][lane] + red[3][i][lane]);
    }
    __syncthreads();  // all reads of red done before the tile overwrites it
    // accumulator tile i = nt*TB + tb, element e: row tb*16 + lane%16, column nt*16 + 4*(lane/16) + e
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const int i = wave + 4 * j;
      if (i < NACC)
        *reinterpret_cast<f32x4*>(&tile[((i % TB) * 16 + lane % 16) * CP + (i / TB) * 16 + 4 * (lane / 16)]) = rs[j];
    }
    __syncthreads();

    bool fin = true;
    if (!full) {
      // ---- split column group: publish the partial, the last contributor reduces ----
      // Partials move as 16-byte device-coherent (sc1) buffer accesses: thread t
      // owns the float4s t, t + 256, ... of the [M][C] partial (C is a multiple of
      // 4, so a float4 never straddles a row).
      const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7fffffff, kBufferRsrcWord3);
      const int my_off = ((w * 2 + which) * MC) * 4;  // byte offset of this partial (< 2^31: the buffer is 16 MiB)
      f32x4 pv[EPT4];  // all tile reads first: the stores would otherwise wait on each
#pragma unroll
      for (int e = 0; e < EPT4; ++e) {
        const int i = 4 * (threadIdx.x + e * kGemmThreads);
        pv[e] = i < R * C ? *reinterpret_cast<const f32x4*>(&tile[(i / C) * CP + i % C]) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int e = 0; e < EPT4; ++e) {
        const int i = 4 * (threadIdx.x + e * kGemmThreads);
        if (i < MC) __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, pv[e]), prs, my_off + 4 * i, 0, kCoherentCpol);
      }
      const int wf = unit_owner((uint32_t)g * KT, KT, G, SC, a.n_wg);
      const int wl = unit_owner((uint32_t)(g + 1) * KT - 1, KT, G, SC, a.n_wg);
      fin = arrive_last(&a.cnt[g * kCntStride], wl - wf + 1, &s_flag);
      if (fin) {
        // contributors added in workgroup order; FB contributors' loads in flight at once
        constexpr int FB = EPT4 >= 8 ? 2 : EPT4 >= 4 ? 4 : 8;
        f32x4 sum[EPT4];
#pragma unroll
        for (int e = 0; e < EPT4; ++e) sum[e] = f32x4{0.f, 0.f, 0.f, 0.f};
        // a contributor published into its slot 0 when g is its share's first group: every contributor but
        // the first, whose share starts inside group g or before it
        const bool wf_first = unit_start(wf, KT, G, SC, a.n_wg) == (uint32_t)g * KT;
        for (int ww = wf; ww <= wl; ww += FB) {
          f32x4 v[FB][EPT4];
#pragma unroll
          for (int q = 0; q < FB; ++q) {
            const int wq = std::min(ww + q, wl);
            const int slot = (wq > wf || wf_first) ? 0 : 1;
            const int src_off = ((wq * 2 + slot) * MC) * 4;
#pragma unroll
            for (int e = 0; e < EPT4; ++e) {
              const int i = 4 * (threadIdx.x + e * kGemmThreads);
              v[q][e] = (ww + q <= wl && i < MC)
                            ? __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(prs, src_off + 4 * i, 0, kCoherentCpol))
                            : f32x4{0.f, 0.f, 0.f, 0.f};
            }
          }
#pragma unroll
          for (int q = 0; q < FB; ++q)
            if (ww + q <= wl)
#pragma unroll
              for (int e = 0; e < EPT4; ++e) sum[e] += v[q][e];
        }
#pragma unroll
        for (int e = 0; e < EPT4; ++e) {
          const int i = 4 * (threadIdx.x + e * kGemmThreads);
          if (i < MC) *reinterpret_cast<f32x4*>(&tile[(i / C) * CP + i % C]) = sum[e];
        }
        __syncthreads();
      }
    }

    // A workgroup whose last segment only contributed a partial is done; it
    // loads the next GEMM's first k-steps into L2 while the group's last
    // arriver reduces and runs the epilogue.
    if (!fin && !more && a.Wn && (int)blockIdx.x < a.nwg_n) prefetch_next(a, wave, lane);
    // ---- epilogue on the final tile of column group g ----
    if (fin) {
      if constexpr (EPI == EPI_QKV) epilogue_qkv<T, NG, R>(a, tile, g, s_rs, s_ri);
      if constexpr (EPI == EPI_RESID) epilogue_resid<T, NG, R>(a, tile, g);
      if constexpr (EPI == EPI_SWIGLU) epilogue_swiglu<T, NG, R>(a, tile, g, s_rs);
      if constexpr (EPI == EPI_LOGITS) epilogue_logits<NG, R>(a, tile, g, s_rs, s_ri);
    }
    if (!more) break;
    s = sn;
  }
}

// ---------------------------------------------------------------------------
// Stream-K GEMM with the segment boundaries taken off the stream (bf16, column
// groups of 8 tiles, the register-only epilogues: SwiGLU and the LM head; at
// most 48 rows).  At a segment boundary the 4-wave kernel above issues no new
// loads until the four waves have summed their accumulators, published or
// finished the group: every boundary delays the workgroup's stream by its
// length.  Here a workgroup is 8 waves.  Waves 0-3 stream exactly as the four
// waves above (same k-steps, same accumulation) and at the end of a segment
// only drop their accumulators into LDS and go on streaming the next one.
// Wave 4 + f (f < TB) owns rows 16 f .. 16 f + 15: per segment it sums the
// four streaming waves' accumulators of that row tile, publishes them or
// finishes the group (its arrival counter is per (group, row tile), so these
// waves never wait for each other) and runs the epilogue in the accumulators'
// register layout.  Every sum is taken in the order of the kernel above, so
// both give the same bits.  The two roles hand over through two LDS counters
// (accumulators filled, released): one segment's accumulators at a time.
// Two waves share a SIMD, so a streaming wave keeps 3 register stages (2 in
// flight) where the 4-wave kernel keeps 4.
constexpr int kWsThreads = 512;
// LDS waits give up after this many polls (about 0.2 s): a broken hand-off
// ends the kernel, with bit3 of the sticky error word set, instead of hanging it
constexpr int kWsSpinMax = 1 << 22;

__device__ inline bool ws_wait_geq(int* p, int target) {
  for (int it = 0; it < kWsSpinMax; ++it) {
    if (__hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) return true;
    __builtin_amdgcn_s_sleep(1);
  }
  return false;
}
// a hand-off that gave up: the call's results are invalid, reported in the sticky error word
__device__ inline void ws_fail(int32_t* err, int lane) {
  if (err && lane == 0) atomicOr(err, 8);
}
// one arrival per wave (lane 0), after the wave's earlier LDS accesses
__device__ inline void ws_signal(int* p, int lane) {
  if (lane == 0) __hip_atomic_fetch_add(p, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// SwiGLU of one row tile in the accumulator layout: lane l holds row 16 f + l % 16 and, of tile nt,
// columns nt * 16 + 4 (l / 16) + e; gate tile 2 t and up tile 2 t + 1 hold the same hidden units, so a
// lane computes 4 consecutive hidden outputs per pair on its own.
__device__ inline void ws_epilogue_swiglu(const GemmArgs& a, const f32x4* v, int g, int f, float r, int lane) {
#pragma clang fp contract(off)
  const int mm = 16 * f + lane % 16;
  if (mm >= a.M) return;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    float hv[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float gt = v[2 * t][e] * r;
      const float up = v[2 * t + 1][e] * r;
      hv[e] = gt / (1.f + expf(-gt)) * up;
    }
    const int64_t off = (int64_t)(a.m0 + mm) * a.dff + (int64_t)g * 64 + t * 16 + 4 * (lane / 16);
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.ffh) + off) =
        make_uint2(pack_bf16x2(hv[0], hv[1]), pack_bf16x2(hv[2], hv[3]));
  }
}

// LM head of one row tile in the accumulator layout: fp32 logits of the valid rows and each row's best
// (value, lowest index) over the group's columns below V (a row's 4 lanes combined by exchanges).
__device__ inline void ws_epilogue_logits(const GemmArgs& a, const f32x4* v, int g, int f, float r, bool valid,
                                          int lane) {
#pragma clang fp contract(off)
  const int mm = 16 * f + lane % 16;
  float bv = -INFINITY;
  int bi = -1;
#pragma unroll
  for (int nt = 0; nt < 8; ++nt) {
    const int n0 = g * 128 + nt * 16 + 4 * (lane / 16);
    float x[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) x[e] = v[nt][e] * r;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (n0 + e < a.V && arg_better(x[e], n0 + e, bv, bi)) {
        bv = x[e];
        bi = n0 + e;
      }
    if (mm < a.M && valid) {
      float* lr = a.logits + (int64_t)(a.m0 + mm) * a.V + n0;
      if ((a.V & 3) == 0 && n0 + 4 <= a.V) {
        *reinterpret_cast<f32x4*>(lr) = f32x4{x[0], x[1], x[2], x[3]};
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n0 + e < a.V) lr[e] = x[e];
      }
    }
  }
#pragma unroll
  for (int o = 16; o <= 32; o *= 2) {
    const float v2 = __shfl_xor(bv, o);
    const int i2 = __shfl_xor(bi, o);
    if (arg_better(v2, i2, bv, bi)) {
      bv = v2;
      bi = i2;
    }
  }
  if (lane < 16 && mm < a.M) {
    a.amax_v[(int64_t)g * a.mp + a.m0 + mm] = bv;
    a.amax_i[(int64_t)g * a.mp + a.m0 + mm] = bi;
  }
}

template <int TB, int EPI>
__global__ void __launch_bounds__(kWsThreads, 1) gemm_ws_kernel(GemmArgs a) {
  static_assert(EPI == EPI_SWIGLU || EPI == EPI_LOGITS, "register-only epilogues");
  static_assert(TB >= 1 && TB <= 3, "at most 48 rows");
  constexpr int NG = 8, C = NG * 16, NACC = NG * TB, EPL = 8, KTILE = 32;
  __shared__ f32x4 red[4][NACC][kWave];
  __shared__ int s_fill, s_free;
  touch_kernargs<GemmArgs>();
  const int w = blockIdx.x;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const uint32_t KT = (uint32_t)a.KT, G = (uint32_t)a.G, SC = (uint32_t)a.segc;
  const uint32_t u0 = unit_start(w, KT, G, SC, a.n_wg), u1 = unit_start(w + 1, KT, G, SC, a.n_wg);
  if (threadIdx.x == 0) {
    s_fill = 0;
    s_free = 0;
  }
  __syncthreads();  // the only workgroup barrier: the roles part here

  if (wv < 4) {
    // ---- streaming waves ----
    const int wave = wv;
    const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char*>(a.X), 0, (a.m0 + a.M) * a.ldx * 2, kBufferRsrcWord3);
    const int xlane = ((a.m0 + lane % 16) * a.ldx + (lane / 16) * EPL) * 2;  // < 2^31: checked on the host
    const int xrow16 = 16 * a.ldx * 2;
    const uint32_t slot_bytes = (uint32_t)NG * kWave * 16, wstride = (uint32_t)a.n_wg * slot_bytes;
    const __amdgpu_buffer_rsrc_t wrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.W), 0, (int)(a.share * wstride), kBufferRsrcWord3);
    const __amdgpu_buffer_rsrc_t nrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.W), 0, 0, kBufferRsrcWord3);
    const uint32_t kstep4w = 4u * wstride, kstep4x = 4u * KTILE * 2;
    const int wlane = lane * 16;
    // local k-step kt of this wave in its segment (as in the 4-wave kernel)
    auto load = [&](uint32_t wo, uint32_t xo, int kt, int kz, uint4* wa, uint4* xb) {
      const bool in = kt < kz;
      const __amdgpu_buffer_rsrc_t wd = in ? wrs : nrs, xd = in ? xrs : nrs;
#pragma unroll
      for (int nt = 0; nt < NG; ++nt)
        wa[nt] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                               wd, wlane, (int)(wo + (uint32_t)kt * kstep4w + (uint32_t)nt * kWave * 16), kNtCpol));
#pragma unroll
      for (int tb = 0; tb < TB; ++tb)
        xb[tb] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xd, xlane + tb * xrow16,
                                                                                   (int)(xo + (uint32_t)kt * kstep4x), 0));
      __builtin_amdgcn_sched_barrier(0);
    };
    struct Seg {
      int kz;
      uint32_t wo, xo, len;
    };
    auto make_seg = [&](uint32_t u) {
      Seg s;
      const int g = (int)(u / KT), kb = (int)(u - (uint32_t)g * KT);
      const int ke = (int)std::min<uint32_t>(KT, kb + (u1 - u));
      const int S = ke - kb;
      s.len = (uint32_t)S;
      s.kz = __builtin_amdgcn_readfirstlane(S > wave ? (S - wave + 3) / 4 : 0);
      s.wo = __builtin_amdgcn_readfirstlane((u - u0 + (uint32_t)wave) * wstride + (uint32_t)w * slot_bytes);
      s.xo = __builtin_amdgcn_readfirstlane((uint32_t)(kb + wave) * KTILE * 2);
      return s;
    };
    uint4 wa0[NG], wa1[NG], wa2[NG], xb0[TB], xb1[TB], xb2[TB];
    auto issue = [&](const Seg& sg) {
      load(sg.wo, sg.xo, 0, sg.kz, wa0, xb0);
      load(sg.wo, sg.xo, 1, sg.kz, wa1, xb1);
    };
    uint32_t u = u0;
    Seg s = make_seg(u);
    issue(s);
    for (int j = 0;; ++j) {
      f32x4 acc[NACC];
#pragma unroll
      for (int i = 0; i < NACC; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
      auto mma = [&](const uint4* wa, const uint4* xb) {
#pragma unroll
        for (int nt = 0; nt < NG; ++nt)
#pragma unroll
          for (int tb = 0; tb < TB; ++tb) mma_tile<uint16_t>(wa[nt], xb[tb], acc[nt * TB + tb]);
      };
      const uint32_t wo = s.wo, xo = s.xo;
      int kt = 0;
      for (; kt + 3 <= s.kz; kt += 3) {
        load(wo, xo, kt + 2, s.kz, wa2, xb2);
        mma(wa0, xb0);
        load(wo, xo, kt + 3, s.kz, wa0, xb0);
        mma(wa1, xb1);
        load(wo, xo, kt + 4, s.kz, wa1, xb1);
        mma(wa2, xb2);
      }
      // 0..2 k-steps left, already loaded in stages 0 and 1
      const int left = s.kz - kt;
      if (left > 0) mma(wa0, xb0);
      if (left > 1) mma(wa1, xb1);
      u += s.len;
      const bool more = u < u1;
      // the next segment's first stages go out before the hand-off (every
      // older load has landed: waiting for them first tells the compiler so)
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      if (more) {
        s = make_seg(u);
        issue(s);
      }
      // hand the accumulators over once the finishing waves have released the previous segment's
      if (!ws_wait_geq(&s_free, TB * j)) return ws_fail(a.err, lane);
#pragma unroll
      for (int i = 0; i < NACC; ++i) red[wave][i][lane] = acc[i];
      ws_signal(&s_fill, lane);
      if (!more) break;
    }
    // this workgroup's stream is done: the next GEMM's first k-steps into L2
    if (a.Wn && (int)blockIdx.x < a.nwg_n) prefetch_next(a, wave, lane);
    return;
  }

  // ---- finishing waves: wave 4 + f owns row tile f ----
  const int f = wv - 4;
  if (f >= TB) return;
  const int row = 16 * f + lane % 16;  // this lane's row (of the padded rows)
  // RMSNorm row scale from the producer's per-group sums of squares, summed as
  // in the 4-wave kernel: four partial sums over every fourth group (lane / 16
  // selects which), then (s0 + s1) + (s2 + s3).  The loads go out in one batch
  // (kPre per lane, groups past 4 kPre in a plain loop): one at a time, at the
  // latency of a memory system the streaming waves keep full, they held the
  // first segment's finishing back by ~45 us.
  float r = 1.f;
  bool valid = false;
  {
    constexpr int kPre = 24;
    const int ng_in = a.ss_in ? a.ss_groups : 0;
    const int q4 = lane / 16;
    const int64_t rr = a.m0 + (row < a.M ? row : 0);
    float pre[kPre];
    if (ng_in > 0) {
#pragma unroll
      for (int j = 0; j < kPre; ++j) pre[j] = a.ss_in[(int64_t)min(q4 + 4 * j, ng_in - 1) * a.mp + rr];
    }
    int vld = 0;
    if constexpr (EPI == EPI_LOGITS) vld = a.rows[rr].valid;
    float ssum = 0.f;
    if (ng_in > 0 && row < a.M) {
#pragma unroll
      for (int j = 0; j < kPre; ++j)
        if (q4 + 4 * j < ng_in) ssum += pre[j];
      for (int gg = q4 + 4 * kPre; gg < ng_in; gg += 4) ssum += a.ss_in[(int64_t)gg * a.mp + rr];
    }
    float t = xor16_op(ssum, [](float x, float y) { return x + y; });
    t = xor32_op(t, [](float x, float y) { return x + y; });
    if (ng_in) r = 1.f / sqrtf(t / (float)a.d_in + a.eps);
    if constexpr (EPI == EPI_LOGITS) valid = row < a.M && vld != 0;
  }
  const int g_first = (int)(u0 / KT);
  const int MC = a.M * C;
  const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7fffffff, kBufferRsrcWord3);
  const bool rin = row < a.M;
  const int elt = row * C + 4 * (lane / 16);  // float offset of the lane's first element (tile 0) in a partial
  uint32_t u = u0;
  for (int j = 0; u < u1; ++j) {
    const int g = (int)(u / KT), kb = (int)(u - (uint32_t)g * KT);
    const int ke = (int)std::min<uint32_t>(KT, kb + (u1 - u));
    u += (uint32_t)(ke - kb);
    if (!ws_wait_geq(&s_fill, 4 * (j + 1))) return ws_fail(a.err, lane);
    f32x4 v[NG];
#pragma unroll
    for (int nt = 0; nt < NG; ++nt) {
      const int i = nt * TB + f;
      v[nt] = (red[0][i][lane] + red[2][i][lane]) + (red[1][i][lane] + red[3][i][lane]);
    }
    ws_signal(&s_free, lane);
    bool fin = true;
    if (!(kb == 0 && ke == (int)KT)) {
      // split group: publish this row tile's partial; the last contributor's wave f finishes it
      const int which = g == g_first ? 0 : 1;
      const int my_off = ((w * 2 + which) * MC) * 4;
#pragma unroll
      for (int nt = 0; nt < NG; ++nt)
        if (rin)
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v[nt]), prs, my_off + 4 * (elt + nt * 16), 0,
                                                 kCoherentCpol);
      const int wf = unit_owner((uint32_t)g * KT, KT, G, SC, a.n_wg);
      const int wl = unit_owner((uint32_t)(g + 1) * KT - 1, KT, G, SC, a.n_wg);
      wait_stores();
      int last = 0;
      if (lane == 0) {
        int* cnt = &a.cnt[(g * 4 + f) * kCntStride];
        const int old = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = old == wl - wf;
        if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      fin = __builtin_amdgcn_readfirstlane(last) != 0;
      if (fin) {
        // contributors added in workgroup order (as the 4-wave kernel), two in flight at once
        const bool wf_first = unit_start(wf, KT, G, SC, a.n_wg) == (uint32_t)g * KT;
#pragma unroll
        for (int nt = 0; nt < NG; ++nt) v[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int ww = wf; ww <= wl; ww += 2) {
          f32x4 p[2][NG];
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int wq = std::min(ww + q, wl);
            const int slot = (wq > wf || wf_first) ? 0 : 1;
            const int src = ((wq * 2 + slot) * MC) * 4;
#pragma unroll
            for (int nt = 0; nt < NG; ++nt)
              p[q][nt] = (rin && ww + q <= wl) ? __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                                                prs, src + 4 * (elt + nt * 16), 0, kCoherentCpol))
                                               : f32x4{0.f, 0.f, 0.f, 0.f};
          }
#pragma unroll
          for (int q = 0; q < 2; ++q)
            if (ww + q <= wl)
#pragma unroll
              for (int nt = 0; nt < NG; ++nt) v[nt] += p[q][nt];
        }
      }
    }
    if (fin) {
      if constexpr (EPI == EPI_SWIGLU) ws_epilogue_swiglu(a, v, g, f, r, lane);
      if constexpr (EPI == EPI_LOGITS) ws_epilogue_logits(a, v, g, f, r, valid, lane);
    }
  }
}

// ---------------------------------------------------------------------------
// Attention, plain VALU version (fp32 models): one workgroup per (row, query
// head).  Scores of a chunk of positions go to LDS; the softmax is carried
// online across chunks.
constexpr int kAttnChunk = 1024;

struct AttnArgs {
  const char* q;  // [rows][hq][hd]
  const char* kc;
  const char* vc;
  char* out;      // [rows][hq*hd]
  const RowInfo* rows;
  int m0, hq, hkv, hd, ld;  // ld: position stride of the caches
  float scale;
};

template <typename T>
__global__ void __launch_bounds__(256) attention_kernel(AttnArgs a) {
  __shared__ float qs[128];
  __shared__ float sc[kAttnChunk];
  __shared__ float red[8];
  __shared__ float acc2[256];
  const int m = a.m0 + blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
  const RowInfo ri = a.rows[m];
  const int hd = a.hd;
  T* outp = reinterpret_cast<T*>(a.out) + ((int64_t)m * a.hq + h) * hd;
  if (!ri.valid) {
    for (int d = tid; d < hd; d += 256) outp[d] = Elem<T>::from_f32(0.f);
    return;
  }
  const int kh = h / (a.hq / a.hkv);
  const T* qp = reinterpret_cast<const T*>(a.q) + ((int64_t)m * a.hq + h) * hd;
  for (int d = tid; d < hd; d += 256) qs[d] = Elem<T>::to_f32(qp[d]) * a.scale;
  __syncthreads();
  const int64_t hb = ((int64_t)ri.seq * a.hkv + kh) * a.ld;
  const T* K = reinterpret_cast<const T*>(a.kc) + hb * hd;
  const T* Vp = reinterpret_cast<const T*>(a.vc) + hb * hd;
  const int npos = ri.pos + 1;
  float run_m = -INFINITY, run_l = 0.f;
  const int dsub = tid / hd, dd = tid % hd;  // PV: (sub-group, dim)
  const int nsub = 256 / hd;
  float acc = 0.f;
  for (int p0 = 0; p0 < npos; p0 += kAttnChunk) {
    const int n = min(kAttnChunk, npos - p0);
    float lmax = -INFINITY;
    for (int i = tid; i < n; i += 256) {
      const T* kr = K + (int64_t)(p0 + i) * hd;
      float s = 0.f;
      for (int d = 0; d < hd; ++d) s += qs[d] * Elem<T>::to_f32(kr[d]);
      sc[i] = s;
      lmax = fmaxf(lmax, s);
    }
    lmax = wave_max(lmax);
    if (lane == 0) red[wave] = lmax;
    __syncthreads();
    float cm = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    const float new_m = fmaxf(run_m, cm);
    float lsum = 0.f;
    for (int i = tid; i < n; i += 256) {
      const float e = expf(sc[i] - new_m);
      sc[i] = e;
      lsum += e;
    }
    lsum = wave_sum(lsum);
    __syncthreads();
    if (lane == 0) red[4 + wave] = lsum;
    __syncthreads();
    const float csum = (red[4] + red[5]) + (red[6] + red[7]);
    const float alpha = expf(run_m - new_m);
    run_l = run_l * alpha + csum;
    run_m = new_m;
    acc *= alpha;
    if (dsub < nsub)
      for (int i = dsub; i < n; i += nsub) acc += sc[i] * Elem<T>::to_f32(Vp[(int64_t)dd * a.ld + p0 + i]);
    __syncthreads();
  }
  if (dsub < nsub) acc2[dsub * hd + dd] = acc;
  __syncthreads();
  if (tid < hd) {
    float o = 0.f;
    for (int s = 0; s < nsub; ++s) o += acc2[s * hd + tid];
    outp[tid] = Elem<T>::from_f32(o / run_l);
  }
}

// ---------------------------------------------------------------------------
// Attention on MFMA (bf16 models).  One workgroup of kAttnWaves waves per (16
// query vectors, sequence x KV head).  The query vectors of one KV head are the
// block's rows times the heads that share it (GQA).  The waves split the cache
// positions into 32-position steps taken round-robin; per step a wave
// computes S^T = K Q^T with K rows as the MFMA A operand, so each lane ends up
// holding scores of its own query column, which is the P^T fragment that
// O^T = V^T P^T takes as its B operand.  Inside a step the K rows are fed in
// the order that leaves lane group g (lane / 16) holding the 8 consecutive
// positions 8g..8g+7, which are the positions of the lane's V^T operand.  The
// caches are stored in these fragments' order (kfrag_index, vfrag_index), so
// every operand load is a contiguous 1 KB block.  Each wave keeps two steps of
// K/V loads in flight.  The softmax is online within a wave; the waves' partial
// (max, sum, O) are combined through LDS in wave order.
constexpr int kAttnWaves = 8;

struct AttnMfmaArgs {
  const uint16_t* q;   // [rows][hq][HD]
  const uint16_t* kc;  // layer base, per (seq, hkv) ld x HD elements, fragment-major
  const uint16_t* vc;  // layer base, per (seq, hkv) ld x HD elements, fragment-major
  uint16_t* out;       // [rows][hq*HD]
  const RowInfo* rows;
  int nb, R, hq, hkv, grp, ld, qblocks;  // ld: position stride of the caches (multiple of 64)
  float scale;
  // workgroups past the n_attn attention ones (n_attn and n_pref multiples of
  // 8) only load into L2 the first k-steps of the next GEMM's workgroups p and
  // p + n_pref (NULL Wn: none)
  int n_attn, n_pref;
  const char* Wn;
  int KTn, Gn, ngn, nwg_n, cn;
};

template <int HD>
__global__ void __launch_bounds__(kAttnWaves * 64) attention_mfma_kernel(AttnMfmaArgs a) {
  constexpr int KK = HD / 32, DB = HD / 16;
  __shared__ float s_o[kAttnWaves][16][HD + 1];
  __shared__ float s_m[kAttnWaves][16], s_l[kAttnWaves][16], s_f[kAttnWaves][16], s_L[16];
  touch_kernargs<AttnMfmaArgs>();
  if ((int)blockIdx.x >= a.n_attn) {
    // on a CU the attention leaves idle: the o_proj's first k-steps into L2,
    // for its workgroups p and p + n_pref (same XCD: n_attn and n_pref are
    // multiples of 8), one per four waves
    const int p = blockIdx.x - a.n_attn, wave4 = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int w = p + (wave4 / 4) * a.n_pref;
    // (six k-steps per wave: about what lands while the attention runs; deeper ones hold it open)
    if (a.Wn && w < a.nwg_n) prefetch_gemm_start<6>(a.Wn, a.KTn, a.Gn, a.cn, a.ngn, a.nwg_n, w, wave4 % 4, threadIdx.x % kWave);
    return;
  }
  // Workgroups are dispatched to the XCDs round-robin by linear id; all query
  // blocks of one (sequence, KV head) get ids of one residue mod kXcds, so they
  // run on one XCD and share its L2 copy of that head's K/V.
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int bk = xcd + kXcds * (slot / a.qblocks), qb = slot % a.qblocks;
  if (bk >= a.nb * a.hkv) return;  // launch larger than the block set
  const int blk = bk / a.hkv, kvh = bk % a.hkv;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const int QV = a.R * a.grp;
  const int qv = qb * 16 + lane % 16;
  const bool qok = qv < QV;
  const int r = qok ? qv / a.grp : 0, hh = qok ? qv % a.grp : 0;
  const int m = blk * a.R + r;
  // row info and this lane's query are independent loads, issued together
  const int r_hi = min(a.R - 1, (qb * 16 + 15) / a.grp);
  const RowInfo first = a.rows[blk * a.R];
  const int pos_hi = a.rows[blk * a.R + r_hi].pos;
  const int qpos = a.rows[m].pos;
  uint4 qf[KK];  // lanes past the last query vector load row 0's (their scores are masked)
  const uint16_t* Q = a.q + ((int64_t)m * a.hq + kvh * a.grp + hh) * HD;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) qf[kk] = load16(Q + 32 * kk + 8 * (lane / 16));
  // positions this query block can see: up to its last row's position
  const int kv_end = __builtin_amdgcn_readfirstlane(first.valid ? pos_hi + 1 : 0);
  const int64_t head = (int64_t)first.seq * a.hkv + kvh;
  const uint16_t* K = a.kc + head * a.ld * HD;
  const uint16_t* Vt = a.vc + head * a.ld * HD;
  const int g8 = 8 * (lane / 16);

  // One step's operands: the K fragments of the two 16-row sub-tiles and the
  // V fragments of the lane's 8 positions, each load one contiguous 1 KB block
  // of the fragment-major caches.  A loaded step starts below kv_end <= ld and
  // ld is a multiple of 64, so its blocks lie inside the head's cache.
  // Entries at positions at or past kv_end hold stale values: their scores are
  // masked, and their V values are zeroed where they are used (P is 0 there,
  // and 0 times a stale non-finite value would not be).
  struct StepRegs {
    uint4 kf[2][KK];
    uint4 vf[DB];
  };
  auto load_step = [&](int p, StepRegs& st) {
    const int64_t so = (int64_t)(p / 32) * 32 * HD + lane * 8;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) st.kf[b][kk] = load16(K + so + (b * KK + kk) * 512);
#pragma unroll
    for (int db = 0; db < DB; ++db) st.vf[db] = load16(Vt + so + db * 512);
  };

  f32x4 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lrun = 0.f;
  auto step = [&](int p, const StepRegs& st) {
    f32x4 sacc[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      sacc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        sacc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, st.kf[b][kk]),
                                                          __builtin_bit_cast(bf16x8, qf[kk]), sacc[b], 0, 0, 0);
    }
    // sacc[b][i]: position p + g8 + 4 b + i, query column lane % 16
    float sv[8];
    float mloc = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kp = p + g8 + 4 * b + i;
        const float v = (qok && kp <= qpos && kp < kv_end) ? sacc[b][i] * a.scale : -INFINITY;
        sv[b * 4 + i] = v;
        mloc = fmaxf(mloc, v);
      }
    mloc = xor16_op(mloc, [](float x, float y) { return fmaxf(x, y); });
    mloc = xor32_op(mloc, [](float x, float y) { return fmaxf(x, y); });
    const float mnew = fmaxf(mrun, mloc);
    const float alpha = mrun == -INFINITY ? 0.f : __expf(mrun - mnew);
    float lsum = 0.f;
    uint16_t pb[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float e = sv[i] == -INFINITY ? 0.f : __expf(sv[i] - mnew);
      lsum += e;
      pb[i] = f32_to_bf16(e);
    }
    lrun = lrun * alpha + lsum;
    mrun = mnew;
    const uint4 pf = make_uint4((uint32_t)pb[0] | ((uint32_t)pb[1] << 16), (uint32_t)pb[2] | ((uint32_t)pb[3] << 16),
                                (uint32_t)pb[4] | ((uint32_t)pb[5] << 16), (uint32_t)pb[6] | ((uint32_t)pb[7] << 16));
    const int nv = kv_end - (p + g8);  // valid positions of the lane's 8 (may be <= 0 or >= 8)
    uint32_t mask[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) mask[i] = (2 * i < nv ? 0xFFFFu : 0u) | (2 * i + 1 < nv ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const uint4 v = st.vf[db];
      const uint4 vm = make_uint4(v.x & mask[0], v.y & mask[1], v.z & mask[2], v.w & mask[3]);
      o[db] *= alpha;
      o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vm), __builtin_bit_cast(bf16x8, pf),
                                                      o[db], 0, 0, 0);
    }
  };
  // Fixed assignment of 32-position steps to waves (step t to wave t % waves),
  // independent of the other rows of the block: a row's result does not
  // depend on how rows are batched, so a block verify reproduces decode steps
  // bit for bit.  Steps past a row's own position are fully masked and leave
  // its running state unchanged, exactly (the rescale factor is 1, or the
  // state is still zero): each wave runs an even number of steps, two per
  // iteration, and every load is unconditional, its step clamped to the last
  // one below kv_end, so that the compiler waits for exactly the step in use
  // while the other one's loads stay in flight.
  constexpr int kStride = 32 * kAttnWaves;
  const int p_last = kv_end > 0 ? (kv_end - 1) / 32 * 32 : 0;  // start of the last step with positions
  const int n_steps = kv_end > 32 * wave ? (kv_end - 32 * wave + kStride - 1) / kStride : 0;
  // The head's query blocks all walk the steps in the same order at about the
  // same time, so they would miss in L2 together.  First each of them loads a
  // different share of the head's cache (step s goes to query block s mod
  // qblocks, its 1 KB blocks spread over the waves) so that the later steps
  // of every query block find it in L2.  Plain (cached) loads whose values
  // are only consumed by an empty asm statement; they are issued before the
  // stream's own loads and land while its first steps wait.
  constexpr int kPre = 4;  // blocks per wave
  // 1 KB blocks of one step: 2 KK of K (the step's 32 x HD elements), then DB of V (the same amount)
  constexpr int kBlk = 2 * KK + DB;
  uint4 pre[kPre];
  {
    const int n_steps_all = (kv_end + 31) / 32;
#pragma unroll
    for (int i = 0; i < kPre; ++i) {
      const int j = wave + kAttnWaves * i;         // this workgroup's j-th block
      const int st = qb + a.qblocks * (j / kBlk);  // the step it belongs to
      const int bi = j % kBlk;                     // its block inside the step
      // past the last step: step 0 again (in range, already wanted).  Step stc lies inside the head's
      // cache: (stc + 1) * 32 <= 32 * ceil(kv_end / 32) <= ld, ld being a multiple of 64 >= kv_end.
      const int stc = st < n_steps_all ? st : 0;
      const uint16_t* src = bi < 2 * KK ? K + bi * 512 : Vt + (bi - 2 * KK) * 512;
      pre[i] = load16(src + (int64_t)stc * 32 * HD + lane * 8);  // unconditional (one load order)
    }
  }
  // The loads sit only inside the loop (a first pass issues them and skips
  // the compute), so that the compiler sees one load order on every path.
  StepRegs s0, s1;
  int p = 32 * wave - 2 * kStride;
  const int t_end = kv_end > 0 ? n_steps : -2;
  for (int t = -2; t < t_end; t += 2, p += 2 * kStride) {
    if (t >= 0) step(p, s0);
    load_step(min(p + 2 * kStride, p_last), s0);
    if (t >= 0) step(p + kStride, s1);
    load_step(min(p + 3 * kStride, p_last), s1);
  }
  {
    uint32_t x = 0;
#pragma unroll
    for (int i = 0; i < kPre; ++i) x ^= pre[i].x ^ pre[i].w;
    asm volatile("" ::"v"(x));  // the values are consumed, so the loads stay
  }
  // softmax denominator of query lane%16 over this wave's positions
  float ltot = xor16_op(lrun, [](float x, float y) { return x + y; });
  ltot = xor32_op(ltot, [](float x, float y) { return x + y; });
  // publish the wave's partial to LDS: o[db][i] is O^T[16 db + 4 (lane / 16) + i][query lane%16]
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int i = 0; i < 4; ++i) s_o[wave][lane % 16][16 * db + 4 * (lane / 16) + i] = o[db][i];
  if (lane < 16) {
    s_m[wave][lane] = mrun;
    s_l[wave][lane] = ltot;
  }
  __syncthreads();
  // per query: the common max, each wave's rescale factor and the total sum,
  // all accumulated in wave order
  if (threadIdx.x < 16) {
    const int q = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) M = fmaxf(M, s_m[w][q]);
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) {
      const float ms = s_m[w][q];
      const float f = (M == -INFINITY || ms == -INFINITY) ? 0.f : __expf(ms - M);
      s_f[w][q] = f;
      L += s_l[w][q] * f;
    }
    s_L[q] = L;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 16 * HD; e += kAttnWaves * 64) {
    const int q = e / HD, dim = e % HD;
    const int qq = qb * 16 + q;
    if (qq >= QV) continue;
    float O = 0.f;
#pragma unroll
    for (int w = 0; w < kAttnWaves; ++w) O += s_o[w][q][dim] * s_f[w][q];
    const float L = s_L[q];
    const int rr = qq / a.grp, hq2 = kvh * a.grp + qq % a.grp;
    a.out[((int64_t)(blk * a.R + rr) * a.hq + hq2) * HD + dim] = f32_to_bf16(L > 0.f ? O / L : 0.f);
  }
}

// ---------------------------------------------------------------------------
struct EmbedArgs {
  const char* E;  // [V][d]
  const float* g; // attention-norm gain of layer 0 (or final norm when there are no layers)
  float* x;
  char* xa;
  float* ss;  // sum of squares of each row (the RMSNorm statistic of layer 0)
  RowInfo* rows;
  int d, V, R, gamma, max_len, max_batch;
  float eps;
  // verify
  const int32_t* seq_ids;
  const int32_t* drafts;
  const int32_t* kv_len;
  const int32_t* pending;
  // prefill
  const int32_t* tokens;
  int seq, pos0, prefill;
  int32_t* err;
};

template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(EmbedArgs a) {
  __shared__ float red[4];
  __shared__ int s_tok;
  const int m = blockIdx.x, tid = threadIdx.x;
  if (tid == 0) {
    int seq, pos, tok, valid;
    if (a.prefill) {
      seq = a.seq;
      pos = a.pos0 + m;
      tok = a.tokens[m];
      valid = pos < a.max_len;
    } else {
      const int s = m / a.R, r = m % a.R;
      seq = a.seq_ids ? a.seq_ids[s] : s;  // no id list: block s is sequence s
      if (seq < 0 || seq >= a.max_batch) {  // refused: no cache slot to read or write
        if (r == 0) atomicOr(a.err, 4);
        seq = 0;
        pos = 0;
        tok = 0;
        valid = 0;
      } else {
        const int len = a.kv_len[seq];
        pos = len + r;
        tok = r == 0 ? a.pending[seq] : a.drafts[(int64_t)s * a.gamma + r - 1];
        valid = len + a.R <= a.max_len;
        if (!valid && r == 0) atomicOr(a.err, 1);
      }
    }
    if (tok < 0 || tok >= a.V) {
      atomicOr(a.err, 2);
      tok = 0;
    }
    RowInfo ri;
    ri.seq = seq;
    ri.pos = valid ? pos : 0;
    ri.valid = valid;
    ri.pad = 0;
    a.rows[m] = ri;
    s_tok = tok;
  }
  __syncthreads();
  // 16-byte vectors of the embedding row and the gains (d is a multiple of 32, rows 16-byte aligned),
  // a round's loads all issued before any is used
  constexpr int EPL = 16 / sizeof(T), kRound = 4;
  const T* e = reinterpret_cast<const T*>(a.E) + (int64_t)s_tok * a.d;
  float* xrow = a.x + (int64_t)m * a.d;
  T* xarow = reinterpret_cast<T*>(a.xa) + (int64_t)m * a.d;
  const int nv = a.d / EPL;
  float ss = 0.f;
  for (int base = 0; base < nv; base += 256 * kRound) {
    uint4 ev[kRound];
    f32x4 gv[kRound][EPL / 4];
#pragma unroll
    for (int j = 0; j < kRound; ++j) {
      const int iv = min(base + j * 256 + tid, nv - 1);
      ev[j] = *reinterpret_cast<const uint4*>(e + iv * EPL);
#pragma unroll
      for (int q = 0; q < EPL / 4; ++q) gv[j][q] = *reinterpret_cast<const f32x4*>(a.g + iv * EPL + 4 * q);
    }
#pragma unroll
    for (int j = 0; j < kRound; ++j) {
      const int iv = base + j * 256 + tid;
      if (iv < nv) {
        const T* ve = reinterpret_cast<const T*>(&ev[j]);
        T xa_out[EPL];
#pragma unroll
        for (int q = 0; q < EPL / 4; ++q) {
          f32x4 xo;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const float v = Elem<T>::to_f32(ve[4 * q + t]);
            xo[t] = v;
            xa_out[4 * q + t] = Elem<T>::from_f32(v * gv[j][q][t]);
            ss += v * v;
          }
          *reinterpret_cast<f32x4*>(xrow + iv * EPL + 4 * q) = xo;
        }
        *reinterpret_cast<uint4*>(xarow + iv * EPL) = *reinterpret_cast<const uint4*>(xa_out);
      }
    }
  }
  ss = wave_sum(ss);
  if (tid % kWave == 0) red[tid / kWave] = ss;
  __syncthreads();
  if (tid == 0) a.ss[m] = (red[0] + red[1]) + (red[2] + red[3]);  // one column group
}

__global__ void commit_kernel(int32_t* len, int32_t* pending, int32_t* err, const int32_t* seq_ids, int n,
                              const int32_t* L, const int32_t* nxt, int max_len, int max_batch, int V) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int s = seq_ids[i];
  if (s < 0 || s >= max_batch) {
    atomicOr(err, 4);
    return;
  }
  const int l = L[i], t = nxt[i];
  if (l < 0 || len[s] + l + 1 > max_len || t < 0 || t >= V) {
    atomicOr(err, 1);
    return;
  }
  len[s] += l + 1;
  pending[s] = t;
}

__global__ void prefill_finish_kernel(int32_t* len, int32_t* pending, int32_t* err, int seq, int n,
                                      const int32_t* tokens, int V) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  int t = tokens[n - 1];
  if (t < 0 || t >= V) {
    atomicOr(err, 2);
    t = 0;
  }
  len[seq] = n - 1;
  pending[seq] = t;
}

__global__ void kv_init_kernel(int32_t* len, int32_t* pending, int32_t* err, int max_batch, float* rope, int max_len,
                               int half, double theta) {
  const int64_t n = (int64_t)max_len * half;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int pos = (int)(i / half), j = (int)(i % half);
    const double inv_freq = pow(theta, -2.0 * j / (2.0 * half));
    const double ang = (double)pos * inv_freq;
    rope[2 * i] = (float)cos(ang);
    rope[2 * i + 1] = (float)sin(ang);
  }
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < max_batch; i += blockDim.x) {
      len[i] = 0;
      pending[i] = 0;
    }
    if (threadIdx.x == 0) *err = 0;
  }
}

// ---------------------------------------------------------------------------
// Host side


// Counter region at the start of every workspace, sized by the model only, so
// that it stays at one place whatever the row count of a call: one arrival
// counter per GEMM column group.

static int64_t gemm_counter_count(const sdd_model* m) {
  return ceil_div(m->cfg.vocab, 16) + ceil_div(2 * (int64_t)m->cfg.d_ff, 16) + ceil_div(m->cfg.d_model, 16) + 64;
}

static size_t counters_bytes(const sdd_model* m) {
  return align_up((size_t)gemm_counter_count(m) * 4 * kCntStride, 256);
}

WsLayout ws_layout(const sdd_model* m, int max_rows) {
  WsLayout L{};
  const sdd_model_config& c = m->cfg;
  const int es = m->es;
  const int mp = (int)align_up((size_t)std::max(1, max_rows), 16);
  const int64_t d = c.d_model, hq = (int64_t)c.n_q_heads * c.head_dim;
  L.mp = mp;
  L.n_wg = m->n_cu;  // one 256-thread GEMM workgroup per compute unit
  L.max_groups = (int)ceil_div(std::max<int64_t>(c.vocab, std::max<int64_t>(2 * (int64_t)c.d_ff, d)), 16);
  size_t off = 0;
  auto take = [&](size_t b) {
    size_t o = off;
    off = align_up(off + b, 256);
    return o;
  };
  L.cnt = take(counters_bytes(m));  // first: survives calls with other row counts
  L.rowinfo = take((size_t)mp * sizeof(RowInfo));
  L.x = take((size_t)mp * d * 4);
  L.xa = take((size_t)mp * d * es);
  L.ss_part = take((size_t)ceil_div(d, 16) * mp * 4);
  L.q = take((size_t)mp * hq * es);
  L.ao = take((size_t)mp * hq * es);
  L.ffh = take((size_t)mp * c.d_ff * es);
  // stream-K partial tiles: [n_wg][2][64 rows][128] for the 33-row kernel; the many-row kernel (bf16, more
  // than 64 rows) keeps its partials in the accumulator layout, kRowsPartBytes per workgroup
  size_t part = (size_t)L.n_wg * 2 * kMaxPassRows * 128 * 4;
  if (es == 2 && max_rows > kMaxPassRows) part = std::max(part, (size_t)L.n_wg * kRowsPartBytes);
  L.part = take(part);
  L.amax = take((size_t)L.max_groups * mp * 8);
  L.total = off;
  return L;
}

struct CallCtx {
  sdd_model* m;
  sdd_kv* kv;
  char* ws;
  WsLayout L;
  hipStream_t st;
};

template <typename T, int NG, int EPI>
static void launch_gemm_tb(int tb, const GemmArgs& a, int nblocks, hipStream_t st) {
  switch (tb) {
    case 1: hipLaunchKernelGGL((gemm_kernel<T, 1, NG, EPI>), dim3(nblocks), dim3(kGemmThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<T, 2, NG, EPI>), dim3(nblocks), dim3(kGemmThreads), 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemm_kernel<T, 3, NG, EPI>), dim3(nblocks), dim3(kGemmThreads), 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_kernel<T, 4, NG, EPI>), dim3(nblocks), dim3(kGemmThreads), 0, st, a); break;
  }
}

// the 8-wave stream-K kernel (bf16, 8-tile groups, SwiGLU or LM head, at most 3 row tiles)
template <int EPI>
static void launch_gemm_ws(int tb, const GemmArgs& a, int nblocks, hipStream_t st) {
  switch (tb) {
    case 1: hipLaunchKernelGGL((gemm_ws_kernel<1, EPI>), dim3(nblocks), dim3(kWsThreads), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemm_ws_kernel<2, EPI>), dim3(nblocks), dim3(kWsThreads), 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_ws_kernel<3, EPI>), dim3(nblocks), dim3(kWsThreads), 0, st, a); break;
  }
}

template <typename T, int EPI>
static void launch_gemm_ng(int ng, int tb, const GemmArgs& a, int nblocks, hipStream_t st) {
  switch (ng) {
    case 8: launch_gemm_tb<T, 8, EPI>(tb, a, nblocks, st); break;
    case 4: launch_gemm_tb<T, 4, EPI>(tb, a, nblocks, st); break;
    default: launch_gemm_tb<T, 2, EPI>(tb, a, nblocks, st); break;
  }
}

// A GEMM of the forward: tiled weights at w_off, N output columns, K inputs,
// column groups of ng tiles.
struct GemmRef {
  size_t w_off;
  int64_t N;
  int K, ng;
};

// The streaming plan of a GEMM of the forward (the order its matrix is stored in).
static MatPlan plan_gemm(const CallCtx& cx, const GemmRef& r) {
  return plan_matrix(r.N, r.K, cx.m->ktile, r.ng, cx.L.n_wg);
}

// Runs one GEMM over rows [0, M) in passes of at most 64 rows; `next` is the
// forward's following GEMM, whose first k-steps the last pass loads into L2.
static int run_gemm(CallCtx& cx, int epi, unsigned prof, size_t w_off, int64_t N, int K, const char* X, GemmArgs a,
                    int M, int ng, const GemmRef* next = nullptr) {
  const sdd_model* m = cx.m;
  const MatPlan plan = plan_gemm(cx, GemmRef{w_off, N, K, ng});
  a.W = m->base + w_off;
  a.KT = plan.KT;
  a.G = plan.G;
  a.N = (int)N;
  a.X = X;
  a.ldx = K;
  a.mp = cx.L.mp;
  a.part = reinterpret_cast<float*>(cx.ws + cx.L.part);
  a.err = cx.kv ? cx.kv->err : nullptr;
  a.cnt = reinterpret_cast<int*>(cx.ws + cx.L.cnt);
  a.rows = reinterpret_cast<const RowInfo*>(cx.ws + cx.L.rowinfo);
  a.eps = m->cfg.rms_eps;
  const int64_t V = (int64_t)a.G * (a.KT + plan.c);
  const int nblocks = plan.n_wg;
  a.n_wg = nblocks;
  a.segc = plan.c;
  a.share = plan.S;
  MatPlan np{};
  if (next) np = plan_gemm(cx, *next);
  if ((V + 1) * nblocks >= (int64_t(1) << 31))
    return fail(SDD_EUNSUPPORTED, "matrix of %lld weight tiles exceeds the 32-bit stream-K bookkeeping",
                (long long)a.G * a.KT);
  // weight buffer offsets, k-steps up to 4 past a wave's range included
  if ((plan_slots(plan) + 4 * (int64_t)plan.n_wg) * ng * 1024 >= (int64_t(1) << 31))
    return fail(SDD_EUNSUPPORTED, "matrix of %lld x %d exceeds the 32-bit buffer offsets", (long long)N, K);
  if ((int64_t)(M + 64) * K * m->es >= (int64_t(1) << 31))
    return fail(SDD_EUNSUPPORTED, "activations of %d rows x %d exceed the 32-bit buffer offsets", M, K);
  if (m->es == 2 && M > kMaxPassRows && (ng == 8 || ng == 4)) {
    // bf16 over more than 64 rows (several sequences' blocks, prefill chunks): the many-row kernel streams
    // the weights once per kRowsMaxRows rows, on the same stream-K partition
    if ((int64_t)(M + kRowsMaxRows) * K * 2 >= (int64_t(1) << 31))
      return fail(SDD_EUNSUPPORTED, "activations of %d rows x %d exceed the 32-bit buffer offsets", M, K);
    a.Wn = nullptr;
    for (int m0 = 0; m0 < M; m0 += kRowsMaxRows) {
      a.m0 = m0;
      a.M = std::min(kRowsMaxRows, M - m0);
      prof_begin(prof, cx.st);
      int rc = launch_gemm_rows(ng, epi, a, nblocks, cx.st);
      prof_end(prof, cx.st);
      if (rc) return rc;
    }
    return SDD_OK;
  }
  for (int m0 = 0; m0 < M; m0 += kMaxPassRows) {
    a.m0 = m0;
    a.M = std::min(kMaxPassRows, M - m0);
    a.Wn = next && m0 + kMaxPassRows >= M ? m->base + next->w_off : nullptr;  // last pass only
    a.KTn = np.KT;
    a.Gn = np.G;
    a.ngn = next ? next->ng : 1;
    a.nwg_n = np.n_wg;
    a.cn = np.c;
    const int tb = (int)ceil_div(a.M, 16);
    prof_begin(prof, cx.st);
    if (m->es == 2) {
      switch (epi) {
        case EPI_QKV: launch_gemm_ng<uint16_t, EPI_QKV>(ng, tb, a, nblocks, cx.st); break;
        case EPI_RESID: launch_gemm_ng<uint16_t, EPI_RESID>(ng, tb, a, nblocks, cx.st); break;
        case EPI_SWIGLU:
          if (ng == 8 && tb <= 3)
            launch_gemm_ws<EPI_SWIGLU>(tb, a, nblocks, cx.st);
          else
            launch_gemm_ng<uint16_t, EPI_SWIGLU>(ng, tb, a, nblocks, cx.st);
          break;
        default:
          if (ng == 8 && tb <= 3)
            launch_gemm_ws<EPI_LOGITS>(tb, a, nblocks, cx.st);
          else
            launch_gemm_ng<uint16_t, EPI_LOGITS>(ng, tb, a, nblocks, cx.st);
          break;
      }
    } else {
      switch (epi) {
        case EPI_QKV: launch_gemm_ng<float, EPI_QKV>(ng, tb, a, nblocks, cx.st); break;
        case EPI_RESID: launch_gemm_ng<float, EPI_RESID>(ng, tb, a, nblocks, cx.st); break;
        case EPI_SWIGLU: launch_gemm_ng<float, EPI_SWIGLU>(ng, tb, a, nblocks, cx.st); break;
        default: launch_gemm_ng<float, EPI_LOGITS>(ng, tb, a, nblocks, cx.st); break;
      }
    }
    prof_end(prof, cx.st);
    int rc = check_launch("gemm_kernel");
    if (rc) return rc;
  }
  return SDD_OK;
}

// Forward of M rows whose RowInfo/x/xa/sum of squares were written by embed_kernel.
static int forward_rows(CallCtx& cx, int nb, int R, float* logits, int32_t* argmax) {
  const int M = nb * R;
  sdd_model* m = cx.m;
  sdd_kv* kv = cx.kv;
  const sdd_model_config& c = m->cfg;
  const int64_t d = c.d_model, hd = c.head_dim, hq = c.n_q_heads * hd, hk = c.n_kv_heads * hd;
  char* ws = cx.ws;
  const WsLayout& L = cx.L;
  float* x = reinterpret_cast<float*>(ws + L.x);
  char* xa = ws + L.xa;
  float* ss = reinterpret_cast<float*>(ws + L.ss_part);
  // column groups of the RMSNorm statistic of the current residual stream
  const int g_resid_o = (int)(d / 16 / m->ng_o), g_resid_down = (int)(d / 16 / m->ng_down);
  int ss_groups = 1;  // from embed_kernel
  int rc;
  for (int l = 0; l < c.n_layers; ++l) {
    const sdd_model::Layer& Ly = m->layers[l];
    // q/k/v + QK-norm + RoPE + cache append
    {
      GemmArgs a{};
      a.ss_in = ss;
      a.ss_groups = ss_groups;
      a.d_in = (int)d;
      a.q_out = ws + L.q;
      a.hq = c.n_q_heads;
      a.hkv = c.n_kv_heads;
      a.hd = c.head_dim;
      a.qk_norm = c.qk_norm;
      a.qn = reinterpret_cast<const float*>(m->base + Ly.q_norm);
      a.kn = reinterpret_cast<const float*>(m->base + Ly.k_norm);
      a.rope = kv->rope;
      a.kv_ld = kv->ld;
      a.kc = kv->k + (size_t)l * kv->layer_stride;
      a.vc = kv->v + (size_t)l * kv->layer_stride;
      const GemmRef nx{Ly.o, d, (int)hq, m->ng_o};
      if ((rc = run_gemm(cx, EPI_QKV, PROF_GEMM_QKV, Ly.qkv, hq + 2 * hk, (int)d, xa, a, M, m->ng_qkv, &nx))) return rc;
    }
    // attention
    if (m->es == 2) {
      AttnMfmaArgs a{};
      a.q = reinterpret_cast<const uint16_t*>(ws + L.q);
      a.kc = reinterpret_cast<const uint16_t*>(kv->k + (size_t)l * kv->layer_stride);
      a.vc = reinterpret_cast<const uint16_t*>(kv->v + (size_t)l * kv->layer_stride);
      a.out = reinterpret_cast<uint16_t*>(ws + L.ao);
      a.rows = reinterpret_cast<const RowInfo*>(ws + L.rowinfo);
      a.nb = nb;
      a.R = R;
      a.hq = c.n_q_heads;
      a.hkv = c.n_kv_heads;
      a.grp = c.n_q_heads / c.n_kv_heads;
      a.ld = kv->ld;
      a.qblocks = (int)ceil_div((int64_t)R * a.grp, 16);
      a.scale = 1.f / sqrtf((float)c.head_dim);
      a.n_attn = kXcds * a.qblocks * (int)ceil_div((int64_t)nb * a.hkv, kXcds);
      // the CUs the attention leaves idle load the o_proj's first k-steps into L2
      const MatPlan op = plan_gemm(cx, GemmRef{Ly.o, d, (int)hq, m->ng_o});
      a.n_pref = std::max(0, std::min((m->n_cu - a.n_attn) / kXcds * kXcds, (op.n_wg + 1) / 2 + kXcds));
      a.n_pref = a.n_pref / kXcds * kXcds;
      a.Wn = a.n_pref > 0 ? m->base + Ly.o : nullptr;
      a.KTn = op.KT;
      a.Gn = op.G;
      a.ngn = m->ng_o;
      a.nwg_n = op.n_wg;
      a.cn = op.c;
      const dim3 grid(a.n_attn + a.n_pref);
      prof_begin(PROF_ATTN, cx.st);
      if (c.head_dim == 128)
        hipLaunchKernelGGL(attention_mfma_kernel<128>, grid, dim3(kAttnWaves * 64), 0, cx.st, a);
      else
        hipLaunchKernelGGL(attention_mfma_kernel<64>, grid, dim3(kAttnWaves * 64), 0, cx.st, a);
      prof_end(PROF_ATTN, cx.st);
      if ((rc = check_launch("attention_mfma_kernel"))) return rc;
    } else {
      AttnArgs a{};
      a.q = ws + L.q;
      a.kc = kv->k + (size_t)l * kv->layer_stride;
      a.vc = kv->v + (size_t)l * kv->layer_stride;
      a.out = ws + L.ao;
      a.rows = reinterpret_cast<const RowInfo*>(ws + L.rowinfo);
      a.m0 = 0;
      a.hq = c.n_q_heads;
      a.hkv = c.n_kv_heads;
      a.hd = c.head_dim;
      a.ld = kv->ld;
      a.scale = 1.f / sqrtf((float)c.head_dim);
      prof_begin(PROF_ATTN, cx.st);
      hipLaunchKernelGGL(attention_kernel<float>, dim3(M, c.n_q_heads), dim3(256), 0, cx.st, a);
      prof_end(PROF_ATTN, cx.st);
      if ((rc = check_launch("attention_kernel"))) return rc;
    }
    // output projection + residual; next input scaled by the FFN norm gain
    {
      GemmArgs a{};
      a.x = x;
      a.xa = xa;
      a.d = (int)d;
      a.g_next = reinterpret_cast<const float*>(m->base + Ly.ffn_norm);
      a.ss_part = ss;
      const GemmRef nx{Ly.gu, 2 * (int64_t)c.d_ff, (int)d, m->ng_gu};
      if ((rc = run_gemm(cx, EPI_RESID, PROF_GEMM_O, Ly.o, d, (int)hq, ws + L.ao, a, M, m->ng_o, &nx))) return rc;
    }
    // gate/up + SwiGLU
    {
      GemmArgs a{};
      a.ss_in = ss;
      a.ss_groups = g_resid_o;
      a.d_in = (int)d;
      a.ffh = ws + L.ffh;
      a.dff = c.d_ff;
      const GemmRef nx{Ly.down, d, c.d_ff, m->ng_down};
      if ((rc = run_gemm(cx, EPI_SWIGLU, PROF_GEMM_GU, Ly.gu, 2 * (int64_t)c.d_ff, (int)d, xa, a, M, m->ng_gu, &nx)))
        return rc;
    }
    // down projection + residual; next input scaled by the next norm gain
    {
      GemmArgs a{};
      a.x = x;
      a.xa = xa;
      a.d = (int)d;
      a.g_next = reinterpret_cast<const float*>(
          m->base + (l + 1 < c.n_layers ? m->layers[l + 1].attn_norm : m->off_final_norm));
      a.ss_part = ss;
      // the next layer's qkv, or the LM head after the last layer
      const GemmRef nq{l + 1 < c.n_layers ? m->layers[l + 1].qkv : 0, hq + 2 * hk, (int)d, m->ng_qkv};
      const GemmRef nl{m->off_lm, c.vocab, (int)d, m->ng_lm};
      const GemmRef* nx = l + 1 < c.n_layers ? &nq : logits ? &nl : nullptr;
      if ((rc = run_gemm(cx, EPI_RESID, PROF_GEMM_DOWN, Ly.down, d, c.d_ff, ws + L.ffh, a, M, m->ng_down, nx))) return rc;
      ss_groups = g_resid_down;
    }
  }
  if (logits) {
    GemmArgs a{};
    a.ss_in = ss;
    a.ss_groups = ss_groups;
    a.d_in = (int)d;
    a.logits = logits;
    a.V = c.vocab;
    a.amax_v = reinterpret_cast<float*>(ws + L.amax);
    a.amax_i = reinterpret_cast<int*>(ws + L.amax + (size_t)L.max_groups * L.mp * 4);
    if ((rc = run_gemm(cx, EPI_LOGITS, PROF_GEMM_LM, m->off_lm, c.vocab, (int)d, xa, a, M, m->ng_lm))) return rc;
    if (argmax) {
      const int G = (int)(c.vocab / 16 / m->ng_lm);
      prof_begin(PROF_GEMM_LM, cx.st);
      hipLaunchKernelGGL(row_argmax_kernel, dim3(M), dim3(256), 0, cx.st, a.amax_v, a.amax_i, G, L.mp,
                         reinterpret_cast<const RowInfo*>(ws + L.rowinfo), argmax);
      prof_end(PROF_GEMM_LM, cx.st);
      if ((rc = check_launch("row_argmax_kernel"))) return rc;
    }
  }
  return SDD_OK;
}

static int launch_embed(CallCtx& cx, EmbedArgs e, int M) {
  sdd_model* m = cx.m;
  const sdd_model_config& c = m->cfg;
  e.E = m->base + m->off_embed;
  e.g = reinterpret_cast<const float*>(m->base + (c.n_layers > 0 ? m->layers[0].attn_norm : m->off_final_norm));
  e.x = reinterpret_cast<float*>(cx.ws + cx.L.x);
  e.xa = cx.ws + cx.L.xa;
  e.ss = reinterpret_cast<float*>(cx.ws + cx.L.ss_part);
  e.rows = reinterpret_cast<RowInfo*>(cx.ws + cx.L.rowinfo);
  e.d = c.d_model;
  e.V = c.vocab;
  e.max_len = cx.kv->max_len;
  e.max_batch = cx.kv->max_batch;
  e.eps = c.rms_eps;
  e.err = cx.kv->err;
  prof_begin(PROF_EMBED, cx.st);
  if (m->es == 2)
    hipLaunchKernelGGL(embed_kernel<uint16_t>, dim3(M), dim3(256), 0, cx.st, e);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, cx.st, e);
  prof_end(PROF_EMBED, cx.st);
  return check_launch("embed_kernel");
}

}  // namespace sdd

using namespace sdd;

extern "C" int sdd_kv_bytes(const sdd_model_config* cfg, int max_batch, int max_len, size_t* bytes) {
  SDD_REQUIRE(cfg && bytes, "NULL pointer");
  SDD_REQUIRE(max_batch > 0 && max_len > 0, "bad max_batch/max_len");
  const int es = cfg->dtype == SDD_BF16 ? 2 : 4;
  size_t hdr = align_up((size_t)(2 * max_batch + 1) * 4, 256);
  size_t rope = align_up((size_t)max_len * cfg->head_dim * 4, 256);
  size_t per_layer = align_up((size_t)max_batch * cfg->n_kv_heads * kv_ld(max_len) * cfg->head_dim * es, 256);
  *bytes = hdr + rope + 2 * per_layer * (size_t)std::max(1, cfg->n_layers);
  return SDD_OK;
}

extern "C" int sdd_kv_create(sdd_model* m, int max_batch, int max_len, void* buf, size_t bytes, sdd_stream_t stream,
                             sdd_kv** out) {
  SDD_REQUIRE(m && buf && out, "NULL pointer");
  size_t need = 0;
  int rc = sdd_kv_bytes(&m->cfg, max_batch, max_len, &need);
  if (rc) return rc;
  if (bytes < need) return fail(SDD_ENOMEM, "KV buffer needs %zu bytes, got %zu", need, bytes);
  SDD_REQUIRE((uintptr_t)buf % 256 == 0, "KV buffer must be 256-byte aligned");
  sdd_kv* kv = new (std::nothrow) sdd_kv();
  if (!kv) return fail(SDD_ENOMEM, "host allocation failed");
  const sdd_model_config& c = m->cfg;
  kv->m = m;
  kv->max_batch = max_batch;
  kv->max_len = max_len;
  kv->base = reinterpret_cast<char*>(buf);
  kv->bytes = bytes;
  kv->len = reinterpret_cast<int32_t*>(kv->base);
  kv->pending = kv->len + max_batch;
  kv->err = kv->pending + max_batch;
  size_t hdr = align_up((size_t)(2 * max_batch + 1) * 4, 256);
  kv->rope = reinterpret_cast<float*>(kv->base + hdr);
  size_t rope = align_up((size_t)max_len * c.head_dim * 4, 256);
  kv->ld = kv_ld(max_len);
  kv->layer_stride = align_up((size_t)max_batch * c.n_kv_heads * kv->ld * c.head_dim * m->es, 256);
  kv->k = kv->base + hdr + rope;
  kv->v = kv->k + kv->layer_stride * (size_t)std::max(1, c.n_layers);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int64_t n = (int64_t)max_len * (c.head_dim / 2);
  hipLaunchKernelGGL(kv_init_kernel, dim3((int)std::min<int64_t>(ceil_div(n, 256), 4096)), dim3(256), 0, st, kv->len,
                     kv->pending, kv->err, max_batch, kv->rope, max_len, c.head_dim / 2, (double)c.rope_theta);
  rc = check_launch("kv_init_kernel");
  if (rc) {
    delete kv;
    return rc;
  }
  *out = kv;
  return SDD_OK;
}

extern "C" int sdd_kv_destroy(sdd_kv* kv) {
  delete kv;
  return SDD_OK;
}

extern "C" int sdd_kv_state(sdd_kv* kv, int32_t* len, int32_t* pending, int32_t* error_bits, sdd_stream_t stream) {
  SDD_REQUIRE(kv != nullptr, "kv is NULL");
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (len) SDD_HIP(hipMemcpyAsync(len, kv->len, (size_t)kv->max_batch * 4, hipMemcpyDeviceToHost, st));
  if (pending) SDD_HIP(hipMemcpyAsync(pending, kv->pending, (size_t)kv->max_batch * 4, hipMemcpyDeviceToHost, st));
  if (error_bits) SDD_HIP(hipMemcpyAsync(error_bits, kv->err, 4, hipMemcpyDeviceToHost, st));
  SDD_HIP(hipStreamSynchronize(st));
  return SDD_OK;
}

extern "C" int sdd_kv_device_state(sdd_kv* kv, const int32_t** len, const int32_t** pending) {
  SDD_REQUIRE(kv != nullptr, "kv is NULL");
  if (len) *len = kv->len;
  if (pending) *pending = kv->pending;
  return SDD_OK;
}

extern "C" int sdd_workspace_bytes(const sdd_model* m, int max_rows, size_t* bytes) {
  SDD_REQUIRE(m && bytes, "NULL pointer");
  SDD_REQUIRE(max_rows > 0 && max_rows <= 65536, "bad max_rows %d", max_rows);
  *bytes = ws_layout(m, max_rows).total;
  return SDD_OK;
}

static int make_ctx(CallCtx& cx, sdd_model* m, sdd_kv* kv, void* ws, size_t ws_bytes, int rows, hipStream_t st) {
  SDD_REQUIRE(m && kv && ws, "NULL pointer");
  SDD_REQUIRE(kv->m == m, "KV cache belongs to another model");
  SDD_REQUIRE((uintptr_t)ws % 256 == 0, "workspace must be 256-byte aligned");
  cx.m = m;
  cx.kv = kv;
  cx.ws = reinterpret_cast<char*>(ws);
  cx.L = ws_layout(m, rows);
  cx.st = st;
  if (cx.L.total > ws_bytes)
    return fail(SDD_ECAPACITY, "workspace of %zu bytes is too small for %d rows (%zu needed)", ws_bytes, rows, cx.L.total);
  return SDD_OK;
}

extern "C" int sdd_kv_prefill(sdd_model* m, sdd_kv* kv, int seq, const int32_t* tokens, int n, void* ws,
                              size_t ws_bytes, sdd_stream_t stream) {
  SDD_REQUIRE(m && kv && tokens, "NULL pointer");
  SDD_REQUIRE(seq >= 0 && seq < kv->max_batch, "bad seq %d", seq);
  SDD_REQUIRE(n >= 1, "prefill needs at least one token");
  if (n - 1 > kv->max_len) return fail(SDD_ECAPACITY, "prompt of %d tokens exceeds max_len %d", n, kv->max_len);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // largest chunk whose layout fits the workspace
  int chunk = 0;
  for (int r : {256, 128, 64, 32, 16}) {
    if (ws_layout(m, r).total <= ws_bytes) {
      chunk = r;
      break;
    }
  }
  if (chunk == 0) return fail(SDD_ECAPACITY, "workspace too small for prefill");
  for (int c0 = 0; c0 < n - 1; c0 += chunk) {
    const int rows = std::min(chunk, n - 1 - c0);
    CallCtx cx;
    int rc = make_ctx(cx, m, kv, ws, ws_bytes, chunk, st);
    if (rc) return rc;
    EmbedArgs e{};
    e.prefill = 1;
    e.seq = seq;
    e.pos0 = c0;
    e.tokens = tokens + c0;
    e.R = rows;
    if ((rc = launch_embed(cx, e, rows))) return rc;
    if ((rc = forward_rows(cx, 1, rows, nullptr, nullptr))) return rc;
  }
  hipLaunchKernelGGL(prefill_finish_kernel, dim3(1), dim3(64), 0, st, kv->len, kv->pending, kv->err, seq, n, tokens,
                     m->cfg.vocab);
  return check_launch("prefill_finish_kernel");
}

extern "C" int sdd_verify_block(sdd_model* m, sdd_kv* kv, const int32_t* seq_ids, int n_seq, const int32_t* drafts,
                                int gamma, float* logits, int32_t* argmax, void* ws, size_t ws_bytes,
                                sdd_stream_t stream) {
  SDD_REQUIRE(m && kv && seq_ids && logits, "NULL pointer");
  SDD_REQUIRE(n_seq > 0 && n_seq <= kv->max_batch, "bad n_seq %d", n_seq);
  SDD_REQUIRE(gamma >= 0 && gamma <= 64, "gamma must be in [0, 64]");
  SDD_REQUIRE(gamma == 0 || drafts, "drafts is NULL");
  if (gamma + 1 > kv->max_len) return fail(SDD_ECAPACITY, "block of %d rows exceeds max_len", gamma + 1);
  const int R = gamma + 1, M = n_seq * R;
  CallCtx cx;
  int rc = make_ctx(cx, m, kv, ws, ws_bytes, M, reinterpret_cast<hipStream_t>(stream));
  if (rc) return rc;
  EmbedArgs e{};
  e.prefill = 0;
  e.seq_ids = seq_ids;
  e.drafts = drafts;
  e.kv_len = kv->len;
  e.pending = kv->pending;
  e.R = R;
  e.gamma = gamma;
  if ((rc = launch_embed(cx, e, M))) return rc;
  return forward_rows(cx, n_seq, R, logits, argmax);
}

extern "C" int sdd_verify_full(sdd_model* m, sdd_kv* scratch, const int32_t* tokens, int n, int gamma, float* logits,
                               int32_t* argmax, void* ws, size_t ws_bytes, sdd_stream_t stream) {
  SDD_REQUIRE(m && scratch && tokens && logits, "NULL pointer");
  SDD_REQUIRE(gamma >= 0 && gamma <= 64, "gamma must be in [0, 64]");
  SDD_REQUIRE(n >= gamma + 1, "%d tokens cannot hold a block of gamma = %d drafts after a context token", n, gamma);
  if (n > scratch->max_len) return fail(SDD_ECAPACITY, "%d tokens exceed the scratch cache's max_len %d", n, scratch->max_len);
  // every position's K/V is recomputed into slot 0 of the scratch cache: the context first (prefill caches
  // positions 0..n-gamma-2 and leaves token n-gamma-1 pending), then the gamma + 1 verify rows
  int rc = sdd_kv_prefill(m, scratch, 0, tokens, n - gamma, ws, ws_bytes, stream);
  if (rc) return rc;
  CallCtx cx;
  if ((rc = make_ctx(cx, m, scratch, ws, ws_bytes, gamma + 1, reinterpret_cast<hipStream_t>(stream)))) return rc;
  EmbedArgs e{};
  e.prefill = 0;
  e.seq_ids = nullptr;  // block 0 is slot 0
  e.drafts = gamma > 0 ? tokens + (n - gamma) : nullptr;
  e.kv_len = scratch->len;
  e.pending = scratch->pending;
  e.R = gamma + 1;
  e.gamma = gamma;
  if ((rc = launch_embed(cx, e, gamma + 1))) return rc;
  return forward_rows(cx, 1, gamma + 1, logits, argmax);
}

extern "C" int sdd_kv_commit(sdd_kv* kv, const int32_t* seq_ids, int n_seq, const int32_t* accepted_len,
                             const int32_t* next_token, sdd_stream_t stream) {
  SDD_REQUIRE(kv && seq_ids && accepted_len && next_token, "NULL pointer");
  SDD_REQUIRE(n_seq > 0 && n_seq <= kv->max_batch, "bad n_seq %d", n_seq);
  hipLaunchKernelGGL(commit_kernel, dim3((n_seq + 255) / 256), dim3(256), 0, reinterpret_cast<hipStream_t>(stream),
                     kv->len, kv->pending, kv->err, seq_ids, n_seq, accepted_len, next_token, kv->max_len,
                     kv->max_batch, kv->m->cfg.vocab);
  return check_launch("commit_kernel");
}
