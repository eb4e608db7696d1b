// Many-row GEMM on gfx950: the projections of a verify call over more than 64
// rows (the blocks of several sequences verified together, Sec. 3.1 per
// sequence) and of prefill chunks.
//
// At 33 rows a projection is bound by streaming its weights once and the
// matrix cores are mostly idle.  At a few hundred rows (8 sequences x 33 rows)
// the same weight bytes feed eight times the MFMA work, so a launch has to
// stream the weights from HBM once at full bandwidth and keep the matrix cores
// busy.  Design:
//  - a workgroup of 8 waves: waves 4-7 only move data, waves 0-3 compute.
//    The movers load every k-step's weight tiles and activation fragments
//    straight into an LDS ring (direct-to-LDS buffer loads: no registers held
//    per load), 4 to 11 k-steps ahead depending on the row count; the
//    computing waves issue no global loads at all, only LDS reads and MFMAs.
//    Measured: the launch is bound by the CU's load throughput (~27 GB/s per
//    CU, as for the 33-row kernel), not by the matrix cores or LDS: every
//    column group re-reads the k-step's activation fragments (M x 64 bytes
//    against NG KiB of weights, twice the weight bytes at 264 rows and 8-tile
//    groups), so wider groups are what would bring it closer to the HBM bound;
//  - one barrier per k-step, without a memory fence: a mover waits for its
//    own loads of the k-step (a memory-counter wait) before it;
//  - the computing waves split the row tiles (wave w owns tiles w, w + 4,
//    ...): each holds NG x TBW accumulator tiles of its own rows, no
//    cross-wave reduction is needed, and a row's sum runs over the k-steps in
//    order whatever the other rows, so a row's result does not depend on how
//    rows are batched (among launches of this kernel);
//  - stream-K over (column group, k-step) units, as in the 33-row kernel; a
//    split group's partials are stored in the accumulator layout and summed
//    by the group's last contributor in workgroup order;
//  - the final tile (up to 288 rows) is staged in LDS, in the space the
//    ring used, and the fused epilogues of the 33-row kernel run on its
//    64-row chunks (16-row pieces for a last partial chunk).
// The wide matrices (gate/up with the SwiGLU epilogue, the LM head) run a
// second kernel, gemm_pair_kernel: a workgroup covers two adjacent 8-tile
// column groups, so each k-step's activation fragments feed 256 columns
// instead of 128, and all 8 waves both load and compute.  Its LDS reads are
// issued by inline assembly with one explicit wait: the compiler cannot tell
// them from reads of the slots the wave's own direct-to-LDS loads are still
// filling, and otherwise waits for every load in flight before them, which
// serialises each k-step on a full memory round trip.
#include "gemm.h"

namespace sdd {
namespace {

constexpr int kRowsThreads = 512;
constexpr size_t kRingBudget = 148 * 1024;  // LDS for the ring (the rest: row info, row scales, the fix-up flag)
// s_waitcnt operand waiting for every LDS operation only (gfx9: vmcnt 63, expcnt 7, lgkmcnt 0)
constexpr int kWaitLgkm0 = 0xC07F;

// A 16-byte-per-lane direct-to-LDS buffer load: lane l's 16 bytes at `lds` + 16 l.  A device function (no host
// compilation of the builtin, which takes an LDS address).
template <int AUX>
__device__ inline void load_lds16(__amdgpu_buffer_rsrc_t rs, void* lds, int voffset, int soffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(lds), 16, voffset, soffset, 0,
                                           AUX);
}

// s_waitcnt operand: vector memory count <= n (0..63), the other counters unconstrained (gfx9 encoding:
// vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int wait_vmcnt(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// 16 bytes from LDS address `addr`, by an instruction the compiler's wait insertion does not track: the caller
// waits for it (lgkmcnt) before using the result.
__device__ inline u32x4 lds_read16(uint32_t addr) {
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr));
  return r;
}

// A workgroup barrier without a memory fence (a fence would wait for every load in flight); LDS
// writes are completed before it by an explicit wait.  The signal fences keep the compiler from
// moving memory accesses across it.
__device__ inline void bare_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int NG, int TBW, int EPI>
__global__ void __launch_bounds__(kRowsThreads, 1) gemm_rows_kernel(GemmArgs a) {
  using T = uint16_t;
  constexpr int C = NG * 16, CP = C + 4;
  static_assert(NG == 8 || NG == 4, "column groups of 8 or 4 tiles");
  static_assert(TBW >= 2 && TBW <= kRowsMaxTBW, "row tiles per wave");
  // ring stage: the k-step's NG weight tiles, then its 4 TBW activation fragments (row tile tb at NG + tb), 1 KiB
  // each, lane l's 16 bytes at 16 l (the layout of both in global memory and in the MFMA operands)
  constexpr int kStage = (NG + 4 * TBW) * 1024;
  constexpr int RS = std::min<int>(12, (int)(kRingBudget / kStage));  // ring stages; RS - 1 k-steps in flight
  constexpr int DW = NG / 4 + TBW;  // loads a mover wave issues per k-step
  static_assert(RS >= 3 && (RS - 2) * DW <= 63, "ring depth within the memory counter");
  // One LDS region serves three phases: the prologue's partial sums of squares [4][kRowsMaxRows] (after the
  // ring, so that the movers' first loads can land while the prologue runs), the k-loop's ring, the epilogue's
  // final tile [kRowsMaxRows][CP] fp32.
  constexpr size_t kPartOff = (size_t)RS * kStage;
  constexpr size_t kBig = std::max((size_t)kRowsMaxRows * CP * 4, kPartOff + (size_t)4 * kRowsMaxRows * 4);
  __shared__ __align__(16) char s_big[kBig];
  __shared__ RowInfo s_ri[kRowsMaxRows];
  __shared__ float s_rs[kRowsMaxRows];
  __shared__ int s_flag;
  float* const s_tile = reinterpret_cast<float*>(s_big);
  float* const s_part = reinterpret_cast<float*>(s_big + kPartOff);
  touch_kernargs<GemmArgs>();
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const bool loader = wv >= 4;
  const int wave = wv & 3;
  const int w = blockIdx.x;
  const uint32_t KT = (uint32_t)a.KT, G = (uint32_t)a.G, SC = (uint32_t)a.segc;
  const uint32_t u0 = unit_start(w, KT, G, SC, a.n_wg), u1 = unit_start(w + 1, KT, G, SC, a.n_wg);
  const int g_first = (int)(u0 / KT);
  const int ntiles = (a.M + 15) / 16;
  // weights, stored in the order of the launch's plan: the i-th unit (NG tiles of 1 KiB, lane l's fragment at
  // 16 l) of workgroup w at slot i * n_wg + w, so this workgroup's consecutive units are kstep_w bytes apart
  const uint32_t kstep_w = (uint32_t)a.n_wg * NG * 1024;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(a.W), 0, (int)(a.share * kstep_w), kBufferRsrcWord3);
  // a descriptor with no range: loads through it return zero without a memory access
  const __amdgpu_buffer_rsrc_t nrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.W), 0, 0, kBufferRsrcWord3);
  // activations: row r of the launch at X + (m0 + r) * ldx elements.  Row tile tb's fragment of k-step kt: lane l
  // reads row 16 tb + l % 16, elements 32 kt + 8 (l / 16) .. + 7.  The descriptor ends at the launch's last row,
  // so the rows of a padded tile read zero without a memory access.
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(a.X), 0, (a.m0 + a.M) * a.ldx * (int)sizeof(T), kBufferRsrcWord3);
  int xl[TBW];  // mover: byte offset of this lane's fragment of row tile wave + 4 j (< 2^31: checked on the host)
#pragma unroll
  for (int j = 0; j < TBW; ++j) xl[j] = ((a.m0 + 16 * (wave + 4 * j) + lane % 16) * a.ldx + (lane / 16) * 8) * 2;

  struct Seg {
    int g, kb, ke, nk;
    uint32_t wo, xo;  // bytes of the segment's first k-step in the weights and in an activation row
  };
  auto make_seg = [&](uint32_t u) {
    Seg s;
    s.g = (int)(u / KT);
    s.kb = (int)(u - (uint32_t)s.g * KT);
    s.ke = (int)std::min<uint32_t>(KT, s.kb + (u1 - u));
    s.nk = s.ke - s.kb;
    s.wo = (u - u0) * kstep_w + (uint32_t)w * NG * 1024;
    s.xo = (uint32_t)s.kb * 64;
    return s;
  };
  // mover: this wave's DW loads of local k-step kt into ring slot kt % RS -- weight tiles wave * NG/4 + i and
  // the fragments of row tiles wave + 4 j.  Every call issues the same loads, a k-step past the segment through
  // the empty descriptor (no memory access), so that the memory-counter waits count alike on every path.
  auto issue = [&](const Seg& s, int kt) {
    char* slot = s_big + (kt % RS) * kStage;
    const bool in = kt < s.nk;
    const __amdgpu_buffer_rsrc_t wd = in ? wrs : nrs, xd = in ? xrs : nrs;
#pragma unroll
    for (int i = 0; i < NG / 4; ++i) {
      const int nt = wave * (NG / 4) + i;
      load_lds16<kNtCpol>(wd, slot + nt * 1024, lane * 16, (int)(s.wo + (uint32_t)kt * kstep_w + (uint32_t)nt * 1024));
    }
#pragma unroll
    for (int j = 0; j < TBW; ++j)
      load_lds16<0>(xd, slot + (NG + wave + 4 * j) * 1024, xl[j], (int)(s.xo + (uint32_t)kt * 64));
  };
  // Row info and RMSNorm row scales of the launch's rows, for the epilogues.  A row's scale sums the producer's
  // per-group sums of squares in the 33-row kernel's order (four threads per row, every fourth group in group
  // order, then (s0 + s1) + (s2 + s3)), so both kernels scale a row alike.
  auto prologue = [&]() {
    const int tid = threadIdx.x;
    if constexpr (EPI == EPI_QKV || EPI == EPI_LOGITS) {
      for (int r = tid; r < a.M; r += kRowsThreads) s_ri[r] = a.rows[a.m0 + r];
    }
    if constexpr (EPI != EPI_RESID) {
      const int ng_in = a.ss_in ? a.ss_groups : 0;
      for (int idx = tid; idx < 4 * a.M; idx += kRowsThreads) {
        const int q4 = idx / a.M, row = idx - q4 * a.M;
        float ssum = 0.f;
        for (int g0 = q4; g0 < ng_in; g0 += 64) {
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
        s_part[q4 * kRowsMaxRows + row] = ssum;
      }
      __syncthreads();
      for (int r = tid; r < a.M; r += kRowsThreads) {
        const float tot = (s_part[r] + s_part[kRowsMaxRows + r]) + (s_part[2 * kRowsMaxRows + r] + s_part[3 * kRowsMaxRows + r]);
        s_rs[r] = ng_in ? 1.f / sqrtf(tot / (float)a.d_in + a.eps) : 1.f;
      }
      __syncthreads();  // the region is the weight slots' next
    }
  };

  // The two roles run their own segment loops (so that the accumulators are not live in the loaders'
  // registers) with the same sequence of barriers: the prologue's on the first segment, one per k-step, two
  // in arrive_last for a split group, two around the final tile's staging, one between segments.
  auto contributors = [&](int g, int& wf, int& wl) {
    wf = unit_owner((uint32_t)g * KT, KT, G, SC, a.n_wg);
    wl = unit_owner((uint32_t)(g + 1) * KT - 1, KT, G, SC, a.n_wg);
  };
  uint32_t u = u0;
  if (loader) {
    for (bool first = true;; first = false) {
      const Seg s = make_seg(u);
      for (int kt = 0; kt < RS - 1; ++kt) issue(s, kt);  // RS - 1 k-steps in flight
      if (first) prologue();
      for (int kt = 0; kt < s.nk; ++kt) {
        __builtin_amdgcn_s_waitcnt(wait_vmcnt((RS - 2) * DW));  // this wave's loads of k-step kt have landed
        bare_barrier();  // ... and every mover's: slot kt % RS is complete; slot (kt - 1) % RS has been read
        issue(s, kt + RS - 1);
      }
      __builtin_amdgcn_s_waitcnt(wait_vmcnt(0));  // the loads past the segment land before the slots are reused
      u += s.nk;
      bool fin = true;
      if (!(s.kb == 0 && s.ke == a.KT)) {
        int wf, wl;
        contributors(s.g, wf, wl);
        fin = arrive_last(&a.cnt[s.g * kCntStride], wl - wf + 1, &s_flag);
      }
      if (fin) {
        __syncthreads();
        __syncthreads();
      }
      if (u >= u1) break;
      __syncthreads();
    }
    return;
  }

  for (bool first = true;; first = false) {
    const Seg s = make_seg(u);
    f32x4 acc[NG][TBW];
#pragma unroll
    for (int nt = 0; nt < NG; ++nt)
#pragma unroll
      for (int j = 0; j < TBW; ++j) acc[nt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (first) prologue();
    for (int kt = 0; kt < s.nk; ++kt) {
      // the previous k-step's LDS reads are complete before the barrier lets the movers refill that slot
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      bare_barrier();  // k-step kt is in slot kt % RS
      const uint4* slot = reinterpret_cast<const uint4*>(s_big + (kt % RS) * kStage);
      uint4 wf[NG], xf[TBW];  // every fragment read first: one LDS latency per k-step
#pragma unroll
      for (int nt = 0; nt < NG; ++nt) wf[nt] = slot[nt * kWave + lane];
#pragma unroll
      for (int j = 0; j < TBW; ++j) xf[j] = slot[(NG + wave + 4 * j) * kWave + lane];
#pragma unroll
      for (int nt = 0; nt < NG; ++nt)
#pragma unroll
        for (int j = 0; j < TBW; ++j) mma_tile<T>(wf[nt], xf[j], acc[nt][j]);
    }
    const int g = s.g;
    const int which = g == g_first ? 0 : 1;
    u += s.nk;

    bool fin = true;
    if (!(s.kb == 0 && s.ke == a.KT)) {
      // split column group: every contributor stores its partial in the accumulator layout with 16-byte
      // device-coherent stores; the last arriver sums all of them in workgroup order
      const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7fffffff, kBufferRsrcWord3);
      auto part_off = [&](int wg, int slot, int j, int nt) {  // bytes (< 2^31: the host sizes the buffer)
        return ((((wg * 2 + slot) * kRowsMaxTBW + j) * NG + nt) * 4 + wave) * 1024 + lane * 16;
      };
#pragma unroll
      for (int j = 0; j < TBW; ++j)
        if (wave + 4 * j < ntiles)
#pragma unroll
          for (int nt = 0; nt < NG; ++nt)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nt][j]), prs, part_off(w, which, j, nt), 0,
                                                   kCoherentCpol);
      int wf, wl;
      contributors(g, wf, wl);
      fin = arrive_last(&a.cnt[g * kCntStride], wl - wf + 1, &s_flag);
      if (fin) {
#pragma unroll
        for (int nt = 0; nt < NG; ++nt)
#pragma unroll
          for (int j = 0; j < TBW; ++j) acc[nt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // a contributor published into its slot 0 when g is its share's first group: every contributor but
        // the first, whose share starts inside group g or before it
        const bool wf_first = unit_start(wf, KT, G, SC, a.n_wg) == (uint32_t)g * KT;
        for (int ww = wf; ww <= wl; ++ww) {
          const int slot = (ww > wf || wf_first) ? 0 : 1;
          // one row tile at a time (NG loads in flight), so that the loaded partials fit beside the sums
#pragma unroll
          for (int j = 0; j < TBW; ++j) {
            f32x4 v[NG];
#pragma unroll
            for (int nt = 0; nt < NG; ++nt)
              v[nt] = (wave + 4 * j < ntiles)
                          ? __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(prs, part_off(ww, slot, j, nt), 0,
                                                                                              kCoherentCpol))
                          : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int nt = 0; nt < NG; ++nt) acc[nt][j] += v[nt];
          }
        }
      }
    }

    if (fin) {
      // the whole final tile into LDS (row tile wave + 4 j of each computing wave at rows 16 (wave + 4 j)), after
      // every wave's last reads of the weight slots that the tile overwrites
      __syncthreads();
      f32x4* trow = reinterpret_cast<f32x4*>(&s_tile[(16 * wave + lane % 16) * CP + 4 * (lane / 16)]);
#pragma unroll
      for (int j = 0; j < TBW; ++j)
        if (wave + 4 * j < ntiles)
#pragma unroll
          for (int nt = 0; nt < NG; ++nt) trow[(64 * j * CP) / 4 + nt * 4] = acc[nt][j];
      __syncthreads();
      // the fused epilogue on 64-row chunks, the last partial chunk in 16-row pieces (the tile holds whole row
      // tiles only)
      const int full = a.M / kMaxPassRows;
      for (int c = 0; c < full; ++c) {
        GemmArgs ac = a;
        ac.m0 = a.m0 + kMaxPassRows * c;
        ac.M = kMaxPassRows;
        const float* t = s_tile + kMaxPassRows * c * CP;
        const int r0 = kMaxPassRows * c;
        if constexpr (EPI == EPI_QKV) epilogue_qkv<T, NG, kMaxPassRows>(ac, t, g, s_rs + r0, s_ri + r0);
        if constexpr (EPI == EPI_RESID) epilogue_resid<T, NG, kMaxPassRows>(ac, t, g);
        if constexpr (EPI == EPI_SWIGLU) epilogue_swiglu<T, NG, kMaxPassRows>(ac, t, g, s_rs + r0);
        if constexpr (EPI == EPI_LOGITS) epilogue_logits<NG, kMaxPassRows>(ac, t, g, s_rs + r0, s_ri + r0);
      }
      for (int r0 = kMaxPassRows * full; r0 < a.M; r0 += 16) {
        GemmArgs ac = a;
        ac.m0 = a.m0 + r0;
        ac.M = min(16, a.M - r0);
        const float* t = s_tile + r0 * CP;
        if constexpr (EPI == EPI_QKV) epilogue_qkv<T, NG, 16>(ac, t, g, s_rs + r0, s_ri + r0);
        if constexpr (EPI == EPI_RESID) epilogue_resid<T, NG, 16>(ac, t, g);
        if constexpr (EPI == EPI_SWIGLU) epilogue_swiglu<T, NG, 16>(ac, t, g, s_rs + r0);
        if constexpr (EPI == EPI_LOGITS) epilogue_logits<NG, 16>(ac, t, g, s_rs + r0, s_ri + r0);
      }
    }
    if (u >= u1) break;
    __syncthreads();  // the epilogue's LDS reads are done before the next segment's loaders write the slots
  }
}

// Column-group pairs (8-tile groups): a workgroup computes the tiles of two adjacent column groups 2p and
// 2p + 1 over its rows, so that every k-step's activation fragments are loaded into LDS once for 256 columns
// instead of once per 128 (halving the activation bytes a launch moves, the bulk of its loads above 64 rows).
// All 8 waves load and compute: wave v computes group v / 4 on row tiles v % 4 + 4 j; the loads into LDS
// are split between the waves as described at the ring constants below.  The pairs are
// partitioned over the launch's workgroups as P x KT stream-K units with equal shares (P = ceil(G / 2) pairs,
// P * split workgroups when P is below the workgroup budget, else that budget); each weight tile is read where
// the matrix's own streaming plan stores it.  A row's sum runs over the k-steps in order, split pairs' partials
// added in workgroup order, so a row's result does not depend on the rows launched with it.
template <int TBW, int EPI>
__global__ void __launch_bounds__(kRowsThreads, 1) gemm_pair_kernel(GemmArgs a) {
  using T = uint16_t;
  constexpr int NG = 8, C = NG * 16, CP = C + 4;
  static_assert(TBW >= 2 && TBW <= kRowsMaxTBW, "row tiles per wave");
  constexpr int NX = 4 * TBW;                     // activation row tiles per k-step
  // Up to 256 rows (TBW <= 4) two rings: waves 0-3 load only weight tiles, into a deep ring, and waves 4-7
  // only activation fragments, into a 3-stage one (a wave's loads complete in order, so separate depths need
  // separate waves): the weights, from HBM, run further ahead.  At 257-288 rows the activation stages are
  // too large for that split and one ring holds both: each wave loads weight tile v of both groups and the
  // fragments of row tiles v, v + 8, ...
  constexpr bool kTwo = TBW <= 4;
  constexpr int kStage = (2 * NG + NX) * 1024;    // one ring: weight tiles of both groups, then the fragments
  constexpr int RS = std::min<int>(12, (int)(kRingBudget / kStage));
  constexpr int XQ = NX / 8, XR = NX % 8;         // one ring: wave v loads XQ + (v < XR) fragments per k-step
  constexpr int DHI = 2 + XQ + (XR ? 1 : 0), DLO = 2 + XQ;
  constexpr int kWS = 2 * NG * 1024, kXS = NX * 1024;  // two rings: weight stage, activation stage
  constexpr int RX = 3;
  constexpr int RW = std::min<int>(12, (int)((kRingBudget - RX * kXS) / kWS));
  static_assert(XR == 0 || XR == 4, "row tiles per stage");
  static_assert(kTwo || (RS >= 3 && (RS - 2) * DHI <= 63), "ring depth within the memory counter");
  static_assert(!kTwo || (RW >= 3 && (RW - 2) * 4 <= 63 && (RX - 2) * TBW <= 63), "ring depths within the memory counter");
  constexpr size_t kXOff = (size_t)RW * kWS;
  constexpr size_t kPartOff = kTwo ? kXOff + (size_t)RX * kXS : (size_t)RS * kStage;
  constexpr size_t kBig = std::max((size_t)kRowsMaxRows * CP * 4, kPartOff + (size_t)4 * kRowsMaxRows * 4);
  __shared__ __align__(16) char s_big[kBig];
  __shared__ RowInfo s_ri[kRowsMaxRows];
  __shared__ float s_rs[kRowsMaxRows];
  __shared__ int s_flag;
  float* const s_tile = reinterpret_cast<float*>(s_big);
  float* const s_part = reinterpret_cast<float*>(s_big + kPartOff);
  const uint32_t lds_ring = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)(s_big);
  touch_kernargs<GemmArgs>();
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = threadIdx.x % kWave;
  const int half = v >> 2, wave = v & 3;
  const bool xhi = v < XR;
  const bool wload = v < 4;                        // two rings: this wave loads weights (else fragments)
  const int RL = kTwo ? (wload ? RW : RX) : RS;    // depth of the ring this wave fills
  const int w = blockIdx.x;
  // storage plan of the matrix (the 33-row kernels' stream-K partition)
  const uint32_t KT = (uint32_t)a.KT, G = (uint32_t)a.G, SC = (uint32_t)a.segc, NW = (uint32_t)a.n_wg;
  // this launch's partition: pairs
  const uint32_t P = (G + 1) / 2, NP = gridDim.x;
  const uint32_t u0 = unit_start(w, KT, P, 0, NP), u1 = unit_start(w + 1, KT, P, 0, NP);
  const int p_first = (int)(u0 / KT);
  const int ntiles = (a.M + 15) / 16;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(a.W), 0, (int)((uint32_t)a.share * NW * NG * 1024), kBufferRsrcWord3);
  const __amdgpu_buffer_rsrc_t nrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(a.W), 0, 0, kBufferRsrcWord3);
  const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(a.X), 0, (a.m0 + a.M) * a.ldx * (int)sizeof(T), kBufferRsrcWord3);
  // byte offset of this lane's fragment of each row tile the wave loads (< 2^31: checked on the host): one
  // ring, row tiles v + 8 j; two rings, row tiles wave + 4 j
  constexpr int NXL = kTwo ? TBW : XQ + 1;
  int xl[NXL];
#pragma unroll
  for (int j = 0; j < NXL; ++j) {
    const int rt = kTwo ? wave + 4 * j : v + 8 * j;
    xl[j] = ((a.m0 + 16 * rt + lane % 16) * a.ldx + (lane / 16) * 8) * 2;
  }

  // Where the storage plan keeps k-step k of column group g: unit g KT + k of owner o at slot
  // (g KT + k - start(o)) n_wg + o.  A tracker follows one group's owners as k rises.
  struct Trk {
    int o, kend, base;  // current owner, the group's first k-step past its share, slot of k-step 0 under it
  };
  auto trk_set = [&](Trk& t, uint32_t g, int o) {
    const uint32_t us = unit_start((uint32_t)o, KT, G, SC, NW), ue = unit_start((uint32_t)o + 1, KT, G, SC, NW);
    t.o = o;
    t.kend = (int)(ue - g * KT);
    t.base = ((int)(g * KT) - (int)us) * (int)NW + o;
  };
  auto trk_at = [&](Trk& t, uint32_t g, int k) { trk_set(t, g, unit_owner(g * KT + (uint32_t)k, KT, G, SC, NW)); };
  auto trk_adv = [&](Trk& t, uint32_t g, int k) {
    while (k >= t.kend) trk_set(t, g, t.o + 1);
  };

  struct Seg {
    int p, kb, ke, nk;
    uint32_t xo;  // bytes of the segment's first k-step in an activation row
  };
  auto make_seg = [&](uint32_t u) {
    Seg s;
    s.p = (int)(u / KT);
    s.kb = (int)(u - (uint32_t)s.p * KT);
    s.ke = (int)std::min<uint32_t>(KT, s.kb + (u1 - u));
    s.nk = s.ke - s.kb;
    s.xo = (uint32_t)s.kb * 64;
    return s;
  };
  // this wave's loads of local k-step kt (one ring: weight tile v of both groups and its fragments; two
  // rings: a weight wave tiles 4 (v & 1) .. + 3 of group 2p + (v >> 1), an activation wave its TBW
  // fragments).  A k-step past the segment goes through the empty descriptor (no memory access) so that the
  // memory-counter waits count alike on every path.
  auto issue = [&](const Seg& s, bool has_b, int kt, Trk& ta, Trk& tb) {
    const bool in = kt < s.nk;
    const int k = s.kb + kt;
    if constexpr (!kTwo) {
      char* slot = s_big + (kt % RS) * kStage;
      int oa = 0, ob = 0;
      if (in) {
        trk_adv(ta, 2 * s.p, k);
        oa = __builtin_amdgcn_readfirstlane((ta.base + k * (int)NW) * NG * 1024 + v * 1024);
        if (has_b) {
          trk_adv(tb, 2 * s.p + 1, k);
          ob = __builtin_amdgcn_readfirstlane((tb.base + k * (int)NW) * NG * 1024 + v * 1024);
        }
      }
      load_lds16<kNtCpol>(in ? wrs : nrs, slot + v * 1024, lane * 16, oa);
      load_lds16<kNtCpol>(in && has_b ? wrs : nrs, slot + (NG + v) * 1024, lane * 16, ob);
      const __amdgpu_buffer_rsrc_t xd = in ? xrs : nrs;
#pragma unroll
      for (int j = 0; j <= XQ; ++j)
        if (j < XQ || xhi) load_lds16<0>(xd, slot + (2 * NG + v + 8 * j) * 1024, xl[j], (int)(s.xo + (uint32_t)kt * 64));
    } else if (wload) {
      char* slot = s_big + (kt % RW) * kWS;
      const int h = v >> 1, q = 4 * (v & 1);
      const bool valid = in && (h == 0 || has_b);
      int off = 0;
      if (valid) {
        Trk& t = h ? tb : ta;
        trk_adv(t, 2 * s.p + h, k);
        off = __builtin_amdgcn_readfirstlane((t.base + k * (int)NW) * NG * 1024 + q * 1024);
      }
      const __amdgpu_buffer_rsrc_t wd = valid ? wrs : nrs;
#pragma unroll
      for (int i = 0; i < 4; ++i) load_lds16<kNtCpol>(wd, slot + (h * NG + q + i) * 1024, lane * 16, off + i * 1024);
    } else {
      char* slot = s_big + kXOff + (kt % RX) * kXS;
      const __amdgpu_buffer_rsrc_t xd = in ? xrs : nrs;
#pragma unroll
      for (int j = 0; j < TBW; ++j) load_lds16<0>(xd, slot + (wave + 4 * j) * 1024, xl[j], (int)(s.xo + (uint32_t)kt * 64));
    }
  };
  // Row info and RMSNorm row scales, as in gemm_rows_kernel (the 33-row kernel's summation order).
  auto prologue = [&]() {
    const int tid = threadIdx.x;
    if constexpr (EPI == EPI_QKV || EPI == EPI_LOGITS) {
      for (int r = tid; r < a.M; r += kRowsThreads) s_ri[r] = a.rows[a.m0 + r];
    }
    if constexpr (EPI != EPI_RESID) {
      const int ng_in = a.ss_in ? a.ss_groups : 0;
      for (int idx = tid; idx < 4 * a.M; idx += kRowsThreads) {
        const int q4 = idx / a.M, row = idx - q4 * a.M;
        float ssum = 0.f;
        for (int g0 = q4; g0 < ng_in; g0 += 64) {
          float vv[16];
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int gg = g0 + 4 * j;
            vv[j] = gg < ng_in ? a.ss_in[(int64_t)gg * a.mp + a.m0 + row] : 0.f;
          }
#pragma unroll
          for (int j = 0; j < 16; ++j)
            if (g0 + 4 * j < ng_in) ssum += vv[j];
        }
        s_part[q4 * kRowsMaxRows + row] = ssum;
      }
      __syncthreads();
      for (int r = tid; r < a.M; r += kRowsThreads) {
        const float tot = (s_part[r] + s_part[kRowsMaxRows + r]) + (s_part[2 * kRowsMaxRows + r] + s_part[3 * kRowsMaxRows + r]);
        s_rs[r] = ng_in ? 1.f / sqrtf(tot / (float)a.d_in + a.eps) : 1.f;
      }
      __syncthreads();
    }
  };
  // the fused epilogue of column group g on the staged tile: 64-row chunks alternate between the two halves
  // of the workgroup (each half's 4 waves run one chunk), then the 16-row pieces of a last partial chunk
  auto epilogue = [&](int g) {
    const int full = a.M / kMaxPassRows;
    for (int c = half; c < full; c += 2) {
      GemmArgs ac = a;
      ac.m0 = a.m0 + kMaxPassRows * c;
      ac.M = kMaxPassRows;
      const float* t = s_tile + kMaxPassRows * c * CP;
      const int r0 = kMaxPassRows * c;
      if constexpr (EPI == EPI_QKV) epilogue_qkv<T, NG, kMaxPassRows>(ac, t, g, s_rs + r0, s_ri + r0);
      if constexpr (EPI == EPI_RESID) epilogue_resid<T, NG, kMaxPassRows>(ac, t, g);
      if constexpr (EPI == EPI_SWIGLU) epilogue_swiglu<T, NG, kMaxPassRows>(ac, t, g, s_rs + r0);
      if constexpr (EPI == EPI_LOGITS) epilogue_logits<NG, kMaxPassRows>(ac, t, g, s_rs + r0, s_ri + r0);
    }
    for (int r0 = kMaxPassRows * full + 16 * half; r0 < a.M; r0 += 32) {
      GemmArgs ac = a;
      ac.m0 = a.m0 + r0;
      ac.M = min(16, a.M - r0);
      const float* t = s_tile + r0 * CP;
      if constexpr (EPI == EPI_QKV) epilogue_qkv<T, NG, 16>(ac, t, g, s_rs + r0, s_ri + r0);
      if constexpr (EPI == EPI_RESID) epilogue_resid<T, NG, 16>(ac, t, g);
      if constexpr (EPI == EPI_SWIGLU) epilogue_swiglu<T, NG, 16>(ac, t, g, s_rs + r0);
      if constexpr (EPI == EPI_LOGITS) epilogue_logits<NG, 16>(ac, t, g, s_rs + r0, s_ri + r0);
    }
  };

  uint32_t u = u0;
  for (bool first = true;; first = false) {
    const Seg s = make_seg(u);
    const bool has_b = (uint32_t)(2 * s.p + 1) < G;
    const bool mine = half == 0 || has_b;  // this wave's group exists
    Trk ta{0, 0, 0}, tb{0, 0, 0};
    if (!kTwo || v < 2) trk_at(ta, 2 * s.p, s.kb);
    if (has_b && (!kTwo || (v >= 2 && v < 4))) trk_at(tb, 2 * s.p + 1, s.kb);
    for (int kt = 0; kt < RL - 1; ++kt) issue(s, has_b, kt, ta, tb);  // RL - 1 k-steps in flight
    if (first) prologue();
    f32x4 acc[NG][TBW];
#pragma unroll
    for (int nt = 0; nt < NG; ++nt)
#pragma unroll
      for (int j = 0; j < TBW; ++j) acc[nt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int kt = 0; kt < s.nk; ++kt) {
      // this wave's loads of k-step kt have landed and its LDS reads of k-step kt - 1 are complete; after the
      // barrier every wave's are: k-step kt is whole in the ring(s) and k-step kt - 1's slots are free
      if constexpr (kTwo) {
        if (wload)
          __builtin_amdgcn_s_waitcnt(wait_vmcnt((RW - 2) * 4));
        else
          __builtin_amdgcn_s_waitcnt(wait_vmcnt((RX - 2) * TBW));
      } else {
        if (xhi)
          __builtin_amdgcn_s_waitcnt(wait_vmcnt((RS - 2) * DHI));
        else
          __builtin_amdgcn_s_waitcnt(wait_vmcnt((RS - 2) * DLO));
      }
      __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
      bare_barrier();
      issue(s, has_b, kt + RL - 1, ta, tb);
      // The fragments are read by LDS instructions the compiler does not see: it cannot tell them from reads of
      // the slots this wave's direct-to-LDS loads are still filling, and would wait for all of those loads
      // (the barrier above already orders them).  One wait for all of them, tied to the registers it fills.
      const uint32_t slw = lds_ring + (uint32_t)(kTwo ? (kt % RW) * kWS : (kt % RS) * kStage) + (uint32_t)lane * 16;
      const uint32_t slx = kTwo ? lds_ring + (uint32_t)(kXOff + (kt % RX) * kXS) + (uint32_t)lane * 16
                                : slw + (uint32_t)(2 * NG * 1024);
      u32x4 wf[NG], xf[TBW];
#pragma unroll
      for (int nt = 0; nt < NG; ++nt) wf[nt] = lds_read16(slw + (uint32_t)((half * NG + nt) * 1024));
#pragma unroll
      for (int j = 0; j < TBW; ++j) xf[j] = lds_read16(slx + (uint32_t)((wave + 4 * j) * 1024));
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int nt = 0; nt < NG; ++nt) asm volatile("" : "+v"(wf[nt]));
#pragma unroll
      for (int j = 0; j < TBW; ++j) asm volatile("" : "+v"(xf[j]));
#pragma unroll
      for (int nt = 0; nt < NG; ++nt)
#pragma unroll
        for (int j = 0; j < TBW; ++j)
          mma_tile<T>(__builtin_bit_cast(uint4, wf[nt]), __builtin_bit_cast(uint4, xf[j]), acc[nt][j]);
    }
    __builtin_amdgcn_s_waitcnt(wait_vmcnt(0));  // the loads past the segment land before the slots are reused
    const int which = s.p == p_first ? 0 : 1;
    u += s.nk;

    bool fin = true;
    if (!(s.kb == 0 && s.ke == (int)KT)) {
      // split pair: every contributor stores its partials (both groups) in the accumulator layout with 16-byte
      // device-coherent stores; the last arriver sums all of them in workgroup order
      const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(a.part, 0, 0x7fffffff, kBufferRsrcWord3);
      auto part_off = [&](int wg, int sl, int j, int nt) {  // bytes (< 2^31: the host sizes the buffer)
        return (((((wg * 2 + sl) * 2 + half) * kRowsMaxTBW + j) * NG + nt) * 4 + wave) * 1024 + lane * 16;
      };
      if (mine)
#pragma unroll
        for (int j = 0; j < TBW; ++j)
          if (wave + 4 * j < ntiles)
#pragma unroll
            for (int nt = 0; nt < NG; ++nt)
              __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, acc[nt][j]), prs, part_off(w, which, j, nt),
                                                     0, kCoherentCpol);
      const int wf = unit_owner((uint32_t)s.p * KT, KT, P, 0, NP);
      const int wl = unit_owner((uint32_t)(s.p + 1) * KT - 1, KT, P, 0, NP);
      fin = arrive_last(&a.cnt[s.p * kCntStride], wl - wf + 1, &s_flag);
      if (fin && mine) {
#pragma unroll
        for (int nt = 0; nt < NG; ++nt)
#pragma unroll
          for (int j = 0; j < TBW; ++j) acc[nt][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // a contributor published into its slot 0 when the pair is its share's first: every contributor but
        // the first, whose share starts at the pair's first unit or before it
        const bool wf_first = unit_start(wf, KT, P, 0, NP) == (uint32_t)s.p * KT;
        for (int ww = wf; ww <= wl; ++ww) {
          const int sl = (ww > wf || wf_first) ? 0 : 1;
#pragma unroll
          for (int j = 0; j < TBW; ++j) {
            f32x4 pv[NG];
#pragma unroll
            for (int nt = 0; nt < NG; ++nt)
              pv[nt] = (wave + 4 * j < ntiles)
                           ? __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(prs, part_off(ww, sl, j, nt), 0,
                                                                                               kCoherentCpol))
                           : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int nt = 0; nt < NG; ++nt) acc[nt][j] += pv[nt];
          }
        }
      }
    }

    if (fin) {
      // each group's final tile in turn: staged in LDS by the waves that hold it (row tile wave + 4 j at rows
      // 16 (wave + 4 j)), then its epilogue on all 8 waves
      for (int h = 0; h < 2; ++h) {
        if (h == 1 && !has_b) break;
        __syncthreads();  // the ring's (or the previous tile's) LDS reads are done
        if (half == h) {
          f32x4* trow = reinterpret_cast<f32x4*>(&s_tile[(16 * wave + lane % 16) * CP + 4 * (lane / 16)]);
#pragma unroll
          for (int j = 0; j < TBW; ++j)
            if (wave + 4 * j < ntiles)
#pragma unroll
              for (int nt = 0; nt < NG; ++nt) trow[(64 * j * CP) / 4 + nt * 4] = acc[nt][j];
        }
        __syncthreads();
        epilogue(2 * s.p + h);
      }
    }
    if (u >= u1) break;
    __syncthreads();  // the epilogue's LDS reads are done before the next segment's loads write the slots
  }
}

template <int EPI>
void launch_pair_tbw(int tbw, const GemmArgs& a, int nb, hipStream_t st) {
  const dim3 grid(nb), block(kRowsThreads);
  switch (tbw) {
    case 2: hipLaunchKernelGGL((gemm_pair_kernel<2, EPI>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemm_pair_kernel<3, EPI>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_pair_kernel<4, EPI>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_pair_kernel<5, EPI>), grid, block, 0, st, a); break;
  }
}

template <int NG, int EPI>
void launch_tbw(int tbw, const GemmArgs& a, int nb, hipStream_t st) {
  const dim3 grid(nb), block(kRowsThreads);
  switch (tbw) {
    case 2: hipLaunchKernelGGL((gemm_rows_kernel<NG, 2, EPI>), grid, block, 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemm_rows_kernel<NG, 3, EPI>), grid, block, 0, st, a); break;
    case 4: hipLaunchKernelGGL((gemm_rows_kernel<NG, 4, EPI>), grid, block, 0, st, a); break;
    default: hipLaunchKernelGGL((gemm_rows_kernel<NG, 5, EPI>), grid, block, 0, st, a); break;
  }
}

template <int NG>
void launch_epi(int epi, int tbw, const GemmArgs& a, int nb, hipStream_t st) {
  switch (epi) {
    case EPI_QKV: launch_tbw<NG, EPI_QKV>(tbw, a, nb, st); break;
    case EPI_RESID: launch_tbw<NG, EPI_RESID>(tbw, a, nb, st); break;
    case EPI_SWIGLU: launch_tbw<NG, EPI_SWIGLU>(tbw, a, nb, st); break;
    default: launch_tbw<NG, EPI_LOGITS>(tbw, a, nb, st); break;
  }
}

}  // namespace

int launch_gemm_rows(int ng, int epi, const GemmArgs& a, int nblocks, hipStream_t st) {
  if (ng != 8 && ng != 4) return fail(SDD_EUNSUPPORTED, "many-row GEMM: column groups of %d tiles", ng);
  if (a.M < 1 || a.M > kRowsMaxRows) return fail(SDD_EUNSUPPORTED, "many-row GEMM: %d rows in one launch", a.M);
  const int tbw = std::max(2, (int)ceil_div(a.M, 4 * 16));
  if (ng == 8 && (epi == EPI_SWIGLU || epi == EPI_LOGITS)) {
    // pairs of 8-tile groups (the wide matrices: gate/up, LM head)
    const int64_t P = (a.G + 1) / 2;
    // each pair on nblocks / P workgroups (split evenly) when there are fewer pairs than workgroups, else
    // stream-K over nblocks: a many-row partial is M x 256 fp32, so splitting a pair further costs more in
    // partial stores and fix-up reads than the idle compute units it would fill
    const int64_t np = P >= nblocks ? nblocks : P * std::min<int64_t>(nblocks / P, a.KT);
    if ((P * a.KT + 1) * np >= (int64_t(1) << 31))
      return fail(SDD_EUNSUPPORTED, "many-row GEMM: %lld x %d units exceed the 32-bit stream-K bookkeeping",
                  (long long)P, a.KT);
    if (epi == EPI_SWIGLU)
      launch_pair_tbw<EPI_SWIGLU>(tbw, a, (int)np, st);
    else
      launch_pair_tbw<EPI_LOGITS>(tbw, a, (int)np, st);
    return check_launch("gemm_pair_kernel");
  }
  if (ng == 8) {
    launch_epi<8>(epi, tbw, a, nblocks, st);
    return check_launch("gemm_rows_kernel");
  }
  launch_epi<4>(epi, tbw, a, nblocks, st);
  return check_launch("gemm_rows_kernel");
}

}  // namespace sdd
