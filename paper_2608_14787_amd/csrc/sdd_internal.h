// Internal helpers shared by the HIP translation units of libsdd (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdarg>
#include <cstdio>
#include <string>

#include "../../include/sdd.h"

namespace sdd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---- error reporting ------------------------------------------------------
void set_error(const char* fmt, ...);
int fail(int code, const char* fmt, ...);
int check_launch(const char* what);

#define SDD_REQUIRE(cond, ...)                   \
  do {                                           \
    if (!(cond)) return sdd::fail(SDD_EINVAL, __VA_ARGS__); \
  } while (0)

#define SDD_HIP(call)                                                             \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess)                                                         \
      return sdd::fail(SDD_EHIP, "%s: %s", #call, hipGetErrorString(e_));         \
  } while (0)

// ---- bf16 <-> fp32 (bit-level; round to nearest even) ----------------------
__host__ __device__ inline float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, (uint32_t)b << 16);
}
// Round to nearest even by the gfx950 conversion instruction (v_cvt_pk_bf16_f32): one branch-free
// instruction, where a bit-level version needs a divergent branch for NaN and infinity.  Finite values and
// infinities round exactly as the bit-level definition (add 0x7fff plus the kept lsb, truncate); a NaN
// stays a quiet NaN.
__device__ inline uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// two values in one instruction: a in the low half, b in the high half
__device__ inline uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((float2v){a, b}, bf16x2));
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static constexpr int kVec = 4;  // elements per 16-byte load
  __device__ static inline float load(const float* p) { return *p; }
  __device__ static inline float to_f32(float x) { return x; }
  __device__ static inline float from_f32(float x) { return x; }
};
template <> struct Elem<uint16_t> {
  static constexpr int kVec = 8;
  __device__ static inline float load(const uint16_t* p) { return bf16_to_f32(*p); }
  __device__ static inline float to_f32(uint16_t x) { return bf16_to_f32(x); }
  __device__ static inline uint16_t from_f32(float x) { return f32_to_bf16(x); }
};

// unpack a 16-byte vector into fp32 values
__device__ inline void unpack16(const uint4& v, float* out, float) {
  out[0] = __builtin_bit_cast(float, v.x);
  out[1] = __builtin_bit_cast(float, v.y);
  out[2] = __builtin_bit_cast(float, v.z);
  out[3] = __builtin_bit_cast(float, v.w);
}
__device__ inline void unpack16(const uint4& v, float* out, uint16_t) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __builtin_bit_cast(float, w[i] << 16);
    out[2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xffff0000u);
  }
}

// 16-byte streaming load that bypasses cache residency (data read once)
__device__ inline uint4 load_nt16(const void* p) {
  u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline uint4 load16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Cross-workgroup hand-off without cache-wide fences.  A device-scope fence on
// this part writes back and invalidates a whole L2 (one per XCD), which costs
// far more than the few kilobytes handed over.  Instead the published data and
// the arrival counters use relaxed device-scope atomic accesses, which the
// compiler maps to accesses coherent across all XCDs of the device; a
// publisher waits for its stores to complete before it arrives, and the last
// arriver reads the data back with the same coherent loads.
template <typename T>
__device__ inline void st_coherent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ inline T ld_coherent(T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Raw buffer accesses with the device-coherent cache policy (sc1, the bits the
// compiler uses for device-scope atomic loads and stores): 16 bytes at a time
// where the relaxed atomics above move 4.  Descriptor word 3 of an untyped
// buffer on this GPU family.
constexpr int kBufferRsrcWord3 = 0x00020000;
constexpr int kCoherentCpol = 16;  // sc1
constexpr int kNtCpol = 2;         // nt: streamed once, no cache residency
// s_waitcnt operand (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8) that waits for
// every vector memory operation and leaves the other counters unconstrained
constexpr int kWaitVmcnt0 = 0x0F70;
// Waits until every memory operation this thread issued has completed.
__device__ inline void wait_stores() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
// Every thread of the block must call this after its coherent stores; returns
// (in all threads) whether this block is the last of `expected` arrivals on
// *cnt.  The last arriver finds the counter back at zero for the next use.
__device__ inline bool arrive_last(int* cnt, int expected, int* s_flag) {
  wait_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = old == expected - 1;
    if (last) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = last;
  }
  __syncthreads();
  return *s_flag != 0;
}

// Kernel arguments are read through the scalar cache on first use; a kernel
// whose argument block spans several 64-byte lines otherwise pays one memory
// round trip per line, one after another, as the compiler spreads the reads.
// Touching every line once at entry overlaps those misses.
template <typename Args>
__device__ inline void touch_kernargs() {
  typedef const __attribute__((address_space(4))) int* kernarg_ptr;
  const kernarg_ptr kp = (kernarg_ptr)__builtin_amdgcn_kernarg_segment_ptr();
  constexpr int n = (int)sizeof(Args) / 4;
  int acc = kp[n - 1];
#pragma unroll
  for (int i = 0; i < n; i += 16) acc ^= kp[i];
  asm volatile("" ::"s"(acc));
}

// Lane permutations inside rows of 16 lanes by DPP (a VALU operand modifier:
// no LDS round trip, unlike a general shuffle).  The wave must be fully active.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <- lane 7-i within each 8
constexpr int kDppMirror = 0x140;     // lane i <- lane 15-i within each 16
constexpr int kDppRor8 = 0x128;       // row rotate by 8: lane i <- lane i ^ 8 within each 16
template <int CTRL>
__device__ inline int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __builtin_bit_cast(float, dpp_i<CTRL>(__builtin_bit_cast(int, v)));
}
__device__ inline float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
// op(v[l], v[l ^ 16]) and op(v[l], v[l ^ 32]) in every lane of a fully active
// wave, by the gfx950 row-swap permutes (no LDS round trip).  With a copy of
// v in both registers, v_permlane16_swap leaves each lane holding its own
// row pair's two values (lower row in the first register) and
// v_permlane32_swap likewise for the two halves, so a commutative op gives
// the butterfly's value in every lane.  Written as inline assembly with both
// registers as in/out operands (the compiler's builtins fold the two results
// into one); the nops cover the permute's VALU read/write hazards.
__device__ inline void permlane16_swap(unsigned& a, unsigned& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
__device__ inline void permlane32_swap(unsigned& a, unsigned& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
template <typename Op>
__device__ inline float xor16_op(float v, Op op) {
  unsigned a = __builtin_bit_cast(unsigned, v), b = a;
  permlane16_swap(a, b);
  return op(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}
template <typename Op>
__device__ inline float xor32_op(float v, Op op) {
  unsigned a = __builtin_bit_cast(unsigned, v), b = a;
  permlane32_swap(a, b);
  return op(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b));
}

// wave-level reductions (64 lanes)
__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace sdd

namespace sdd {
// Kernel classes for launch timing (sdd_profile_*).
enum ProfClass : unsigned {
  PROF_EMBED = 1u, PROF_GEMM_QKV = 2u, PROF_ATTN = 4u, PROF_GEMM_O = 8u, PROF_GEMM_GU = 16u,
  PROF_GEMM_DOWN = 32u, PROF_GEMM_LM = 64u, PROF_ACCEPT = 128u, PROF_CONF = 256u,
  PROF_SCHED = 512u, PROF_MLP = 1024u
};
// Bracket a launch with events on its stream when timing of cls is enabled.
void prof_begin(unsigned cls, hipStream_t st);
void prof_end(unsigned cls, hipStream_t st);
}  // namespace sdd
