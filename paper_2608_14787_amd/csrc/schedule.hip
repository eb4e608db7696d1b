// Skip scheduler: the two-gate candidate skip length, the commit guards and the staleness counter
// (Sec. 4.1 "Skip Policy": candidate skip length and commit rule; Sec. 4.2: raw confidence, marginal and
// conditional survival as prefix scores; Appendix "Baselines and Sweep Settings": the guard list).
//
// One lane per sequence.  The block's position scores and drafts are staged into LDS with coalesced loads
// (rows padded by one word so the per-lane sequential reads hit distinct banks); each lane then walks its
// row in position order.  The running sum of log-scores is accumulated strictly left to right in fp32, so
// every gate decision is the same fp32 comparison for every launch shape.
#include "sdd_internal.h"

namespace sdd {
namespace {

constexpr int kSchedThreads = 64;
constexpr int kMaxGamma = 64;
constexpr int kMaxSpecial = 256;
constexpr int kPad = kMaxGamma + 1;

struct SchedArgs {
  const float* log_q;
  const int32_t* draft;
  const int32_t* block_len;
  const int32_t* special;
  int32_t* D;
  int32_t* K;
  int32_t* K_hat;
  int32_t* reason;
  int B, gamma, signal, k_min, s_max, n_special, rep_max;
  float log_eta_b, log_eta_c;
};

#pragma clang fp contract(off)
__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(SchedArgs a) {
  __shared__ float s_lq[kSchedThreads * kPad];
  __shared__ int32_t s_x[kSchedThreads * kPad];
  __shared__ int32_t s_special[kMaxSpecial];
  const int b0 = blockIdx.x * kSchedThreads;
  const int nb = min(kSchedThreads, a.B - b0);
  const int n = nb * a.gamma;
  const bool need_draft = a.n_special > 0 || a.rep_max >= 2;
  // batches of kU loads per thread issued before any is used (n <= 64 x 64)
  constexpr int kU = 16;
  for (int i0 = 0; i0 < n; i0 += kSchedThreads * kU) {
    float v[kU];
    int32_t x[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = i0 + u * kSchedThreads + (int)threadIdx.x;
      v[u] = i < n ? a.log_q[(size_t)b0 * a.gamma + i] : 0.f;
      x[u] = (need_draft && i < n) ? a.draft[(size_t)b0 * a.gamma + i] : 0;
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int i = i0 + u * kSchedThreads + (int)threadIdx.x;
      if (i < n) {
        const int r = i / a.gamma, c = i - r * a.gamma;
        s_lq[r * kPad + c] = v[u];
        s_x[r * kPad + c] = x[u];
      }
    }
  }
  for (int i = threadIdx.x; i < a.n_special; i += kSchedThreads) s_special[i] = a.special[i];
  __syncthreads();
  if ((int)threadIdx.x >= nb) return;
  const int b = b0 + threadIdx.x;
  const float* lq = s_lq + threadIdx.x * kPad;
  const int32_t* x = s_x + threadIdx.x * kPad;

  // candidate skip length: the longest prefix whose local and prefix gates both pass
  int khat = 0;
  float bk = INFINITY, sum = 0.f;
  for (int k = 1; k <= a.gamma; ++k) {
    const float v = lq[k - 1];
    if (__builtin_isnan(v) || v == INFINITY) break;  // invalid score: no longer prefix can pass
    bk = v < bk ? v : bk;
    sum = sum + v;
    const float c = a.signal == SDD_SIG_RAW        ? __fdiv_rn(sum, (float)k)  // log geometric mean
                    : a.signal == SDD_SIG_MARGINAL ? bk                        // running minimum
                                                   : sum;                      // log product
    if (bk >= a.log_eta_b && c >= a.log_eta_c) khat = k;
  }

  int d = a.D[b];
  int r;
  if (d >= a.s_max) r = SDD_SKIP_STALE;
  else if (khat == 0) r = SDD_SKIP_NO_CANDIDATE;
  else if (khat < a.k_min) r = SDD_SKIP_SHORT;
  else if (a.block_len && a.block_len[b] < a.gamma) r = SDD_SKIP_SHORT_BLOCK;
  else {
    r = SDD_SKIP_OK;
    for (int j = 0; j < khat && r == SDD_SKIP_OK && a.n_special > 0; ++j)
      for (int s = 0; s < a.n_special; ++s)
        if (x[j] == s_special[s]) r = SDD_SKIP_SPECIAL;
    if (r == SDD_SKIP_OK && a.rep_max >= 2) {
      int run = 1;
      for (int j = 1; j < khat; ++j) {
        run = x[j] == x[j - 1] ? run + 1 : 1;
        if (run >= a.rep_max) {
          r = SDD_SKIP_REPEAT;
          break;
        }
      }
    }
  }
  const int K = r == SDD_SKIP_OK ? khat : 0;
  a.K[b] = K;
  if (a.K_hat) a.K_hat[b] = khat;
  if (a.reason) a.reason[b] = r;
  a.D[b] = K > 0 ? d + K : 0;  // every verifier call resets the count of unverified tokens
}
#pragma clang fp contract(on)

float log_threshold(double eta) { return eta > 0.0 ? (float)std::log(eta) : -INFINITY; }

// Agreement counters over the rounds that commit an unverified prefix (K > 0): |A|, sum K, sum min(K, L),
// count K <= L.  Integer atomics: the totals do not depend on the order of the additions.
__global__ void audit_kernel(const int32_t* K, const int32_t* L, int B, unsigned long long* acc) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int k = K[b], l = L[b];
  if (k <= 0) return;
  atomicAdd(&acc[0], 1ull);
  atomicAdd(&acc[1], (unsigned long long)k);
  atomicAdd(&acc[2], (unsigned long long)(k < l ? k : (l > 0 ? l : 0)));
  if (k <= l) atomicAdd(&acc[3], 1ull);
}

}  // namespace
}  // namespace sdd

using namespace sdd;

extern "C" int sdd_schedule(const float* log_q, const int32_t* draft, const int32_t* block_len, int B,
                            int gamma, int signal, double eta_b, double eta_c, int k_min, int s_max,
                            const int32_t* special, int n_special, int rep_max, int32_t* D, int32_t* K,
                            int32_t* K_hat, int32_t* reason, sdd_stream_t stream) {
  SDD_REQUIRE(D && K && (gamma == 0 || log_q), "NULL required pointer");
  SDD_REQUIRE(B > 0 && gamma >= 0 && gamma <= kMaxGamma, "bad shape B=%d gamma=%d", B, gamma);
  SDD_REQUIRE(signal >= SDD_SIG_RAW && signal <= SDD_SIG_CONDITIONAL, "bad signal %d", signal);
  SDD_REQUIRE(!std::isnan(eta_b) && !std::isnan(eta_c), "threshold is NaN");
  SDD_REQUIRE(n_special >= 0 && n_special <= kMaxSpecial, "n_special=%d outside [0, %d]", n_special, kMaxSpecial);
  SDD_REQUIRE(n_special == 0 || special, "special is NULL");
  SDD_REQUIRE((n_special == 0 && rep_max < 2) || gamma == 0 || draft, "draft is NULL");
  SchedArgs a{};
  a.log_q = log_q;
  a.draft = draft;
  a.block_len = block_len;
  a.special = special;
  a.D = D;
  a.K = K;
  a.K_hat = K_hat;
  a.reason = reason;
  a.B = B;
  a.gamma = gamma;
  a.signal = signal;
  a.k_min = k_min;
  a.s_max = s_max;
  a.n_special = n_special;
  a.rep_max = rep_max;
  a.log_eta_b = log_threshold(eta_b);
  a.log_eta_c = log_threshold(eta_c);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  prof_begin(PROF_SCHED, st);
  hipLaunchKernelGGL(schedule_kernel, dim3((B + kSchedThreads - 1) / kSchedThreads), dim3(kSchedThreads), 0, st, a);
  prof_end(PROF_SCHED, st);
  return check_launch("schedule_kernel");
}

extern "C" int sdd_audit_accumulate(const int32_t* K, const int32_t* L, int B, int64_t* acc, sdd_stream_t stream) {
  SDD_REQUIRE(K && L && acc, "NULL pointer");
  SDD_REQUIRE(B >= 0, "B = %d", B);
  if (B == 0) return SDD_OK;
  hipLaunchKernelGGL(audit_kernel, dim3((B + 255) / 256), dim3(256), 0, reinterpret_cast<hipStream_t>(stream), K, L, B,
                     reinterpret_cast<unsigned long long*>(acc));
  return check_launch("audit_kernel");
}
