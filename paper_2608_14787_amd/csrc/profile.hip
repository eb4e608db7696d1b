// Launch timing for benchmarks: while enabled, every n-th launch of the
// selected kernel classes is bracketed with HIP events on its own stream (an
// event pair costs a few microseconds of stream time, so sampling keeps the
// timed work close to the untimed one).  Single-threaded use; the events are
// recorded into a fixed pool allocated at start.
#include <vector>

#include "sdd_internal.h"

namespace sdd {
namespace {
struct Rec {
  unsigned cls;
  hipEvent_t a, b;
};
unsigned g_mask = 0;
int g_every = 1;
long long g_seen = 0;
std::vector<hipEvent_t> g_pool;
std::vector<Rec> g_recs;
size_t g_next = 0;
bool g_open = false;
Rec g_cur;
}  // namespace

void prof_begin(unsigned cls, hipStream_t st) {
  if (!(g_mask & cls) || g_next + 2 > g_pool.size()) return;
  if (g_seen++ % g_every) return;
  g_cur.cls = cls;
  g_cur.a = g_pool[g_next++];
  g_cur.b = g_pool[g_next++];
  (void)hipEventRecord(g_cur.a, st);
  g_open = true;
}

void prof_end(unsigned cls, hipStream_t st) {
  if (!g_open || g_cur.cls != cls) return;
  (void)hipEventRecord(g_cur.b, st);
  g_recs.push_back(g_cur);
  g_open = false;
}
}  // namespace sdd

using namespace sdd;

extern "C" int sdd_profile_start(unsigned class_mask, int max_launches, int every) {
  SDD_REQUIRE(max_launches > 0 && max_launches <= (1 << 20), "bad max_launches");
  SDD_REQUIRE(every >= 1, "bad sampling interval");
  g_every = every;
  g_seen = 0;
  for (hipEvent_t e : g_pool) (void)hipEventDestroy(e);
  g_pool.clear();
  g_recs.clear();
  g_next = 0;
  g_open = false;
  g_pool.resize(2 * (size_t)max_launches);
  for (auto& e : g_pool) SDD_HIP(hipEventCreate(&e));
  g_mask = class_mask;
  return SDD_OK;
}

extern "C" int sdd_profile_read(unsigned cls, int* launches, double* total_ms, double* min_ms, double* max_ms) {
  SDD_REQUIRE(launches && total_ms, "NULL pointer");
  int n = 0;
  double tot = 0, mn = 1e30, mx = 0;
  for (const Rec& r : g_recs) {
    if (!(r.cls & cls)) continue;
    SDD_HIP(hipEventSynchronize(r.b));
    float ms = 0.f;
    SDD_HIP(hipEventElapsedTime(&ms, r.a, r.b));
    ++n;
    tot += ms;
    mn = ms < mn ? ms : mn;
    mx = ms > mx ? ms : mx;
  }
  *launches = n;
  *total_ms = tot;
  if (min_ms) *min_ms = n ? mn : 0;
  if (max_ms) *max_ms = mx;
  return SDD_OK;
}

extern "C" int sdd_profile_stop(void) {
  g_mask = 0;
  g_recs.clear();
  g_next = 0;
  g_open = false;
  for (hipEvent_t e : g_pool) (void)hipEventDestroy(e);
  g_pool.clear();
  return SDD_OK;
}
