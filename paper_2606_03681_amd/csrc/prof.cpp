// Per-step HIP-event timing of launch steps (include/tfm_prof.h).
#include "prof.h"

#include <hip/hip_runtime.h>

#include <map>
#include <string>
#include <vector>

#include "tfm_prof.h"

namespace {

struct Rec {
  const char* name;
  hipEvent_t a, b;
};

bool g_on = false;
std::vector<hipEvent_t> g_pool;
size_t g_used = 0;
std::vector<Rec> g_recs;
const char* g_open = nullptr;
hipEvent_t g_open_ev = nullptr;
struct Agg {
  const char* name;
  long long n;
  double ms;
};
std::vector<Agg> g_agg;

hipEvent_t take_event() {
  if (g_used == g_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    g_pool.push_back(e);
  }
  return g_pool[g_used++];
}

}  // namespace

namespace tfm {

void prof_begin(const char* name, hipStream_t s) {
  if (!g_on) return;
  g_open = name;
  g_open_ev = take_event();
  if (g_open_ev && hipEventRecord(g_open_ev, s) != hipSuccess) g_open_ev = nullptr;
}

void prof_end(hipStream_t s) {
  if (!g_on || !g_open || !g_open_ev) return;
  hipEvent_t b = take_event();
  if (!b) return;
  if (hipEventRecord(b, s) != hipSuccess) return;
  g_recs.push_back(Rec{g_open, g_open_ev, b});
  g_open = nullptr;
}

}  // namespace tfm

extern "C" {

int tfm_prof_enable(int on) {
  g_on = on != 0;
  g_used = 0;
  g_recs.clear();
  g_agg.clear();
  g_open = nullptr;
  return 0;
}

int tfm_prof_collect(void) {
  std::map<std::string, size_t> idx;
  g_agg.clear();
  for (const Rec& r : g_recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return -6;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return -6;
    auto it = idx.find(r.name);
    if (it == idx.end()) {
      idx[r.name] = g_agg.size();
      g_agg.push_back(Agg{r.name, 1, ms});
    } else {
      g_agg[it->second].n += 1;
      g_agg[it->second].ms += ms;
    }
  }
  return (int)g_agg.size();
}

int tfm_prof_step(int i, const char** name, long long* launches, double* total_ms) {
  if (i < 0 || (size_t)i >= g_agg.size()) return -1;
  if (name) *name = g_agg[i].name;
  if (launches) *launches = g_agg[i].n;
  if (total_ms) *total_ms = g_agg[i].ms;
  return 0;
}

}  // extern "C"
