// Per-phase timing with HIP events (diagnostics entry points of include/alto.h).
#include "profile.h"

#include <vector>

namespace {
struct Rec {
  int phase;
  hipEvent_t a, b;
};
bool g_on = false;
uint32_t g_mask = ~0u;   // phases recorded
std::vector<Rec> g_recs;
size_t g_used = 0;
int g_open[PH_COUNT];
}  // namespace

void prof_begin(int phase, hipStream_t st) {
  if (!g_on || g_used >= g_recs.size() || !((g_mask >> phase) & 1u)) {
    g_open[phase] = -1;
    return;
  }
  g_open[phase] = (int)g_used;
  Rec& r = g_recs[g_used++];
  r.phase = phase;
  (void)hipEventRecord(r.a, st);
}

void prof_end(int phase, hipStream_t st) {
  if (!g_on || g_open[phase] < 0) return;
  (void)hipEventRecord(g_recs[g_open[phase]].b, st);
  g_open[phase] = -1;
}

extern "C" {

int alto_profile_phases(uint32_t mask) {
  if (g_on) return ALTO_E_ARG;
  g_mask = mask;
  return ALTO_OK;
}

int alto_profile_begin(int32_t max_records) {
  if (g_on || max_records < 1) return ALTO_E_ARG;
  g_recs.resize((size_t)max_records);
  for (auto& r : g_recs) {
    if (hipEventCreate(&r.a) != hipSuccess || hipEventCreate(&r.b) != hipSuccess) return ALTO_E_HIP;
  }
  g_used = 0;
  for (int i = 0; i < PH_COUNT; ++i) g_open[i] = -1;
  g_on = true;
  return ALTO_OK;
}

int alto_profile_end(float* ms, int32_t* calls, int32_t nphase) {
  if (!g_on) return ALTO_E_ARG;
  g_on = false;
  for (int i = 0; i < nphase; ++i) {
    if (ms) ms[i] = 0.f;
    if (calls) calls[i] = 0;
  }
  int rc = ALTO_OK;
  for (size_t k = 0; k < g_used; ++k) {
    Rec& r = g_recs[k];
    if (hipEventSynchronize(r.b) != hipSuccess) rc = ALTO_E_HIP;
    float t = 0.f;
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) rc = ALTO_E_HIP;
    if (r.phase < nphase) {
      if (ms) ms[r.phase] += t;
      if (calls) calls[r.phase] += 1;
    }
  }
  for (auto& r : g_recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_recs.clear();
  g_used = 0;
  return rc;
}

}  // extern "C"
