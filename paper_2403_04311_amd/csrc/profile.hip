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

// A plain streaming read (diagnostics): every block streams one contiguous chunk
// with 16-byte non-temporal loads, RU in flight per thread (measured on MI355X:
// contiguous chunks per block read ~2% faster than a grid-stride loop), and stores
// the XOR of its words with a plain store (device-scope atomics at the end of every
// block, all ending together, cost ~17% of the bandwidth).
namespace {
constexpr int RU = 8;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void k_read_probe(const u32x4* __restrict__ p, int64_t n16, int64_t per_block,
                                                    uint64_t* out) {
  __shared__ uint32_t s_x[256 / ALTO_WAVE];
  uint32_t x = 0;
  const int64_t b0 = (int64_t)blockIdx.x * per_block;
  const int64_t b1 = b0 + per_block < n16 ? b0 + per_block : n16;
  for (int64_t i0 = b0 + threadIdx.x; i0 < b1; i0 += 256 * RU) {
    u32x4 v[RU];
#pragma unroll
    for (int u = 0; u < RU; ++u) {
      const int64_t i = i0 + u * 256;
      v[u] = i < b1 ? __builtin_nontemporal_load(p + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < RU; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (int o = ALTO_WAVE / 2; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
  if (lane_id() == 0) s_x[threadIdx.x / ALTO_WAVE] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < 256 / ALTO_WAVE; ++w) t ^= s_x[w];
    out[blockIdx.x] = t;
  }
  if (blockIdx.x == 0)
    for (int b = gridDim.x + threadIdx.x; b < ALTO_READ_PROBE_WORDS; b += blockDim.x) out[b] = 0;
}
}  // namespace

extern "C" {

int alto_read_probe(const void* p, int64_t bytes, uint64_t* out, hipStream_t stream) {
  if (!p || !out || bytes < 16 || (bytes & 15) || ((uintptr_t)p & 15)) return ALTO_E_ARG;
  const int64_t n16 = bytes / 16;
  int64_t grid = cdiv(n16, 256 * RU);
  grid = grid < ALTO_READ_PROBE_WORDS ? grid : ALTO_READ_PROBE_WORDS;
  const int64_t per_block = cdiv(n16, grid);
  k_read_probe<<<(int)grid, 256, 0, stream>>>(reinterpret_cast<const u32x4*>(p), n16, per_block, out);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

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
