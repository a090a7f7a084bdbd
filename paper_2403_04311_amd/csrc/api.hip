// Host entry points of the C ABI declared in include/alto.h.
#include <limits.h>
#include <mutex>
#include <string.h>

#include <atomic>
#include <random>

#include "aggregate.h"

// Workspace of alto_aggregate_noalloc: one array per GPU, held until the process
// ends. Host code never uses this name as an address (on the host it only stands
// for the symbol); each device's address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[ALTO_NOALLOC_SCRATCH_BYTES];

// Fingerprint keys: SplitMix64 outputs of a counter that starts at a value drawn
// from the operating system's entropy source when the library first needs one.
uint64_t fresh_fp_key() {
  static std::atomic<uint64_t> next{0};
  static const uint64_t base = [] {
    std::random_device rd;
    return ((uint64_t)rd() << 32) ^ (uint64_t)rd();
  }();
  return mix64(base + 0x9E3779B97F4A7C15ull * next.fetch_add(1, std::memory_order_relaxed));
}

KeyGeom make_geom(const alto_layout* l) {
  KeyGeom g;
  memset(&g, 0, sizeof(g));
  g.fkey = fresh_fp_key();
  g.depth = l->depth;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) total += l->bits[i];
  g.total = total;
  g.shift[0] = total;
  int below = total;
  for (int lev = 1; lev <= l->depth; ++lev) {
    below -= l->bits[lev - 1];
    g.shift[lev] = below;
    g.tagmask[lev] = (uint32_t)((1ull << l->bits[lev - 1]) - 1ull);
  }
  return g;
}

RouteGeom make_route(const KeyGeom& g, int route_level, int num_dest) {
  RouteGeom r;
  r.shift = route_level <= 0 ? 64 : g.shift[route_level];
  r.num_dest = (uint32_t)(num_dest < 1 ? 1 : num_dest);
  return r;
}

namespace {

__global__ void k_pack(const int32_t* __restrict__ path, int64_t ld, int64_t n, KeyGeom g, uint64_t* keys,
                       int32_t* status) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    uint64_t k = 0;
    for (int l = 1; l <= g.depth; ++l) {
      const int32_t t = path[(int64_t)(l - 1) * ld + i];
      bad |= (t < 0) || ((uint32_t)t > g.tagmask[l]);
      k |= ((uint64_t)(uint32_t)t & (uint64_t)g.tagmask[l]) << g.shift[l];
    }
    keys[i] = k;
  }
  if (bad) raise_status(status, ALTO_E_LAYOUT);
}

bool layout_ok(const alto_layout* l) {
  if (!l || l->depth < 2 || l->depth > ALTO_MAX_LEVELS) return false;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) {
    if (l->bits[i] < 1 || l->bits[i] > 32) return false;
    total += l->bits[i];
  }
  return total <= 63;
}

bool agg_ok(const alto_layout* l, const alto_agg* a, int route_level, int num_dest) {
  if (!a) return false;
  const int d = l->depth;
  if (a->level < 1 || a->level > d - 1) return false;
  if (a->mask_level < 0 || a->mask_level > d - 1) return false;
  if (a->op != ALTO_CONCAT_I32 && a->op != ALTO_MEAN_F32) return false;
  if (a->op == ALTO_MEAN_F32 && (a->dim < 1 || a->dim > (1 << 20))) return false;
  if (a->release != ALTO_RELEASE_COMPLETE && a->release != ALTO_RELEASE_IN_ORDER) return false;
  if (route_level < 0 || route_level > a->level) return false;
  if (route_level == 0 && num_dest != 1) return false;
  return true;
}

const int64_t N_LIMIT = (int64_t)INT_MAX - 1;

GroupOut to_dev_out(const alto_groups* o) {
  GroupOut g;
  g.cap_groups = o->cap_groups;
  g.cap_tokens = o->cap_tokens;
  g.cap_mask = o->cap_mask;
  g.key = o->key;
  g.dest = o->dest;
  g.count = o->count;
  g.first_i32 = o->first_i32;
  g.fan_up = o->fan_up;
  g.tok_off = o->tok_off;
  g.tok = o->tok;
  g.mean = o->mean;
  g.mask_key = o->mask_key;
  g.mask = o->mask;
  g.pend_key = o->pend_key;
  g.pend_count = o->pend_count;
  g.counts = o->counts;
  return g;
}

}  // namespace

namespace {
constexpr int NOALLOC_MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[NOALLOC_MAX_DEVICES];

// Device address of the scratch array on the current device, looked up once per
// device (with that device current); null if the lookup fails.
void* scratch_on_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= NOALLOC_MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" {

size_t alto_workspace_bytes(const alto_layout* layout, int64_t n_max, int32_t num_dest, const alto_agg* agg) {
  if (!layout_ok(layout) || n_max < 0 || n_max > N_LIMIT || num_dest < 1 || num_dest > (1 << 24)) return 0;
  KeyGeom g = make_geom(layout);
  // size for the widest case the aggregation allows (route level 1 gives the most
  // segmented levels when a mask sits above the route level)
  size_t worst = 0;
  const int lr_max = agg ? agg->level : layout->depth;
  for (int lr = (agg ? 0 : 1); lr <= lr_max; ++lr) {
    if (agg && !agg_ok(layout, agg, lr, lr == 0 ? 1 : num_dest)) continue;
    WsCarver c{nullptr, (size_t)-1, 0, true};
    AggBufs b;
    plan_buffers(g, n_max, make_route(g, lr, num_dest), agg, lr, c, b);
    if (c.off > worst) worst = c.off;
  }
  return worst;
}

int alto_pack_keys(const int32_t* path, int64_t path_ld, int64_t n, const alto_layout* layout, uint64_t* keys,
                   int32_t* status, hipStream_t stream) {
  if (!layout_ok(layout) || n < 0 || n > N_LIMIT || path_ld < n || !status) return ALTO_E_ARG;
  if (n == 0) return ALTO_OK;
  if (!path || !keys) return ALTO_E_ARG;
  KeyGeom g = make_geom(layout);
  int64_t blocks = cdiv(n, 256 * 4);
  if (blocks > 4096) blocks = 4096;
  k_pack<<<(int)blocks, 256, 0, stream>>>(path, path_ld, n, g, keys, status);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

int alto_route(const uint64_t* keys, int64_t n, const alto_layout* layout, int32_t route_level, int32_t num_dest,
               int32_t* perm, int64_t* dest_offsets, int32_t* dest, int32_t* status, void* ws, size_t ws_bytes,
               hipStream_t stream) {
  if (!layout_ok(layout) || n < 0 || n > N_LIMIT || route_level < 1 || route_level > layout->depth || num_dest < 1 ||
      num_dest > (1 << 24) || !status || !perm || !dest_offsets)
    return ALTO_E_ARG;
  KeyGeom g = make_geom(layout);
  RouteGeom rg = make_route(g, route_level, num_dest);
  if (n == 0) {
    zero_offsets(dest_offsets, num_dest, stream);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  if (!keys || !ws) return ALTO_E_ARG;
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  AggBufs b;
  plan_buffers(g, n, rg, nullptr, route_level, c, b);
  if (!c.ok) return ALTO_E_ARG;
  return route_run(g, rg, keys, n, b, perm, dest_offsets, dest, nullptr, 0, 1, 0, status, stream);
}

int alto_aggregate_dev(const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* payload_i32,
                       const float* payload_f32, int64_t n, const int64_t* n_dev, const alto_layout* layout,
                       const alto_agg* agg, int32_t route_level, int32_t num_dest, int32_t* perm,
                       int64_t* dest_offsets, int32_t* dest, alto_groups* out, int32_t* status, void* ws,
                       size_t ws_bytes, hipStream_t stream) {
  // n: the batch's count (n_dev null) or its bound (the count is *n_dev on the device)
  if (!layout_ok(layout) || n < 0 || n > N_LIMIT || num_dest < 1 || num_dest > (1 << 24) || !status || !out ||
      !out->counts || !agg_ok(layout, agg, route_level, num_dest) || out->cap_groups < 0 || out->cap_tokens < 0 ||
      out->cap_mask < 0)
    return ALTO_E_ARG;
  if (agg->release != ALTO_RELEASE_COMPLETE) return ALTO_E_ARG;   // an order of release needs a stream
  if (agg->op == ALTO_CONCAT_I32 && !payload_i32 && n > 0) return ALTO_E_ARG;
  if (agg->op == ALTO_MEAN_F32 && !payload_f32 && n > 0) return ALTO_E_ARG;
  GroupOut o = to_dev_out(out);
  if (n == 0) {
    empty_outputs(o, dest_offsets, num_dest, stream);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  if (!keys || !fan || fan_ld < n || !ws) return ALTO_E_ARG;
  KeyGeom g = make_geom(layout);
  RouteGeom rg = make_route(g, route_level, num_dest);
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  AggBufs b;
  plan_buffers(g, n, rg, agg, route_level, c, b);
  if (!c.ok) return ALTO_E_ARG;
  return aggregate_run(g, rg, route_level, *agg, keys, fan, fan_ld, payload_i32, payload_f32, n, b, perm,
                       dest_offsets, dest, o, status, stream, n_dev);
}

int alto_aggregate_overlap(const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* payload_i32,
                           const float* payload_f32, int64_t n, const alto_layout* layout, const alto_agg* agg,
                           int32_t route_level, int32_t num_dest, int32_t* perm, int64_t* dest_offsets,
                           int32_t* dest, alto_groups* out, int32_t* status, void* ws, size_t ws_bytes,
                           hipStream_t stream, hipStream_t gather_stream) {
  if (!layout_ok(layout) || n < 0 || n > N_LIMIT || num_dest < 1 || num_dest > (1 << 24) || !status || !out ||
      !out->counts || !agg_ok(layout, agg, route_level, num_dest) || out->cap_groups < 0 || out->cap_tokens < 0 ||
      out->cap_mask < 0)
    return ALTO_E_ARG;
  if (agg->release != ALTO_RELEASE_COMPLETE) return ALTO_E_ARG;
  if (agg->op == ALTO_CONCAT_I32 && !payload_i32 && n > 0) return ALTO_E_ARG;
  if (agg->op == ALTO_MEAN_F32 && !payload_f32 && n > 0) return ALTO_E_ARG;
  GroupOut o = to_dev_out(out);
  if (n == 0) {
    empty_outputs(o, dest_offsets, num_dest, stream);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  if (!keys || !fan || fan_ld < n || !ws) return ALTO_E_ARG;
  KeyGeom g = make_geom(layout);
  RouteGeom rg = make_route(g, route_level, num_dest);
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  AggBufs b;
  plan_buffers(g, n, rg, agg, route_level, c, b);
  if (!c.ok) return ALTO_E_ARG;
  return aggregate_run(g, rg, route_level, *agg, keys, fan, fan_ld, payload_i32, payload_f32, n, b, perm,
                       dest_offsets, dest, o, status, stream, nullptr, gather_stream);
}

int alto_aggregate(const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* payload_i32,
                   const float* payload_f32, int64_t n, const alto_layout* layout, const alto_agg* agg,
                   int32_t route_level, int32_t num_dest, int32_t* perm, int64_t* dest_offsets, int32_t* dest,
                   alto_groups* out, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream) {
  return alto_aggregate_dev(keys, fan, fan_ld, payload_i32, payload_f32, n, nullptr, layout, agg, route_level,
                            num_dest, perm, dest_offsets, dest, out, status, ws, ws_bytes, stream);
}


int alto_aggregate_noalloc(const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* payload_i32,
                           const float* payload_f32, int64_t n, const alto_layout* layout, const alto_agg* agg,
                           int32_t route_level, int32_t num_dest, int32_t* perm, int64_t* dest_offsets,
                           int32_t* dest, alto_groups* out, int32_t* status, hipStream_t stream) {
  if (!layout_ok(layout) || n < 0 || n > N_LIMIT || num_dest < 1 || num_dest > (1 << 24) ||
      !agg_ok(layout, agg, route_level, num_dest))
    return ALTO_E_ARG;
  const size_t need = alto_workspace_bytes(layout, n, num_dest, agg);
  if (need == 0 || need > (size_t)ALTO_NOALLOC_SCRATCH_BYTES) return ALTO_E_ARG;   // too large for the scratch
  void* ws = scratch_on_current_device();
  if (!ws) return ALTO_E_HIP;
  return alto_aggregate(keys, fan, fan_ld, payload_i32, payload_f32, n, layout, agg, route_level, num_dest, perm,
                        dest_offsets, dest, out, status, ws, (size_t)ALTO_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
