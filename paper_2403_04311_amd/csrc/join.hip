// pcombine (Section 3.2 of the paper): objects that two parallel branches produce
// under the same ancestry are combined. The left branch gives one object per node
// of the join level (its prefix); the right branch gives fragments. The left
// prefixes are sorted once (radix sort, keys = prefixes, values = left indices);
// every right fragment then finds its ancestor's object by binary search over the
// sorted prefixes, which stay in the caches.
#include "sort.h"

#include <limits.h>
#include <string.h>

namespace {

struct JoinBufs {
  uint64_t* skey;      // [n] sorted left prefixes
  uint32_t* sidx;      // [n] left index of each
  uint64_t* tmp_keys;  // [n] sort scratch
  uint32_t* tmp_vals;
  SortCtl* ctl;
  uint32_t* os_status;
  uint32_t* os_ctr;
  uint32_t* os_hist;
  int64_t os_ntiles;
  int32_t* hits;       // [n] when the caller passes none
};

void plan_join(int64_t n_max, WsCarver& c, JoinBufs& b) {
  const int64_t n = n_max < 1 ? 1 : n_max;
  b.skey = c.take<uint64_t>(n);
  b.sidx = c.take<uint32_t>(n);
  b.tmp_keys = c.take<uint64_t>(n);
  b.tmp_vals = c.take<uint32_t>(n);
  b.ctl = c.take<SortCtl>(1);
  b.os_ntiles = sort_tiles(n);
  b.os_status = c.take<uint32_t>(2 * b.os_ntiles * SORT_BUCKETS);
  b.os_ctr = c.take<uint32_t>(SORT_MAX_PASSES);
  b.os_hist = c.take<uint32_t>((int64_t)SORT_MAX_PASSES * SORT_BUCKETS);
  b.hits = c.take<int32_t>(n);
}


// Counts and hits cleared; left prefixes wider than their levels are LAYOUT.
__global__ void k_join_init(const uint64_t* __restrict__ left, int64_t nl, int lbits, int32_t* hits, int64_t* counts,
                            int32_t* status) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nl; i += (int64_t)gridDim.x * blockDim.x) {
    hits[i] = 0;
    bad |= (left[i] >> lbits) != 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) counts[0] = counts[1] = 0;
  if (bad) raise_status(status, ALTO_E_LAYOUT);
}

// Two left objects for one node: adjacent after the sort.
__global__ void k_join_dups(const uint64_t* __restrict__ skey, int64_t nl, int32_t* status) {
  bool dup = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x + 1; i < nl; i += (int64_t)gridDim.x * blockDim.x)
    dup |= skey[i] == skey[i - 1];
  if (dup) raise_status(status, ALTO_E_DUPLICATE);
}

// Right fragments, JU per thread in flight (independent binary searches): the
// level prefix, a binary search over the sorted left prefixes, the match, the
// object's hit count; paired fragments counted per block. Persistent grid.
// MODE 0: prefixes read through the caches, one global atomic per paired fragment.
// MODE 1: hit counts in an LDS histogram of the nl objects, added to the global
//         counts once per block (many fragments share an object: a global atomic
//         per fragment serialises on the popular ones).
// MODE 2: as 1, and the sorted prefixes and their indices copied into LDS too.
constexpr int JU = 4;
constexpr int JOIN_LDS_HITS = 8192;   // MODE 1: 32 KB
constexpr int JOIN_LDS_KEYS = 4096;   // MODE 2: 64 KB (8-byte prefix, 4-byte index, 4-byte count)

template <int MODE>
__global__ __launch_bounds__(256) void k_join_probe(const uint64_t* __restrict__ right, int64_t nr, int total, int shift,
                                                    const uint64_t* __restrict__ skey_g, const uint32_t* __restrict__ sidx_g,
                                                    int64_t nl, int32_t* match, int32_t* hits, int64_t* counts,
                                                    int32_t* status) {
  __shared__ uint64_t s_n[256 / ALTO_WAVE];
  extern __shared__ uint64_t s_dyn[];
  uint32_t* s_hits = reinterpret_cast<uint32_t*>(MODE == 2 ? s_dyn + nl : s_dyn);
  uint32_t* s_idx = s_hits + nl;
  const uint64_t* skey = MODE == 2 ? s_dyn : skey_g;
  if (MODE >= 1) {
    for (int64_t i = threadIdx.x; i < nl; i += blockDim.x) {
      s_hits[i] = 0;
      if (MODE == 2) {
        s_dyn[i] = skey_g[i];
        s_idx[i] = sidx_g[i];
      }
    }
    __syncthreads();
  }
  uint64_t paired = 0;
  bool bad = false;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < nr; i0 += stride * JU) {
    uint64_t p[JU];
    int64_t lo[JU], hi[JU];
#pragma unroll
    for (int u = 0; u < JU; ++u) {
      const int64_t i = i0 + u * stride;
      const uint64_t k = i < nr ? right[i] : 0ull;
      bad |= (k >> total) != 0;
      p[u] = key_prefix(k, shift);
      lo[u] = 0;
      hi[u] = i < nr ? nl : 0;
    }
    // first sorted prefix >= p, the JU searches advancing together
    for (int64_t w = nl; w > 0; w >>= 1) {
#pragma unroll
      for (int u = 0; u < JU; ++u) {
        if (lo[u] < hi[u]) {
          const int64_t mid = (lo[u] + hi[u]) >> 1;
          if (skey[mid] < p[u]) lo[u] = mid + 1; else hi[u] = mid;
        }
      }
    }
#pragma unroll
    for (int u = 0; u < JU; ++u) {
      const int64_t i = i0 + u * stride;
      if (i >= nr) continue;
      int32_t m = -1;
      if (lo[u] < nl && skey[lo[u]] == p[u]) {
        m = (int32_t)(MODE == 2 ? s_idx[lo[u]] : sidx_g[lo[u]]);
        if (MODE >= 1) atomicAdd(&s_hits[m], 1u);
        else atomicAdd(&hits[m], 1);
        ++paired;
      }
      match[i] = m;
    }
  }
  if (bad) raise_status(status, ALTO_E_LAYOUT);
  const uint64_t v = wave_sum(paired);
  if (lane_id() == 0) s_n[threadIdx.x / ALTO_WAVE] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int w = 0; w < 256 / ALTO_WAVE; ++w) t += s_n[w];
    if (t) atomicAdd((unsigned long long*)&counts[0], (unsigned long long)t);
  }
  if (MODE >= 1) {
    for (int64_t i = threadIdx.x; i < nl; i += blockDim.x)
      if (s_hits[i]) atomicAdd(&hits[i], (int32_t)s_hits[i]);
  }
}

// Left objects with at least one paired fragment.
__global__ __launch_bounds__(256) void k_join_count(const int32_t* __restrict__ hits, int64_t nl, int64_t* counts) {
  __shared__ uint64_t s_n[256 / ALTO_WAVE];
  uint64_t c = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nl; i += (int64_t)gridDim.x * blockDim.x)
    c += hits[i] > 0 ? 1 : 0;
  const uint64_t v = wave_sum(c);
  if (lane_id() == 0) s_n[threadIdx.x / ALTO_WAVE] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int w = 0; w < 256 / ALTO_WAVE; ++w) t += s_n[w];
    if (t) atomicAdd((unsigned long long*)&counts[1], (unsigned long long)t);
  }
}

bool join_layout_ok(const alto_layout* l) {
  if (!l || l->depth < 1 || l->depth > ALTO_MAX_LEVELS) return false;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) {
    if (l->bits[i] < 1 || l->bits[i] > 32) return false;
    total += l->bits[i];
  }
  return total <= 63;
}

const int64_t JOIN_N_LIMIT = (int64_t)INT_MAX - 1;

}  // namespace

extern "C" {

size_t alto_join_workspace_bytes(const alto_layout* layout, int64_t n_left_max) {
  if (!join_layout_ok(layout) || n_left_max < 0 || n_left_max > JOIN_N_LIMIT) return 0;
  WsCarver c{nullptr, (size_t)-1, 0, true};
  JoinBufs b;
  plan_join(n_left_max, c, b);
  return c.off;
}

int alto_join(const uint64_t* left, int64_t n_left, const uint64_t* right_keys, int64_t n_right,
              const alto_layout* layout, int32_t level, int32_t* match, int32_t* hits, int64_t* counts,
              int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!join_layout_ok(layout) || level < 1 || level > layout->depth || n_left < 0 || n_left > JOIN_N_LIMIT ||
      n_right < 0 || n_right > JOIN_N_LIMIT || !counts || !status || !ws)
    return ALTO_E_ARG;
  if ((n_left > 0 && !left) || (n_right > 0 && (!right_keys || !match))) return ALTO_E_ARG;
  const KeyGeom g = make_geom(layout);
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  JoinBufs b;
  plan_join(n_left, c, b);
  if (!c.ok) return ALTO_E_ARG;
  int32_t* h = hits ? hits : b.hits;
  const int lbits = g.total - g.shift[level];
  k_join_init<<<grid_for(n_left, 256), 256, 0, stream>>>(left, n_left, lbits, h, counts, status);
  if (n_left > 0) {
    SortBufs sb;
    memset(&sb, 0, sizeof(sb));
    sb.in_keys = left;
    sb.tmp_keys = b.tmp_keys;
    sb.tmp_vals = b.tmp_vals;
    sb.out_keys = b.skey;
    sb.out_vals = b.sidx;
    sb.ctl = b.ctl;
    sb.os_status = b.os_status;
    sb.os_ctr = b.os_ctr;
    sb.os_hist = b.os_hist;
    sb.os_ntiles = b.os_ntiles;
    sb.status = status;
    RouteGeom none;
    none.shift = 64;
    none.num_dest = 1;
    int rc = sort_pairs(sb, n_left, nullptr, none, lbits, false, stream);
    if (rc) return rc;
    k_join_dups<<<grid_for(n_left, 256), 256, 0, stream>>>(b.skey, n_left, status);
  }
  if (n_right > 0) {
    const int grid = grid_for(n_right, 256 * JU, 1024);
    if (n_left <= JOIN_LDS_KEYS)
      k_join_probe<2><<<grid, 256, (size_t)n_left * 16, stream>>>(right_keys, n_right, g.total, g.shift[level], b.skey,
                                                                  b.sidx, n_left, match, h, counts, status);
    else if (n_left <= JOIN_LDS_HITS)
      k_join_probe<1><<<grid, 256, (size_t)n_left * 4, stream>>>(right_keys, n_right, g.total, g.shift[level], b.skey,
                                                                 b.sidx, n_left, match, h, counts, status);
    else
      k_join_probe<0><<<grid, 256, 0, stream>>>(right_keys, n_right, g.total, g.shift[level], b.skey, b.sidx, n_left,
                                                match, h, counts, status);
  }
  if (n_left > 0) k_join_count<<<grid_for(n_left, 256), 256, 0, stream>>>(h, n_left, counts);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

}  // extern "C"
