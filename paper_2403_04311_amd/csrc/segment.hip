// Segmentation of sorted elements into the ancestry nodes of several levels, and
// the completion cascade.
//
// Ancestry levels (Section 4.2 of the paper) nest: when elements are ordered by
// key, every node is a contiguous run, and a boundary of a level-m node is also a
// boundary at every deeper level. One pass counts the boundaries of each level per
// tile, a scan turns them into node ids, and a second pass writes each node's
// first element, first child and parent. Completion (Section 3.1: the extent of a
// stream is known only at its end, so each node declares its child count) is then
// evaluated bottom-up, one level per launch: a node is complete when it has as many
// children as it declares and none of them is incomplete.
#include "segment.h"
#include "sort.h"

namespace {

constexpr int NT = SEG_NT;
constexpr int IT = SEG_IT;
constexpr int TILE = SEG_TILE;

__device__ inline int64_t nelem(const SegJob& j) { return j.n_dev ? *j.n_dev : j.n_host; }

__device__ inline int es_of(const KeyGeom& g, const SegJob& j, int m) { return g.shift[m] - g.shift[j.elem_level]; }

__device__ inline int32_t fan_at(const SegJob& j, int m, int64_t e) {
  if (j.src) {
    const int64_t r = j.src[e];
    return r >= 0 ? j.fan[(int64_t)(m - j.fan_base) * j.fan_ld + r]
                  : j.fan2[(int64_t)(m - j.fan_base) * j.fan2_ld + (-1 - r)];
  }
  return j.fan[(int64_t)(m - j.fan_base) * j.fan_ld + j.idx[e]];
}

// Loads the tile's keys plus the key before the tile into LDS.
__device__ inline void load_tile(const SegJob& j, int64_t tile0, int64_t n, uint64_t* s_key) {
  for (int t = threadIdx.x; t <= TILE; t += NT) {
    int64_t e = tile0 - 1 + t;
    s_key[t] = (e >= 0 && e < n) ? j.keys[e] : 0ull;
  }
  __syncthreads();
}

__global__ __launch_bounds__(NT) void k_seg_count(KeyGeom g, SegJob j, int nblk) {
  __shared__ uint64_t s_key[TILE + 1];
  __shared__ int32_t s_w[NT / ALTO_WAVE];
  const int64_t n = nelem(j);
  const int64_t tile0 = (int64_t)blockIdx.x * TILE;
  const int K = j.elem_level - j.lo;
  if (blockIdx.x == 0 && threadIdx.x == 0) j.blkcnt[(int64_t)K * nblk] = 0;
  if (tile0 >= n) {
    if (threadIdx.x < K) j.blkcnt[(int64_t)threadIdx.x * nblk + blockIdx.x] = 0;
    return;
  }
  load_tile(j, tile0, n, s_key);
  for (int m = j.lo; m < j.elem_level; ++m) {
    const int es = es_of(g, j, m);
    int32_t c = 0;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      int t = threadIdx.x * IT + i;
      int64_t e = tile0 + t;
      if (e < n) c += (e == 0) || (key_prefix(s_key[t + 1], es) != key_prefix(s_key[t], es));
    }
    c = wave_sum(c);
    if (lane_id() == 0) s_w[threadIdx.x / ALTO_WAVE] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
      int32_t t = 0;
      for (int w = 0; w < NT / ALTO_WAVE; ++w) t += s_w[w];
      j.blkcnt[(int64_t)(m - j.lo) * nblk + blockIdx.x] = t;
    }
    __syncthreads();
  }
}

// Node counts per level from the scanned block counts; sentinels.
__global__ void k_seg_totals(SegJob j, int nblk, int64_t total_len) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int K = j.elem_level - j.lo;
  // blkcnt has been scanned in place; the sum sits in the scan partials (part[nb])
  for (int m = j.lo; m < j.elem_level; ++m) {
    int64_t base = j.blkcnt[(int64_t)(m - j.lo) * nblk];
    int64_t next = (m + 1 < j.elem_level) ? (int64_t)j.blkcnt[(int64_t)(m + 1 - j.lo) * nblk] : (int64_t)j.blkcnt[(int64_t)K * nblk];
    j.nnodes[m] = next - base;
  }
}

__global__ __launch_bounds__(NT) void k_seg_write(KeyGeom g, SegJob j, int nblk) {
  __shared__ uint64_t s_key[TILE + 1];
  __shared__ int32_t s_w[NT / ALTO_WAVE];
  const int64_t n = nelem(j);
  const int64_t tile0 = (int64_t)blockIdx.x * TILE;
  if (tile0 >= n) return;
  load_tile(j, tile0, n, s_key);
  const int lo = j.lo, E = j.elem_level;
  int32_t cur[ALTO_MAX_LEVELS + 1];
  // per level: node id of the element before this thread's first element
  for (int m = lo; m < E; ++m) {
    const int es = es_of(g, j, m);
    int32_t c = 0;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      int t = threadIdx.x * IT + i;
      int64_t e = tile0 + t;
      if (e < n) c += (e == 0) || (key_prefix(s_key[t + 1], es) != key_prefix(s_key[t], es));
    }
    int32_t tot;
    int32_t ex = block_excl_scan<int32_t, NT>(c, s_w, &tot);
    const int32_t lvl_base = j.blkcnt[(int64_t)(m - lo) * nblk];
    const int32_t blk_off = j.blkcnt[(int64_t)(m - lo) * nblk + blockIdx.x] - lvl_base;
    cur[m] = blk_off + ex - 1;
  }
  for (int i = 0; i < IT; ++i) {
    int t = threadIdx.x * IT + i;
    int64_t e = tile0 + t;
    if (e >= n) break;
    const uint64_t k = s_key[t + 1], kp = s_key[t];
    uint32_t flags = 0;
    for (int m = lo; m < E; ++m) {
      const int es = es_of(g, j, m);
      bool f = (e == 0) || (key_prefix(k, es) != key_prefix(kp, es));
      if (f) {
        flags |= 1u << m;
        ++cur[m];
      }
    }
    if (j.check_dup && e > 0 && k == kp) raise_status(j.status, ALTO_E_DUPLICATE);
    for (int m = lo; m < E; ++m) {
      if (flags & (1u << m)) {
        const int32_t id = cur[m];
        LevelNodes& L = j.lv[m];
        L.start[id] = (int32_t)e;
        if (m + 1 < E) L.fc[id] = cur[m + 1];
        if (m > lo) L.par[id] = cur[m - 1];
        L.nfan[id] = fan_at(j, m, e);
        L.bad[id] = 0;
        if (m == lo && j.carry_fan) {
          for (int mm = j.carry_lo; mm < lo; ++mm)
            j.carry_fan[(int64_t)(mm - j.carry_lo) * j.carry_ld + id] = fan_at(j, mm, e);
        }
      } else if (j.chain_check) {
        if (fan_at(j, m, e) != fan_at(j, m, e - 1)) raise_status(j.status, ALTO_E_FANOUT);
      }
    }
  }
}

__global__ void k_seg_sentinels(SegJob j) {
  const int64_t n = nelem(j);
  const int m = j.lo + (int)threadIdx.x;
  if (blockIdx.x != 0 || m >= j.elem_level) return;
  const int64_t N = j.nnodes[m];
  j.lv[m].start[N] = (int32_t)n;
  if (m + 1 < j.elem_level) j.lv[m].fc[N] = (int32_t)j.nnodes[m + 1];
}

// Completion of the level-m nodes (children are level m+1 nodes, or elements when
// m = elem_level - 1), and the node side of the fan fingerprint.
__global__ __launch_bounds__(256) void k_seg_nodes(KeyGeom g, SegJob j, int m) {
  const int64_t N = j.nnodes[m];
  const LevelNodes L = j.lv[m];
  const bool leafy = (m + 1 == j.elem_level);
  const int es = es_of(g, j, m);
  uint64_t fp[ALTO_MAX_LEVELS + 1];
  const int clo = (m == j.lo && j.carry_fan) ? j.carry_lo : m;
  for (int mm = clo; mm <= m; ++mm) fp[mm] = 0;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < N; u += (int64_t)gridDim.x * blockDim.x) {
    const int32_t s = L.start[u], e = L.start[u + 1];
    const int32_t cnt = e - s;
    int32_t nchild;
    bool allok = true;
    if (leafy) {
      nchild = cnt;
      if (j.elem_ok)
        for (int32_t x = s; x < e; ++x) allok = allok && j.elem_ok[j.idx[x]];
    } else {
      nchild = L.fc[u + 1] - L.fc[u];
    }
    const bool ok = (nchild == L.nfan[u]) && !L.bad[u] && allok;
    L.ok[u] = ok ? 1 : 0;
    if (!ok && m > j.lo) j.lv[m - 1].bad[L.par[u]] = 1;
    if (j.fp_nodes) {
      const uint64_t k = j.keys[s];
      fp[m] += (uint64_t)cnt * fan_term(m, key_prefix(k, es), (uint32_t)L.nfan[u]);
      for (int mm = clo; mm < m; ++mm)
        fp[mm] += (uint64_t)cnt * fan_term(mm, key_prefix(k, es_of(g, j, mm)),
                                           (uint32_t)j.carry_fan[(int64_t)(mm - j.carry_lo) * j.carry_ld + u]);
    }
  }
  if (j.fp_nodes) {
    for (int mm = clo; mm <= m; ++mm) {
      uint64_t v = wave_sum(fp[mm]);
      if (lane_id() == 0 && v) atomicAdd((unsigned long long*)&j.fp_nodes[mm], (unsigned long long)v);
    }
  }
}

}  // namespace

int seg_blocks(int64_t n_max) { return (int)(n_max < 1 ? 1 : cdiv(n_max, SEG_TILE)); }

int seg_run(const KeyGeom& g, SegJob& job, hipStream_t st) {
  const int nblk = seg_blocks(job.n_max);
  const int K = job.elem_level - job.lo;
  if (K <= 0) return ALTO_OK;
  k_seg_count<<<nblk, NT, 0, st>>>(g, job, nblk);
  // one scan over all levels' block counts; level m's ids are relative to its first entry
  const int64_t len = (int64_t)K * nblk;
  int rc = scan_exclusive<int32_t>(job.blkcnt, job.blkcnt, len + 1, nullptr, job.scan_part, nullptr, st);
  if (rc) return rc;
  k_seg_totals<<<1, 1, 0, st>>>(job, nblk, len);
  k_seg_write<<<nblk, NT, 0, st>>>(g, job, nblk);
  k_seg_sentinels<<<1, 64, 0, st>>>(job);
  for (int m = job.elem_level - 1; m >= job.lo; --m) k_seg_nodes<<<NODE_GRID, 256, 0, st>>>(g, job, m);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}
