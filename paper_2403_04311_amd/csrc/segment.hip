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
  if (j.dest_offsets) {
    // destination offsets from the sorted keys: each change of destination fills
    // the starts of the destinations it passes
    const uint32_t D = j.rg.num_dest;
    int64_t* offs = j.dest_offsets;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int t = threadIdx.x * IT + i;
      const int64_t e = tile0 + t;
      if (e >= n) break;
      const uint32_t d = dest_of_key(j.rg, s_key[t + 1]);
      if (e == 0) {
        for (uint32_t x = 0; x <= d; ++x) offs[x] = 0;
      } else {
        const uint32_t dp = dest_of_key(j.rg, s_key[t]);
        if (d != dp)
          for (uint32_t x = dp + 1; x <= d; ++x) offs[x] = e;
      }
      if (e == n - 1)
        for (uint32_t x = d + 1; x <= D; ++x) offs[x] = n;
    }
  }
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

template <int KM>
__global__ __launch_bounds__(NT) void k_seg_write(KeyGeom g, SegJob j, int nblk) {
  __shared__ uint64_t s_key[TILE + 1];
  __shared__ int32_t s_w[NT / ALTO_WAVE];
  const int64_t n = nelem(j);
  const int64_t tile0 = (int64_t)blockIdx.x * TILE;
  if (tile0 >= n) return;
  load_tile(j, tile0, n, s_key);
  const int lo = j.lo, E = j.elem_level, K = E - lo;
  // slot q holds level lo + q; every loop below is fully unrolled so that the
  // per-level arrays stay in registers
  int32_t cur[KM];
  int es[KM];
#pragma unroll
  for (int q = 0; q < KM; ++q) {
    cur[q] = 0;
    es[q] = q < K ? es_of(g, j, lo + q) : 64;
  }
  // per level: node id of the element before this thread's first element
#pragma unroll
  for (int q = 0; q < KM; ++q) {
    if (q < K) {
      int32_t c = 0;
#pragma unroll
      for (int i = 0; i < IT; ++i) {
        const int t = threadIdx.x * IT + i;
        const int64_t e = tile0 + t;
        if (e < n) c += (e == 0) || (key_prefix(s_key[t + 1], es[q]) != key_prefix(s_key[t], es[q]));
      }
      int32_t tot;
      const int32_t ex = block_excl_scan<int32_t, NT>(c, s_w, &tot);
      const int32_t lvl_base = j.blkcnt[(int64_t)q * nblk];
      const int32_t blk_off = j.blkcnt[(int64_t)q * nblk + blockIdx.x] - lvl_base;
      cur[q] = blk_off + ex - 1;
    }
  }
  for (int i = 0; i < IT; ++i) {
    const int t = threadIdx.x * IT + i;
    const int64_t e = tile0 + t;
    if (e >= n) break;
    const uint64_t k = s_key[t + 1], kp = s_key[t];
    uint32_t flags = 0;
#pragma unroll
    for (int q = 0; q < KM; ++q) {
      if (q < K && ((e == 0) || (key_prefix(k, es[q]) != key_prefix(kp, es[q])))) {
        flags |= 1u << q;
        ++cur[q];
      }
    }
    if (j.check_dup && e > 0 && k == kp) raise_status(j.status, ALTO_E_DUPLICATE);
#pragma unroll
    for (int q = 0; q < KM; ++q) {
      if (q >= K) continue;
      const int m = lo + q;
      if (flags & (1u << q)) {
        const int32_t id = cur[q];
        const LevelNodes& L = j.lv[m];
        L.start[id] = (int32_t)e;
        if (q + 1 < K) L.fc[id] = cur[q + 1 < KM ? q + 1 : q];
        if (q > 0) L.par[id] = cur[q > 0 ? q - 1 : 0];
        L.nfan[id] = fan_at(j, m, e);
        L.bad[id] = 0;
        if (q == 0 && j.carry_fan) {
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
  const int clo = (m == j.lo && j.carry_fan) ? j.carry_lo : m;
  const int nc = m - clo;   // carried levels handled here (clo .. m-1)
  uint64_t fpm = 0;
  uint64_t fpc[ALTO_MAX_LEVELS];
  int esc[ALTO_MAX_LEVELS];
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
    fpc[q] = 0;
    esc[q] = q < nc ? es_of(g, j, clo + q) : 64;
  }
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < N; u += (int64_t)gridDim.x * blockDim.x) {
    const int32_t s = L.start[u], e = L.start[u + 1];
    const int32_t cnt = e - s;
    int32_t nchild;
    if (leafy) {
      nchild = cnt;   // incomplete element records were pushed into bad by k_elem_bad
    } else {
      nchild = L.fc[u + 1] - L.fc[u];
    }
    const bool ok = (nchild == L.nfan[u]) && !L.bad[u];
    L.ok[u] = ok ? 1 : 0;
    if (!ok && m > j.lo) j.lv[m - 1].bad[L.par[u]] = 1;
    if (j.fp_nodes) {
      const uint64_t k = j.keys[s];
      fpm += (uint64_t)cnt * fan_term(m, key_prefix(k, es), (uint32_t)L.nfan[u]);
#pragma unroll
      for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
        if (q < nc)
          fpc[q] += (uint64_t)cnt * fan_term(clo + q, key_prefix(k, esc[q]),
                                             (uint32_t)j.carry_fan[(int64_t)q * j.carry_ld + u]);
    }
  }
  if (j.fp_nodes) {
    // block sums first: one atomic per block and level
    __shared__ uint64_t s_fp[256 / ALTO_WAVE][ALTO_MAX_LEVELS + 1];
    const int w = threadIdx.x / ALTO_WAVE;
    const uint64_t v = wave_sum(fpm);
    if (lane_id() == 0) s_fp[w][ALTO_MAX_LEVELS] = v;
#pragma unroll
    for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
      if (q < nc) {
        const uint64_t vc = wave_sum(fpc[q]);
        if (lane_id() == 0) s_fp[w][q] = vc;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t t = 0;
      for (int ww = 0; ww < 256 / ALTO_WAVE; ++ww) t += s_fp[ww][ALTO_MAX_LEVELS];
      if (t) atomicAdd((unsigned long long*)&j.fp_nodes[m], (unsigned long long)t);
      for (int q = 0; q < nc; ++q) {
        uint64_t tc = 0;
        for (int ww = 0; ww < 256 / ALTO_WAVE; ++ww) tc += s_fp[ww][q];
        if (tc) atomicAdd((unsigned long long*)&j.fp_nodes[clo + q], (unsigned long long)tc);
      }
    }
  }
}

// Records that are themselves incomplete make their parent incomplete: one thread
// per record finds its parent node by binary search over the node starts.
__global__ __launch_bounds__(256) void k_elem_bad(SegJob j) {
  const int64_t n = nelem(j);
  const int m = j.elem_level - 1;
  const int64_t N = j.nnodes[m];
  const LevelNodes L = j.lv[m];
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n; e += (int64_t)gridDim.x * blockDim.x) {
    if (j.elem_ok[j.idx[e]]) continue;
    int64_t lo = 0, hi = N - 1;   // last node with start <= e
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (L.start[mid] <= e) lo = mid; else hi = mid - 1;
    }
    if (N > 0) L.bad[lo] = 1;
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
  if (K <= 2) k_seg_write<2><<<nblk, NT, 0, st>>>(g, job, nblk);
  else if (K <= 4) k_seg_write<4><<<nblk, NT, 0, st>>>(g, job, nblk);
  else k_seg_write<ALTO_MAX_LEVELS><<<nblk, NT, 0, st>>>(g, job, nblk);
  k_seg_sentinels<<<1, 64, 0, st>>>(job);
  if (job.elem_ok) k_elem_bad<<<NODE_GRID, 256, 0, st>>>(job);
  for (int m = job.elem_level - 1; m >= job.lo; --m) k_seg_nodes<<<NODE_GRID, 256, 0, st>>>(g, job, m);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}
