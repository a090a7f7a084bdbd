// Segmentation of sorted elements into the ancestry nodes of several levels, and
// the completion cascade.
//
// Ancestry levels (Section 4.2 of the paper) nest: when elements are ordered by
// key, every node is a contiguous run, and a boundary of a level-m node is also a
// boundary at every deeper level. One pass counts the boundaries of each level per
// tile; a look-back over earlier tiles turns them into node ids in the same pass,
// which writes each node's first element, first child and parent. Completion
// (Section 3.1: the extent of a stream is known only at its end, so each node
// declares its child count) is then
// evaluated bottom-up, one level per launch: a node is complete when it has as many
// children as it declares and none of them is incomplete.
#include "segment.h"
#include "sort.h"

namespace {

constexpr int NT = SEG_NT;
constexpr int IT = SEG_IT;
constexpr int TILE = SEG_TILE;
constexpr int SEG_SPEC_BLOCKS = 64;   // blocks that load their tile before the count arrives

__device__ inline int64_t nelem(const SegJob& j) { return j.n_dev ? *j.n_dev : j.n_host; }

__device__ inline bool skipped(const SegJob& j) { return j.skip_ctl && j.skip_ctl->dp; }

__device__ inline int es_of(const KeyGeom& g, const SegJob& j, int m) { return g.shift[m] - g.shift[j.elem_level]; }

__device__ inline int32_t fan_at(const SegJob& j, int m, int64_t e) {
  if (j.src) {
    const int64_t r = j.src[e];
    return r >= 0 ? j.fan[(int64_t)(m - j.fan_base) * j.fan_ld + r]
                  : j.fan2[(int64_t)(m - j.fan_base) * j.fan2_ld + (-1 - r)];
  }
  return j.fan[(int64_t)(m - j.fan_base) * j.fan_ld + j.idx[e]];
}

// Clears the look-back words and the ticket; with no elements, writes the empty
// node counts and sentinels.
__global__ void k_seg_prep(SegJob j) {
  if (skipped(j)) return;
  // with no element (a count known on the device only) every destination is empty
  seg_prep_device(j, nelem(j), (int64_t)blockIdx.x * blockDim.x + threadIdx.x, (int64_t)gridDim.x * blockDim.x);
}

// One pass over the sorted elements: per tile, the boundary flags of every level
// (a boundary of a level is also one of every deeper level), node counts by block
// scan, node ids by look-back over earlier tiles, then the node records (first
// element, first child, parent, declared fan). Also: duplicate keys (fragments),
// the exact fan chain check (records), destination offsets at route-prefix changes.
// Persistent; tiles by ticket. Up to four levels share one 64-bit scan (16-bit
// counts; a tile has at most SEG_TILE < 2^16 elements).
template <int KM>
__global__ __launch_bounds__(NT) void k_seg_pass(KeyGeom g, SegJob j) {
  if (skipped(j)) return;
  constexpr int NP = (KM + 3) / 4;
  const int64_t n = nelem(j);
  const int64_t ntiles = cdiv(n, TILE);
  const int lo = j.lo, E = j.elem_level, K = E - lo;
  __shared__ uint64_t s_w[NT / ALTO_WAVE];
  __shared__ uint32_t s_excl[KM], s_tot[KM];
  __shared__ uint32_t s_tile;
  int es[KM];
#pragma unroll
  for (int q = 0; q < KM; ++q) es[q] = q < K ? es_of(g, j, lo + q) : 64;
  const int lane = lane_id();
  const bool vec_ok = (reinterpret_cast<uintptr_t>(j.keys) & 15) == 0;
  // with j.prefetch, the keys of the tile this block most likely takes first (its
  // own index) are loaded before the element count and the ticket have arrived
  // (within the key buffer's n_max elements; those past the count are masked)
  const int64_t gt = blockIdx.x;
  const bool spec = j.prefetch && blockIdx.x < SEG_SPEC_BLOCKS;   // the grid is sized for the largest count
  uint64_t kg[IT], pg = 0;
  if (spec) {
    const int64_t eg = gt * TILE + (int64_t)threadIdx.x * IT;
    if (vec_ok && eg + IT <= j.n_max) {
      const ulonglong2* p = reinterpret_cast<const ulonglong2*>(j.keys + eg);
#pragma unroll
      for (int i = 0; i < IT / 2; ++i) {
        const ulonglong2 v = p[i];
        kg[2 * i] = v.x;
        kg[2 * i + 1] = v.y;
      }
    } else {
#pragma unroll
      for (int i = 0; i < IT; ++i) kg[i] = eg + i < j.n_max ? j.keys[eg + i] : 0ull;
    }
    if (lane == 0 && eg > 0 && eg - 1 < j.n_max) pg = j.keys[eg - 1];
  }
  // blocks past the tile count would only contend for tickets (the grid is sized
  // for the largest count, the count may be known on the device only)
  if ((int64_t)blockIdx.x >= ntiles) return;
  bool first = true;
  while (true) {
    // a single tile is block 0's without a ticket (it waits for no other tile)
    if (ntiles > 1 && threadIdx.x == 0) s_tile = atomicAdd(j.lb_ctr, 1u);
    __syncthreads();
    const int64_t tile = ntiles > 1 ? (int64_t)__builtin_amdgcn_readfirstlane(s_tile) : (first ? 0 : 1);
    first = false;
    if (tile >= ntiles) break;   // uniform across the block
    const int64_t e0 = tile * TILE + (int64_t)threadIdx.x * IT;
    uint64_t k[IT];
    const bool pre = spec && tile == gt;   // uniform
    if (pre) {
#pragma unroll
      for (int i = 0; i < IT; ++i) k[i] = e0 + i < n ? kg[i] : 0ull;
    } else if (vec_ok && e0 + IT <= n) {
      const ulonglong2* p = reinterpret_cast<const ulonglong2*>(j.keys + e0);
#pragma unroll
      for (int i = 0; i < IT / 2; ++i) {
        const ulonglong2 v = p[i];
        k[2 * i] = v.x;
        k[2 * i + 1] = v.y;
      }
    } else {
#pragma unroll
      for (int i = 0; i < IT; ++i) k[i] = e0 + i < n ? j.keys[e0 + i] : 0ull;
    }
    uint64_t prev = __shfl_up(k[IT - 1], 1);
    if (lane == 0) prev = (e0 > 0 && e0 - 1 < n) ? (pre ? pg : j.keys[e0 - 1]) : 0ull;
    // boundary bits of this thread's elements per level (bit i = element e0 + i),
    // route-prefix changes, duplicate keys
    uint32_t fl[KM];
#pragma unroll
    for (int q = 0; q < KM; ++q) fl[q] = 0;
    uint32_t rbits = 0;
    bool dup = false;
#pragma unroll
    for (int i = 0; i < IT; ++i) {
      const int64_t e = e0 + i;
      if (e >= n) continue;
      const uint64_t kp = i == 0 ? prev : k[i - 1];
#pragma unroll
      for (int q = 0; q < KM; ++q)
        if (q < K && (e == 0 || key_prefix(k[i], es[q]) != key_prefix(kp, es[q]))) fl[q] |= 1u << i;
      if (e == 0 || (j.rg.shift < 64 && (k[i] >> j.rg.shift) != (kp >> j.rg.shift)) || e == n - 1) rbits |= 1u << i;
      dup |= e > 0 && k[i] == kp;
    }
    if (j.check_dup && dup) raise_status(j.status, ALTO_E_DUPLICATE);
    // node counts: four levels per 64-bit word, 16-bit fields
    uint64_t pw[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) pw[p] = 0;
#pragma unroll
    for (int q = 0; q < KM; ++q) pw[q / 4] += (uint64_t)__popc(fl[q]) << (16 * (q % 4));
    uint64_t ex[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      uint64_t tot;
      ex[p] = block_excl_scan<uint64_t, NT>(pw[p], s_w, &tot);
      if (threadIdx.x < KM && threadIdx.x / 4 == p) s_tot[threadIdx.x] = (uint32_t)((tot >> (16 * (threadIdx.x % 4))) & 0xFFFFu);
    }
    __syncthreads();
    if (threadIdx.x < K) {
      const int q = threadIdx.x;
      lb_publish(j.lb_status + q, tile, SEG_LB_STRIDE, s_tot[q]);
      const uint32_t excl = lb_resolve(j.lb_status + q, tile, SEG_LB_STRIDE, s_tot[q], j.status);
      s_excl[q] = excl;
      if (tile == ntiles - 1) {
        s_tot[q] = excl + s_tot[q];   // node count of the level
        j.nnodes[lo + q] = (int64_t)s_tot[q];
      }
    }
    __syncthreads();
    // ids: base[q] = level-q boundaries before this thread's first element
    int32_t base[KM];
#pragma unroll
    for (int q = 0; q < KM; ++q)
      base[q] = q < K ? (int32_t)(s_excl[q] + (uint32_t)((ex[q / 4] >> (16 * (q % 4))) & 0xFFFFu)) : 0;
    if (j.gw && e0 < n) j.gw[e0 / IT] = make_uint2((uint32_t)base[0], fl[0]);
    // destination offsets, where the route prefix changes (keys reloaded: rare)
    if (j.dest_offsets) {
      int64_t* offs = j.dest_offsets;
      for (uint32_t r = rbits; r; r &= r - 1) {
        const int i = __builtin_ctz(r);
        const int64_t e = e0 + i;
        const uint64_t kk = j.keys[e];
        const uint32_t d = dest_of_key(j.rg, kk);
        const bool change = e == 0 || (j.rg.shift < 64 && (kk >> j.rg.shift) != (j.keys[e - 1] >> j.rg.shift));
        if (e == 0) {
          for (uint32_t x = 0; x <= d; ++x) offs[x] = 0;
        } else if (change) {
          const uint32_t dp = dest_of_key(j.rg, j.keys[e - 1]);
          for (uint32_t x = dp + 1; x <= d; ++x) offs[x] = e;
        }
        if (e == n - 1)
          for (uint32_t x = d + 1; x <= j.rg.num_dest; ++x) offs[x] = n;
      }
    }
    // node records at the boundaries
#pragma unroll
    for (int q = 0; q < KM; ++q) {
      if (q >= K) continue;
      const int m = lo + q;
      const LevelNodes& L = j.lv[m];
      for (uint32_t r = fl[q]; r;) {
        // up to four boundaries at a time, their declared fans loaded together
        constexpr int NBF = 4;
        int ib[NBF];   // element offsets of the next boundaries (-1: none)
#pragma unroll
        for (int bq = 0; bq < NBF; ++bq) {
          ib[bq] = r ? __builtin_ctz(r) : -1;
          r &= r - 1;
        }
        int32_t fb[NBF];
#pragma unroll
        for (int bq = 0; bq < NBF; ++bq) fb[bq] = ib[bq] >= 0 ? fan_at(j, m, e0 + ib[bq]) : 0;
#pragma unroll
        for (int bq = 0; bq < NBF; ++bq) {
          if (ib[bq] < 0) break;
          const int i = ib[bq];
          const int64_t e = e0 + i;
          const uint32_t below = (1u << i) - 1u;
          const int32_t id = base[q] + __popc(fl[q] & below);
          L.start[id] = (int32_t)e;
          // a boundary of this level is one of the next: the first child starts here
          if (q + 1 < K) L.fc[id] = base[q + 1 < KM ? q + 1 : q] + __popc(fl[q + 1 < KM ? q + 1 : q] & below);
          if (q > 0) L.par[id] = base[q > 0 ? q - 1 : 0] + __popc(fl[q > 0 ? q - 1 : 0] & (below | (1u << i))) - 1;
          L.nfan[id] = fb[bq];
          L.bad[id] = 0;
          if (L.nkey) L.nkey[id] = k[i];
          if (q == 0 && j.carry_fan) {
            for (int mm = j.carry_lo; mm < lo; ++mm)
              j.carry_fan[(int64_t)(mm - j.carry_lo) * j.carry_ld + id] = fan_at(j, mm, e);
          }
        }
      }
      if (j.chain_check) {
        // records: carriers of one node must declare the same fan
        for (int i = 0; i < IT; ++i) {
          const int64_t e = e0 + i;
          if (e >= n) break;
          if (!((fl[q] >> i) & 1u) && fan_at(j, m, e) != fan_at(j, m, e - 1)) raise_status(j.status, ALTO_E_FANOUT);
        }
      }
    }
    if (tile == ntiles - 1 && threadIdx.x == 0) {
      // sentinels: start[N] = element count, fc[N] = node count of the next level
      for (int q = 0; q < K; ++q) {
        const LevelNodes& L = j.lv[lo + q];
        L.start[s_tot[q]] = (int32_t)n;
        if (q + 1 < K) L.fc[s_tot[q]] = (int32_t)s_tot[q + 1];
      }
    }
    __syncthreads();   // shared words and the ticket are reused by the next tile
  }
}

// Completion of the level-m nodes (children are level m+1 nodes, or elements when
// m = elem_level - 1), and the node side of the fan fingerprint.
__global__ __launch_bounds__(256) void k_seg_nodes(KeyGeom g, SegJob j, int m) {
  if (skipped(j)) return;
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
      fpm += (uint64_t)cnt * fan_term(g.fkey, m, key_prefix(k, es), (uint32_t)L.nfan[u]);
#pragma unroll
      for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
        if (q < nc)
          fpc[q] += (uint64_t)cnt * fan_term(g.fkey, clo + q, key_prefix(k, esc[q]),
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
  if (skipped(j)) return;
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

int seg_tiles(int64_t n_max) { return (int)(n_max < 1 ? 1 : cdiv(n_max, SEG_TILE)); }

int seg_run(const KeyGeom& g, SegJob& job, hipStream_t st) {
  const int K = job.elem_level - job.lo;
  if (K <= 0) return ALTO_OK;
  const int tiles = seg_tiles(job.n_max);
  if (!job.lb_status || !job.lb_ctr || job.lb_tiles < tiles) return ALTO_E_ARG;
  const int64_t pb = cdiv((int64_t)tiles * SEG_LB_STRIDE, 256);
  if (!job.no_prep) k_seg_prep<<<(int)(pb < 1024 ? pb : 1024), 256, 0, st>>>(job);
  const int grid = tiles < 1024 ? tiles : 1024;
  if (K <= 2) k_seg_pass<2><<<grid, NT, 0, st>>>(g, job);
  else if (K <= 4) k_seg_pass<4><<<grid, NT, 0, st>>>(g, job);
  else k_seg_pass<ALTO_MAX_LEVELS><<<grid, NT, 0, st>>>(g, job);
  if (job.elem_ok) k_elem_bad<<<NODE_GRID, 256, 0, st>>>(job);
  for (int m = job.elem_level - 1; m >= job.lo + (job.fold_lo ? 1 : 0); --m)
    k_seg_nodes<<<NODE_GRID, 256, 0, st>>>(g, job, m);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}
