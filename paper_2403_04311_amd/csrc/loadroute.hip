// Load-aware routing (Section 4.3: because elements are produced slowly, the
// destination of a new flow of tags can be chosen by load instead of by a hash;
// Section 5: the controller picks replicas by queue length). A flow is a distinct
// route-level prefix. It keeps the destination it is first given (all fragments
// with the same tags reach the same instance), held in a device flow table that
// lives across calls. Per batch, the fragments of known flows join their queues
// first; the new flows then go, in ascending prefix order, each to the shortest
// queue (lowest index among ties), which grows by the flow's fragments.
//
// Steps: the keys are sorted by the routing sort of alto_route with one destination
// (the flows ranked in prefix order, packed words); flow runs are found with a
// head-flag scan; run
// heads look their prefix up in the table; known runs add their lengths to a
// per-destination delta; the new runs are compacted in prefix order. One wave then
// assigns the new flows in order: the queue lengths sit in LDS, each lane keeps the
// minimum over the queues it owns (d = lane mod 64), and a wave reduction picks the
// shortest queue per flow, so only the owner lane rescans after an update. The new
// flows enter the table. A flow's fragments share its destination and form one run
// of the key order, so the (destination, key) order of perm only needs the runs
// sorted by (destination, prefix) (a small sort) and a segmented copy of each run
// to its offset; the input-order destinations are looked up in a table of the
// batch's flows built in LDS.
#include "aggregate.h"
#include "sort.h"

#include <limits.h>
#include <string.h>

#include <new>

#define LR_MAX_DEST 4096
#define LR_CHUNK 2048   // new flows staged in LDS per round of the assignment wave

struct alto_router {
  KeyGeom g;
  int32_t route_level, num_dest;
  int64_t max_flows, hcap;
  uint64_t* tkey;    // [hcap] flow prefixes, ~0 = empty
  int32_t* tdest;    // [hcap] their destinations
  int64_t* nflows;   // flows stored
};

namespace {

struct LrBufs {
  AggBufs ab;           // the key sort: ab.sk sorted keys, ab.perm input index of each;
                        // its scratch serves the destination sort afterwards
  uint32_t* hs;         // [n + 1] run heads before each sorted position
  uint32_t* part;       // [SCAN_MAX_BLOCKS + 1]
  uint32_t* run_start;  // [n] first sorted position of each run
  uint64_t* run_pfx;    // [n] flow prefix of each run
  int32_t* rank;        // [n] flow rank of every input element (packed routing sort)
  int32_t* run_dest;    // [n] destination of each run (-1: new, until assigned)
  uint32_t* nf;         // [n + 1] new-flow flag of each run, then their exclusive scan
  uint32_t* new_run;    // [n] runs of the new flows, in prefix order
  int64_t* nrun1;       // runs + 1 (the length of the new-flow scan)
  int64_t* nrun;        // runs (device count of the run sort)
  int64_t* delta;       // [D] fragments of known flows per destination
  uint64_t* rkey;       // [n] (destination << 32 | run) of each run
  uint64_t* rsk;        // [n] the same, sorted
  uint32_t* rval;       // [n] run of each sorted entry
  int64_t* roff;        // [n + 1] output offset of each run (scan in sorted-run order)
  int64_t* rpart;       // [SCAN_MAX_BLOCKS + 1]
  int64_t* rbase;       // [n] output offset by run index
};

void plan_lr(const KeyGeom& g, int Lr, int64_t n_max, int D, WsCarver& c, LrBufs& b) {
  const int64_t n = n_max < 1 ? 1 : n_max;
  plan_buffers(g, n, make_route(g, Lr, 1), nullptr, Lr, c, b.ab);
  b.hs = c.take<uint32_t>(n + 1);
  b.part = c.take<uint32_t>(SCAN_MAX_BLOCKS + 1);
  b.run_start = c.take<uint32_t>(n);
  b.run_pfx = c.take<uint64_t>(n);
  b.rank = c.take<int32_t>(n);
  b.run_dest = c.take<int32_t>(n);
  b.nf = c.take<uint32_t>(n + 1);
  b.new_run = c.take<uint32_t>(n);
  b.nrun1 = c.take<int64_t>(1);
  b.nrun = c.take<int64_t>(1);
  b.delta = c.take<int64_t>(D);
  b.rkey = c.take<uint64_t>(n);
  b.rsk = c.take<uint64_t>(n);
  b.rval = c.take<uint32_t>(n);
  b.roff = c.take<int64_t>(n + 1);
  b.rpart = c.take<int64_t>(SCAN_MAX_BLOCKS + 1);
  b.rbase = c.take<int64_t>(n);
}


__device__ inline int read_status(const int32_t* st) {
  return __hip_atomic_load(st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline uint64_t lr_hash(uint64_t p, int64_t hcap) {
  return mix64(p ^ 0x5851F42D4C957F2Dull) & (uint64_t)(hcap - 1);
}

__global__ void k_lr_clear(uint64_t* tkey, int64_t hcap, int64_t* nflows) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < hcap; i += (int64_t)gridDim.x * blockDim.x)
    tkey[i] = ~0ull;
  if (blockIdx.x == 0 && threadIdx.x == 0) *nflows = 0;
}

__global__ void k_lr_init(int64_t* counts, int64_t* delta, int D, uint32_t* hs_end) {
  for (int d = threadIdx.x; d < D; d += blockDim.x) delta[d] = 0;
  if (threadIdx.x == 0) {
    counts[0] = counts[1] = 0;
    *hs_end = 0;
  }
}

// Run heads (a new route prefix in sorted order); layout and duplicate checks.
__global__ __launch_bounds__(256) void k_lr_heads(const uint64_t* __restrict__ skey, int64_t n, int total, int sh,
                                                  uint32_t* __restrict__ hs, int32_t* status) {
  bool bad = false, dup = false;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t k = skey[j];
    bad |= (k >> total) != 0;
    bool head = true;
    if (j > 0) {
      const uint64_t kp = skey[j - 1];
      dup |= kp == k;
      head = key_prefix(k, sh) != key_prefix(kp, sh);
    }
    hs[j] = head ? 1u : 0u;
  }
  if (bad) raise_status(status, ALTO_E_LAYOUT);
  if (dup) raise_status(status, ALTO_E_DUPLICATE);
}

// Each run head looks its flow up in the table; the new-flow flags of the R runs
// (and a zero at R) are written for a scan of R + 1 entries.
__global__ __launch_bounds__(256) void k_lr_runs(const uint64_t* __restrict__ skey, int64_t n, int sh,
                                                 const uint32_t* __restrict__ hs, const uint64_t* __restrict__ tkey,
                                                 const int32_t* __restrict__ tdest, int64_t hcap,
                                                 uint32_t* __restrict__ run_start, uint64_t* __restrict__ run_pfx,
                                                 int32_t* __restrict__ run_dest, uint32_t* __restrict__ nf,
                                                 int64_t* nrun1, int64_t* nrun, int64_t* counts) {
  __shared__ uint64_t s_n[256 / ALTO_WAVE];
  uint64_t known = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    const uint32_t R = hs[n];
    nf[R] = 0u;
    *nrun1 = (int64_t)R + 1;
    *nrun = (int64_t)R;
  }
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t r = hs[j];
    if (hs[j + 1] == r) continue;   // not a head
    run_start[r] = (uint32_t)j;
    const uint64_t p = key_prefix(skey[j], sh);
    run_pfx[r] = p;
    uint64_t h = lr_hash(p, hcap);
    int32_t d = -1;
    for (int64_t probe = 0; probe < hcap; ++probe) {
      const uint64_t v = tkey[h];
      if (v == p) {
        d = tdest[h];
        break;
      }
      if (v == ~0ull) break;
      h = (h + 1) & (uint64_t)(hcap - 1);
    }
    run_dest[r] = d;
    nf[r] = d < 0 ? 1u : 0u;
    known += d >= 0 ? 1 : 0;
  }
  const uint64_t v = wave_sum(known);
  if (lane_id() == 0) s_n[threadIdx.x / ALTO_WAVE] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int w = 0; w < 256 / ALTO_WAVE; ++w) t += s_n[w];
    if (t) atomicAdd((unsigned long long*)&counts[1], (unsigned long long)t);
  }
}

__device__ inline int64_t run_len(const uint32_t* run_start, uint32_t r, uint32_t R, int64_t n) {
  return (r + 1 < R ? (int64_t)run_start[r + 1] : n) - (int64_t)run_start[r];
}

// Known runs add their fragments to their destination (through an LDS histogram);
// new runs are listed in prefix order.
__global__ __launch_bounds__(256) void k_lr_known(int64_t n, const uint32_t* __restrict__ hs,
                                                  const uint32_t* __restrict__ run_start,
                                                  const int32_t* __restrict__ run_dest, const uint32_t* __restrict__ nf,
                                                  uint32_t* __restrict__ new_run, int64_t* delta, int D) {
  __shared__ unsigned long long s_d[LR_MAX_DEST];
  for (int d = threadIdx.x; d < D; d += blockDim.x) s_d[d] = 0ull;
  __syncthreads();
  const uint32_t R = hs[n];
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < R; r += (int64_t)gridDim.x * blockDim.x) {
    const int32_t d = run_dest[r];
    if (d >= 0) {
      if (d < D) atomicAdd(&s_d[d], (unsigned long long)run_len(run_start, (uint32_t)r, R, n));
    } else {
      new_run[nf[r]] = (uint32_t)r;
    }
  }
  __syncthreads();
  for (int d = threadIdx.x; d < D; d += blockDim.x)
    if (s_d[d]) atomicAdd((unsigned long long*)&delta[d], s_d[d]);
}

__device__ inline void lr_better(int64_t& v, int32_t& i, int64_t ov, int32_t oi) {
  if (ov < v || (ov == v && oi < i)) {
    v = ov;
    i = oi;
  }
}

// One wave: the new flows in prefix order, each to the shortest queue. Nothing
// changes if this call has raised an error or the flows do not fit the table.
__global__ __launch_bounds__(ALTO_WAVE) void k_lr_assign(int64_t n, const uint32_t* __restrict__ hs,
                                                         const uint32_t* __restrict__ run_start,
                                                         int32_t* __restrict__ run_dest,
                                                         const uint32_t* __restrict__ nf,
                                                         const uint32_t* __restrict__ new_run,
                                                         const int64_t* __restrict__ delta, int64_t* load, int D,
                                                         int64_t* nflows, int64_t max_flows, int64_t* counts,
                                                         int32_t* status) {
  __shared__ int64_t s_load[LR_MAX_DEST];
  __shared__ int32_t s_len[LR_CHUNK];
  __shared__ int32_t s_dst[LR_CHUNK];
  const int lane = threadIdx.x;
  if (read_status(status) != ALTO_OK) return;
  const uint32_t R = hs[n];
  const int64_t F = nf[R];
  const int64_t stored = *nflows;
  if (stored + F > max_flows) {
    if (lane == 0) raise_status(status, ALTO_E_CAPACITY);
    return;
  }
  for (int d = lane; d < D; d += ALTO_WAVE) s_load[d] = load[d] + delta[d];
  // the lane's shortest queue among d = lane, lane + 64, ...
  int64_t lv = INT64_MAX;
  int32_t li = INT32_MAX;
  for (int d = lane; d < D; d += ALTO_WAVE) lr_better(lv, li, s_load[d], d);
  for (int64_t base = 0; base < F; base += LR_CHUNK) {
    const int cnt = (int)(F - base < LR_CHUNK ? F - base : LR_CHUNK);
    for (int k = lane; k < cnt; k += ALTO_WAVE) s_len[k] = (int32_t)run_len(run_start, new_run[base + k], R, n);
    __syncthreads();
    for (int k = 0; k < cnt; ++k) {
      int64_t gv = lv;
      int32_t gi = li;
#pragma unroll
      for (int o = ALTO_WAVE / 2; o > 0; o >>= 1) {
        const int64_t ov = __shfl_xor(gv, o);
        const int32_t oi = __shfl_xor(gi, o);
        lr_better(gv, gi, ov, oi);
      }
      if (lane == 0) s_dst[k] = gi;
      if (lane == (gi & (ALTO_WAVE - 1))) {
        s_load[gi] += s_len[k];
        lv = INT64_MAX;
        li = INT32_MAX;
        for (int d = lane; d < D; d += ALTO_WAVE) lr_better(lv, li, s_load[d], d);
      }
      __syncthreads();
    }
    for (int k = lane; k < cnt; k += ALTO_WAVE) run_dest[new_run[base + k]] = s_dst[k];
    __syncthreads();
  }
  for (int d = lane; d < D; d += ALTO_WAVE) load[d] = s_load[d];
  if (lane == 0) {
    *nflows = stored + F;
    counts[0] = F;
  }
}

// The new flows enter the table (distinct prefixes: one run each).
__global__ __launch_bounds__(256) void k_lr_insert(int64_t n, const uint32_t* __restrict__ hs,
                                                   const uint32_t* __restrict__ nf,
                                                   const uint32_t* __restrict__ new_run,
                                                   const uint32_t* __restrict__ run_start,
                                                   const int32_t* __restrict__ run_dest,
                                                   const uint64_t* __restrict__ skey, int sh, uint64_t* tkey,
                                                   int32_t* tdest, int64_t hcap, const int32_t* status) {
  if (read_status(status) != ALTO_OK) return;
  const int64_t F = nf[hs[n]];
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < F; k += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t r = new_run[k];
    const uint64_t p = key_prefix(skey[run_start[r]], sh);
    uint64_t h = lr_hash(p, hcap);
    for (int64_t probe = 0; probe < hcap; ++probe) {
      const uint64_t old = atomicCAS((unsigned long long*)&tkey[h], ~0ull, (unsigned long long)p);
      if (old == ~0ull || old == p) {
        tdest[h] = run_dest[r];
        break;
      }
      h = (h + 1) & (uint64_t)(hcap - 1);
    }
  }
}

// Sort key of every run: (destination, run), the run index being prefix order.
__global__ __launch_bounds__(256) void k_lr_runkeys(const int64_t* __restrict__ nrun,
                                                    const int32_t* __restrict__ run_dest, int D,
                                                    uint64_t* __restrict__ rkey) {
  const int64_t R = *nrun;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < R; r += (int64_t)gridDim.x * blockDim.x) {
    int32_t d = run_dest[r];
    d = (d < 0 || d >= D) ? 0 : d;   // only after an error (outputs undefined, accesses in bounds)
    rkey[r] = ((uint64_t)d << 32) | (uint64_t)r;
  }
}

// Fragments of each run in sorted-run order (the input of the offset scan).
__global__ __launch_bounds__(256) void k_lr_runlen(int64_t n, const int64_t* __restrict__ nrun,
                                                   const uint32_t* __restrict__ rval,
                                                   const uint32_t* __restrict__ run_start,
                                                   int64_t* __restrict__ roff) {
  const int64_t R = *nrun;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q <= R; q += (int64_t)gridDim.x * blockDim.x)
    roff[q] = q < R ? run_len(run_start, rval[q], (uint32_t)R, n) : 0;
}

// Output offset by run index, and the destination offsets (from the first run of
// every destination in sorted-run order).
__global__ __launch_bounds__(256) void k_lr_runoff(int64_t n, const int64_t* __restrict__ nrun,
                                                   const uint64_t* __restrict__ rsk,
                                                   const uint32_t* __restrict__ rval,
                                                   const int64_t* __restrict__ roff, int D,
                                                   int64_t* __restrict__ rbase, int64_t* __restrict__ offs) {
  const int64_t R = *nrun;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < R; q += (int64_t)gridDim.x * blockDim.x) {
    rbase[rval[q]] = roff[q];
    if (!offs) continue;
    const uint32_t d = (uint32_t)(rsk[q] >> 32);
    if (q == 0) {
      for (uint32_t x = 0; x <= d; ++x) offs[x] = 0;
    } else {
      const uint32_t dp = (uint32_t)(rsk[q - 1] >> 32);
      for (uint32_t x = dp + 1; x <= d; ++x) offs[x] = roff[q];
    }
    if (q == R - 1)
      for (uint32_t x = d + 1; x <= (uint32_t)D; ++x) offs[x] = n;
  }
}

// perm: every run copied to its offset (reads and writes contiguous within runs).
__global__ __launch_bounds__(256) void k_lr_copy(int64_t n, const uint32_t* __restrict__ hs,
                                                 const uint32_t* __restrict__ run_start,
                                                 const int64_t* __restrict__ rbase,
                                                 const uint32_t* __restrict__ sidx, int32_t* __restrict__ perm) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t r = hs[j + 1] - 1;
    int64_t o = rbase[r] + (j - (int64_t)run_start[r]);
    o = o < 0 ? 0 : (o >= n ? n - 1 : o);   // in bounds whatever an error left behind
    perm[o] = (int32_t)sidx[j];
  }
}

// Destination of every input fragment, in input order (coalesced reads and
// writes), when the key sort did not run packed (then k_lr_dest_rank below has it
// from the flow ranks). With at most LR_LDS_FLOWS runs, every block first builds an
// open-addressing table of the batch's flows in LDS from the runs (prefix, run
// destination); otherwise the lookups go to the flow table (L2). LU lookups per
// thread are in flight together.
constexpr int LU = 8;
constexpr int LR_LDS_FLOWS = 2048;
constexpr int LR_LDS_SLOTS = 4096;

template <typename KT, typename DT>
__device__ inline void lr_lookup(const uint64_t* __restrict__ keys, int64_t n, int sh, KT tk, DT td, int64_t cap,
                                 int32_t* __restrict__ dest) {
  const uint64_t mask = (uint64_t)(cap - 1);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += stride * LU) {
    uint64_t p[LU], h[LU];
    int32_t d[LU];
    bool done[LU];
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      const int64_t i = i0 + u * stride;
      p[u] = i < n ? keys[i] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      p[u] = key_prefix(p[u], sh);
      h[u] = lr_hash(p[u], cap);
      d[u] = 0;   // a flow missing from the table only after an error
      done[u] = i0 + u * stride >= n;
    }
    for (uint64_t probe = 0; probe <= mask; ++probe) {
      bool all = true;
#pragma unroll
      for (int u = 0; u < LU; ++u) {
        if (done[u]) continue;
        const uint64_t v = tk[h[u]];
        if (v == p[u]) {
          d[u] = td[h[u]];
          done[u] = true;
        } else if (v == ~0ull) {
          done[u] = true;
        } else {
          h[u] = (h[u] + 1) & mask;
        }
        all = all && done[u];
      }
      if (all) break;
    }
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      const int64_t i = i0 + u * stride;
      if (i < n) dest[i] = d[u];
    }
  }
}

__global__ __launch_bounds__(256) void k_lr_dest_in(const uint64_t* __restrict__ keys, int64_t n, int sh,
                                                    const uint64_t* __restrict__ run_pfx,
                                                    const int32_t* __restrict__ run_dest,
                                                    const int64_t* __restrict__ nrun,
                                                    const uint64_t* __restrict__ tkey,
                                                    const int32_t* __restrict__ tdest, int64_t hcap,
                                                    const SortCtl* ctl, const int32_t* __restrict__ rank,
                                                    int32_t* __restrict__ dest) {
  __shared__ uint64_t s_k[LR_LDS_SLOTS];
  __shared__ int32_t s_d[LR_LDS_SLOTS];
  const int64_t R = *nrun;
  if (rank && ctl->mode == SORT_PACKED) return;   // k_lr_dest_rank does it
  if (R > LR_LDS_FLOWS) {   // uniform
    lr_lookup(keys, n, sh, tkey, tdest, hcap, dest);
    return;
  }
  for (int i = threadIdx.x; i < LR_LDS_SLOTS; i += blockDim.x) s_k[i] = ~0ull;
  __syncthreads();
  for (int64_t r = threadIdx.x; r < R; r += blockDim.x) {
    const uint64_t p = run_pfx[r];
    uint64_t h = lr_hash(p, LR_LDS_SLOTS);
    for (int probe = 0; probe < LR_LDS_SLOTS; ++probe) {
      const unsigned long long old =
          atomicCAS(reinterpret_cast<unsigned long long*>(&s_k[h]), ~0ull, (unsigned long long)p);
      if (old == ~0ull || old == p) {
        s_d[h] = run_dest[r];
        break;
      }
      h = (h + 1) & (uint64_t)(LR_LDS_SLOTS - 1);
    }
  }
  __syncthreads();
  lr_lookup(keys, n, sh, s_k, s_d, LR_LDS_SLOTS, dest);
}

// The same from the flow ranks of the packed key sort: dest = run_dest[rank], LU
// elements per thread in flight (no LDS, full occupancy).
__global__ __launch_bounds__(256) void k_lr_dest_rank(int64_t n, const int64_t* __restrict__ nrun,
                                                      const int32_t* __restrict__ run_dest, const SortCtl* ctl,
                                                      const int32_t* __restrict__ rank, int32_t* __restrict__ dest) {
  if (ctl->mode != SORT_PACKED) return;   // k_lr_dest_in does it
  const int64_t R = *nrun;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += stride * LU) {
    int64_t q[LU];
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      const int64_t i = i0 + u * stride;
      q[u] = i < n ? rank[i] : 0;
    }
#pragma unroll
    for (int u = 0; u < LU; ++u) {
      const int64_t i = i0 + u * stride;
      const int64_t r = q[u] < 0 ? 0 : (q[u] >= R ? R - 1 : q[u]);   // in bounds whatever an error left behind
      if (i < n) dest[i] = run_dest[r];
    }
  }
}

__global__ void k_lr_zero_offsets(int64_t* offs, int D) {
  for (int d = threadIdx.x; d <= D; d += blockDim.x) offs[d] = 0;
}

bool lr_layout_ok(const alto_layout* l) {
  if (!l || l->depth < 2 || l->depth > ALTO_MAX_LEVELS) return false;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) {
    if (l->bits[i] < 1 || l->bits[i] > 32) return false;
    total += l->bits[i];
  }
  return total <= 63;
}

int64_t lr_hcap(int64_t max_flows) {
  int64_t h = 64;
  while (h < 2 * max_flows) h <<= 1;
  return h;
}

const int64_t LR_N_LIMIT = (int64_t)INT_MAX - 1;
const int64_t LR_FLOWS_LIMIT = (int64_t)1 << 30;

}  // namespace

extern "C" {

size_t alto_router_state_bytes(int64_t max_flows) {
  if (max_flows < 1 || max_flows > LR_FLOWS_LIMIT) return 0;
  WsCarver c{nullptr, (size_t)-1, 0, true};
  const int64_t h = lr_hcap(max_flows);
  c.take<uint64_t>(h);
  c.take<int32_t>(h);
  c.take<int64_t>(1);
  return c.off;
}

int alto_router_create(const alto_layout* layout, int32_t route_level, int32_t num_dest, int64_t max_flows,
                       void* state, size_t state_bytes, hipStream_t stream, alto_router** out) {
  if (!out || !lr_layout_ok(layout) || route_level < 1 || route_level > layout->depth || num_dest < 1 ||
      num_dest > LR_MAX_DEST || max_flows < 1 || max_flows > LR_FLOWS_LIMIT || !state)
    return ALTO_E_ARG;
  const int64_t h = lr_hcap(max_flows);
  WsCarver c{(char*)state, state_bytes, 0, true};
  uint64_t* tkey = c.take<uint64_t>(h);
  int32_t* tdest = c.take<int32_t>(h);
  int64_t* nflows = c.take<int64_t>(1);
  if (!c.ok) return ALTO_E_ARG;
  alto_router* r = new (std::nothrow) alto_router;
  if (!r) return ALTO_E_ARG;
  r->g = make_geom(layout);
  r->route_level = route_level;
  r->num_dest = num_dest;
  r->max_flows = max_flows;
  r->hcap = h;
  r->tkey = tkey;
  r->tdest = tdest;
  r->nflows = nflows;
  k_lr_clear<<<grid_for(h, 256), 256, 0, stream>>>(tkey, h, nflows);
  if (hipGetLastError() != hipSuccess) {
    delete r;
    return ALTO_E_HIP;
  }
  *out = r;
  return ALTO_OK;
}

int alto_router_destroy(alto_router* r) {
  delete r;
  return ALTO_OK;
}

size_t alto_route_load_workspace_bytes(const alto_layout* layout, int32_t route_level, int64_t n_max,
                                       int32_t num_dest) {
  if (!lr_layout_ok(layout) || route_level < 1 || route_level > layout->depth || n_max < 0 || n_max > LR_N_LIMIT ||
      num_dest < 1 || num_dest > LR_MAX_DEST)
    return 0;
  WsCarver c{nullptr, (size_t)-1, 0, true};
  LrBufs b;
  plan_lr(make_geom(layout), route_level, n_max, num_dest, c, b);
  return c.off;
}

int alto_route_load(alto_router* r, const uint64_t* keys, int64_t n, int64_t* load, int32_t* perm,
                    int64_t* dest_offsets, int32_t* dest, int64_t* counts, int32_t* status, void* ws,
                    size_t ws_bytes, hipStream_t stream) {
  if (!r || n < 0 || n > LR_N_LIMIT || !load || !counts || !status || !ws || (n > 0 && !keys)) return ALTO_E_ARG;
  const int D = r->num_dest;
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  LrBufs b;
  plan_lr(r->g, r->route_level, n, D, c, b);
  if (!c.ok) return ALTO_E_ARG;
  k_lr_init<<<1, 256, 0, stream>>>(counts, b.delta, D, b.hs + n);
  if (n == 0) {
    if (dest_offsets) k_lr_zero_offsets<<<1, 256, 0, stream>>>(dest_offsets, D);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  const int total = r->g.total;
  const int sh = r->g.shift[r->route_level];
  // duplicates are reported by k_lr_heads (the routing sort's own offset pass is skipped)
  // with flows, the counting sweep writes every element's flow rank into b.rank
  const bool flows = b.ab.fl.hcap > 0 && n > SORT_SMALL_MAX;
  b.ab.fl.rank_dest = 1;
  int rc = route_run(r->g, make_route(r->g, r->route_level, 1), keys, n, b.ab, nullptr, nullptr,
                     flows ? b.rank : nullptr, nullptr, 0, 1, 0, status, stream, true);
  if (rc) return rc;
  const uint64_t* skey = b.ab.sk;
  const uint32_t* sidx = b.ab.perm;
  k_lr_heads<<<grid_for(n, 256), 256, 0, stream>>>(skey, n, total, sh, b.hs, status);
  rc = scan_exclusive<uint32_t>(b.hs, b.hs, n + 1, nullptr, b.part, nullptr, stream);
  if (rc) return rc;
  k_lr_runs<<<grid_for(n, 256), 256, 0, stream>>>(skey, n, sh, b.hs, r->tkey, r->tdest, r->hcap, b.run_start, b.run_pfx,
                                            b.run_dest, b.nf, b.nrun1, b.nrun, counts);
  rc = scan_exclusive<uint32_t>(b.nf, b.nf, n + 1, b.nrun1, b.part, nullptr, stream);
  if (rc) return rc;
  k_lr_known<<<grid_for(n, 256, 1024), 256, 0, stream>>>(n, b.hs, b.run_start, b.run_dest, b.nf, b.new_run, b.delta,
                                                        D);
  k_lr_assign<<<1, ALTO_WAVE, 0, stream>>>(n, b.hs, b.run_start, b.run_dest, b.nf, b.new_run, b.delta, load, D,
                                           r->nflows, r->max_flows, counts, status);
  k_lr_insert<<<grid_for(n, 256, 1024), 256, 0, stream>>>(n, b.hs, b.nf, b.new_run, b.run_start, b.run_dest, skey, sh,
                                                         r->tkey, r->tdest, r->hcap, status);
  if (dest) {
    // one of the two does the work, as the key sort ran packed or not
    if (flows) k_lr_dest_rank<<<grid_for(n, 256 * LU), 256, 0, stream>>>(n, b.nrun, b.run_dest, b.ab.ctl, b.rank, dest);
    k_lr_dest_in<<<grid_for(n, 256 * LU, 1024), 256, 0, stream>>>(keys, n, sh, b.run_pfx, b.run_dest, b.nrun, r->tkey,
                                                                  r->tdest, r->hcap, b.ab.ctl, flows ? b.rank : nullptr,
                                                                  dest);
  }
  if (perm || dest_offsets) {
    // the runs in (destination, prefix) order, their offsets, then the runs copied
    k_lr_runkeys<<<grid_for(n, 256, 1024), 256, 0, stream>>>(b.nrun, b.run_dest, D, b.rkey);
    SortBufs db;
    memset(&db, 0, sizeof(db));
    db.in_keys = b.rkey;
    db.tmp_keys = b.ab.tmp_keys;
    db.tmp_vals = b.ab.tmp_vals;
    db.out_keys = b.rsk;
    db.out_vals = b.rval;
    db.ctl = b.ab.rctl;
    db.os_status = b.ab.os_status;
    db.os_ctr = b.ab.os_ctr;
    db.os_hist = b.ab.os_hist;
    db.os_ntiles = b.ab.os_ntiles;
    db.status = status;
    RouteGeom none;
    none.shift = 64;
    none.num_dest = 1;
    rc = sort_pairs(db, n, b.nrun, none, 32 + bits_for(D - 1), false, stream);
    if (rc) return rc;
    k_lr_runlen<<<grid_for(n, 256, 1024), 256, 0, stream>>>(n, b.nrun, b.rval, b.run_start, b.roff);
    rc = scan_exclusive<int64_t>(b.roff, b.roff, n + 1, b.nrun1, b.rpart, nullptr, stream);
    if (rc) return rc;
    k_lr_runoff<<<grid_for(n, 256, 1024), 256, 0, stream>>>(n, b.nrun, b.rsk, b.rval, b.roff, D, b.rbase,
                                                           dest_offsets);
    if (perm) k_lr_copy<<<grid_for(n, 256), 256, 0, stream>>>(n, b.hs, b.run_start, b.rbase, sidx, perm);
  }
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

}  // extern "C"
