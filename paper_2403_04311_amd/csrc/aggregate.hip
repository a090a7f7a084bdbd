// Routing (Section 4.3 of the paper) and aggregation at a pmap exit (Sections 3.3
// and 4.3) of one batch: kernels and their orchestration.
#include "aggregate.h"
#include "profile.h"

#include <string.h>

namespace {

constexpr int PREP_NT = 1024;
constexpr int GRID_CAP = 4096;
constexpr int MEAN_GRID = 2048;   // 8 blocks of 256 threads per CU

__device__ inline int64_t dev_or(const int64_t* p, int64_t h) { return p ? *p : h; }

// Input order, one pass: layout check, destination, OR/AND of keys and
// destinations for the sort, flow-set inserts, per-fragment fan-out checks, and
// the carrier-agreement checks of the declared child counts. NL = number of count
// levels read (flo .. flo + NL - 1). Levels xlo..xhi (the route level and up to
// two levels above it: functions of the flow) are checked exactly: the block's LDS
// flow set keeps, per flow and level, the first count seen, every later carrier
// compares against it, and the block's flows are merged into the global set (and
// their counts compared there) when the block ends. The other levels add their
// terms to the fan fingerprint (sums stay in registers). Each thread keeps PU
// elements in flight; each block leaves one record of partial results.
constexpr int PU = 2;
constexpr int PREP_GRID = PREP_BLOCKS_MAX;   // two blocks of PREP_NT threads per CU
constexpr int PREP_SLOTS = 3072;        // LDS flow set of a block (open addressing)
constexpr int PREP_PROBES = 4;          // then the global set directly: when the flows outnumber the
                                        // slots the block's set fills up, and a long walk over it
                                        // costs more than the cached global lookup
constexpr int PREP_NX = FLOW_EXACT_LEVELS;

__device__ inline uint32_t prep_slot(uint64_t p) {
  uint32_t x = ((uint32_t)p ^ ((uint32_t)(p >> 32) * 0x9E3779B1u)) * 0x85EBCA6Bu;
  x ^= x >> 15;
  return (uint32_t)(((uint64_t)(x * 0xC2B2AE35u) * PREP_SLOTS) >> 32);
}

// The count of level x of the flow in global slot s: set by the first carrier
// (0 = unset), compared by every later one. Returns false on a disagreement.
__device__ inline bool flow_fan_check(const FlowBufs& fl, int x, int nx, int64_t s, uint32_t f) {
  uint32_t* w = (x == nx - 1 && fl.x_route) ? &fl.ht_fan[s] : &fl.ht_anc[(int64_t)x * fl.hcap + s];
  const uint32_t cur = *w;   // a count changes once, from 0; the CAS settles a stale 0
  if (cur == f) return true;
  if (cur != 0u) return false;
  const uint32_t old = atomicCAS(w, 0u, f);
  return old == 0u || old == f;
}

template <int NL>
__global__ __launch_bounds__(PREP_NT, 8) void k_prep(const uint64_t* __restrict__ keys, int64_t n, KeyGeom g,
                                                  RouteGeom rg, int32_t* dest, const int32_t* __restrict__ fan,
                                                  int64_t fan_ld, int flo, FlowBufs fl, PrepPartial* part, int qx0,
                                                  int nx, int skip_fp, const int64_t* n_dev) {
  n = dev_n(n_dev, n);
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u;
  uint64_t fp[NL > 0 ? NL : 1];
  int sh[NL > 0 ? NL : 1], shc[NL > 0 ? NL : 1];
  uint32_t tm[NL > 0 ? NL : 1];
#pragma unroll
  for (int q = 0; q < NL; ++q) {
    fp[q] = 0;
    sh[q] = g.shift[flo + q];
    shc[q] = g.shift[flo + q + 1];
    tm[q] = g.tagmask[flo + q + 1];
  }
  bool bad_layout = false, bad_fan = false, flow_full = false;
  __shared__ uint64_t s_fl[PREP_SLOTS];
  __shared__ uint32_t s_ff[PREP_NX][PREP_SLOTS];
  __shared__ uint32_t s_mk;
  if (threadIdx.x == 0) s_mk = 0u;
  if (fl.hcap) {
    for (int i = threadIdx.x; i < PREP_SLOTS; i += PREP_NT) {
      s_fl[i] = ~0ull;
#pragma unroll
      for (int x = 0; x < PREP_NX; ++x) s_ff[x][i] = 0u;
    }
    __syncthreads();
  }
  const int total = g.total;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i0 < n; i0 += stride * PU) {
    uint64_t k[PU];
    int32_t f[PU][NL > 0 ? NL : 1];
#pragma unroll
    for (int u = 0; u < PU; ++u) {
      const int64_t i = i0 + u * stride;
      k[u] = i < n ? keys[i] : 0ull;
#pragma unroll
      for (int q = 0; q < NL; ++q) f[u][q] = i < n ? fan[(int64_t)(flo + q - 1) * fan_ld + i] : 1;
    }
#pragma unroll
    for (int u = 0; u < PU; ++u) {
      const int64_t i = i0 + u * stride;
      if (i >= n) continue;
      bad_layout |= (k[u] >> total) != 0;
      if (!fl.hcap) {
        // without flows the destinations are computed here; with flows the
        // sort's counting sweep takes them from the ranked flows
        const uint32_t d = dest_of_key(rg, k[u]);
        if (dest) dest[i] = (int32_t)d;
        dor |= d;
        dand &= d;
      } else {
        dor = ~0u;   // unknown here: a fallback plan covers every destination bit
        dand = 0u;
      }
      kor |= k[u];
      kand &= k[u];
      if (fl.hcap) {
        const uint64_t p = k[u] >> fl.shift;
        uint32_t h = prep_slot(p);
        uint64_t v = s_fl[h];
        int probes = 0;
        while (v != p) {
          if (v == ~0ull) {
            const uint64_t old = atomicCAS((unsigned long long*)&s_fl[h], ~0ull, (unsigned long long)p);
            if (old == ~0ull || old == p) break;
          }
          if (++probes >= PREP_PROBES) {
            h = PREP_SLOTS;   // crowded: this element goes to the global set itself
            break;
          }
          h = h + 1 == PREP_SLOTS ? 0 : h + 1;
          v = s_fl[h];
        }
        if (h < PREP_SLOTS) {
#pragma unroll
          for (int q = 0; q < NL; ++q) {
            if (q < qx0 || q >= qx0 + nx) continue;   // uniform
            const uint32_t fx = (uint32_t)f[u][q];
            uint32_t* w = &s_ff[q - qx0][h];
            const uint32_t cur = *w;
            if (cur != fx) {
              const uint32_t old = cur == 0u ? atomicCAS(w, 0u, fx) : cur;
              bad_fan |= old != 0u && old != fx;
            }
          }
        } else {
          const int64_t s = flow_insert(fl, p, &flow_full);
          if (s >= 0) {
#pragma unroll
            for (int q = 0; q < NL; ++q)
              if (q >= qx0 && q < qx0 + nx) bad_fan |= !flow_fan_check(fl, q - qx0, nx, s, (uint32_t)f[u][q]);
          }
        }
      }
#pragma unroll
      for (int q = 0; q < NL; ++q) {
        const uint32_t child = (uint32_t)((k[u] >> shc[q]) & (uint64_t)tm[q]);
        bad_fan |= (f[u][q] < 1) || ((int64_t)child >= (int64_t)f[u][q]);
        if (!skip_fp || q < qx0 || q >= qx0 + nx) fp[q] += fan_term(g.fkey, flo + q, key_prefix(k[u], sh[q]), (uint32_t)f[u][q]);
      }
      if (NL > 0 && fl.dp) {
        // markers (direct placement): leaves whose tag is their parent's count - 1,
        // listed in the block's own region (an LDS counter: few markers per block)
        const int32_t fl_ = f[u][NL > 0 ? NL - 1 : 0];
        const uint32_t leaf = (uint32_t)((k[u] >> shc[NL > 0 ? NL - 1 : 0]) & (uint64_t)tm[NL > 0 ? NL - 1 : 0]);
        if (fl_ >= 1 && leaf == (uint32_t)(fl_ - 1)) {
          const uint32_t j = atomicAdd(&s_mk, 1u);
          if (j < (uint32_t)fl.mk_per) {
            const int64_t at = (int64_t)blockIdx.x * fl.mk_per + j;
            fl.mk_key[at] = k[u];
            fl.mk_fan[at] = (uint32_t)fl_;
          }
        }
      }
    }
  }
  if (fl.dp) {
    __syncthreads();
    if (threadIdx.x == 0) fl.mk_cnt[blockIdx.x] = s_mk;
  }
  if (fl.hcap) {
    // the block's flows into the global set, with their counts
    __syncthreads();
    for (int h = threadIdx.x; h < PREP_SLOTS; h += PREP_NT) {
      const uint64_t p = s_fl[h];
      if (p == ~0ull) continue;
      const int64_t s = flow_insert(fl, p, &flow_full);
      if (s < 0) continue;
      for (int x = 0; x < nx; ++x) bad_fan |= !flow_fan_check(fl, x, nx, s, s_ff[x][h]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kor |= __shfl_xor(kor, o);
    kand &= __shfl_xor(kand, o);
    dor |= __shfl_xor(dor, o);
    dand &= __shfl_xor(dand, o);
  }
#pragma unroll
  for (int q = 0; q < NL; ++q) fp[q] = wave_sum(fp[q]);
  uint32_t flags = (bad_layout ? 1u : 0u) | (bad_fan ? 2u : 0u) | (flow_full ? 4u : 0u);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) flags |= __shfl_xor(flags, o);
  __shared__ PrepPartial s_w[PREP_NT / ALTO_WAVE];
  const int w = threadIdx.x / ALTO_WAVE;
  if (lane_id() == 0) {
    s_w[w].kor = kor;
    s_w[w].kand = kand;
    s_w[w].dor = dor;
    s_w[w].dand = dand;
    s_w[w].flags = flags;
#pragma unroll
    for (int q = 0; q < NL; ++q) s_w[w].fp[q] = fp[q];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    PrepPartial r = s_w[0];
    for (int ww = 1; ww < PREP_NT / ALTO_WAVE; ++ww) {
      r.kor |= s_w[ww].kor;
      r.kand &= s_w[ww].kand;
      r.dor |= s_w[ww].dor;
      r.dand &= s_w[ww].dand;
      r.flags |= s_w[ww].flags;
#pragma unroll
      for (int q = 0; q < NL; ++q) r.fp[q] += s_w[ww].fp[q];
    }
    part[blockIdx.x] = r;
  }
}

// When the flow set overflowed, some fragments had no exact check: the exactly
// checked levels then join the fingerprint (their terms over every fragment).
__global__ __launch_bounds__(256) void k_prep_fp(const uint64_t* __restrict__ keys, int64_t n, KeyGeom g,
                                                 const int32_t* __restrict__ fan, int64_t fan_ld, int xlo, int xhi,
                                                 const SortCtl* ctl, uint64_t* fp_in, const int64_t* n_dev) {
  if (!ctl->flow_overflow) return;
  n = dev_n(n_dev, n);
  uint64_t fp[FLOW_EXACT_LEVELS];
#pragma unroll
  for (int x = 0; x < FLOW_EXACT_LEVELS; ++x) fp[x] = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t k = keys[i];
#pragma unroll
    for (int x = 0; x < FLOW_EXACT_LEVELS; ++x) {
      const int m = xlo + x;
      if (m <= xhi) fp[x] += fan_term(g.fkey, m, key_prefix(k, g.shift[m]), (uint32_t)fan[(int64_t)(m - 1) * fan_ld + i]);
    }
  }
#pragma unroll
  for (int x = 0; x < FLOW_EXACT_LEVELS; ++x) {
    const uint64_t v = wave_sum(fp[x]);
    if (lane_id() == 0 && v && xlo + x <= xhi) atomicAdd((unsigned long long*)&fp_in[xlo + x], (unsigned long long)v);
  }
}

// Folds the per-block records of k_prep into the sort control block, the
// fingerprint sums and the status word (strided per thread, then a wave
// reduction, then the 4 wave results).
__global__ __launch_bounds__(256) void k_prep_fold(const PrepPartial* part, int nblocks, int flo, int nl, SortCtl* ctl,
                                                   uint64_t* fp_in, int32_t* status) {
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u, flags = 0;
  uint64_t fp[ALTO_MAX_LEVELS];
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) fp[q] = 0;
  for (int b = threadIdx.x; b < nblocks; b += blockDim.x) {
    const PrepPartial& x = part[b];
    kor |= x.kor;
    kand &= x.kand;
    dor |= x.dor;
    dand &= x.dand;
    flags |= x.flags;
#pragma unroll
    for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
      if (q < nl) fp[q] += x.fp[q];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kor |= __shfl_xor(kor, o);
    kand &= __shfl_xor(kand, o);
    dor |= __shfl_xor(dor, o);
    dand &= __shfl_xor(dand, o);
    flags |= __shfl_xor(flags, o);
  }
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
    if (q < nl) fp[q] = wave_sum(fp[q]);
  __shared__ PrepPartial s_w[256 / ALTO_WAVE];
  const int w = threadIdx.x / ALTO_WAVE;
  if (lane_id() == 0) {
    s_w[w].kor = kor;
    s_w[w].kand = kand;
    s_w[w].dor = dor;
    s_w[w].dand = dand;
    s_w[w].flags = flags;
#pragma unroll
    for (int q = 0; q < ALTO_MAX_LEVELS; ++q) s_w[w].fp[q] = fp[q];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int ww = 1; ww < 256 / ALTO_WAVE; ++ww) {
      kor |= s_w[ww].kor;
      kand &= s_w[ww].kand;
      dor |= s_w[ww].dor;
      dand &= s_w[ww].dand;
      flags |= s_w[ww].flags;
      for (int q = 0; q < nl; ++q) fp[q] += s_w[ww].fp[q];
    }
    ctl->key_or = kor;
    ctl->key_and = kand;
    ctl->dest_or = dor;
    ctl->dest_and = dand;
    if (flags & 4u) ctl->flow_overflow = 1;
    for (int q = 0; q < nl; ++q) fp_in[flo + q] = fp[q];
    if (flags & 1u) raise_status(status, ALTO_E_LAYOUT);
    if (flags & 2u) raise_status(status, ALTO_E_FANOUT);
  }
}

// Start of a routing call: control block, fingerprint sums and the flow set.
__global__ void k_route_init(SortCtl* ctl, uint64_t* fp_in, uint64_t* fp_nodes, FlowBufs fl, const int64_t* n_dev,
                             int64_t n_max, int32_t* status) {
  if (blockIdx.x == 0) {
    if (threadIdx.x == 0) {
      if (n_dev && (*n_dev < 0 || *n_dev > n_max)) raise_status(status, ALTO_E_CAPACITY);
      ctl->key_or = 0;
      ctl->key_and = ~0ull;
      ctl->dest_or = 0;
      ctl->dest_and = ~0u;
      ctl->mode = SORT_GENERAL;
      ctl->flow_overflow = 0;
      ctl->nflows = 0;
      ctl->nflows_c = 0;
      ctl->cmode = 0;
      ctl->dp = 0;
      ctl->dbits = -1;
    }
    for (int i = threadIdx.x; i <= ALTO_MAX_LEVELS; i += blockDim.x) {
      fp_in[i] = 0;
      fp_nodes[i] = 0;
    }
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < fl.hcap; i += (int64_t)gridDim.x * blockDim.x) {
    fl.ht_key[i] = ~0ull;
    fl.ct_key[i] = ~0ull;
    fl.ht_fan[i] = 0u;
#pragma unroll
    for (int x = 0; x < FLOW_EXACT_LEVELS; ++x) fl.ht_anc[(int64_t)x * fl.hcap + i] = 0u;
  }
}

// Direct placement (see FlowBufs.dp), after the sort: the groups are the flows,
// their bounds the child-rank bases of their first children (with check_all, also
// the search for positions left unplaced, when no gather reads them all). Writes what the segmentation pass writes for the group level:
// node starts, complete flags, declared and carried counts, the node side of the
// fingerprints of those levels, destination offsets, and the sorted key at each
// group start (its prefix bits: the group's key and destination come from it).
__global__ __launch_bounds__(256) void k_dp_groups(KeyGeom g, FlowBufs fl, const SortCtl* ctl, int64_t n, int La,
                                                   LevelNodes L, int64_t* nnodes, int64_t* dest_offsets,
                                                   uint32_t num_dest, uint64_t* sk, const uint32_t* perm,
                                                   const int32_t* fan, int64_t fan_ld, int carry_lo,
                                                   int32_t* carry_fan, int64_t carry_ld, uint64_t* fp_nodes,
                                                   int32_t* status, int check_all) {
  if (!ctl->dp) return;
  const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (check_all) {
    // no gather reads the whole permutation in this call: look for unplaced
    // positions here
    bool hole = false;
    for (int64_t i = gtid; i < n; i += stride) hole |= perm[i] == DP_UNPLACED;
    if (__ballot(hole) && lane_id() == 0) raise_status(status, ALTO_E_DUPLICATE);
  }
  const int64_t F = ctl->nflows_c;
  const int nc = La - carry_lo;   // carried levels carry_lo .. La-1
  uint64_t fpm = 0;
  uint64_t fpc[ALTO_MAX_LEVELS];
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) fpc[q] = 0;
  for (int64_t r = gtid; r < F; r += stride) {
    // with direct placement chosen, cbase rises strictly (every count >= 1) from 0 to
    // n; the clamps only keep every later index in bounds
    int64_t s = fl.cbase[fl.fbase[r]], e = fl.cbase[fl.fbase[r + 1]];
    s = s < n ? s : n;
    e = e < n ? e : n;
    const int64_t cnt = e > s ? e - s : 0;
    L.start[r] = (int32_t)s;
    L.ok[r] = 1;
    L.bad[r] = 0;
    if (cnt == 0) {
      L.nfan[r] = 0;
      continue;
    }
    // the first leaf's row (a position left unwritten holds no row: duplicate keys,
    // reported by whoever reads the permutation; any row in bounds serves then)
    const uint32_t row0 = perm[s];
    const uint32_t row = (int64_t)row0 < n ? row0 : 0u;
    const uint64_t pk = fl.flow_sorted[r] << fl.shift;
    const int32_t nf = fan[(int64_t)(La - 1) * fan_ld + row];
    L.nfan[r] = nf;
    sk[s] = pk;
    fpm += (uint64_t)cnt * fan_term(g.fkey, La, key_prefix(pk, g.shift[La]), (uint32_t)nf);
#pragma unroll
    for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
      if (q >= nc) break;
      const int m = carry_lo + q;
      const int32_t cf = fan[(int64_t)(m - 1) * fan_ld + row];
      if (carry_fan) carry_fan[(int64_t)q * carry_ld + r] = cf;
      fpc[q] += (uint64_t)cnt * fan_term(g.fkey, m, key_prefix(pk, g.shift[m]), (uint32_t)cf);
    }
    if (dest_offsets) {
      const uint32_t d = fl.fdest[r];
      if (r == 0) {
        for (uint32_t x = 0; x <= d; ++x) dest_offsets[x] = 0;
      } else {
        const uint32_t dp = fl.fdest[r - 1];
        for (uint32_t x = dp + 1; x <= d; ++x) dest_offsets[x] = s;
      }
      if (r == F - 1)
        for (uint32_t x = d + 1; x <= num_dest; ++x) dest_offsets[x] = n;
    }
  }
  if (gtid == 0) {
    nnodes[La] = F;
    L.start[F] = (int32_t)n;
  }
  fpm = wave_sum(fpm);
  if (lane_id() == 0 && fpm) atomicAdd((unsigned long long*)&fp_nodes[La], (unsigned long long)fpm);
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
    if (q >= nc) break;
    const uint64_t v = wave_sum(fpc[q]);
    if (lane_id() == 0 && v) atomicAdd((unsigned long long*)&fp_nodes[carry_lo + q], (unsigned long long)v);
  }
}

// dest_offsets from the sorted keys; duplicate keys are adjacent after the sort.
__global__ __launch_bounds__(256) void k_dest_offsets(const uint64_t* __restrict__ sk, int64_t n, RouteGeom rg,
                                                      int64_t* offs, int32_t* status, const int64_t* n_dev) {
  const uint32_t D = rg.num_dest;
  n = dev_n(n_dev, n);
  if (n == 0) {
    if (offs && blockIdx.x == 0)
      for (uint32_t x = threadIdx.x; x <= D; x += blockDim.x) offs[x] = 0;
    return;
  }
  bool dup = false;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t k = sk[j];
    const uint32_t d = dest_of_key(rg, k);
    uint32_t dp = 0;
    if (j > 0) {
      const uint64_t kp = sk[j - 1];
      dup |= (kp == k);
      dp = dest_of_key(rg, kp);
    }
    if (offs) {
      if (j == 0) {
        for (uint32_t x = 0; x <= d; ++x) offs[x] = 0;
      } else if (d != dp) {
        for (uint32_t x = dp + 1; x <= d; ++x) offs[x] = j;
      }
      if (j == n - 1)
        for (uint32_t x = d + 1; x <= D; ++x) offs[x] = n;
    }
  }
  if (dup) raise_status(status, ALTO_E_DUPLICATE);
}

// The groups of the aggregation level in one kernel. Per tile of groups: the
// exclusive sums over groups u = 0..G (entry G holds the totals) of emitted
// (complete) flags, emitted tokens, long-group chunks, chunk partials (groups of
// more than one chunk) and short groups; tiles by ticket, sums across tiles by
// look-back (64-bit words: token sums may exceed 2^30). Then, with the tile's
// groups strided over the threads, each group's outputs: records (emitted groups)
// or pending entries, and its chunk descriptors. Groups of more than
// MEAN_SMALL_ROWS rows are cut into chunks of chunk_rows, at chunks[first long
// chunk of the group ...]; each shorter group is one chunk at chunks[short_base +
// its short-group index], so no position depends on the totals. Emitted groups
// enter the emitted set (ex.ht). The thread holding entry G writes the call's
// counts and the chunk totals the gathers read (capacity checked there), and,
// unless the fold accumulates fingerprint terms in this same kernel, compares the
// fan fingerprints.
constexpr int GS_NT = 256;
constexpr int GS_IT = 4;
constexpr int GS_TILE = GS_NT * GS_IT;
static_assert(GS_TILE == GROUP_SCAN_TILE, "group scan tile");
static_assert(GS_IT <= 32, "a thread's groups in one flag word");
static_assert(GS_NT * GS_IT < (1 << 21), "a tile's group counts fit 21 bits");

constexpr int GS_NV = GROUP_SCAN_WORDS;   // scanned values per group
constexpr int GS_SPEC_BLOCKS = 8;         // blocks that load their tile before the count arrives

__global__ void k_group_scan_prep(const int64_t* Gp, uint64_t* st, uint32_t* ctr, GroupsExtra ex) {
  const int64_t len = cdiv(*Gp + 1, GS_TILE) * GS_NV;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = t0; i < len; i += stride) st[i] = 0;
  if (ex.xst) {
    const int64_t xl = cdiv(*ex.xlen, ex.xtile) * ex.xper;
    for (int64_t i = t0; i < xl; i += stride) ex.xst[i] = 0;
  }
  if (t0 == 0) {
    *ctr = 0;
    if (ex.xst) *ex.xctr = 0;
  }
}

// The completion of the group-level nodes, when the group kernel evaluates it (as
// k_seg_nodes would for that level).
struct GroupFold {
  int32_t on, leafy, level, es;
  uint64_t fkey;
  const uint64_t* keys;
  uint64_t* fp;   // nullable: fingerprint sums per level
};

// The node fields a thread of the group kernel reads for its groups of a tile
// (group g0 + k GS_NT + threadIdx.x for k < GS_IT), below bound.
struct GroupTileLoad {
  int32_t sv[GS_IT], sn[GS_IT], cv[GS_IT], cn[GS_IT], nf[GS_IT];
  uint8_t bd[GS_IT], okf[GS_IT];
  uint64_t nk[GS_IT];   // first keys, when the pass recorded them
};

__device__ inline void group_tile_load(const LevelNodes& L, const GroupFold& f, int64_t g0, int64_t bound,
                                       GroupTileLoad& t) {
#pragma unroll
  for (int k = 0; k < GS_IT; ++k) {
    const int64_t u = g0 + k * GS_NT + threadIdx.x;
    const bool in = u < bound;
    t.sv[k] = in ? L.start[u] : 0;
    t.sn[k] = in ? L.start[u + 1] : 0;
    t.cv[k] = (in && f.on && !f.leafy) ? L.fc[u] : 0;
    t.cn[k] = (in && f.on && !f.leafy) ? L.fc[u + 1] : 0;
    t.nf[k] = (in && f.on) ? L.nfan[u] : 0;
    t.bd[k] = (in && f.on) ? L.bad[u] : 1;
    t.okf[k] = (in && !f.on) ? L.ok[u] : 0;
    t.nk[k] = (in && L.nkey) ? L.nkey[u] : 0ull;
  }
}

template <typename Src>
__global__ __launch_bounds__(GS_NT) void k_groups(KeyGeom g, RouteGeom rg, int La, LevelNodes L, const int64_t* Gp,
                                                  const uint64_t* __restrict__ sk, Src src, Chunk* chunks,
                                                  int64_t short_base, int chunk_rows, GroupOut out, int concat,
                                                  const int64_t* Mp, int64_t* scal, GroupsExtra ex, uint64_t* st,
                                                  uint32_t* ctr, GroupFold f, int64_t ucap, int32_t* status) {
  // the fields of the tile this block most likely takes first (its own index),
  // loaded before the group count and the ticket have arrived (the node arrays
  // hold ucap + 1 entries; groups past the count are not used). Only the first
  // GS_SPEC_BLOCKS blocks do so: the grid is sized for the largest count, and
  // blocks past the actual tile count would only load in vain.
  const int64_t gt = blockIdx.x;
  const bool spec = blockIdx.x < GS_SPEC_BLOCKS;
  GroupTileLoad pre;
  if (spec) group_tile_load(L, f, gt * GS_TILE, ucap, pre);
  const int64_t G = *Gp;
  const int64_t ntiles = cdiv(G + 1, GS_TILE);
  __shared__ uint64_t s_w[GS_NT / ALTO_WAVE];
  __shared__ int64_t s_ex[GS_NV];
  __shared__ uint32_t s_tile;
  // per group of the tile: the fold's flags and row counts, then the exclusive sums
  __shared__ uint8_t s_okf[GS_TILE];
  __shared__ int32_t s_cnt[GS_TILE];
  __shared__ int32_t s_em[GS_TILE], s_cb[GS_TILE], s_pb[GS_TILE], s_sb[GS_TILE];
  __shared__ int64_t s_tb[GS_TILE];
  if ((int64_t)blockIdx.x >= ntiles) return;   // no tile would be left for this block
  const int lane = lane_id();
  uint64_t fpm = 0;     // fingerprint terms of the groups this thread evaluated
  int64_t fresh = 0;    // keys new to the emitted set
  bool full = false;
  bool first = true;
  while (true) {
    // a single tile is block 0's without a ticket (it waits for no other tile)
    if (ntiles > 1 && threadIdx.x == 0) s_tile = atomicAdd(ctr, 1u);
    __syncthreads();
    const int64_t tile = ntiles > 1 ? (int64_t)s_tile : (first ? 0 : 1);
    first = false;
    if (tile >= ntiles) break;   // uniform
    const int64_t g0 = tile * GS_TILE;
    const int64_t u0 = g0 + (int64_t)threadIdx.x * GS_IT;
    // the tile's groups strided over the threads (group g0 + k GS_NT + threadIdx.x):
    // first element and its key, for the fold and the outputs
    int32_t sv[GS_IT];
    uint64_t kk[GS_IT];
    int64_t v[GS_IT][GS_NV];
    int64_t sum[GS_NV] = {0, 0, 0, 0, 0};
    uint32_t okm = 0;         // bit i: group u0 + i is complete
    int32_t cnv[GS_IT] = {};  // rows of the groups u0 + i
    if (f.on) {
      // complete: as many children as declared, none of them incomplete. Every load
      // first, then the flags, fingerprint terms and stores; the scan reads the
      // flags and row counts back from LDS.
      GroupTileLoad t;
      if (spec && tile == gt) t = pre;
      else group_tile_load(L, f, g0, G, t);
      const int32_t* sn = t.sn;
      const int32_t* cv = t.cv;
      const int32_t* cn = t.cn;
      const int32_t* nf = t.nf;
      const uint8_t* bd = t.bd;
#pragma unroll
      for (int k = 0; k < GS_IT; ++k) sv[k] = t.sv[k];
#pragma unroll
      for (int k = 0; k < GS_IT; ++k)
        kk[k] = g0 + k * GS_NT + threadIdx.x < G ? (L.nkey ? t.nk[k] : f.keys[sv[k]]) : 0ull;
#pragma unroll
      for (int k = 0; k < GS_IT; ++k) {
        const int64_t u = g0 + k * GS_NT + threadIdx.x;
        const int idx = k * GS_NT + threadIdx.x;
        if (u >= G) {
          s_okf[idx] = 0;
          s_cnt[idx] = 0;
          continue;
        }
        const int32_t n0 = sn[k] - sv[k];
        const int32_t nchild = f.leafy ? n0 : cn[k] - cv[k];
        const bool ok = nchild == nf[k] && !bd[k];
        s_okf[idx] = ok ? 1 : 0;
        s_cnt[idx] = n0;
        L.ok[u] = ok ? 1 : 0;
        if (f.fp) fpm += (uint64_t)n0 * fan_term(f.fkey, f.level, key_prefix(kk[k], f.es), (uint32_t)nf[k]);
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < GS_IT; ++i) {
        const int idx = threadIdx.x * GS_IT + i;
        okm |= (uint32_t)s_okf[idx] << i;
        cnv[i] = s_cnt[idx];
      }
    } else {
      GroupTileLoad t;
      if (spec && tile == gt) t = pre;
      else group_tile_load(L, f, g0, G, t);
#pragma unroll
      for (int k = 0; k < GS_IT; ++k) {
        const bool in = g0 + k * GS_NT + threadIdx.x < G;
        sv[k] = t.sv[k];
        s_okf[k * GS_NT + threadIdx.x] = (in && t.okf[k]) ? 1 : 0;
        s_cnt[k * GS_NT + threadIdx.x] = in ? t.sn[k] - t.sv[k] : 0;
      }
#pragma unroll
      for (int k = 0; k < GS_IT; ++k)
        kk[k] = g0 + k * GS_NT + threadIdx.x < G ? (L.nkey ? t.nk[k] : sk[sv[k]]) : 0ull;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < GS_IT; ++i) {
        const int idx = threadIdx.x * GS_IT + i;
        okm |= (uint32_t)s_okf[idx] << i;
        cnv[i] = s_cnt[idx];
      }
    }
#pragma unroll
    for (int i = 0; i < GS_IT; ++i) {
      const bool ok = (okm >> i) & 1u;
      const int64_t cnt = ok ? (int64_t)cnv[i] : 0;
      const bool small = ok && cnt <= MEAN_SMALL_ROWS;
      const int64_t c = ok && !small ? cdiv(cnt, chunk_rows) : 0;
      v[i][0] = ok ? 1 : 0;
      v[i][1] = cnt;
      v[i][2] = c;
      v[i][3] = c > 1 ? c : 0;
      v[i][4] = small ? 1 : 0;
#pragma unroll
      for (int q = 0; q < GS_NV; ++q) sum[q] += v[i][q];
    }
    // two block scans of packed words: emitted groups, short groups and long-group
    // chunks in 21-bit fields (a tile holds GS_TILE < 2^21 groups and fewer than
    // 2^31 / MEAN_CHUNK_ROWS + GS_TILE < 2^21 chunks), rows (below 2^31) and partial
    // slots (below 2^21) in 32-bit fields: no field carries into the next
    constexpr uint64_t F21 = (1ull << 21) - 1ull, F32 = (1ull << 32) - 1ull;
    const uint64_t wa = (uint64_t)sum[0] | ((uint64_t)sum[4] << 21) | ((uint64_t)sum[2] << 42);
    const uint64_t wb = (uint64_t)sum[1] | ((uint64_t)sum[3] << 32);
    uint64_t ta, tb;
    const uint64_t xa = block_excl_scan<uint64_t, GS_NT>(wa, s_w, &ta);
    const uint64_t xb = block_excl_scan<uint64_t, GS_NT>(wb, s_w, &tb);
    int64_t exs[GS_NV], tot[GS_NV];
    exs[0] = (int64_t)(xa & F21);
    exs[1] = (int64_t)(xb & F32);
    exs[2] = (int64_t)(xa >> 42);
    exs[3] = (int64_t)(xb >> 32);
    exs[4] = (int64_t)((xa >> 21) & F21);
    tot[0] = (int64_t)(ta & F21);
    tot[1] = (int64_t)(tb & F32);
    tot[2] = (int64_t)(ta >> 42);
    tot[3] = (int64_t)(tb >> 32);
    tot[4] = (int64_t)((ta >> 21) & F21);
    if (threadIdx.x < GS_NV) {
      const int q = threadIdx.x;
      int64_t t = tot[0];
#pragma unroll
      for (int qq = 1; qq < GS_NV; ++qq)
        if (q == qq) t = tot[qq];
      lb64_publish(st + q, tile, GS_NV, (uint64_t)t);
      s_ex[q] = (int64_t)lb64_resolve(st + q, tile, GS_NV, (uint64_t)t, status);
    }
    __syncthreads();
    int64_t run[GS_NV];
#pragma unroll
    for (int q = 0; q < GS_NV; ++q) run[q] = s_ex[q] + exs[q];
#pragma unroll
    for (int i = 0; i < GS_IT; ++i) {
      const int64_t u = u0 + i;
      const int idx = threadIdx.x * GS_IT + i;
      s_em[idx] = (int32_t)run[0];
      s_tb[idx] = run[1];
      s_cb[idx] = (int32_t)run[2];
      s_pb[idx] = (int32_t)run[3];
      s_sb[idx] = (int32_t)run[4];
      if (u == G) {
        // the totals: the call's counts, the chunk totals of the gathers, capacity
        const int64_t E = run[0], T = concat ? run[1] : 0, M = Mp ? *Mp : 0, P = G - E;
        scal[1] = run[2];   // long-group chunks: chunks[0, scal[1])
        scal[2] = 0;        // block tickets of the mean gather (long groups)
        scal[3] = run[4];   // short groups: chunks[short_base, short_base + scal[3])
        out.counts[0] = E;
        out.counts[1] = T;
        out.counts[2] = M;
        out.counts[3] = P;
        if (out.tok_off && E <= out.cap_groups) out.tok_off[E] = T;
        if (E > out.cap_groups || P > out.cap_groups || T > out.cap_tokens || M > out.cap_mask)
          raise_status(status, ALTO_E_CAPACITY);
        if (ex.fp_in) {
          const bool all = ex.ctl == nullptr || ex.ctl->flow_overflow;
          for (int m = ex.flo; m <= ex.fhi; ++m)
            if ((all || m < ex.xlo || m > ex.xhi) && ex.fp_in[m] != ex.fp_nodes[m]) raise_status(status, ALTO_E_FANOUT);
        }
      }
#pragma unroll
      for (int q = 0; q < GS_NV; ++q) run[q] += v[i][q];
    }
    __syncthreads();   // the tile's sums are in LDS
    // the outputs of the tile's groups (strided, as loaded above): records or pending
    // entries, the emitted set, and each complete group's first chunk by its own
    // lane; the further chunks of long groups by the whole wave, group by group
    const bool need_first = out.first_i32 || (out.fan_up && La > 1);
    int64_t fr[GS_IT];
#pragma unroll
    for (int k = 0; k < GS_IT; ++k) {
      const int idx = k * GS_NT + threadIdx.x;
      fr[k] = (need_first && g0 + k * GS_NT + threadIdx.x < G && s_okf[idx]) ? src.row(sv[k]) : 0;
    }
#pragma unroll
    for (int k = 0; k < GS_IT; ++k) {
      const int64_t u = g0 + k * GS_NT + threadIdx.x;
      const int idx = k * GS_NT + threadIdx.x;
      const bool in = u < G;
      const bool ok = in && s_okf[idx];
      const int32_t s = sv[k], cnt = s_cnt[idx];
      const int64_t e = s_em[idx], o = s_tb[idx];
      const bool small = cnt <= MEAN_SMALL_ROWS;
      const int64_t nc = ok ? (small ? 1 : cdiv(cnt, chunk_rows)) : 0;
      const int64_t c0 = small ? short_base + s_sb[idx] : (int64_t)s_cb[idx];
      const int64_t part = nc > 1 ? (int64_t)s_pb[idx] : -1;
      if (in) {
        const uint64_t gk = key_prefix(kk[k], g.shift[La]);
        if (ok) {
          if (e < out.cap_groups) {
            if (out.key) out.key[e] = gk;
            if (out.dest) out.dest[e] = (int32_t)dest_of_key(rg, kk[k]);
            if (out.count) out.count[e] = cnt;
            if (out.first_i32) out.first_i32[e] = src.p32_of(fr[k]);
            if (out.fan_up)
              for (int l = 1; l < La; ++l) out.fan_up[(int64_t)(l - 1) * out.cap_groups + e] = src.fan_of(l, fr[k]);
            if (out.tok_off) out.tok_off[e] = o;
          }
          if (ex.ht) {
            const int r = emitted_insert(gk, ex.ht, ex.htcap);
            if (r < 0) full = true;
            else fresh += r;
          }
          Chunk ch;
          ch.e = e;
          ch.begin = s;
          ch.len = cnt < chunk_rows ? cnt : chunk_rows;
          ch.k = 0;
          ch.nch = (int32_t)nc;
          ch.count = cnt;
          ch.part = part;
          ch.out = o;
          ch.pad = 0;
          chunks[c0] = ch;
        } else {
          const int64_t p = u - e;
          if (p < out.cap_groups) {
            if (out.pend_key) out.pend_key[p] = gk;
            if (out.pend_count) out.pend_count[p] = cnt;
          }
        }
      }
      // chunks 1 .. nc-1 of the wave's long groups, one group at a time
      for (uint64_t many = __ballot(nc > 1); many; many &= many - 1) {
        const int l = __builtin_ctzll(many);
        const int64_t le = __shfl(e, l), lo = __shfl(o, l), lc0 = __shfl(c0, l), lpart = __shfl(part, l);
        const int32_t ls = __shfl(s, l), lcnt = __shfl(cnt, l);
        const int64_t lnc = __shfl(nc, l);
        for (int64_t c = 1 + lane; c < lnc; c += ALTO_WAVE) {
          Chunk ch;
          ch.e = le;
          ch.begin = ls + (int32_t)(c * chunk_rows);
          ch.len = (int32_t)((lcnt - c * chunk_rows) < chunk_rows ? (lcnt - c * chunk_rows) : chunk_rows);
          ch.k = (int32_t)c;
          ch.nch = (int32_t)lnc;
          ch.count = lcnt;
          ch.part = lpart;
          ch.out = lo + c * chunk_rows;
          ch.pad = 0;
          chunks[lc0 + c] = ch;
        }
      }
    }
    __syncthreads();   // s_ex, the tile's LDS and the ticket are reused by the next tile
  }
  if (f.on && f.fp) {
    // one atomic per block
    __shared__ uint64_t s_fp[GS_NT / ALTO_WAVE];
    const uint64_t w = wave_sum(fpm);
    if (lane == 0) s_fp[threadIdx.x / ALTO_WAVE] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t t = 0;
      for (int ww = 0; ww < GS_NT / ALTO_WAVE; ++ww) t += s_fp[ww];
      if (t) atomicAdd((unsigned long long*)&f.fp[f.level], (unsigned long long)t);
    }
  }
  if (ex.ht) {
    // one count update per wave (the caller's next kernel compares the total with
    // its limit)
    const int64_t w = wave_sum(fresh);
    if (lane == 0 && w) atomicAdd((unsigned long long*)ex.emit_count, (unsigned long long)w);
    if (full) raise_status(status, ALTO_E_CAPACITY);
  }
}

template <typename Src>
__global__ __launch_bounds__(256) void k_concat(const Chunk* __restrict__ chunks, const int64_t* nlong,
                                                const Chunk* __restrict__ chunks_s, const int64_t* nshort, Src src,
                                                int32_t* tok, int64_t cap_tokens) {
  concat_chunks<Src>(chunks, *nlong, chunks_s, *nshort, src, tok, cap_tokens, blockIdx.x, gridDim.x);
}

// fp64 sum of the rows of one chunk of a group, in a fixed order: each lane sums
// its rows sequentially (U independent row loads in flight), then lanes holding the
// same columns are combined in lane order, then the waves in wave order. Groups of
// one chunk are finished here; the others leave a partial sum per chunk.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
// buffer resource word 3 for raw (untyped) buffer access on gfx9-family GPUs, and the
// cache-policy operand of a device-scope (sc1) store
constexpr int BUFFER_RSRC_WORD3 = 0x00020000;
constexpr int BUFFER_STORE_SC1 = 16;

// One short group (a single chunk of at most MEAN_SMALL_ROWS rows) gathered by one
// wave: rows in batches of 64 (one coalesced index load each), UW rows per lane in
// flight, lanes holding the same columns combined in lane order; the mean is
// written directly.
template <int VEC, int CPL, typename Src>
__device__ inline void mean_short_chunk(const Chunk& ch, const Src& srcp, int dim, int C, int lpr, float* mean,
                                        int64_t cap_groups) {
  constexpr int UW = 4;
  const int lane = lane_id();
  const int rpw = ALTO_WAVE / lpr, sub = lane / lpr, cl = lane % lpr;
  const int32_t row_safe = (int32_t)srcp.row(ch.begin);
  for (int col0 = 0; col0 < C; col0 += lpr * CPL) {
    double acc[CPL][VEC];
#pragma unroll
    for (int q = 0; q < CPL; ++q)
#pragma unroll
      for (int v = 0; v < VEC; ++v) acc[q][v] = 0.0;
    for (int b0 = 0; b0 < ch.len; b0 += ALTO_WAVE) {
      const int nr = ch.len - b0 < ALTO_WAVE ? ch.len - b0 : ALTO_WAVE;
      const int32_t myrow = lane < nr ? (int32_t)srcp.row(ch.begin + b0 + lane) : 0;
      const int steps = (int)cdiv(nr, rpw);
      for (int it0 = 0; it0 < steps; it0 += UW) {
        float x[UW][CPL][VEC];
#pragma unroll
        for (int u = 0; u < UW; ++u) {
          const int r = (it0 + u) * rpw + sub;
          const int32_t rr = __shfl(myrow, r & (ALTO_WAVE - 1));
          const bool ok = (it0 + u < steps) && r < nr;
          const float* src = srcp.pay_of(ok ? rr : row_safe);
#pragma unroll
          for (int q = 0; q < CPL; ++q) {
            const int col = col0 + cl + q * lpr;
            const bool okc = ok && col < C;
            const int colc = col < C ? col : C - 1;
            if constexpr (VEC == 4) {
              const f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + (int64_t)colc * 4));
              x[u][q][0] = okc ? t[0] : 0.f;
              x[u][q][1] = okc ? t[1] : 0.f;
              x[u][q][2] = okc ? t[2] : 0.f;
              x[u][q][3] = okc ? t[3] : 0.f;
            } else {
              const float t = __builtin_nontemporal_load(src + colc);
              x[u][q][0] = okc ? t : 0.f;
            }
          }
        }
#pragma unroll
        for (int u = 0; u < UW; ++u)
#pragma unroll
          for (int q = 0; q < CPL; ++q)
#pragma unroll
            for (int v = 0; v < VEC; ++v) acc[q][v] += (double)x[u][q][v];
      }
    }
    for (int o = lpr; o < ALTO_WAVE; o <<= 1)
#pragma unroll
      for (int q = 0; q < CPL; ++q)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[q][v] += __shfl_xor(acc[q][v], o);
    if constexpr (VEC == 4) {
      // write-through (device scope) 16-byte stores: dirty mean lines evicted from L2
      // by the row stream cost the gather more than lines written through at once
      // (measured on 768-float means: 2-4% of the gather). The row's base is the
      // wave's (one group per wave), held in scalar registers.
      const uint64_t ba = (uint64_t)(uintptr_t)(mean + ch.e * (int64_t)dim);
      const uint32_t blo = __builtin_amdgcn_readfirstlane((uint32_t)ba);
      const uint32_t bhi = __builtin_amdgcn_readfirstlane((uint32_t)(ba >> 32));
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          reinterpret_cast<void*>((uintptr_t)(((uint64_t)bhi << 32) | blo)), 0, dim * 4, BUFFER_RSRC_WORD3);
      if (sub == 0 && ch.e < cap_groups) {
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
          const int col = col0 + cl + q * lpr;
          if (col >= C) continue;
          i32x4 w;
#pragma unroll
          for (int v = 0; v < 4; ++v) w[v] = __float_as_int((float)(acc[q][v] / (double)ch.count));
          __builtin_amdgcn_raw_buffer_store_b128(w, rs, col * 16, 0, BUFFER_STORE_SC1);
        }
      }
    } else if (sub == 0 && ch.e < cap_groups) {
#pragma unroll
      for (int q = 0; q < CPL; ++q) {
        const int col = col0 + cl + q * lpr;
        if (col >= C) continue;
#pragma unroll
        for (int v = 0; v < VEC; ++v)
          mean[ch.e * (int64_t)dim + (int64_t)col * VEC + v] = (float)(acc[q][v] / (double)ch.count);
      }
    }
  }
}

// Chunks [0, NB) belong to long groups and are gathered a block each (first phase);
// chunks_s [0, NS) are short groups, gathered a wave each (second phase).
template <int VEC, int CPL, typename Src>
__global__ __launch_bounds__(256) void k_mean(const Chunk* __restrict__ chunks, const int64_t* nblock,
                                              const Chunk* __restrict__ chunks_s, const int64_t* nshort, Src srcp,
                                              int dim, int lpr, double* part, float* mean, int64_t cap_groups,
                                              unsigned long long* ticket) {
  constexpr int NW = 4;
  constexpr int U = 2;   // row loads in flight per lane (more lowers occupancy)
  __shared__ double red[NW][64 * CPL * VEC];
  const int C = dim / VEC;
  const int lane = lane_id(), w = threadIdx.x / ALTO_WAVE;
  const int rpw = ALTO_WAVE / lpr, sub = lane / lpr, cl = lane % lpr;
  const int64_t NB = *nblock, NS = *nshort;
  __shared__ int64_t s_c;
  // chunks are taken by ticket: groups have very different sizes, and a block that
  // finishes early takes the next chunk (the sum of a chunk does not depend on
  // which block computes it). Blocks past the chunk count take none (no contention).
  while ((int64_t)blockIdx.x < NB) {
    if (threadIdx.x == 0) s_c = (int64_t)atomicAdd(ticket, 1ull);
    __syncthreads();
    const int64_t c = s_c;
    if (c >= NB) break;   // uniform
    const Chunk ch = chunks[c];
    // a row of the chunk that exists: lanes past the end load it and discard it, so
    // that no load sits behind a branch (which would wait for each load in turn)
    const int32_t row_safe = (int32_t)srcp.row(ch.begin);
    for (int col0 = 0; col0 < C; col0 += lpr * CPL) {
      double acc[CPL][VEC];
#pragma unroll
      for (int q = 0; q < CPL; ++q)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[q][v] = 0.0;
      // the block takes batches of NW x 64 rows; in a batch, step `it` loads rows
      // b0 + (it x NW + w) x rpw + sub (rpw rows per wave and step, the waves
      // interleaved, so that a short chunk still spreads over every wave). Each wave
      // first reads the row indices of its 64 rows with one load and passes them to
      // the lanes that load the rows, so the payload loads do not wait on index loads.
      for (int b0 = 0; b0 < ch.len; b0 += NW * ALTO_WAVE) {
        const int mine = b0 + ((lane / rpw) * NW + w) * rpw + lane % rpw;   // row of index slot `lane`
        const int32_t myrow = mine < ch.len ? (int32_t)srcp.row(ch.begin + mine) : 0;
        // steps holding a row of this wave: b0 + (it x NW + w) x rpw < len
        const int left = ch.len - b0 - w * rpw;
        const int steps = left <= 0 ? 0 : (int)cdiv(left, NW * rpw) < lpr ? (int)cdiv(left, NW * rpw) : lpr;
        for (int it0 = 0; it0 < steps; it0 += U) {
          float x[U][CPL][VEC];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int r = (it0 + u) * rpw + sub;   // index slot
            const int32_t rr = __shfl(myrow, r & (ALTO_WAVE - 1));
            const bool ok = (it0 + u < steps) && b0 + ((it0 + u) * NW + w) * rpw + sub < ch.len;
            const float* src = srcp.pay_of(ok ? rr : row_safe);
#pragma unroll
            for (int q = 0; q < CPL; ++q) {
              const int col = col0 + cl + q * lpr;
              const bool okc = ok && col < C;
              const int colc = col < C ? col : C - 1;
              // payload rows are read once: non-temporal loads keep them from
              // displacing reusable lines in the caches
              if constexpr (VEC == 4) {
                const f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(src + (int64_t)colc * 4));
                x[u][q][0] = okc ? t[0] : 0.f;
                x[u][q][1] = okc ? t[1] : 0.f;
                x[u][q][2] = okc ? t[2] : 0.f;
                x[u][q][3] = okc ? t[3] : 0.f;
              } else {
                const float t = __builtin_nontemporal_load(src + colc);
                x[u][q][0] = okc ? t : 0.f;
              }
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < CPL; ++q)
#pragma unroll
              for (int v = 0; v < VEC; ++v) acc[q][v] += (double)x[u][q][v];
        }
      }
      // combine the sub-rows of the wave (lanes with equal cl), in a fixed order
      for (int o = lpr; o < ALTO_WAVE; o <<= 1)
#pragma unroll
        for (int q = 0; q < CPL; ++q)
#pragma unroll
          for (int v = 0; v < VEC; ++v) acc[q][v] += __shfl_xor(acc[q][v], o);
      if (sub == 0)
#pragma unroll
        for (int q = 0; q < CPL; ++q)
#pragma unroll
          for (int v = 0; v < VEC; ++v) red[w][(q * lpr + cl) * VEC + v] = acc[q][v];
      __syncthreads();
      const int ncol = lpr * CPL * VEC;
      for (int t = threadIdx.x; t < ncol; t += blockDim.x) {
        const int q = t / (lpr * VEC), rem = t % (lpr * VEC);
        const int col = col0 + q * lpr + rem / VEC;
        if (col >= C) continue;
        double s = 0.0;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) s += red[ww][t];
        const int64_t x = (int64_t)col * VEC + rem % VEC;
        if (ch.nch == 1) {
          if (ch.e < cap_groups) mean[ch.e * (int64_t)dim + x] = (float)(s / (double)ch.count);
        } else {
          part[(ch.part + ch.k) * (int64_t)dim + x] = s;
        }
      }
      __syncthreads();
    }
    __syncthreads();   // s_c is rewritten by the next ticket
  }
  // short groups: one wave each, assigned round robin (they have similar sizes, and
  // tickets would serialise on one counter: one atomic per short group)
  for (int64_t c = (int64_t)blockIdx.x * NW + w; c < NS; c += (int64_t)gridDim.x * NW) {
    const Chunk ch = chunks_s[c];
    mean_short_chunk<VEC, CPL, Src>(ch, srcp, dim, C, lpr, mean, cap_groups);
  }
}

// The means of the groups of several chunks (mean_combine_chunks).
__global__ __launch_bounds__(256) void k_mean_combine(const Chunk* __restrict__ chunks, const int64_t* nchunks,
                                                      const double* __restrict__ part, int dim, float* mean,
                                                      int64_t cap_groups) {
  mean_combine_chunks(chunks, *nchunks, part, dim, mean, cap_groups, blockIdx.x, gridDim.x);
}

__global__ void k_mask_out(LevelNodes L, const int64_t* Np, const uint64_t* __restrict__ keys, int shift,
                           uint64_t* mask_key, uint8_t* mask, int64_t cap_mask) {
  const int64_t N = *Np;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < N && u < cap_mask; u += (int64_t)gridDim.x * blockDim.x) {
    if (mask_key) mask_key[u] = key_prefix(keys[L.start[u]], shift);
    if (mask) mask[u] = L.ok[u];
  }
}

__global__ void k_record_keys(LevelNodes L, const int64_t* Np, const uint64_t* __restrict__ sk, int shift,
                              uint64_t* rkey) {
  const int64_t N = *Np;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < N; u += (int64_t)gridDim.x * blockDim.x)
    rkey[u] = key_prefix(sk[L.start[u]], shift);
}

inline bool src_rows_aligned16(const BatchSrc& s) { return (reinterpret_cast<uintptr_t>(s.pf) & 15) == 0; }
inline bool src_rows_aligned16(const MergedSrc& s) {
  return ((reinterpret_cast<uintptr_t>(s.spf) | reinterpret_cast<uintptr_t>(s.arena)) & 15) == 0;
}


}  // namespace

// ---------------------------------------------------------------------------
// workspace plan
// ---------------------------------------------------------------------------
void agg_levels(const KeyGeom& g, int La, int Lm, int Lr, int* Lt, int* Lseg) {
  *Lt = (Lm > 0 && Lm < La) ? Lm : La;
  *Lseg = Lr > *Lt ? Lr : *Lt;
}

void plan_buffers(const KeyGeom& g, int64_t n_max, const RouteGeom& rg, const alto_agg* agg, int Lr, WsCarver& c,
                  AggBufs& b, int64_t flow_cap) {
  memset(&b, 0, sizeof(b));
  const int64_t n = n_max < 1 ? 1 : n_max;
  b.ctl = c.take<SortCtl>(1);
  b.rctl = c.take<SortCtl>(1);
  b.fp_in = c.take<uint64_t>(ALTO_MAX_LEVELS + 1);
  b.fp_nodes = c.take<uint64_t>(ALTO_MAX_LEVELS + 1);
  b.nnodes = c.take<int64_t>(ALTO_MAX_LEVELS + 1);
  b.scal = c.take<int64_t>(8);
  b.prep_part = c.take<PrepPartial>(PREP_GRID);
  b.tmp_keys = c.take<uint64_t>(n);
  b.tmp_vals = c.take<uint32_t>(n);
  b.sk = c.take<uint64_t>(n);
  b.perm = c.take<uint32_t>(n);
  b.os_ntiles = sort_tiles(n);
  b.os_status = c.take<uint32_t>(2 * b.os_ntiles * SORT_BUCKETS);
  b.os_ctr = c.take<uint32_t>(SORT_MAX_PASSES);
  b.os_hist = c.take<uint32_t>((int64_t)SORT_MAX_PASSES * SORT_BUCKETS);
  b.scan_i32 = c.take<int32_t>(SCAN_MAX_BLOCKS + 1);
  b.scan_i64 = c.take<int64_t>(SCAN_MAX_BLOCKS + 1);
  b.gw = c.take<uint2>(cdiv(n, SEG_IT));
  memset(&b.fl, 0, sizeof(b.fl));
  if (n_max > SORT_SMALL_MAX && Lr >= 1) {
    // flows of the route level, ranked in (dest, prefix) order (packed sort)
    FlowBufs& f = b.fl;
    f.fcap = n < flow_cap ? n : flow_cap;
    int64_t h = 1024;
    while (h < 2 * f.fcap) h <<= 1;
    f.hcap = h;
    f.shift = g.shift[Lr];
    f.ib = bits_for(n - 1);
    f.ht_key = c.take<uint64_t>(h);
    f.ht_rank = c.take<uint32_t>(h);
    f.ct_key = c.take<uint64_t>(h);
    f.ct_rank = c.take<uint32_t>(h);
    f.drank = c.take<uint16_t>((int64_t)1 << FLOW_DIRECT_BITS);
    f.fdest = c.take<uint32_t>(f.fcap);
    f.ht_fan = c.take<uint32_t>(h);
    f.ht_anc = c.take<uint32_t>((int64_t)FLOW_EXACT_LEVELS * h);
    f.fbase = c.take<uint32_t>(f.fcap + 1);
    f.ctab_cap = n < ((int64_t)1 << 22) ? n : ((int64_t)1 << 22);
    f.ctab = c.take<uint64_t>(f.ctab_cap);
    // the child level (route level + 1); none when routing by the full key
    f.cshift = Lr < g.depth ? g.shift[Lr + 1] : 0;
    f.cmask = Lr < g.depth ? g.tagmask[Lr + 1] : 0u;
    f.child_ok = 0;                 // set per call
    f.flow_key = c.take<uint64_t>(f.fcap);
    f.flow_slot = c.take<uint32_t>(f.fcap);
    f.flow_sorted = c.take<uint64_t>(f.fcap);
    f.flow_order = c.take<uint32_t>(f.fcap);
    f.ftmp_keys = c.take<uint64_t>(f.fcap);
    f.ftmp_vals = c.take<uint32_t>(f.fcap);
    f.fctl = c.take<SortCtl>(1);
  }
  if (!agg) return;
  int Lt, Lseg;
  agg_levels(g, agg->level, agg->mask_level, Lr, &Lt, &Lseg);
  const int d = g.depth;
  if (b.fl.hcap && agg->level == Lr && d == Lr + 2 && (agg->mask_level == 0 || agg->mask_level <= agg->level)) {
    // direct placement: groups are the flows, leaves one level below their children
    FlowBufs& f = b.fl;
    f.mk_cap = n < ((int64_t)1 << 22) ? n : ((int64_t)1 << 22);
    f.mk_key = c.take<uint64_t>(f.mk_cap);
    f.mk_fan = c.take<uint32_t>(f.mk_cap);
    f.mk_cnt = c.take<uint32_t>(PREP_GRID);
    f.cfan = c.take<uint32_t>(f.ctab_cap);
    f.cmk = c.take<uint32_t>(f.ctab_cap);
    f.cbase = c.take<uint32_t>(f.ctab_cap + 1);
    f.dp_part = c.take<uint64_t>(3 * (DP_MAX_BLOCKS + 1));
  }
  for (int m = Lt; m < d; ++m) {
    LevelNodes& L = b.lv[m];
    L.start = c.take<int32_t>(n + 1);
    L.fc = c.take<int32_t>(n + 1);
    L.par = c.take<int32_t>(n);
    L.nfan = c.take<int32_t>(n);
    L.ok = c.take<uint8_t>(n);
    L.bad = c.take<uint8_t>(n);
  }
  if (Lt < Lseg) b.carry_fan = c.take<int32_t>((int64_t)(Lseg - Lt) * n);
  if (Lt < Lseg || agg->release == ALTO_RELEASE_IN_ORDER) {
    // node records re-sorted by key (a mask above the route level; release order)
    b.rkey = c.take<uint64_t>(n);
    b.rsk = c.take<uint64_t>(n);
    b.ridx = c.take<uint32_t>(n);
  }
  b.em = c.take<int32_t>(n + 1);
  b.tokc = c.take<int64_t>(n + 1);
  // long groups (more than MEAN_SMALL_ROWS rows) have at most n / MEAN_CHUNK_ROWS +
  // n / (MEAN_SMALL_ROWS + 1) chunks; short groups (one chunk each) at most n
  b.short_base = n / MEAN_CHUNK_ROWS + n / (MEAN_SMALL_ROWS + 1) + 1;
  b.chunks = c.take<Chunk>(b.short_base + n + 1);
  if (agg->op == ALTO_MEAN_F32) b.part = c.take<double>((2 * cdiv(n, MEAN_CHUNK_ROWS) + 2) * (int64_t)agg->dim);
}

// ---------------------------------------------------------------------------
// orchestration
// ---------------------------------------------------------------------------
int route_run(const KeyGeom& g, const RouteGeom& rg, const uint64_t* keys, int64_t n, AggBufs& b, int32_t* perm_out,
              int64_t* dest_offsets, int32_t* dest, const int32_t* fan, int64_t fan_ld, int flo, int fhi,
              int32_t* status, hipStream_t st, bool offsets_later, bool exact_flow_levels, bool allow_dp,
              const int64_t* n_dev) {
  // flows (packed sort) only when the sort runs its multi-block passes
  FlowBufs fl;
  if (n > SORT_SMALL_MAX) fl = b.fl;
  else memset(&fl, 0, sizeof(fl));
  // direct placement: the child level's counts (level depth - 1) are among those read
  fl.dp = (allow_dp && !n_dev && fl.hcap && fl.mk_key && fan && fhi == g.depth - 1 && flo <= fhi) ? 1 : 0;
  fl.dp_level = g.depth - 1;
  fl.fp_child = b.fp_nodes + (g.depth - 1);
  fl.fkey = g.fkey;
  b.fl.dp = fl.dp;
  // child ranks need the route level's declared child counts, read here when the
  // route level is among the levels whose counts are checked
  int fq = -1;
  for (int m = flo; fan && m <= fhi; ++m)
    if (rg.shift < 64 && g.shift[m] == rg.shift) fq = m - flo;
  fl.child_ok = (fl.hcap && fq >= 0 && fl.cmask != 0u) ? 1 : 0;
  // count levels that are functions of the flow (the route level and the ones
  // above it, at most FLOW_EXACT_LEVELS of them) are checked exactly per flow;
  // with exact_flow_levels they also leave the fingerprint
  int xhi = 0, xlo = 1;
  if (fl.hcap && fan && fhi >= flo && rg.shift < 64) {
    int lr = 0;   // the route level
    for (int m = 1; m <= g.depth; ++m)
      if (g.shift[m] == rg.shift) lr = m;
    xhi = lr < fhi ? lr : fhi;
    xlo = xhi - FLOW_EXACT_LEVELS + 1 > flo ? xhi - FLOW_EXACT_LEVELS + 1 : flo;
    if (xhi < flo) { xhi = 0; xlo = 1; }
    fl.x_route = (xhi == lr) ? 1 : 0;
  }
  const int nx = xhi >= xlo ? xhi - xlo + 1 : 0;
  b.fx_lo = exact_flow_levels ? xlo : 1;
  b.fx_hi = exact_flow_levels ? xhi : 0;
  // a call that fits one workgroup: the sort does the preparation too
  const bool small = n <= SORT_SMALL_MAX && !fl.hcap;
  if (!small) {
    ProfScope ps(PH_PREP, st);
    const int64_t cb = fl.hcap > 0 ? cdiv(fl.hcap, 256) : 1;
    k_route_init<<<(int)(cb < 2048 ? cb : 2048), 256, 0, st>>>(b.ctl, b.fp_in, b.fp_nodes, fl, n_dev, n, status);
    const int nl = fhi >= flo ? fhi - flo + 1 : 0;
    const int grid = grid_for(n, PREP_NT * PU, PREP_GRID);
    fl.mk_blocks = grid;
    fl.mk_per = fl.dp ? (int32_t)(fl.mk_cap / grid) : 0;
#define ALTO_PREP_CASE(NLV)                                                                                   \
  case NLV:                                                                                                   \
    k_prep<NLV><<<grid, PREP_NT, 0, st>>>(keys, n, g, rg, dest, fan, fan_ld, flo, fl, b.prep_part, xlo - flo, nx, \
                                          exact_flow_levels ? 1 : 0, n_dev);                                   \
    break;
    switch (nl) {
      ALTO_PREP_CASE(0) ALTO_PREP_CASE(1) ALTO_PREP_CASE(2) ALTO_PREP_CASE(3) ALTO_PREP_CASE(4)
      ALTO_PREP_CASE(5) ALTO_PREP_CASE(6) ALTO_PREP_CASE(7) ALTO_PREP_CASE(8) ALTO_PREP_CASE(9)
      ALTO_PREP_CASE(10) ALTO_PREP_CASE(11) ALTO_PREP_CASE(12) ALTO_PREP_CASE(13) ALTO_PREP_CASE(14)
      default: return ALTO_E_ARG;
    }
#undef ALTO_PREP_CASE
    k_prep_fold<<<1, 256, 0, st>>>(b.prep_part, grid, flo, nl, b.ctl, b.fp_in, status);
    if (exact_flow_levels && nx > 0)
      k_prep_fp<<<grid_for(n, 256 * 8, 2048), 256, 0, st>>>(keys, n, g, fan, fan_ld, xlo, xhi, b.ctl, b.fp_in, n_dev);
    ALTO_LAUNCH_CHECK();
  }
  ProfScope ps_sort(PH_SORT, st);
  SortBufs sb;
  memset(&sb, 0, sizeof(sb));
  sb.in_keys = keys;
  sb.tmp_keys = b.tmp_keys;
  sb.tmp_vals = b.tmp_vals;
  sb.out_keys = b.sk;
  sb.out_vals = perm_out ? reinterpret_cast<uint32_t*>(perm_out) : b.perm;
  sb.ctl = b.ctl;
  sb.fl = fl;
  sb.os_status = b.os_status;
  sb.os_ctr = b.os_ctr;
  sb.os_hist = b.os_hist;
  sb.os_ntiles = b.os_ntiles;
  sb.status = status;
  sb.dest_out = fl.hcap ? dest : nullptr;   // with flows the counting sweep writes them
  if (small) {
    sb.prep.ctl = b.ctl;
    sb.prep.fp_in = b.fp_in;
    sb.prep.fp_nodes = b.fp_nodes;
    sb.prep.fan = fan;
    sb.prep.fan_ld = fan_ld;
    sb.prep.flo = flo;
    sb.prep.fhi = fhi;
    sb.prep.dest = dest;
    sb.prep.status = status;
    sb.prep.g = g;
  }
  b.perm_used = sb.out_vals;
  int rc = sort_pairs(sb, n, n_dev, rg, g.total, true, st);
  if (rc) return rc;
  // destination offsets and duplicate keys; aggregation does both in its
  // segmentation pass over the same sorted keys
  if (!offsets_later) k_dest_offsets<<<grid_for(n, 256), 256, 0, st>>>(b.sk, n, rg, dest_offsets, status, n_dev);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

int aggregate_run(const KeyGeom& g, const RouteGeom& rg, int Lr, const alto_agg& agg, const uint64_t* keys,
                  const int32_t* fan, int64_t fan_ld, const int32_t* p32, const float* pf, int64_t n, AggBufs& b,
                  int32_t* perm_out, int64_t* dest_offsets, int32_t* dest, const GroupOut& out, int32_t* status,
                  hipStream_t st, const int64_t* n_dev, hipStream_t gather_st) {
  const int d = g.depth, La = agg.level, Lm = agg.mask_level;
  int Lt, Lseg;
  agg_levels(g, La, Lm, Lr, &Lt, &Lseg);
  ProfScope ps_total(PH_TOTAL, st);
  int rc = route_run(g, rg, keys, n, b, perm_out, dest_offsets, dest, fan, fan_ld, Lt, d - 1, status, st, true, true,
                     true, n_dev);
  if (rc) return rc;
  const uint32_t* perm = b.perm_used;
  prof_begin(PH_SEGMENT, st);
  if (b.fl.dp) {
    // direct placement chosen on the device: the group level from the child ranks
    // (the segmentation kernels below then return at once)
    k_dp_groups<<<grid_for(n, 256 * 16, 1024), 256, 0, st>>>(
        g, b.fl, b.ctl, n, La, b.lv[La], b.nnodes, dest_offsets, rg.num_dest, b.sk, perm, fan, fan_ld, Lt,
        (Lt < Lseg) ? b.carry_fan : nullptr, n < 1 ? 1 : n, b.fp_nodes, status,
        (agg.op == ALTO_MEAN_F32 ? out.mean == nullptr : out.tok == nullptr) ? 1 : 0);
  }

  // fragments: levels Lseg..d-1 are contiguous in (dest, key) order
  SegJob fj;
  memset(&fj, 0, sizeof(fj));
  fj.keys = b.sk;
  fj.idx = perm;
  fj.n_host = n;
  fj.n_dev = n_dev;
  fj.n_max = n;
  fj.elem_level = d;
  fj.lo = Lseg;
  fj.fan = fan;
  fj.fan_ld = fan_ld;
  fj.fan_base = 1;
  fj.check_dup = 1;
  fj.dest_offsets = dest_offsets;
  fj.rg = rg;
  fj.carry_lo = Lt;
  fj.carry_fan = (Lt < Lseg) ? b.carry_fan : nullptr;
  fj.carry_ld = n < 1 ? 1 : n;
  for (int m = 0; m <= ALTO_MAX_LEVELS; ++m) fj.lv[m] = b.lv[m];
  fj.nnodes = b.nnodes;
  fj.lb_status = b.os_status;
  fj.lb_ctr = b.os_ctr;
  fj.lb_tiles = b.os_ntiles * 2 * SORT_BUCKETS / SEG_LB_STRIDE;   // the sort's status words, free by now
  fj.fp_nodes = b.fp_nodes;
  fj.status = status;
  fj.skip_ctl = b.fl.dp ? b.ctl : nullptr;
  rc = seg_run(g, fj, st);
  if (rc) return rc;

  const int64_t* Mp = nullptr;
  if (Lm > 0 && Lm < Lseg) {
    // mask levels above the route level: node records of level Lseg, re-sorted by key
    const int64_t* Rp = b.nnodes + Lseg;
    k_record_keys<<<grid_for(n, 256), 256, 0, st>>>(b.lv[Lseg], Rp, b.sk, g.shift[Lseg], b.rkey);
    SortBufs rb;
    memset(&rb, 0, sizeof(rb));   // no flows: records sort by key only
    rb.in_keys = b.rkey;
    rb.tmp_keys = b.tmp_keys;
    rb.tmp_vals = b.tmp_vals;
    rb.out_keys = b.rsk;
    rb.out_vals = b.ridx;
    rb.ctl = b.rctl;
    rb.os_status = b.os_status;
    rb.os_ctr = b.os_ctr;
    rb.os_hist = b.os_hist;
    rb.os_ntiles = b.os_ntiles;
    rb.status = status;
    RouteGeom none;
    none.shift = 64;
    none.num_dest = 1;
    rc = sort_pairs(rb, n, Rp, none, g.total - g.shift[Lseg], false, st);
    if (rc) return rc;
    SegJob rj;
    memset(&rj, 0, sizeof(rj));
    rj.keys = b.rsk;
    rj.idx = b.ridx;
    rj.n_dev = Rp;
    rj.n_max = n;
    rj.elem_level = Lseg;
    rj.lo = Lt;
    rj.fan = b.carry_fan;
    rj.fan_ld = n < 1 ? 1 : n;
    rj.fan_base = Lt;
    rj.elem_ok = b.lv[Lseg].ok;
    rj.chain_check = 1;
    for (int m = 0; m <= ALTO_MAX_LEVELS; ++m) rj.lv[m] = b.lv[m];
    rj.nnodes = b.nnodes;
    rj.lb_status = b.os_status;
    rj.lb_ctr = b.os_ctr;
    rj.lb_tiles = b.os_ntiles * 2 * SORT_BUCKETS / SEG_LB_STRIDE;   // the sort's status words, free by now
    rj.status = status;
    rc = seg_run(g, rj, st);
    if (rc) return rc;
    Mp = b.nnodes + Lm;
    k_mask_out<<<grid_for(n, 256), 256, 0, st>>>(b.lv[Lm], Mp, b.rsk, g.shift[Lm] - g.shift[Lseg], out.mask_key,
                                                 out.mask, out.cap_mask);
  } else if (Lm > 0) {
    Mp = b.nnodes + Lm;
    k_mask_out<<<grid_for(n, 256), 256, 0, st>>>(b.lv[Lm], Mp, b.sk, g.shift[Lm], out.mask_key, out.mask, out.cap_mask);
  }
  prof_end(PH_SEGMENT, st);

  // groups (their record kernel also compares the fan fingerprints)
  GroupsExtra ex;
  memset(&ex, 0, sizeof(ex));
  ex.fp_in = b.fp_in;
  ex.fp_nodes = b.fp_nodes;
  ex.flo = Lt;
  ex.fhi = d - 1;
  ex.xlo = b.fx_lo;
  ex.xhi = b.fx_hi;
  ex.ctl = b.ctl;
  ex.gather_st = gather_st;
  BatchSrc src{perm, p32, fan, fan_ld, pf, agg.dim, n, status};
  return groups_run<BatchSrc>(g, rg, agg, src, b.sk, n, b, Mp, out, status, st, &ex);
}

template <typename Src>
int groups_run(const KeyGeom& g, const RouteGeom& rg, const alto_agg& agg, const Src& src, const uint64_t* sk,
               int64_t n_max, AggBufs& b, const int64_t* Mp, const GroupOut& out, int32_t* status, hipStream_t st,
               const GroupsExtra* ex) {
  const int La = agg.level;
  const int64_t n = n_max;
  prof_begin(PH_GROUPS, st);
  const int64_t* Gp = b.nnodes + La;
  const LevelNodes& GL = b.lv[La];
  GroupsExtra none;
  memset(&none, 0, sizeof(none));
  const GroupsExtra& x = ex ? *ex : none;
  // the sort's status words and a ticket word are free by now (or the caller's)
  uint64_t* gst = x.gst ? x.gst : reinterpret_cast<uint64_t*>(b.os_status);
  uint32_t* gctr = x.gctr ? x.gctr : b.os_ctr;
  {
    const int64_t tiles = cdiv(n + 1, GS_TILE);
    const int64_t xwords = x.xst ? cdiv(n + 1, x.xtile) * x.xper : 0;   // the caller's, after ours
    if (!x.gst && (tiles * GS_NV + xwords) * 2 > (int64_t)b.os_ntiles * 2 * SORT_BUCKETS)
      return ALTO_E_ARG;   // never: words to spare
    const int64_t pb = cdiv(tiles * GS_NV, 256);
    if (!x.cleared) k_group_scan_prep<<<(int)(pb < 1024 ? pb : 1024), 256, 0, st>>>(Gp, gst, gctr, x);
    GroupFold f{x.fold, x.fold_leafy, x.fold_level, x.fold_es, g.fkey, x.fold_keys, x.fold_fp};
    k_groups<Src><<<grid_for(n + 1, GS_TILE, 1024), GS_NT, 0, st>>>(
        g, rg, La, GL, Gp, sk, src, b.chunks, b.short_base, MEAN_CHUNK_ROWS, out, agg.op == ALTO_CONCAT_I32 ? 1 : 0,
        Mp, b.scal, x, gst, gctr, f, n, status);
  }
  ALTO_LAUNCH_CHECK();
  prof_end(PH_GROUPS, st);
  // the gathers, on another stream if asked (after the records, through an event
  // that is released once the device has passed it)
  if (x.gather_st && x.gather_st != st) {
    hipEvent_t ev;
    if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return ALTO_E_HIP;
    const bool ok = hipEventRecord(ev, st) == hipSuccess && hipStreamWaitEvent(x.gather_st, ev, 0) == hipSuccess;
    (void)hipEventDestroy(ev);
    if (!ok) return ALTO_E_HIP;
    st = x.gather_st;
  }
  ProfScope ps_gather(PH_GATHER, st);
  const int64_t* NBp = b.scal + 1;   // chunks of long groups
  const int64_t* NSp = b.scal + 3;   // short groups (one chunk each, from short_base)
  if (agg.op == ALTO_CONCAT_I32) {
    if (out.tok && !x.defer_concat)
      k_concat<Src><<<GRID_CAP, 256, 0, st>>>(b.chunks, NBp, b.chunks + b.short_base, NSp, src, out.tok,
                                              out.cap_tokens);
  } else if (out.mean) {
    const int dim = agg.dim;
    const bool v4 = (dim % 4 == 0) && src_rows_aligned16(src);
    const int C = v4 ? dim / 4 : dim;
    int lpr = 1;
    while (lpr < C && lpr < 64) lpr <<= 1;
    const int cpl_need = (int)cdiv(C, lpr);
    const int cpl = cpl_need >= 4 ? 4 : cpl_need;
    const int grid = MEAN_GRID;   // persistent: chunks by ticket
#define ALTO_MEAN_CASE(V, P)                                                                                 \
  do {                                                                                                       \
    ProfScope ps_mean(PH_MEAN, st);                                                                          \
    k_mean<V, P, Src><<<grid, 256, 0, st>>>(b.chunks, NBp, b.chunks + b.short_base, NSp, src, dim, lpr, b.part, \
                                            out.mean, out.cap_groups,                                          \
                                            reinterpret_cast<unsigned long long*>(b.scal + 2));                \
  } while (0)
    if (v4) {
      if (cpl == 1) ALTO_MEAN_CASE(4, 1);
      else if (cpl == 2) ALTO_MEAN_CASE(4, 2);
      else if (cpl == 3) ALTO_MEAN_CASE(4, 3);
      else ALTO_MEAN_CASE(4, 4);
    } else {
      if (cpl == 1) ALTO_MEAN_CASE(1, 1);
      else if (cpl == 2) ALTO_MEAN_CASE(1, 2);
      else if (cpl == 3) ALTO_MEAN_CASE(1, 3);
      else ALTO_MEAN_CASE(1, 4);
    }
#undef ALTO_MEAN_CASE
    if (!x.defer_combine)
      k_mean_combine<<<GRID_CAP, 256, 0, st>>>(b.chunks, NBp, b.part, dim, out.mean, out.cap_groups);
  }
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

template int groups_run<BatchSrc>(const KeyGeom&, const RouteGeom&, const alto_agg&, const BatchSrc&, const uint64_t*,
                                  int64_t, AggBufs&, const int64_t*, const GroupOut&, int32_t*, hipStream_t,
                                  const GroupsExtra*);
template int groups_run<MergedSrc>(const KeyGeom&, const RouteGeom&, const alto_agg&, const MergedSrc&,
                                   const uint64_t*, int64_t, AggBufs&, const int64_t*, const GroupOut&, int32_t*,
                                   hipStream_t, const GroupsExtra*);

namespace {
__global__ void k_empty(GroupOut out, int64_t* offs, int num_dest) {
  for (int i = threadIdx.x; i <= num_dest; i += blockDim.x)
    if (offs) offs[i] = 0;
  if (threadIdx.x == 0) {
    out.counts[0] = out.counts[1] = out.counts[2] = out.counts[3] = 0;
    if (out.tok_off) out.tok_off[0] = 0;
  }
}
}  // namespace

void empty_outputs(const GroupOut& out, int64_t* dest_offsets, int num_dest, hipStream_t st) {
  k_empty<<<1, 256, 0, st>>>(out, dest_offsets, num_dest);
}

namespace {
__global__ void k_zero_offsets(int64_t* offs, int num_dest) {
  for (int i = threadIdx.x; i <= num_dest; i += blockDim.x) offs[i] = 0;
}
}  // namespace

void zero_offsets(int64_t* dest_offsets, int num_dest, hipStream_t st) {
  if (dest_offsets) k_zero_offsets<<<1, 256, 0, st>>>(dest_offsets, num_dest);
}

