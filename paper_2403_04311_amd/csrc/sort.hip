// LSD radix sort of (uint64 key, uint32 value) pairs by (destination, key), and a
// device-wide exclusive scan.
//
// The sort realises the order of Sections 3.2 and 4.1 of the paper (elements of a
// parallelised stream are put back in their original order) inside each
// destination of Section 4.3. Each pass sorts stably by one 8-bit digit taken from
// a window of key bits or of destination bits; windows are placed on device over
// the bits that actually vary across the input (OR xor AND of all keys), so a
// layout with sparse tags costs only the passes its data needs. Within a block,
// digits are ranked stably with wavefront ballots (8 ballots give the lanes holding
// the same digit; mbcnt-style popcount gives the rank), then the tile is staged in
// LDS in digit order so that the global scatter writes contiguous runs.
#include "sort.h"

#include <string.h>

namespace {

constexpr int NT = SORT_NT;
constexpr int IT = SORT_IT;
constexpr int OS_IT = SORT_OS_IT;
constexpr int OS_TILE = SORT_OS_TILE;
constexpr int TILE = SORT_TILE;
constexpr int NW = NT / ALTO_WAVE;

__device__ inline int64_t load_n(int64_t n_host, const int64_t* n_dev) { return n_dev ? *n_dev : n_host; }

__global__ void k_sort_init(SortCtl* ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
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
}

// OR / AND of the keys and destinations (which bits vary). Waves reduce with shuffles, blocks in
// LDS, and each block adds one atomic per value: the four words are shared by the
// whole grid, and same-address atomics serialise.
__global__ __launch_bounds__(256) void k_sort_reduce(const uint64_t* __restrict__ keys, int64_t n_host,
                                                     const int64_t* n_dev, RouteGeom rg, SortCtl* ctl) {
  __shared__ uint64_t s_or[256 / ALTO_WAVE], s_and[256 / ALTO_WAVE];
  __shared__ uint32_t s_dor[256 / ALTO_WAVE], s_dand[256 / ALTO_WAVE];
  const int64_t n = load_n(n_host, n_dev);
  if ((int64_t)blockIdx.x * blockDim.x >= n) return;   // block-uniform
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u;
#pragma unroll 4
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    uint64_t k = keys[i];
    kor |= k;
    kand &= k;
    uint32_t d = dest_of_key(rg, k);
    dor |= d;
    dand &= d;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kor |= __shfl_xor(kor, o);
    kand &= __shfl_xor(kand, o);
    dor |= __shfl_xor(dor, o);
    dand &= __shfl_xor(dand, o);
  }
  const int w = threadIdx.x / ALTO_WAVE;
  if (lane_id() == 0) {
    s_or[w] = kor;
    s_and[w] = kand;
    s_dor[w] = dor;
    s_dand[w] = dand;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int v = 1; v < 256 / ALTO_WAVE; ++v) {
      kor |= s_or[v];
      kand &= s_and[v];
      dor |= s_dor[v];
      dand &= s_dand[v];
    }
    atomicOr((unsigned long long*)&ctl->key_or, (unsigned long long)kor);
    atomicAnd((unsigned long long*)&ctl->key_and, (unsigned long long)kand);
    atomicOr(&ctl->dest_or, dor);
    atomicAnd(&ctl->dest_and, dand);
  }
}

__device__ inline int greedy_windows(uint64_t v, int limit, int from_dest, SortPass* out, int np) {
  const int start = np;
  while (v && np < start + limit) {
    const int lo = __builtin_ctzll(v);
    out[np].from_dest = from_dest;
    out[np].lo = lo;
    ++np;
    v = (lo + SORT_RADIX >= 64) ? 0ull : (v & ~((1ull << (lo + SORT_RADIX)) - 1ull));
  }
  return np;
}

// Digit windows: a greedy cover of the varying bits with 8-bit windows (optimal
// for fixed-width interval cover). General mode: key windows, then destination
// windows. Packed mode: windows over the (flow rank, suffix) bits. Then the buffer
// ping-pong so that the last pass lands in the final buffers. With a device-side
// count of at most SORT_SMALL_MAX the one-workgroup sort has done the work.
__global__ void k_sort_plan(SortCtl* ctl, int64_t n_host, const int64_t* n_dev, int max_key_windows,
                            int max_dest_windows, int packed_slots) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int64_t n = load_n(n_host, n_dev);
  SortPlan p;
  SortPass win[SORT_MAX_PASSES];
  int np = 0;
  p.idle = (n_dev && n <= SORT_SMALL_MAX) ? 1 : 0;
  const bool packed = ctl->mode == SORT_PACKED;
  p.direct = (packed && ctl->cmode && ctl->dp && !p.idle) ? 1 : 0;
  if (!p.idle) {
    if (packed) {
      const int S = ctl->sbits, R = ctl->rbits;
      // with direct placement the leaf tags (the suffix bits) are not sorted: the
      // last pass puts each element at its child's start + its tag
      uint64_t vs = p.direct ? 0ull : (ctl->key_or ^ ctl->key_and) & (S >= 64 ? ~0ull : ((1ull << S) - 1ull));
      uint64_t vr = R > 0 ? (((1ull << R) - 1ull) << S) : 0ull;
      np = greedy_windows(vs | vr, SORT_MAX_PASSES, 0, win, np);
      if (np == 0) p.direct = 0;
    } else {
      np = greedy_windows(ctl->key_or ^ ctl->key_and, max_key_windows, 0, win, np);
      np = greedy_windows((uint64_t)(ctl->dest_or ^ ctl->dest_and), max_dest_windows, 1, win, np);
    }
  }
  // packed passes end at the host's last packed slot, whose kernel also unpacks
  const int first = (packed && packed_slots >= np) ? packed_slots - np : 0;
  for (int k = 0; k < SORT_MAX_PASSES; ++k) {
    p.pass[k].active = 0;
    p.pass[k].src = p.pass[k].dst = 0;
    p.pass[k].from_dest = p.pass[k].lo = 0;
  }
  for (int k = 0; k < np; ++k) {
    SortPass& q = p.pass[first + k];
    q.active = 1;
    q.from_dest = win[k].from_dest;
    q.lo = win[k].lo;
    q.dst = ((np - 1 - k) % 2 == 0) ? SORT_BUF_FINAL : SORT_BUF_TMP;
    q.src = (k == 0) ? SORT_BUF_INPUT : p.pass[first + k - 1].dst;
  }
  p.npass = np;
  p.first = first;
  ctl->plan = p;
}

__device__ inline uint32_t digit_of(const SortPass& ps, const RouteGeom& rg, uint64_t k) {
  uint64_t src = ps.from_dest ? (uint64_t)dest_of_key(rg, k) : k;
  return (uint32_t)((src >> ps.lo) & (SORT_BUCKETS - 1));
}

// ---- flows (packed mode) ----------------------------------------------------
// Compact rank table: the ranked flows in a table of about twice their number, so
// that the lookups of the first pass stay in the caches.
__global__ void k_ct_insert(FlowBufs fl, const SortCtl* ctl, uint32_t num_dest) {
  const int64_t F = ctl->nflows_c;
  const uint64_t mask = (uint64_t)ctl->ct_mask;
  const int dlo = ctl->dlo, dbits = ctl->dbits;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < F; r += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t p = fl.flow_sorted[r];
    fl.fdest[r] = fl.rank_dest ? (uint32_t)r : dest_of_prefix(p, num_dest);
    if (dbits >= 0) {
      fl.drank[(p >> dlo) & ((1ull << dbits) - 1ull)] = (uint16_t)r;
      continue;
    }
    uint64_t h = mix64(p ^ 0xD6E8FEB86659FD93ull) & mask;
    for (uint64_t probe = 0; probe <= mask; ++probe) {
      const uint64_t old = atomicCAS((unsigned long long*)&fl.ct_key[h], ~0ull, (unsigned long long)p);
      if (old == ~0ull) {
        fl.ct_rank[h] = (uint32_t)r;
        break;
      }
      h = (h + 1) & mask;
    }
  }
}

// Compaction of the flow set; one atomic per wave.
__global__ __launch_bounds__(256) void k_flow_compact(FlowBufs fl, SortCtl* ctl) {
  for (int64_t base = (int64_t)blockIdx.x * blockDim.x; base < fl.hcap; base += (int64_t)gridDim.x * blockDim.x) {
    const int64_t s = base + threadIdx.x;
    const uint64_t v = s < fl.hcap ? fl.ht_key[s] : ~0ull;
    const bool has = v != ~0ull;
    const uint64_t ball = __ballot(has);
    int64_t first = 0;
    if (lane_id() == 0 && ball) first = (int64_t)atomicAdd((unsigned long long*)&ctl->nflows, (unsigned long long)__popcll(ball));
    first = __shfl(first, 0);
    if (has) {
      const int64_t i = first + __popcll(ball & lanemask_lt());
      if (i < fl.fcap) {
        fl.flow_key[i] = v;
        fl.flow_slot[i] = (uint32_t)s;
      }
    }
  }
}

__global__ void k_flow_count(FlowBufs fl, SortCtl* ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    const int64_t F = ctl->nflows;
    ctl->nflows_c = F < fl.fcap ? F : fl.fcap;
    if (F > fl.fcap) ctl->flow_overflow = 1;
  }
}

// Rank of every flow in (destination, prefix) order, and the choice of mode.
__global__ void k_flow_rank(FlowBufs fl, SortCtl* ctl, int64_t n, int allow_packed) {
  const int64_t F = ctl->nflows_c;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < F; r += (int64_t)gridDim.x * blockDim.x)
    fl.ht_rank[fl.flow_slot[fl.flow_order[r]]] = (uint32_t)r;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    int R = 0;
    while (R < 63 && ((int64_t)1 << R) < F) ++R;
    const bool fits = allow_packed && !ctl->flow_overflow && ctl->nflows <= fl.fcap && F >= 1 &&
                      R + fl.shift + fl.ib <= 64;
    ctl->mode = fits ? SORT_PACKED : SORT_GENERAL;
    int64_t t = 64;
    while (t < 2 * F && t < fl.hcap) t <<= 1;
    ctl->ct_mask = t - 1;
    // prefixes whose varying bits span at most FLOW_DIRECT_BITS bits index a direct
    // table (a prefix is fixed by those bits, the others being common to all keys)
    const uint64_t vm = fl.shift >= 64 ? 0ull : ((ctl->key_or ^ ctl->key_and) >> fl.shift);
    const int lo = vm ? __builtin_ctzll(vm) : 0;
    const int span = vm ? 64 - __builtin_clzll(vm) - lo : 0;
    ctl->dlo = lo;
    ctl->dbits = span <= FLOW_DIRECT_BITS ? span : -1;
    ctl->rbits = R;
    ctl->sbits = fl.shift;
    ctl->ib = fl.ib;
  }
}

// Child ranks (packed mode with a direct rank table): the children of flow r (the
// nodes one level below the route level) take the ranks fbase[r] .. fbase[r] +
// count - 1 in tag order, with count the flow's declared child count. A packed word
// then holds (child rank | key bits below the child level | index): the ranks of
// all children together need fewer bits than (flow rank, child tag), since a tag
// field must hold the largest child count. Used when every count is >= 1, the
// ranks fit the lookup table and the word fits 64 bits; a child tag >= its declared
// count is a FANOUT error, reported by the input pass (the order is then undefined).
// One workgroup; flows <= 2^FLOW_DIRECT_BITS here.
__global__ __launch_bounds__(1024) void k_flow_base(FlowBufs fl, SortCtl* ctl) {
  __shared__ uint32_t s_w[1024 / ALTO_WAVE];
  __shared__ int s_bad;
  if (threadIdx.x == 0) {
    ctl->cmode = 0;
    s_bad = 0;
  }
  __syncthreads();
  if (ctl->mode != SORT_PACKED || ctl->dbits < 0 || !fl.child_ok) return;   // uniform
  const int F = (int)ctl->nflows_c;   // <= 2^FLOW_DIRECT_BITS = 4 per thread
  uint32_t c[4], sum = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = threadIdx.x * 4 + k;
    c[k] = r < F ? fl.ht_fan[fl.flow_slot[fl.flow_order[r]]] : 0u;
    if (r < F && (c[k] < 1u || c[k] > (1u << 24))) s_bad = 1;
    sum += c[k];
  }
  uint32_t tot;
  uint32_t run = block_excl_scan<uint32_t, 1024>(sum, s_w, &tot);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = threadIdx.x * 4 + k;
    if (r < F) fl.fbase[r] = run;
    run += c[k];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    fl.fbase[F] = tot;
    int R = 0;
    while (R < 63 && ((int64_t)1 << R) < (int64_t)tot) ++R;
    if (!s_bad && (int64_t)tot <= fl.ctab_cap && R + fl.cshift + fl.ib <= 64) {
      ctl->cmode = 1;
      ctl->ctotal = tot;
      ctl->rbits = R;
      ctl->sbits = fl.cshift;
    }
  }
}

// Child rank -> the key's bits above the child level's suffix (child-rank packing):
// the flow r is the last whose first child rank is <= t (binary search over fbase),
// the child tag is t - fbase[r]; the last pass then rebuilds a key with one lookup.
__global__ void k_ctab_fill(FlowBufs fl, const SortCtl* ctl) {
  if (!ctl->cmode) return;
  const int64_t C = ctl->ctotal;
  const int F = (int)ctl->nflows_c;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < C; t += (int64_t)gridDim.x * blockDim.x) {
    int lo = 0, hi = F - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((int64_t)fl.fbase[mid] <= t) lo = mid; else hi = mid - 1;
    }
    fl.ctab[t] = (fl.flow_sorted[lo] << fl.shift) | ((uint64_t)(t - fl.fbase[lo]) << fl.cshift);
    if (fl.dp) {
      fl.cfan[t] = 0u;
      fl.cmk[t] = 0u;
    }
  }
}

// ---- direct placement (see FlowBufs.dp) --------------------------------------
// The markers into the child-rank table: declared count (one marker's) and the
// number of markers per child rank.
__global__ __launch_bounds__(256) void k_dp_table(FlowBufs fl, const SortCtl* ctl) {
  if (!ctl->cmode || ctl->mode != SORT_PACKED || ctl->dbits < 0 || fl.mk_per <= 0) return;
  const int64_t C = ctl->ctotal, F = ctl->nflows_c;
  const uint64_t dm = (1ull << ctl->dbits) - 1ull;
  const int dlo = ctl->dlo;
  // one block per region of the input pass, over its markers only
  for (int blk = blockIdx.x; blk < fl.mk_blocks; blk += gridDim.x) {
    const uint32_t mc = fl.mk_cnt[blk] < (uint32_t)fl.mk_per ? fl.mk_cnt[blk] : (uint32_t)fl.mk_per;
    for (uint32_t i = threadIdx.x; i < mc; i += blockDim.x) {
      const int64_t j = (int64_t)blk * fl.mk_per + i;
      const uint64_t k = fl.mk_key[j];
      const uint64_t pfx = k >> fl.shift;
      const uint32_t r = fl.drank[(pfx >> dlo) & dm];
      if ((int64_t)r >= F || fl.flow_sorted[r] != pfx) continue;   // a key of no flow: the input had errors
      const uint32_t tag = (uint32_t)((k >> fl.cshift) & fl.cmask);
      const uint64_t cr = (uint64_t)fl.fbase[r] + tag;
      if (tag >= fl.fbase[r + 1] - fl.fbase[r] || (int64_t)cr >= C) continue;   // a FANOUT error (input pass)
      fl.cfan[cr] = fl.mk_fan[j];
      atomicAdd(&fl.cmk[cr], 1u);
    }
  }
}

// Per block of DP_CHUNK child ranks: the sum of declared counts, whether some rank
// has no or several markers, and the node side of the child level's fingerprint
// (each complete child contributes its count x its term). dp_part holds three
// arrays of DP_MAX_BLOCKS + 1 words.
__global__ __launch_bounds__(256) void k_dp_sums(FlowBufs fl, const SortCtl* ctl) {
  if (!ctl->cmode || ctl->mode != SORT_PACKED || ctl->dbits < 0) return;
  const int64_t C = ctl->ctotal;
  const int64_t nb = cdiv(C, DP_CHUNK);
  __shared__ uint64_t s_s[256 / ALTO_WAVE], s_f[256 / ALTO_WAVE];
  __shared__ uint32_t s_b[256 / ALTO_WAVE];
  for (int64_t blk = blockIdx.x; blk < nb; blk += gridDim.x) {
    uint64_t sum = 0, fp = 0;
    uint32_t bad = 0;
    const int64_t c1 = (blk + 1) * DP_CHUNK < C ? (blk + 1) * DP_CHUNK : C;
    for (int64_t c = blk * DP_CHUNK + threadIdx.x; c < c1; c += blockDim.x) {
      const uint32_t f = fl.cfan[c];
      sum += f;
      bad |= fl.cmk[c] != 1u;
      fp += (uint64_t)f * fan_term(fl.fkey, fl.dp_level, fl.ctab[c] >> fl.cshift, f);
    }
    sum = wave_sum(sum);
    fp = wave_sum(fp);
    const uint64_t ball = __ballot(bad != 0);
    const int w = threadIdx.x / ALTO_WAVE;
    if (lane_id() == 0) {
      s_s[w] = sum;
      s_f[w] = fp;
      s_b[w] = ball ? 1u : 0u;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      uint64_t ts = 0, tf = 0;
      uint32_t tb = 0;
      for (int i = 0; i < 256 / ALTO_WAVE; ++i) {
        ts += s_s[i];
        tf += s_f[i];
        tb |= s_b[i];
      }
      fl.dp_part[blk] = ts;
      fl.dp_part[(DP_MAX_BLOCKS + 1) + blk] = tb;
      fl.dp_part[2 * (DP_MAX_BLOCKS + 1) + blk] = tf;
    }
    __syncthreads();
  }
}

// One block: the block sums become exclusive block prefixes, and the choice. Direct
// placement needs child ranks, at most mk_cap markers, exactly one marker per child
// rank (ctotal of them) and declared counts adding up to n.
__global__ __launch_bounds__(1024) void k_dp_decide(FlowBufs fl, SortCtl* ctl, int64_t n) {
  __shared__ uint64_t s_w[1024 / ALTO_WAVE];
  __shared__ uint32_t s_bad;
  const bool can = ctl->cmode && ctl->mode == SORT_PACKED && ctl->dbits >= 0;
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  if (!can) {
    if (threadIdx.x == 0) ctl->dp = 0;
    return;
  }
  const int64_t C = ctl->ctotal;
  const int nb = (int)cdiv(C, DP_CHUNK);   // <= DP_MAX_BLOCKS = the block size
  const int b = threadIdx.x;
  const uint64_t v = b < nb ? fl.dp_part[b] : 0ull;
  const uint64_t f = b < nb ? fl.dp_part[2 * (DP_MAX_BLOCKS + 1) + b] : 0ull;
  if (b < nb && fl.dp_part[(DP_MAX_BLOCKS + 1) + b]) s_bad = 1u;
  uint64_t tot;
  const uint64_t ex = block_excl_scan<uint64_t, 1024>(v, s_w, &tot);
  __syncthreads();
  uint64_t ftot;
  (void)block_excl_scan<uint64_t, 1024>(f, s_w, &ftot);
  if (b < nb) fl.dp_part[b] = ex;
  // markers: every block within its region, C of them in all
  __shared__ uint64_t s_m;
  __shared__ uint32_t s_over;
  if (threadIdx.x == 0) {
    s_m = 0;
    s_over = 0;
  }
  __syncthreads();
  if (threadIdx.x < fl.mk_blocks) {
    const uint32_t mc = fl.mk_cnt[threadIdx.x];
    atomicAdd((unsigned long long*)&s_m, (unsigned long long)mc);
    if (mc > (uint32_t)fl.mk_per) s_over = 1u;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint64_t m = s_m;
    const bool ok = C >= 1 && !s_bad && !s_over && m == (uint64_t)C && tot == (uint64_t)n;
    ctl->dp = ok ? 1 : 0;
    if (ok) {
      fl.cbase[C] = (uint32_t)n;
      *fl.fp_child = ftot;
    }
  }
}

// cbase: exclusive scan of the declared counts over child ranks (direct placement).
__global__ __launch_bounds__(256) void k_dp_base(FlowBufs fl, const SortCtl* ctl) {
  if (!ctl->dp) return;
  constexpr int PER = DP_CHUNK / 256;
  const int64_t C = ctl->ctotal;
  const int64_t nb = cdiv(C, DP_CHUNK);
  __shared__ uint32_t s_w[256 / ALTO_WAVE];
  for (int64_t blk = blockIdx.x; blk < nb; blk += gridDim.x) {
    const int64_t c0 = blk * DP_CHUNK + (int64_t)threadIdx.x * PER;
    uint32_t v[PER], sum = 0;
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      v[k] = c0 + k < C ? fl.cfan[c0 + k] : 0u;
      sum += v[k];
    }
    uint32_t tot;
    uint32_t run = (uint32_t)fl.dp_part[blk] + block_excl_scan<uint32_t, 256>(sum, s_w, &tot);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      if (c0 + k < C) fl.cbase[c0 + k] = run;
      run += v[k];
    }
    __syncthreads();
  }
}

// What a pass kernel needs from the control block (kept in scalars, not a copy of
// the whole block).
struct PassView {
  SortPass ps;
  int32_t mode, ib, sbits, npass;
  int32_t dlo, dbits;
  int32_t cmode;
  int32_t first;
  int32_t direct;
  uint64_t ct_mask;
  uint64_t ctotal;
};

__device__ inline PassView read_pass(const SortCtl* ctl, int slot) {
  PassView v;
  v.ps = ctl->plan.pass[slot];
  v.mode = ctl->mode;
  v.ib = ctl->ib;
  v.sbits = ctl->sbits;
  v.npass = ctl->plan.npass;
  v.ct_mask = (uint64_t)ctl->ct_mask;
  v.dlo = ctl->dlo;
  v.dbits = ctl->dbits;
  v.cmode = ctl->cmode;
  v.first = ctl->plan.first;
  v.direct = ctl->plan.direct;
  v.ctotal = (uint64_t)ctl->ctotal;
  return v;
}

__device__ inline uint64_t unpack_key(const FlowBufs& fl, const uint64_t* flow_sorted, const PassView& c,
                                      uint64_t e) {
  const int S = c.sbits, hi = S + c.ib;
  const uint64_t top = hi >= 64 ? 0ull : (e >> hi);
  const uint64_t suffix = S == 0 ? 0ull : ((e >> c.ib) & ((1ull << S) - 1ull));
  // child rank -> (prefix, child tag); a rank past the table comes only from a child
  // tag beyond its declared count (a FANOUT error, order undefined): kept in bounds
  if (c.cmode) return fl.ctab[top < c.ctotal ? top : 0] | suffix;
  return (flow_sorted[top] << S) | suffix;
}

// A pointer value hidden from the optimiser: selecting between buffers of the
// by-value argument struct then selects values, not addresses inside the struct
// (which would force a copy of the struct into scratch memory). The pointers are
// device (global) memory.
template <typename T>
__device__ inline T* opaque(T* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  // rebuilt as a global-memory pointer, so that accesses stay global (not flat)
  typedef __attribute__((address_space(1))) T GlobalT;
  return (T*)(GlobalT*)(((uint64_t)hi << 32) | lo);
}

// Stable in-wave ranking of one row of 64 digits: the lane mask of the valid lanes
// holding the same digit as this lane. Per digit bit, one ballot; each lane keeps
// the OR over bits of (ballot XOR its own bit spread over 32 lanes), a lane whose
// bits all agree being a peer. One v_bitop3 per half-mask (truth table 0xF6 is
// a | (b ^ c), with the operands weighted 0xF0, 0xCC, 0xAA).
__device__ inline uint64_t match_digit(uint32_t dig, bool valid) {
  uint32_t lo = 0, hi = 0;
#pragma unroll
  for (int b = 0; b < SORT_RADIX; ++b) {
    const uint32_t sx = (uint32_t)((int32_t)(dig << (31 - b)) >> 31);   // 0 or ~0
    const uint64_t m = __ballot(sx != 0);
    lo = __builtin_amdgcn_bitop3_b32(lo, (uint32_t)m, sx, 0xF6);
    hi = __builtin_amdgcn_bitop3_b32(hi, (uint32_t)(m >> 32), sx, 0xF6);
  }
  return __ballot(valid) & ~(((uint64_t)hi << 32) | lo);
}

// Stable in-wave rank of one row of 64 digits against the wave's running digit
// counters `cnt` (LDS): the number of earlier elements with the same digit (rows
// before this one, then lower lanes of this row); the counters advance past the
// row. Every lane reads its digit's counter before the lowest lane of each digit
// writes it back (one instruction after the other, in the wave's order), so no
// broadcast is needed. Invalid lanes (digit 0) read but neither count nor write.
__device__ inline uint32_t wave_rank(uint16_t* cnt, uint32_t dig, bool valid) {
  const uint64_t peers = match_digit(dig, valid);
  const uint32_t below =
      __builtin_amdgcn_mbcnt_hi((uint32_t)(peers >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)peers, 0u));
  const uint32_t old = cnt[dig];
  if (valid && below == 0) cnt[dig] = (uint16_t)(old + (uint32_t)__popcll(peers));
  return old + below;
}

// ---- packed passes: one 64-bit word per element, (rank | suffix | index) --------
// The digit is a plain bit field of the word, so LDS holds only the staged words and
// 16-bit per-wave counters. The words are composed once from the input keys and
// staged in the ping-pong buffer that the first pass does not write.
// Packs IT input keys with their ranks: the first probe of every item is issued
// before any is resolved (independent loads), collisions are resolved afterwards.
template <int NI>
__device__ inline void pack_items(const SortBufs& b, const PassView& c, const int64_t* gi, int64_t n,
                                  const uint64_t* key, uint64_t* out, const uint16_t* s_drank, const uint32_t* s_fbase,
                                  uint32_t* rank_out) {
  const int S = c.sbits;
  const int hi = S + c.ib;
  if (s_drank) {
    // direct table in LDS; with child ranks, S is the bits below the child level and
    // the route prefix sits above the child tag
    const uint64_t dm = (1ull << c.dbits) - 1ull;
    const int SR = c.cmode ? b.fl.shift : S;   // bits below the route level
#pragma unroll
    for (int j = 0; j < NI; ++j) {
      const uint32_t rank0 = gi[j] < n ? s_drank[((key[j] >> SR) >> c.dlo) & dm] : 0u;
      rank_out[j] = rank0;
      const uint32_t rank = c.cmode ? s_fbase[rank0] + (uint32_t)((key[j] >> S) & b.fl.cmask) : rank0;
      const uint64_t suffix = S == 0 ? 0ull : (key[j] & ((1ull << S) - 1ull));
      const uint64_t r = hi >= 64 ? 0ull : ((uint64_t)rank << hi);
      out[j] = gi[j] < n ? (r | (suffix << c.ib) | (uint64_t)gi[j]) : 0ull;
    }
    return;
  }
  const uint64_t mask = c.ct_mask;
  uint64_t p[NI], h[NI], v[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    p[j] = key[j] >> S;
    h[j] = mix64(p[j] ^ 0xD6E8FEB86659FD93ull) & mask;
  }
#pragma unroll
  for (int j = 0; j < NI; ++j) v[j] = b.fl.ct_key[h[j]];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    if (gi[j] >= n) {
      out[j] = 0;
      rank_out[j] = 0;
      continue;
    }
    uint64_t hh = h[j], vv = v[j];
    for (uint64_t probe = 0; vv != p[j] && vv != ~0ull && probe < mask; ++probe) {
      hh = (hh + 1) & mask;
      vv = b.fl.ct_key[hh];
    }
    const uint32_t rank = vv == p[j] ? b.fl.ct_rank[hh] : 0u;
    rank_out[j] = rank;
    const uint64_t suffix = S == 0 ? 0ull : (key[j] & ((1ull << S) - 1ull));
    const uint64_t r = hi >= 64 ? 0ull : ((uint64_t)rank << hi);
    out[j] = r | (suffix << c.ib) | (uint64_t)gi[j];
  }
}

// ---- single-pass passes (decoupled look-back) -----------------------------------
// Each pass is one persistent kernel. A block takes tile tickets in order; for a
// tile it ranks the digits locally, publishes the tile's per-digit counts, and looks
// back over earlier tiles (lb_publish / lb_resolve) for the exclusive prefix of
// every digit; global digit bases come from counts taken for all passes in one
// earlier sweep over the input. Two status regions alternate between passes; a
// pass clears the other region at its own tiles for the next pass.
#define OS_GRID 1024

// Counter copies of the digit counting sweep: 16-bit counters, two digits to a word,
// `copies` copies picked by lane so that a row whose lanes share one digit (common
// for flow-rank digits) makes at most 64 / copies same-address LDS atomics; copies
// sit in consecutive words (banks).
__host__ __device__ inline int os_copies(int passes) { return passes <= 6 ? 16 : 4; }
__host__ __device__ inline int os_hist_max_tiles(int copies) { return 65535 / (SORT_TILE / copies); }

__global__ void k_os_prep(SortBufs b, int64_t n_host, const int64_t* n_dev, int64_t region) {
  const int64_t n = load_n(n_host, n_dev);
  const int64_t len = cdiv(n, OS_TILE) * SORT_BUCKETS;   // status words of the first pass
  uint32_t* st = b.os_status + (b.ctl->plan.first & 1) * region;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < len; i += (int64_t)gridDim.x * blockDim.x)
    st[i] = 0;
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < SORT_MAX_PASSES * SORT_BUCKETS; i += blockDim.x) b.os_hist[i] = 0;
    if (threadIdx.x < SORT_MAX_PASSES) b.os_ctr[threadIdx.x] = 0;
  }
}

// Digit counts of every pass, in one sweep over the input. Packed mode also
// composes the words and stages them for the first pass. Persistent.
__global__ __launch_bounds__(NT) void k_sort_hist(SortBufs b, int64_t n_host, const int64_t* n_dev, RouteGeom rg,
                                                  int max_passes, int copies_h) {
  const int first = b.ctl->plan.first;
  const PassView c = read_pass(b.ctl, first);
  int32_t* const dest_out = b.dest_out ? opaque(b.dest_out) : nullptr;
  if (c.npass == 0 && (!dest_out || b.ctl->plan.idle)) return;   // nothing varies, or sorted in one workgroup
  const int64_t n = load_n(n_host, n_dev);
  const int64_t ntiles = cdiv(n, TILE);
  const bool packed = c.mode == SORT_PACKED && c.npass > 0;
  extern __shared__ uint32_t s_hw[];
  __shared__ int s_sh[SORT_MAX_PASSES], s_fd[SORT_MAX_PASSES];
  const int np = c.npass < max_passes ? c.npass : max_passes;   // npass <= max_passes by the plan
  // the counters were sized for max_passes passes of copies_h copies; fewer passes
  // take more copies (up to 16) in the same words
  int copies = copies_h;
  while (copies < 16 && 2 * copies * np <= copies_h * max_passes) copies *= 2;
  const int wpp = 128 * copies;   // words per pass
  for (int i = threadIdx.x; i < np * wpp; i += NT) s_hw[i] = 0;
  // packed mode with a direct rank table: the table follows the counters
  const int cwords = max_passes * 128 * copies_h;
  uint16_t* const s_drank = (packed && c.dbits >= 0) ? reinterpret_cast<uint16_t*>(s_hw + cwords) : nullptr;
  // and the flows' destinations (ranks < 2^dbits), after the rank table
  uint32_t* const s_fdest = s_drank ? s_hw + cwords + (1 << FLOW_DIRECT_BITS) / 2 : nullptr;
  // and the child-rank bases (child-rank packing)
  uint32_t* const s_fbase = s_drank ? s_fdest + (1 << FLOW_DIRECT_BITS) : nullptr;
  if (s_drank) {
    const uint16_t* dr = opaque(b.fl.drank);
    for (int i = threadIdx.x; i < (1 << c.dbits); i += NT) s_drank[i] = dr[i];
    const int F = (int)b.ctl->nflows_c;
    if (dest_out) {
      const uint32_t* fd = opaque(b.fl.fdest);
      for (int i = threadIdx.x; i < F; i += NT) s_fdest[i] = fd[i];
    }
    if (c.cmode) {
      const uint32_t* fb = opaque(b.fl.fbase);
      for (int i = threadIdx.x; i < F; i += NT) s_fbase[i] = fb[i];
    }
  }
  const uint32_t* const g_fdest = packed ? opaque(b.fl.fdest) : nullptr;
  if (threadIdx.x < SORT_MAX_PASSES) {
    const SortPass ps = b.ctl->plan.pass[first + threadIdx.x < SORT_MAX_PASSES ? first + threadIdx.x : 0];
    s_sh[threadIdx.x] = (packed ? c.ib : 0) + ps.lo;
    s_fd[threadIdx.x] = packed ? 0 : ps.from_dest;
  }
  __syncthreads();
  bool any_dest = false;
  for (int q = 0; q < np; ++q) any_dest |= s_fd[q] != 0;
  uint64_t* const stage = packed ? (c.ps.dst == SORT_BUF_TMP ? opaque(b.out_keys) : opaque(b.tmp_keys)) : nullptr;
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  const int copy = lane & (copies - 1);
  const int lofs = w * (IT * ALTO_WAVE) + lane;   // tile-local index of item 0
  // the input keys of the block's next tile are loaded while it works on the current
  // one (the loads stay in flight across the counting)
  const uint64_t* const ik = opaque(b.in_keys);
  uint64_t nkey[IT];
  auto load_keys = [&](int64_t t) {
    const int64_t t0 = t * TILE;
    if (t0 + TILE <= n) {
#pragma unroll
      for (int j = 0; j < IT; ++j) nkey[j] = ik[t0 + lofs + j * ALTO_WAVE];
    } else {
#pragma unroll
      for (int j = 0; j < IT; ++j) nkey[j] = t0 + lofs + j * ALTO_WAVE < n ? ik[t0 + lofs + j * ALTO_WAVE] : 0ull;
    }
  };
  if ((int64_t)blockIdx.x < ntiles) load_keys(blockIdx.x);
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t tile0 = t * TILE;
    int64_t gi[IT];
    uint64_t key[IT];
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      gi[j] = tile0 + lofs + j * ALTO_WAVE;
      key[j] = nkey[j];
    }
    if (t + gridDim.x < ntiles) load_keys(t + gridDim.x);
    uint32_t dv[IT];
    if (packed) {
      uint32_t rank[IT];
      pack_items<IT>(b, c, gi, n, key, key, s_drank, s_fbase, rank);
#pragma unroll
      for (int j = 0; j < IT; ++j)
        if (gi[j] < n) stage[gi[j]] = key[j];
      if (c.direct) {
        // the last pass writes every position of the permutation once (unless a key
        // is given twice): positions it misses keep this value
        uint32_t* const pv = opaque(b.out_vals);
#pragma unroll
        for (int j = 0; j < IT; ++j)
          if (gi[j] < n) pv[gi[j]] = DP_UNPLACED;
      }
      if (dest_out) {
        // the element's destination is its flow's (ranks follow (destination, prefix))
#pragma unroll
        for (int j = 0; j < IT; ++j)
          if (gi[j] < n) dest_out[gi[j]] = (int32_t)(s_fdest ? s_fdest[rank[j]] : g_fdest[rank[j]]);
      }
    } else {
#pragma unroll
      for (int j = 0; j < IT; ++j) dv[j] = (any_dest || dest_out) ? dest_of_key(rg, key[j]) : 0u;
      if (dest_out) {
#pragma unroll
        for (int j = 0; j < IT; ++j)
          if (gi[j] < n) dest_out[gi[j]] = (int32_t)dv[j];
      }
    }
    for (int q = 0; q < np; ++q) {
      const int sh = s_sh[q];
      const bool fd = s_fd[q] != 0;
      uint32_t* hq = s_hw + q * wpp;
#pragma unroll
      for (int j = 0; j < IT; ++j) {
        if (gi[j] >= n) continue;
        const uint64_t src = fd ? (uint64_t)dv[j] : key[j];
        const uint32_t dig = (uint32_t)((src >> sh) & (SORT_BUCKETS - 1));
        atomicAdd(&hq[(dig >> 1) * copies + copy], (dig & 1u) ? 65536u : 1u);
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < np * SORT_BUCKETS; i += NT) {
    const int q = i / SORT_BUCKETS, d = i % SORT_BUCKETS;
    const uint32_t* hq = s_hw + q * wpp + (d >> 1) * copies;
    uint32_t v = 0;
    for (int k = 0; k < copies; ++k) v += (hq[k] >> ((d & 1) * 16)) & 0xFFFFu;
    if (v) atomicAdd(&b.os_hist[(first + q) * SORT_BUCKETS + d], v);
  }
}

// Exclusive scan of each pass's 256 global digit counts (one wave per pass).
__global__ void k_os_bases(SortBufs b) {
  const int q = threadIdx.x / ALTO_WAVE, lane = lane_id();
  if (q >= SORT_MAX_PASSES) return;
  uint32_t* h = b.os_hist + q * SORT_BUCKETS;
  uint32_t v[4], s = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[k] = h[lane * 4 + k];
    s += v[k];
  }
  const uint32_t inc = wave_incl_scan(s);
  uint32_t run = inc - s;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[lane * 4 + k] = run;
    run += v[k];
  }
}

__device__ inline uint32_t pass_digit(bool packed, const SortPass& ps, int sh, const RouteGeom& rg, uint64_t el) {
  return packed ? (uint32_t)((el >> sh) & (SORT_BUCKETS - 1)) : digit_of(ps, rg, el);
}

// One pass over all tiles. Packed mode moves one word per element (the last pass
// unpacks it into key and input index); general mode moves a key and a value. One
// instantiation per mode (each exits when the device chose the other), so that the
// packed one keeps the registers of its simpler digits.
// Packed passes: LAST is the instantiation launched for the host's last packed slot,
// where the plan puts the final pass; only it unpacks (keeping the unpacking code
// and its registers out of the other passes).
template <bool PACKED, bool LAST = false>
__global__ __launch_bounds__(NT, PACKED ? (OS_IT <= 8 ? 6 : 4) : 2) void k_onesweep(SortBufs b, int64_t n_host, const int64_t* n_dev, RouteGeom rg,
                                                 int slot, int64_t region) {
  const PassView c = read_pass(b.ctl, slot);
  if (!c.ps.active || (c.mode == SORT_PACKED) != PACKED) return;
  const int64_t n = load_n(n_host, n_dev);
  const int64_t ntiles = cdiv(n, OS_TILE);
  if ((int64_t)blockIdx.x >= ntiles) return;   // the grid covers the largest count; no tile for this block
  constexpr bool packed = PACKED;
  const bool last = PACKED ? LAST : (slot + 1 == c.first + c.npass);
  const int sh = c.ib + c.ps.lo;
  __shared__ uint16_t s_cnt[NW][SORT_BUCKETS];
  __shared__ uint32_t s_base[SORT_BUCKETS];
  __shared__ uint32_t s_gbase[SORT_BUCKETS];
  __shared__ uint32_t s_wsum[NT / ALTO_WAVE];
  __shared__ uint64_t s_key[OS_TILE];
  __shared__ uint16_t s_slot[OS_TILE];   // general mode: position of the element in its tile
  __shared__ int64_t s_tile;
  uint32_t* st = b.os_status + (slot & 1) * region;
  uint32_t* st_next = b.os_status + ((slot + 1) & 1) * region;
  uint64_t* const tk = opaque(b.tmp_keys);
  uint64_t* const ok = opaque(b.out_keys);
  uint32_t* const tv = opaque(b.tmp_vals);
  uint32_t* const ov = opaque(b.out_vals);
  const uint64_t* const ik = opaque(b.in_keys);
  // source: the input keys (general), the staged words (packed, first pass, in the
  // buffer the pass does not write), or the previous pass's output
  const uint64_t* sk = c.ps.src == SORT_BUF_TMP ? tk : ok;
  const uint32_t* sv = c.ps.src == SORT_BUF_TMP ? tv : ov;
  if (c.ps.src == SORT_BUF_INPUT) {
    sk = packed ? (c.ps.dst == SORT_BUF_TMP ? ok : tk) : ik;
    sv = nullptr;
  }
  uint64_t* const dk = c.ps.dst == SORT_BUF_TMP ? tk : ok;
  uint32_t* const dvals = c.ps.dst == SORT_BUF_TMP ? tv : ov;
  const uint64_t* const fsorted = opaque(b.fl.flow_sorted);
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  while (true) {
    if (threadIdx.x == 0) s_tile = (int64_t)atomicAdd(&b.os_ctr[slot], 1u);
    for (int i = threadIdx.x; i < NW * SORT_BUCKETS; i += NT) (&s_cnt[0][0])[i] = 0;
    __syncthreads();
    // uniform across the block: kept in scalar registers (scalar-based addressing)
    const int64_t tile = (int64_t)__builtin_amdgcn_readfirstlane((uint32_t)s_tile);
    if (tile >= ntiles) break;   // uniform across the block
    const int64_t tile0 = tile * OS_TILE;
    const int rem = (int)(n - tile0 < OS_TILE ? n - tile0 : OS_TILE);   // elements in this tile
    const uint64_t* const tsk = sk + tile0;
    const int lbase = w * (OS_IT * ALTO_WAVE) + lane;               // tile-local index of item 0
    uint64_t key[OS_IT];
    uint32_t dof[OS_IT];   // digit | in-wave offset << 8 (offsets < OS_IT * 64)
#pragma unroll
    for (int j = 0; j < OS_IT; ++j) key[j] = lbase + j * ALTO_WAVE < rem ? tsk[lbase + j * ALTO_WAVE] : 0ull;
#pragma unroll
    for (int j = 0; j < OS_IT; ++j) {
      const bool valid = lbase + j * ALTO_WAVE < rem;
      const uint32_t dig = valid ? pass_digit(packed, c.ps, sh, rg, key[j]) : 0u;
      dof[j] = dig | (wave_rank(s_cnt[w], dig, valid) << 8);
    }
    __syncthreads();
    // per-wave offsets of every digit, the tile's count published at once (so that
    // later tiles can pass this one), then the LDS scatter; the look-back comes
    // after it, when the elements no longer occupy registers
    const int d = threadIdx.x;
    uint32_t run = 0;
    // direct placement (last pass): positions come from the child ranks, no look-back
    const bool direct = PACKED && LAST && c.direct;
    if (d < SORT_BUCKETS) {
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) {
        const uint32_t cc = s_cnt[ww][d];
        s_cnt[ww][d] = (uint16_t)run;
        run += cc;
      }
      if (!direct) lb_publish(st + d, tile, SORT_BUCKETS, run);
    }
    uint32_t tot;
    {
      const uint32_t ex = block_excl_scan<uint32_t, NT>(run, s_wsum, &tot);
      if (d < SORT_BUCKETS) s_base[d] = ex;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < OS_IT; ++j) {
      if (lbase + j * ALTO_WAVE < rem) {
        const uint32_t dg = dof[j] & 0xFFu;
        const uint32_t r = s_base[dg] + (uint32_t)s_cnt[w][dg] + (dof[j] >> 8);
        s_key[r] = key[j];
        if (!packed) s_slot[r] = (uint16_t)(lbase + j * ALTO_WAVE);
      }
    }
    if (d < SORT_BUCKETS && !direct) {
      const uint32_t excl = lb_resolve(st + d, tile, SORT_BUCKETS, run, b.status);
      s_gbase[d] = b.os_hist[slot * SORT_BUCKETS + d] + excl;
      st_next[tile * SORT_BUCKETS + d] = 0;   // the next pass's status of this tile
    }
    __syncthreads();
    if (packed && !LAST) {
      for (uint32_t e = threadIdx.x; e < tot; e += NT) {
        const uint64_t el = s_key[e];
        const uint32_t dg = (uint32_t)((el >> sh) & (SORT_BUCKETS - 1));
        dk[(uint64_t)s_gbase[dg] + (e - s_base[dg])] = el;
      }
    } else if (direct) {
      // element (child rank cr, leaf tag t) goes to cbase[cr] + t; only the
      // permutation is written (the sorted keys are not needed: group bounds come
      // from cbase). A rank past the table comes only from an input error and is not
      // written.
      const uint64_t imask = c.ib >= 64 ? ~0ull : ((1ull << c.ib) - 1ull);
      const int S = c.sbits;
      const uint64_t tmask = S >= 64 ? ~0ull : ((1ull << S) - 1ull);
      const uint32_t* const cbase = opaque(b.fl.cbase);
      // the base lookups of all of a thread's elements are issued before any is used
      // (their latency is not hidden by other waves). A tag past its child's count (an
      // input error) lands in a neighbour's range: a position is then written twice
      // and another left at DP_UNPLACED.
      constexpr int DH = OS_IT / 2;   // two halves: fewer registers live
#pragma unroll 1
      for (int h = 0; h < 2; ++h) {
        uint64_t el[DH];
        uint32_t gb[DH];
#pragma unroll
        for (int u = 0; u < DH; ++u) {
          const uint32_t e = threadIdx.x + (uint32_t)(h * DH + u) * NT;
          el[u] = e < tot ? s_key[e] : 0ull;
        }
#pragma unroll
        for (int u = 0; u < DH; ++u) {
          const uint32_t e = threadIdx.x + (uint32_t)(h * DH + u) * NT;
          const uint64_t cr = (S + c.ib >= 64) ? 0ull : (el[u] >> (S + c.ib));
          gb[u] = (e < tot && cr < c.ctotal) ? cbase[cr] : 0xFFFFFFFFu;
        }
#pragma unroll
        for (int u = 0; u < DH; ++u) {
          const uint64_t g = (uint64_t)gb[u] + ((el[u] >> c.ib) & tmask);
          if (gb[u] == 0xFFFFFFFFu || g >= (uint64_t)n) continue;
          ov[g] = (uint32_t)(el[u] & imask);
        }
      }
    } else if (packed && LAST) {
      const uint64_t imask = c.ib >= 64 ? ~0ull : ((1ull << c.ib) - 1ull);
      for (uint32_t e = threadIdx.x; e < tot; e += NT) {
        const uint64_t el = s_key[e];
        const uint32_t dg = (uint32_t)((el >> sh) & (SORT_BUCKETS - 1));
        const uint64_t g = (uint64_t)s_gbase[dg] + (e - s_base[dg]);
        ok[g] = unpack_key(b.fl, fsorted, c, el);
        ov[g] = (uint32_t)(el & imask);
      }
    } else {
      for (uint32_t e = threadIdx.x; e < tot; e += NT) {
        const uint64_t el = s_key[e];
        const uint32_t dg = digit_of(c.ps, rg, el);
        const uint64_t g = (uint64_t)s_gbase[dg] + (e - s_base[dg]);
        const int64_t gi = tile0 + s_slot[e];
        dk[g] = el;
        dvals[g] = sv ? sv[gi] : (uint32_t)gi;
      }
    }
    __syncthreads();   // LDS and the ticket are reused by the next tile
  }
}

__global__ void k_sort_identity(SortBufs b, int64_t n_host, const int64_t* n_dev) {
  if (b.ctl->plan.npass != 0 || b.ctl->plan.idle) return;
  const int64_t n = load_n(n_host, n_dev);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    b.out_keys[i] = b.in_keys[i];
    b.out_vals[i] = (uint32_t)i;
  }
}

// ---------------------------------------------------------------------------
// device-wide exclusive scan: per-block sums, one-block scan of the sums, apply
// ---------------------------------------------------------------------------
constexpr int SCAN_NT = 256;
constexpr int SCAN_IT = 4;

template <typename T>
__global__ __launch_bounds__(SCAN_NT) void k_scan_sums(const T* __restrict__ in, int64_t len_host, const int64_t* len_dev,
                                                      T* part, int nb) {
  const int64_t len = load_n(len_host, len_dev);
  const int64_t chunk = (len + nb - 1) / nb;
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = lo + chunk < len ? lo + chunk : len;
  T s = 0;
  for (int64_t i = lo + threadIdx.x; i < hi; i += SCAN_NT) s += in[i];
  __shared__ T sh[SCAN_NT / ALTO_WAVE];
  s = wave_sum(s);
  if (lane_id() == 0) sh[threadIdx.x / ALTO_WAVE] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    T t = 0;
    for (int i = 0; i < SCAN_NT / ALTO_WAVE; ++i) t += sh[i];
    part[blockIdx.x] = t;
  }
}

template <typename T>
__global__ __launch_bounds__(1024) void k_scan_part(T* part, int nb, T* total) {
  __shared__ T sh[1024 / ALTO_WAVE];
  T v = threadIdx.x < (unsigned)nb ? part[threadIdx.x] : 0;
  T tot;
  T ex = block_excl_scan<T, 1024>(v, sh, &tot);
  if (threadIdx.x < (unsigned)nb) part[threadIdx.x] = ex;
  if (threadIdx.x == 0) {
    part[nb] = tot;
    if (total) *total = tot;
  }
}

template <typename T>
__global__ __launch_bounds__(SCAN_NT) void k_scan_apply(const T* in, T* out, int64_t len_host, const int64_t* len_dev,
                                                       const T* part, int nb) {
  const int64_t len = load_n(len_host, len_dev);
  const int64_t chunk = (len + nb - 1) / nb;
  const int64_t lo = (int64_t)blockIdx.x * chunk, hi = lo + chunk < len ? lo + chunk : len;
  __shared__ T sh[SCAN_NT / ALTO_WAVE];
  T run = part[blockIdx.x];
  for (int64_t base = lo; base < hi; base += SCAN_NT * SCAN_IT) {
    T v[SCAN_IT];
    T s = 0;
#pragma unroll
    for (int k = 0; k < SCAN_IT; ++k) {
      int64_t i = base + (int64_t)threadIdx.x * SCAN_IT + k;
      v[k] = i < hi ? in[i] : 0;
      s += v[k];
    }
    T tot;
    T ex = block_excl_scan<T, SCAN_NT>(s, sh, &tot);
    T r = run + ex;
#pragma unroll
    for (int k = 0; k < SCAN_IT; ++k) {
      int64_t i = base + (int64_t)threadIdx.x * SCAN_IT + k;
      if (i < hi) out[i] = r;
      r += v[k];
    }
    run += tot;
  }
}


// ---------------------------------------------------------------------------
// whole sort in one workgroup for n <= SORT_SMALL_MAX: keys stay in LDS between
// passes; the digit windows are planned in the block from its own OR/AND.
// ---------------------------------------------------------------------------
constexpr int SM_NT = 1024;
constexpr int SM_NW = SM_NT / ALTO_WAVE;
static_assert(SM_NT == 4 * SORT_BUCKETS && SM_NW == 16, "the count scan gives each thread 4 waves of one digit");

// The routing call's preparation (SmallPrep), by the whole workgroup, in two parts
// around the sort's own read of the keys (which also writes the destinations and
// checks the layout): the control block and the fingerprint sums are reset first.
__device__ inline void small_prep_begin(const SmallPrep& pp, int64_t n_host, const int64_t* n_dev,
                                        unsigned long long* s_fp, uint32_t* s_flags) {
  if (threadIdx.x == 0) {
    *s_flags = 0u;
    if (n_dev && (*n_dev < 0 || *n_dev > n_host)) raise_status(pp.status, ALTO_E_CAPACITY);
    SortCtl* c = pp.ctl;
    c->key_or = 0;
    c->key_and = ~0ull;
    c->dest_or = 0;
    c->dest_and = ~0u;
    c->mode = SORT_GENERAL;
    c->flow_overflow = 0;
    c->nflows = 0;
    c->nflows_c = 0;
    c->cmode = 0;
    c->dp = 0;
    c->dbits = -1;
  }
  const int flo = pp.flo, fhi = pp.fan ? pp.fhi : pp.flo - 1;
  for (int i = threadIdx.x; i <= ALTO_MAX_LEVELS; i += SM_NT) {
    s_fp[i] = 0ull;
    pp.fp_nodes[i] = 0;
    if (i < flo || i > fhi) pp.fp_in[i] = 0;
  }
}

// Second part, with the keys in LDS (s_key[e] & kmask is element e's key): the
// declared-count checks and the fragment side of the fan fingerprint, one level at
// a time (a scalar sum per level, a wave sum, one LDS add per wave).
__device__ inline void small_prep_levels(const SmallPrep& pp, const uint64_t* s_key, uint64_t kmask, int64_t n,
                                         bool bad_layout, unsigned long long* s_fp, uint32_t* s_flags) {
  const KeyGeom& g = pp.g;
  const int flo = pp.flo, fhi = pp.fan ? pp.fhi : pp.flo - 1;
  bool bad_fan = false;
  for (int m = flo; m <= fhi; ++m) {
    const int sh = g.shift[m], shc = g.shift[m + 1];
    const uint64_t tm = (uint64_t)g.tagmask[m + 1];
    uint64_t acc = 0;
    for (int64_t e = threadIdx.x; e < n; e += SM_NT) {
      const uint64_t k = s_key[e] & kmask;
      const int32_t f = pp.fan[(int64_t)(m - 1) * pp.fan_ld + e];
      bad_fan |= (f < 1) || ((int64_t)((k >> shc) & tm) >= (int64_t)f);
      acc += fan_term(g.fkey, m, key_prefix(k, sh), (uint32_t)f);
    }
    acc = wave_sum(acc);
    if (lane_id() == 0 && acc) atomicAdd(&s_fp[m], (unsigned long long)acc);
  }
  if (bad_layout) atomicOr(s_flags, 1u);
  if (bad_fan) atomicOr(s_flags, 2u);
  __syncthreads();
  for (int m = flo + (int)threadIdx.x; m <= fhi; m += SM_NT) pp.fp_in[m] = (uint64_t)s_fp[m];
  if (threadIdx.x == 0) {
    if (*s_flags & 1u) raise_status(pp.status, ALTO_E_LAYOUT);
    if (*s_flags & 2u) raise_status(pp.status, ALTO_E_FANOUT);
  }
}

// IT items per thread (IT * SM_NT elements at most): launched with the smallest IT
// that holds the host's bound on the count, so small sorts rank fewer items per pass.
// dshift >= 0: the destination is placed above the key bits (dshift = key bits; the
// host checked that both fit 64 bits), so the destination takes no pass of its own
// and is hashed once per element; the key is unpacked when written out.
template <int IT>
__global__ __launch_bounds__(SM_NT) void k_sort_small(SortBufs b, int64_t n_host, const int64_t* n_dev, RouteGeom rg,
                                                      int max_key_windows, int max_dest_windows, int dshift) {
  __shared__ uint64_t s_key[IT * SM_NT];
  __shared__ uint32_t s_val[IT * SM_NT];
  __shared__ uint16_t s_cnt[SM_NW][SORT_BUCKETS];
  __shared__ uint32_t s_wsum[SM_NW];
  __shared__ uint64_t s_or[SM_NW], s_and[SM_NW];
  __shared__ uint32_t s_dor[SM_NW], s_dand[SM_NW];
  __shared__ int s_np;
  __shared__ int s_lo[SORT_MAX_PASSES], s_fd[SORT_MAX_PASSES];
  __shared__ unsigned long long s_fp[ALTO_MAX_LEVELS + 1];
  __shared__ uint32_t s_flags;
  int64_t n = load_n(n_host, n_dev);
  // the call's only sort (its bound fits here): a device count outside [0, bound]
  // is clamped (and reported by the preparation); otherwise larger counts are the
  // multi-block path's
  if (n_host <= IT * SM_NT) n = n < 0 ? 0 : (n > n_host ? n_host : n);
  const bool prep = b.prep.ctl != nullptr;
  if (prep) small_prep_begin(b.prep, n_host, n_dev, s_fp, &s_flags);
  if (n > IT * SM_NT) return;   // block-uniform
  const bool packed = dshift >= 0;
  const uint64_t kmask = packed ? ((1ull << dshift) - 1ull) : ~0ull;
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u;
  bool bad_layout = false;
  for (int j = 0; j < IT; ++j) {
    const int e = w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    if (e < n) {
      const uint64_t k = b.in_keys[e];
      const uint32_t d = dest_of_key(rg, k);
      const uint64_t word = packed ? (k | ((uint64_t)d << dshift)) : k;
      s_key[e] = word;
      s_val[e] = (uint32_t)e;
      kor |= word;
      kand &= word;
      dor |= d;
      dand &= d;
      if (prep) {
        bad_layout |= (k >> b.prep.g.total) != 0;
        if (b.prep.dest) b.prep.dest[e] = (int32_t)d;
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    kor |= __shfl_xor(kor, o);
    kand &= __shfl_xor(kand, o);
    dor |= __shfl_xor(dor, o);
    dand &= __shfl_xor(dand, o);
  }
  if (lane == 0) {
    s_or[w] = kor;
    s_and[w] = kand;
    s_dor[w] = dor;
    s_dand[w] = dand;
  }
  __syncthreads();
  if (prep) small_prep_levels(b.prep, s_key, kmask, n, bad_layout, s_fp, &s_flags);
  if (threadIdx.x == 0) {
    uint64_t a = 0, c = ~0ull;
    uint32_t da = 0, dc = ~0u;
    for (int i = 0; i < SM_NW; ++i) {
      a |= s_or[i];
      c &= s_and[i];
      da |= s_dor[i];
      dc &= s_dand[i];
    }
    int np = 0;
    uint64_t vk = a ^ c;
    while (vk && np < max_key_windows) {
      const int lo = __builtin_ctzll(vk);
      s_lo[np] = lo;
      s_fd[np] = 0;
      ++np;
      vk = (lo + SORT_RADIX >= 64) ? 0ull : (vk & ~((1ull << (lo + SORT_RADIX)) - 1ull));
    }
    uint32_t vd = packed ? 0u : (da ^ dc);
    const int nk = np;
    while (vd && np < nk + max_dest_windows) {
      const int lo = __builtin_ctz(vd);
      s_lo[np] = lo;
      s_fd[np] = 1;
      ++np;
      vd = (lo + SORT_RADIX >= 32) ? 0u : (vd & ~((1u << (lo + SORT_RADIX)) - 1u));
    }
    s_np = np;
  }
  __syncthreads();
  const int np = s_np;
  for (int p = 0; p < np; ++p) {
    SortPass ps;
    ps.from_dest = s_fd[p];
    ps.lo = s_lo[p];
    for (int i = threadIdx.x; i < SM_NW * SORT_BUCKETS; i += SM_NT) (&s_cnt[0][0])[i] = 0;
    uint64_t key[IT];
    uint32_t val[IT], dig[IT], off[IT];
    // rows of 64 elements past the count are skipped by the whole wave (a count far
    // below the host's bound leaves most waves without work, and the sort is bound
    // by the one CU's vector instructions)
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int e = w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      const bool valid = e < n;
      key[j] = 0ull;
      val[j] = 0u;
      dig[j] = 0u;
      off[j] = 0u;
      if (w * (IT * ALTO_WAVE) + j * ALTO_WAVE < n) {   // wave-uniform
        key[j] = valid ? s_key[e] : 0ull;
        val[j] = valid ? s_val[e] : 0u;
        dig[j] = valid ? digit_of(ps, rg, key[j]) : 0u;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int e = w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      const bool valid = e < n;
      if (w * (IT * ALTO_WAVE) + j * ALTO_WAVE < n) off[j] = wave_rank(s_cnt[w], dig[j], valid);
    }
    __syncthreads();
    {
      // the per-wave digit counts in (digit, wave) order, scanned by the whole block:
      // thread t holds digit t / 4, waves 4 (t % 4) .. 4 (t % 4) + 3; the counters
      // become the wave's first position for the digit
      const int d = threadIdx.x >> 2, q0 = (threadIdx.x & 3) * 4;
      uint32_t c[4], sum = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        c[k] = s_cnt[q0 + k][d];
        sum += c[k];
      }
      uint32_t tot;
      uint32_t ex = block_excl_scan<uint32_t, SM_NT>(sum, s_wsum, &tot);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        s_cnt[q0 + k][d] = (uint16_t)ex;
        ex += c[k];
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IT; ++j) {
      const int e = w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      if (e < n) {
        const uint32_t pos = (uint32_t)s_cnt[w][dig[j]] + off[j];
        s_key[pos] = key[j];
        s_val[pos] = val[j];
      }
    }
    __syncthreads();
  }
  for (int e = threadIdx.x; e < n; e += SM_NT) {
    b.out_keys[e] = s_key[e] & kmask;
    b.out_vals[e] = s_val[e];
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// host launchers
// ---------------------------------------------------------------------------
template <typename T>
int scan_exclusive(const T* in, T* out, int64_t len_max, const int64_t* len_dev, T* part, T* total,
                   hipStream_t st) {
  int nb = (int)(len_max < 1 ? 1 : cdiv(len_max, SCAN_NT * SCAN_IT * 4));
  if (nb > SCAN_MAX_BLOCKS) nb = SCAN_MAX_BLOCKS;
  k_scan_sums<T><<<nb, SCAN_NT, 0, st>>>(in, len_max, len_dev, part, nb);
  k_scan_part<T><<<1, 1024, 0, st>>>(part, nb, total);
  k_scan_apply<T><<<nb, SCAN_NT, 0, st>>>(in, out, len_max, len_dev, part, nb);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

template int scan_exclusive<uint32_t>(const uint32_t*, uint32_t*, int64_t, const int64_t*, uint32_t*, uint32_t*, hipStream_t);
template int scan_exclusive<int32_t>(const int32_t*, int32_t*, int64_t, const int64_t*, int32_t*, int32_t*, hipStream_t);
template int scan_exclusive<int64_t>(const int64_t*, int64_t*, int64_t, const int64_t*, int64_t*, int64_t*, hipStream_t);

int sort_tiles(int64_t n_max) { return (int)(n_max < 1 ? 1 : cdiv(n_max, SORT_OS_TILE)); }

int sort_max_key_windows(int key_bits) { return (int)cdiv(key_bits, SORT_RADIX); }

int sort_max_dest_windows(const RouteGeom& rg) {
  if (rg.shift >= 64 || rg.num_dest <= 1) return 0;
  int bits = 0;
  while (bits < 32 && ((uint64_t)1 << bits) < rg.num_dest) ++bits;
  return (int)cdiv(bits, SORT_RADIX);
}

int bits_for(int64_t v) {
  int b = 0;
  while (b < 63 && ((int64_t)1 << b) <= v) ++b;
  return b;
}

// The one-workgroup sort with the fewest items per thread that holds n_max elements.
static void launch_sort_small(const SortBufs& b, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg,
                              int key_bits, hipStream_t st) {
  // the destination above the key bits when both fit one word
  int dbits = 0;
  if (rg.shift < 64 && rg.num_dest > 1)
    while (dbits < 32 && ((uint64_t)1 << dbits) < rg.num_dest) ++dbits;
  const bool pack = dbits > 0 && key_bits + dbits <= 64;
  const int dshift = pack ? key_bits : -1;
  const int kw = sort_max_key_windows(pack ? key_bits + dbits : key_bits), dw = pack ? 0 : sort_max_dest_windows(rg);
  if (n_max <= SM_NT) k_sort_small<1><<<1, SM_NT, 0, st>>>(b, n_max, n_dev, rg, kw, dw, dshift);
  else if (n_max <= 2 * SM_NT) k_sort_small<2><<<1, SM_NT, 0, st>>>(b, n_max, n_dev, rg, kw, dw, dshift);
  else if (n_max <= 4 * SM_NT) k_sort_small<4><<<1, SM_NT, 0, st>>>(b, n_max, n_dev, rg, kw, dw, dshift);
  else k_sort_small<SORT_SMALL_MAX / SM_NT><<<1, SM_NT, 0, st>>>(b, n_max, n_dev, rg, kw, dw, dshift);
}

int sort_pairs(const SortBufs& b, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, int key_bits,
               bool ctl_has_reduction, hipStream_t st) {
  if (n_max <= SORT_SMALL_MAX) {
    launch_sort_small(b, n_max, n_dev, rg, key_bits, st);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  const int ostiles = sort_tiles(n_max);                   // tiles of the look-back passes
  const int htiles = (int)cdiv(n_max, SORT_TILE);          // tiles of the counting sweep
  if (!b.os_status || !b.os_ctr || !b.os_hist || b.os_ntiles < ostiles) return ALTO_E_ARG;
  const int grid_r = (int)(cdiv(n_max, 256 * 8) < 2048 ? cdiv(n_max, 256 * 8) : 2048);
  if (n_dev) {
    // the count is known on the device only: small counts go to one workgroup
    launch_sort_small(b, n_max, n_dev, rg, key_bits, st);
  }
  if (!ctl_has_reduction) {
    k_sort_init<<<1, 1, 0, st>>>(b.ctl);
    k_sort_reduce<<<grid_r < 512 ? grid_r : 512, 256, 0, st>>>(b.in_keys, n_max, n_dev, rg, b.ctl);
  }
  // packed words need a host-known count (the index bits are fixed on the host)
  const bool packable = b.fl.hcap > 0 && n_dev == nullptr;
  if (b.fl.hcap > 0) {
    // rank the flows in (destination, prefix) order
    const FlowBufs& fl = b.fl;
    const int64_t cb = cdiv(fl.hcap, 256);
    k_flow_compact<<<(int)(cb < 2048 ? cb : 2048), 256, 0, st>>>(fl, b.ctl);
    k_flow_count<<<1, 1, 0, st>>>(fl, b.ctl);
    SortBufs fb;
    memset(&fb, 0, sizeof(fb));
    fb.in_keys = fl.flow_key;
    fb.tmp_keys = fl.ftmp_keys;
    fb.tmp_vals = fl.ftmp_vals;
    fb.out_keys = fl.flow_sorted;
    fb.out_vals = fl.flow_order;
    fb.ctl = fl.fctl;
    fb.os_status = b.os_status;
    fb.os_ctr = b.os_ctr;
    fb.os_hist = b.os_hist;
    fb.os_ntiles = b.os_ntiles;
    fb.status = b.status;
    RouteGeom frg = rg;
    frg.shift = 0;   // the flow keys are already prefixes of the route level
    int rc = sort_pairs(fb, fl.fcap, &b.ctl->nflows_c, frg, key_bits - fl.shift, false, st);
    if (rc) return rc;
    const int64_t rb = cdiv(fl.fcap, 256);
    k_flow_rank<<<(int)(rb < 1024 ? rb : 1024), 256, 0, st>>>(fl, b.ctl, n_max, packable ? 1 : 0);
    k_flow_base<<<1, 1024, 0, st>>>(fl, b.ctl);
    k_ct_insert<<<(int)(rb < 1024 ? rb : 1024), 256, 0, st>>>(fl, b.ctl, rg.num_dest);
    const int64_t cb2 = cdiv(fl.ctab_cap, 256);
    k_ctab_fill<<<(int)(cb2 < 1024 ? cb2 : 1024), 256, 0, st>>>(fl, b.ctl);
    if (fl.dp && packable) {
      k_dp_table<<<PREP_BLOCKS_MAX, 256, 0, st>>>(fl, b.ctl);
      const int64_t db = cdiv(fl.ctab_cap, DP_CHUNK);
      k_dp_sums<<<(int)(db < 1024 ? db : 1024), 256, 0, st>>>(fl, b.ctl);
      k_dp_decide<<<1, 1024, 0, st>>>(fl, b.ctl, n_max);
      k_dp_base<<<(int)(db < 1024 ? db : 1024), 256, 0, st>>>(fl, b.ctl);
    }
  }
  const int mk = sort_max_key_windows(key_bits), md = sort_max_dest_windows(rg);
  int maxp = mk + md;   // general passes
  if (maxp > SORT_MAX_PASSES) maxp = SORT_MAX_PASSES;
  const int mp_slots = packable ? (int)cdiv(64 - b.fl.ib, SORT_RADIX) : 0;
  k_sort_plan<<<1, 1, 0, st>>>(b.ctl, n_max, n_dev, mk, md, mp_slots < SORT_MAX_PASSES ? mp_slots : SORT_MAX_PASSES);
  ALTO_LAUNCH_CHECK();
  // passes at most: general windows, or packed windows over 64 - index bits
  const int mp = mp_slots < SORT_MAX_PASSES ? mp_slots : SORT_MAX_PASSES;
  const int passes = mp > maxp ? mp : maxp;
  const int copies = os_copies(passes);
  const int64_t g0 = cdiv(htiles, os_hist_max_tiles(copies));
  const int grid_h = (int)(g0 > 1024 ? g0 : (htiles < 1024 ? htiles : 1024));
  const size_t lds = (size_t)passes * 128 * copies * sizeof(uint32_t) +
                     (packable ? ((size_t)1 << FLOW_DIRECT_BITS) * (sizeof(uint16_t) + 2 * sizeof(uint32_t)) : 0);
  const int64_t pb = cdiv((int64_t)ostiles * SORT_BUCKETS, 256);
  const int64_t region = (int64_t)b.os_ntiles * SORT_BUCKETS;
  k_os_prep<<<(int)(pb < 1024 ? pb : 1024), 256, 0, st>>>(b, n_max, n_dev, region);
  k_sort_hist<<<grid_h, NT, lds, st>>>(b, n_max, n_dev, rg, passes, copies);
  k_os_bases<<<1, SORT_MAX_PASSES * ALTO_WAVE, 0, st>>>(b);
  const int grid_o = ostiles < OS_GRID ? ostiles : OS_GRID;
  for (int slot = 0; slot < passes; ++slot) {
    if (slot + 1 == mp) k_onesweep<true, true><<<grid_o, NT, 0, st>>>(b, n_max, n_dev, rg, slot, region);
    else if (slot < mp) k_onesweep<true, false><<<grid_o, NT, 0, st>>>(b, n_max, n_dev, rg, slot, region);
    if (slot < maxp) k_onesweep<false><<<grid_o, NT, 0, st>>>(b, n_max, n_dev, rg, slot, region);
  }
  k_sort_identity<<<grid_r, 256, 0, st>>>(b, n_max, n_dev);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

void sort_reduce_launch(const uint64_t* keys, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, SortCtl* ctl,
                        hipStream_t st) {
  const int grid_r = (int)(n_max < 1 ? 1 : (cdiv(n_max, 256 * 8) < 2048 ? cdiv(n_max, 256 * 8) : 2048));
  k_sort_init<<<1, 1, 0, st>>>(ctl);
  k_sort_reduce<<<grid_r < 512 ? grid_r : 512, 256, 0, st>>>(keys, n_max, n_dev, rg, ctl);
}
