// Streams: partial groups carried across steps (paper Section 3.1: outputs are
// streamed before inputs are complete; Section 4.2: aggregation at pmap exit).
//
// Device state, in caller memory:
//   live set   the arrived leaves of groups not yet emitted, kept sorted by
//              (destination, key): key, int32 payload, all declared child counts,
//              and (MEAN) the slot of the leaf's row in the arena; two copies,
//              written alternately;
//   arena      MEAN: one float32 row per live leaf, with a stack of free slots;
//   emitted    an insert-only open-addressing set of emitted group keys, to
//              report fragments that arrive after their group was released;
//   parents    with in-order release: each parent's next child to release, in an
//              insert-only open-addressing table keyed by the parent's prefix.
// A step sorts its own fragments, merges them with the live set by binary search
// (merge path), segments the merged run into nodes, evaluates completion, emits the
// complete groups with the batch kernels, and writes the survivors as the new live
// set.
#include <string.h>

#include "aggregate.h"
#include "profile.h"

namespace {

constexpr uint64_t HT_EMPTY = EMIT_EMPTY;

struct StreamCtl {
  int32_t error;     // data error of an earlier step (the handle is poisoned)
  int32_t pad;
  int64_t live;      // carried leaves
  int64_t top[2];    // free slots on the stack (MEAN), by step parity: read [p], written [p ^ 1]
  int64_t emitted;   // keys in the emitted set
  int64_t merged;    // live + step, this step
  int64_t merged1;   // merged + 1
  // this step's totals, from the last tile of the live-set update: kept leaves,
  // freed arena slots, slots needed (MEAN)
  int64_t knext, ftot, atot;
};

// live-set update: tiles of LU_TILE merged elements, LU_IT consecutive ones per thread
constexpr int LU_NT = 256;
constexpr int LU_IT = 8;
constexpr int LU_TILE = LU_NT * LU_IT;
constexpr int LU_SPEC_BLOCKS = 64;   // blocks that load their tile before the merged count arrives

// sampled keys per run in the merge's LDS search
constexpr int MERGE_SAMPLES = 2048;
static_assert(MERGE_SAMPLES % 256 == 0, "whole sample rows per merge block");

struct LiveSet {
  uint64_t* key;
  int32_t* p32;
  int32_t* fan;    // [(depth-1)][cap]
  int32_t* slot;   // MEAN
};


__device__ inline bool dk_less(const RouteGeom& rg, uint64_t a, uint64_t b) {
  const uint32_t da = dest_of_key(rg, a), db = dest_of_key(rg, b);
  return da < db || (da == db && a < b);
}

__global__ void k_stream_init(StreamCtl* ctl, int32_t* stack, int64_t cap, uint64_t* ht, int64_t htcap, uint64_t* pht,
                              int32_t* pcur) {
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (int64_t)gridDim.x * blockDim.x;
  if (stack)
    for (int64_t i = t0; i < cap; i += stride) stack[i] = (int32_t)i;
  for (int64_t i = t0; i < htcap; i += stride) ht[i] = HT_EMPTY;
  if (pht)
    for (int64_t i = t0; i < htcap; i += stride) {
      pht[i] = HT_EMPTY;
      pcur[i] = 0;
    }
  if (t0 == 0) {
    ctl->error = 0;
    ctl->live = 0;
    ctl->top[0] = ctl->top[1] = stack ? cap : 0;
    ctl->emitted = 0;
    ctl->merged = 0;
    ctl->merged1 = 1;
  }
}

__global__ void k_stream_begin(const StreamCtl* ctl, int32_t* status) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && ctl->error) raise_status(status, ctl->error);
}

// Steps routed on another HIP stream: the routing's end is published in a word of
// the handle's state (one per workspace, each on its own 256-byte line) rather
// than with a HIP event, whose cross-queue wait costs the host about 10 us per
// step and the step's queue a barrier packet. The signal kernel runs on the
// routing stream after the routing's kernels, whose writes are released at their
// ends; the merge waits for the word to hold the step's sequence number (a
// per-handle random base plus a count, compared for equality, so a stale word of
// an earlier handle in the same memory never matches) and then acquires.
constexpr int64_t ROUTE_FLAG_STRIDE = 32;      // uint64 words: 256 bytes
constexpr int ROUTE_WAIT_LIMIT = 1 << 22;      // polls of ~0.3-1.2 us: 1-5 s, then ALTO_E_INTERNAL

__global__ void k_route_signal(uint64_t* flag, uint64_t seq) {
  if (threadIdx.x == 0) __hip_atomic_store(flag, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Bounded wait of a block for its step's routing (rflag null: the routing ran
// before on the same stream). On giving up the status word gets ALTO_E_INTERNAL
// and the block goes on; whatever it then reads of the routing's outputs is used
// only within bounds (the merge clamps the permutation's source indices).
__device__ inline void route_wait(const uint64_t* rflag, uint64_t rseq, int32_t* status) {
  if (!rflag) return;
  if (threadIdx.x == 0) {
    int spin = 0;
    while (__hip_atomic_load(rflag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != rseq) {
      if (++spin > ROUTE_WAIT_LIMIT) {
        raise_status(status, ALTO_E_INTERNAL);
        break;
      }
      __builtin_amdgcn_s_sleep(8);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

// Merge path: every element finds its place by binary search in the other run.
// Live elements go before equal step keys (which are duplicates, reported later).
// The searches start in LDS: each block that holds merged elements first copies
// every s-th key of both runs (at most MERGE_SAMPLES of each, s the smallest stride
// that fits), which narrows a search to s consecutive keys before it reads global
// memory (log2 s dependent loads instead of log2 of the run length).
// Also adds the live leaves' terms of the fan fingerprint.
// Also, so that the step launches fewer kernels: reports a poisoned handle, finds
// late fragments (their group is in the emitted set), writes the step's destination
// offsets (from its sorted keys) and does the segmentation pass's preparation for
// the merged run (seg_prep_device), and clears the look-back words and tickets of
// the group scan (gst, ctr[0]) and the live-set update (lst, ctr[1]). When the
// routing ran on another HIP stream, it also writes the step's permutation and
// destinations (perm_out, dest_out; null: the routing wrote them), after waiting
// for the routing's signal (rflag, rseq; null: no wait).
__global__ __launch_bounds__(256) void k_merge(KeyGeom g, RouteGeom rg, StreamCtl* ctl, int64_t cap, LiveSet live,
                                               const uint64_t* __restrict__ sk, const uint32_t* __restrict__ sperm,
                                               int64_t n, int flo, int fhi, uint64_t* mkey, int32_t* msrc,
                                               uint64_t* fp_in, const int64_t* n_dev, int shiftLa,
                                               const uint64_t* __restrict__ ht, int64_t htcap, int64_t* dest_offsets,
                                               SegJob sj, uint64_t* gst, uint64_t* lst, uint32_t* ctr,
                                               int32_t* perm_out, int32_t* dest_out, const uint64_t* rflag,
                                               uint64_t rseq, int32_t* status) {
  const int64_t nb = n;   // the host's count, or with n_dev its bound
  int64_t Lc = ctl->live;
  Lc = Lc < 0 ? 0 : (Lc > cap ? cap : Lc);
  // blocks past the merged run (the grid is sized for the largest count) leave at
  // once: only blocks that may hold elements wait for the routing, and they also do
  // the grid-stride clearing below
  const int64_t nwork_ = cdiv(Lc + nb, (int64_t)blockDim.x);
  const int64_t nwork = nwork_ < 1 ? 1 : (nwork_ > (int64_t)gridDim.x ? (int64_t)gridDim.x : nwork_);
  if ((int64_t)blockIdx.x >= nwork) return;
  const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, gstride = nwork * blockDim.x;
  // the live set's loads first (this thread's first element, the sampled keys): they
  // do not depend on the routing, whose signal may still be on its way; nothing in
  // the workspace and none of the step's inputs (not even its device count) is read
  // or written before the wait
  const int64_t t1 = gtid;
  uint64_t k1 = 0;
  uint32_t p1 = 0;
  if (t1 < Lc) k1 = live.key[t1];
  // sampled keys of both runs: the step's every s1-th (c1 of them), the live set's
  // every s2-th (c2); blocks past the merged run load none
  __shared__ uint64_t s_sk[MERGE_SAMPLES], s_lk[MERGE_SAMPLES];
  const int64_t s2 = Lc > MERGE_SAMPLES ? cdiv(Lc, MERGE_SAMPLES) : 1, c2 = cdiv(Lc, s2);
  constexpr int PER = MERGE_SAMPLES / 256;
  uint64_t a[PER], b[PER];
  if ((int64_t)blockIdx.x * blockDim.x < Lc + nb) {   // uniform across the block
#pragma unroll
    for (int r = 0; r < PER; ++r) {
      const int64_t i = threadIdx.x + r * 256;
      b[r] = i < c2 ? live.key[i * s2] : 0ull;
    }
  }
  route_wait(rflag, rseq, status);
  n = dev_n(n_dev, nb);
  const int64_t s1 = n > MERGE_SAMPLES ? cdiv(n, MERGE_SAMPLES) : 1, c1 = cdiv(n, s1);
  const bool sampling = (int64_t)blockIdx.x * blockDim.x < Lc + n;   // uniform across the block
  if (gtid == 0) {
    ctl->merged = Lc + n;
    ctl->merged1 = Lc + n + 1;
    ctl->knext = 0;
    ctl->ftot = 0;
    ctl->atot = 0;
    ctr[0] = 0;
    ctr[1] = 0;
    if (ctl->error) raise_status(status, ctl->error);
  }
  seg_prep_device(sj, Lc + n, gtid, gstride);
  if (gst) {
    const int64_t gl = cdiv(Lc + n + 1, GROUP_SCAN_TILE) * GROUP_SCAN_WORDS;
    for (int64_t i = gtid; i < gl; i += gstride) gst[i] = 0;
    const int64_t ll = cdiv(Lc + n, LU_TILE) * 3;
    for (int64_t i = gtid; i < ll; i += gstride) lst[i] = 0;
  }
  if (dest_offsets && n == 0 && gtid == 0)
    for (uint32_t x = 0; x <= rg.num_dest; ++x) dest_offsets[x] = 0;
  bool late = false;
  if (t1 >= Lc && t1 < Lc + n) {
    k1 = sk[t1 - Lc];
    p1 = sperm[t1 - Lc];
    p1 = p1 < (uint32_t)n ? p1 : 0u;
  }
  if (sampling) {
    // all of a thread's sample loads first (independent, in flight together)
#pragma unroll
    for (int r = 0; r < PER; ++r) {
      const int64_t i = threadIdx.x + r * 256;
      a[r] = i < c1 ? sk[i * s1] : 0ull;
    }
#pragma unroll
    for (int r = 0; r < PER; ++r) {
      const int64_t i = threadIdx.x + r * 256;
      if (i < c1) s_sk[i] = a[r];
      if (i < c2) s_lk[i] = b[r];
    }
    __syncthreads();
  }
  const int nl = fhi - flo + 1;
  uint64_t fp[ALTO_MAX_LEVELS];
  int sh[ALTO_MAX_LEVELS];
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
    fp[q] = 0;
    sh[q] = q < nl ? g.shift[flo + q] : 64;
  }
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < Lc + n; t += (int64_t)gridDim.x * blockDim.x) {
    if (t < Lc) {
      const uint64_t k = t == t1 ? k1 : live.key[t];
#pragma unroll
      for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
        if (q < nl)
          fp[q] += fan_term(g.fkey, flo + q, key_prefix(k, sh[q]), (uint32_t)live.fan[(int64_t)(flo + q - 1) * cap + t]);
      // number of step keys < k: c sampled ones, so between (c - 1) s1 + 1 and c s1
      int64_t a = 0, b = c1;
      while (a < b) {
        const int64_t mid = (a + b) >> 1;
        if (dk_less(rg, s_sk[mid], k)) a = mid + 1; else b = mid;
      }
      int64_t lo = a == 0 ? 0 : (a - 1) * s1 + 1, hi = a < c1 ? a * s1 : n;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (dk_less(rg, sk[mid], k)) lo = mid + 1; else hi = mid;
      }
      mkey[t + lo] = k;
      msrc[t + lo] = (int32_t)(-1 - t);
    } else {
      const int64_t j = t - Lc;
      const uint64_t k = t == t1 ? k1 : sk[j];
      const uint32_t pr = t == t1 ? p1 : sperm[j];
      const uint32_t pj = pr < (uint32_t)n ? pr : 0u;   // always, unless a routing wait gave up
      late |= emitted_has(key_prefix(k, shiftLa), ht, htcap);
      // number of live keys <= k: c sampled ones, so between (c - 1) s2 + 1 and c s2
      int64_t a = 0, b = c2;
      while (a < b) {
        const int64_t mid = (a + b) >> 1;
        if (!dk_less(rg, k, s_lk[mid])) a = mid + 1; else b = mid;
      }
      int64_t lo = a == 0 ? 0 : (a - 1) * s2 + 1, hi = a < c2 ? a * s2 : Lc;
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (!dk_less(rg, k, live.key[mid])) lo = mid + 1; else hi = mid;
      }
      mkey[j + lo] = k;
      msrc[j + lo] = (int32_t)pj;
      if (perm_out) perm_out[j] = (int32_t)pj;
      if (dest_out) dest_out[pj] = (int32_t)dest_of_key(rg, k);
      if (dest_offsets) {
        // the step's destination offsets, where the destination changes in its sorted keys
        const uint32_t d = dest_of_key(rg, k);
        if (j == 0) {
          for (uint32_t x = 0; x <= d; ++x) dest_offsets[x] = 0;
        } else {
          const uint32_t dp = dest_of_key(rg, sk[j - 1]);
          for (uint32_t x = dp + 1; x <= d; ++x) dest_offsets[x] = j;
        }
        if (j == n - 1)
          for (uint32_t x = d + 1; x <= rg.num_dest; ++x) dest_offsets[x] = n;
      }
    }
  }
  if (late) raise_status(status, ALTO_E_LATE);
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
    if (q < nl) {
      const uint64_t v = wave_sum(fp[q]);
      if (lane_id() == 0 && v) atomicAdd((unsigned long long*)&fp_in[flo + q], (unsigned long long)v);
    }
  }
}

// The step's end, by one thread once every error of the step that can still be
// raised is known: the handle is poisoned if the step reported an error.
__device__ inline void stream_poison(StreamCtl* ctl, int32_t* status) {
  const int32_t sv = __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (sv != 0 && ctl->error == 0) ctl->error = sv;
}

// The live-set update. Per merged element: kept (its group is not released) or
// not. A kept element goes to the new live set at its rank among the kept ones
// (exclusive scan over the merged run in one pass: tiles by ticket, a block scan,
// a look-back over earlier tiles by one wave per scanned value). MEAN: a released
// carried element frees its arena slot (listed in fslot, in scan order) and a kept
// step element needs one (listed in alist with its live position and step row,
// for k_arena_slots). The group of each element comes from the segmentation
// pass's boundary words (gw). The last tile writes the totals and the new live
// count; a live set over capacity is found from the total (the elements past it
// are not written), so with CONCAT the last tile also ends the step.
// The kept elements' fields are loaded before the scan (they do not depend on the
// ranks), all of a thread's elements at once; fans of the first NFP levels too, the
// others level by level after it.
static_assert(SEG_IT % LU_IT == 0, "a thread's elements lie in one boundary word");

// CONCAT: the same kernel also copies the emitted groups' tokens (the chunks that
// the group kernel listed), one wave per chunk, in the blocks that have no tile
// (beside the tiles, not after them); only when every block has a tile, after the
// tiles.
struct ConcatJob {
  const Chunk* chunks;     // long groups' chunks (long_cap entries)
  const int64_t* nlong;
  const Chunk* chunks_s;   // short groups' chunks (short_cap entries)
  const int64_t* nshort;
  int64_t long_cap, short_cap;
  MergedSrc src;
  int32_t* tok;            // null: no concatenation here
  int64_t cap_tokens;
};

// The concatenation by the blocks without a tile: wave cw of nw (numbered from the
// grid's end) copies chunks cw, cw + nw, ... of the long then the short groups;
// its first chunk was loaded before the counts were known (c0l = chunks[cw],
// c0s = chunks_s[cw]: used when the counts place chunk cw there).
__device__ inline void concat_role(const ConcatJob& cj, int64_t cw, int64_t nw, const Chunk& c0l, const Chunk& c0s) {
  const int64_t NB = *cj.nlong, NS = *cj.nshort;
  const int lane = lane_id();
  for (int64_t c = cw; c < NB + NS; c += nw) {
    Chunk ch;
    if (c == cw && c < NB) ch = c0l;
    else if (c == cw && NB == 0) ch = c0s;
    else ch = c < NB ? cj.chunks[c] : cj.chunks_s[c - NB];
    for (int r = lane; r < ch.len; r += ALTO_WAVE) {
      const int64_t o = ch.out + r;
      if (o < cj.cap_tokens) cj.tok[o] = cj.src.p32_of(cj.src.row(ch.begin + r));
    }
  }
}

// The fan fingerprint comparison when the group kernel accumulated the group
// level's node terms itself (so it cannot compare them): done by the live-set
// update's last tile, before it ends the step (levels lo..hi, in: null = none).
struct FpCheck {
  const uint64_t* in;
  const uint64_t* nodes;
  int32_t lo, hi;
};

template <int NFP>
__global__ __launch_bounds__(LU_NT) void k_live_update(KeyGeom g, LevelNodes L, const uint2* __restrict__ gw,
                                                       const uint64_t* __restrict__ mkey,
                                                       const int32_t* __restrict__ msrc, StreamCtl* ctl,
                                                       int64_t cap, LiveSet old, LiveSet nw,
                                                       const int32_t* __restrict__ sp32,
                                                       const int32_t* __restrict__ sfan, int64_t sfan_ld, int mean,
                                                       int32_t* fslot, int64_t* alist, uint64_t* st, uint32_t* ctr,
                                                       ConcatJob cj, FpCheck fpc, int64_t max_emit, int64_t ncap,
                                                       int32_t* status) {
  constexpr uint64_t F21 = (1ull << 21) - 1ull;   // a tile's counts fit 21 bits (LU_TILE < 2^21)
  // the sources, keys and boundary word of the tile this block most likely takes
  // first (its own index), loaded before the merged count and the ticket have
  // arrived (the merged run's buffers hold ncap elements; those past the count are
  // not used)
  const int64_t gt = blockIdx.x;
  const bool spec = blockIdx.x < LU_SPEC_BLOCKS;   // the grid is sized for the largest count
  // the first chunk of this block's waves in the concatenation, if it has no tile
  const int64_t cw = ((int64_t)gridDim.x - 1 - (int64_t)blockIdx.x) * (LU_NT / ALTO_WAVE) + threadIdx.x / ALTO_WAVE;
  Chunk c0l{}, c0s{};
  if (cj.tok) {
    if (cw < cj.long_cap) c0l = cj.chunks[cw];
    if (cw < cj.short_cap) c0s = cj.chunks_s[cw];
  }
  int32_t msg[LU_IT];
  uint64_t kkg[LU_IT];
  uint2 wg = make_uint2(0u, 0u);
  if (spec) {
    const int64_t eg = gt * LU_TILE + (int64_t)threadIdx.x * LU_IT;
#pragma unroll
    for (int i = 0; i < LU_IT; ++i) {
      msg[i] = eg + i < ncap ? msrc[eg + i] : 0;
      kkg[i] = eg + i < ncap ? mkey[eg + i] : 0ull;
    }
    if (eg < ncap) wg = gw[eg / SEG_IT];
  }
  const int64_t M = ctl->merged;
  const int64_t ntiles = cdiv(M, LU_TILE);
  const int nf = g.depth - 1;
  __shared__ uint64_t s_w[LU_NT / ALTO_WAVE];
  __shared__ int64_t s_ex[3];
  __shared__ uint32_t s_tile;
  const int64_t idle = (int64_t)gridDim.x - ntiles;   // blocks without a tile
  if (cj.tok && idle > 0 && (int64_t)blockIdx.x >= ntiles) concat_role(cj, cw, idle * (LU_NT / ALTO_WAVE), c0l, c0s);
  if (ntiles == 0) {
    // nothing carried and nothing arrived
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      ctl->live = 0;
      if (!mean) stream_poison(ctl, status);
    }
    return;
  }
  if ((int64_t)blockIdx.x < ntiles) {
    bool first = true;
    while (true) {
      // a single tile is block 0's without a ticket (it waits for no other tile)
      if (ntiles > 1 && threadIdx.x == 0) s_tile = atomicAdd(ctr, 1u);
      __syncthreads();
      const int64_t tile = ntiles > 1 ? (int64_t)s_tile : (first ? 0 : 1);
      first = false;
      if (tile >= ntiles) break;   // uniform
      const int64_t e0 = tile * LU_TILE + (int64_t)threadIdx.x * LU_IT;
      int32_t ms[LU_IT];
      uint32_t km = 0, fm = 0, am = 0;   // bit i: element e0 + i is kept / frees a slot / needs one
      // the fields of a kept element are loaded with the flags (they depend on its
      // source only), and used only if it is kept
      uint64_t kk[LU_IT];
      int32_t pv[LU_IT], sv[LU_IT], fv[NFP > 0 ? NFP : 1][LU_IT];
#pragma unroll
      for (int i = 0; i < LU_IT; ++i) {
        kk[i] = 0;
        pv[i] = sv[i] = 0;
#pragma unroll
        for (int l = 0; l < NFP; ++l) fv[l][i] = 0;
      }
      if (e0 < M) {
        const bool pre = spec && tile == gt;   // uniform
        uint2 w;
        if (pre) {
#pragma unroll
          for (int i = 0; i < LU_IT; ++i) {
            ms[i] = e0 + i < M ? msg[i] : 0;
            kk[i] = e0 + i < M ? kkg[i] : 0ull;
          }
          w = wg;
        } else {
          if (e0 + LU_IT <= M) {
            const int4* p = reinterpret_cast<const int4*>(msrc + e0);
#pragma unroll
            for (int v = 0; v < LU_IT / 4; ++v) {
              const int4 q = p[v];
              ms[4 * v] = q.x;
              ms[4 * v + 1] = q.y;
              ms[4 * v + 2] = q.z;
              ms[4 * v + 3] = q.w;
            }
          } else {
#pragma unroll
            for (int i = 0; i < LU_IT; ++i) ms[i] = e0 + i < M ? msrc[e0 + i] : 0;
          }
#pragma unroll
          for (int i = 0; i < LU_IT; ++i) kk[i] = e0 + i < M ? mkey[e0 + i] : 0ull;
          w = gw[e0 / SEG_IT];
        }
        const int off = (int)(e0 % SEG_IT);
        const uint32_t fs = w.y >> off;                                          // bit i: e0 + i starts a group
        const int32_t u0 = (int32_t)w.x + __popc(w.y & ((1u << off) - 1u));      // groups started before e0
        bool okv[LU_IT];
#pragma unroll
        for (int i = 0; i < LU_IT; ++i) {
          const int32_t u = u0 + __popc(fs & ((2u << i) - 1u)) - 1;
          const bool in = e0 + i < M;
          okv[i] = in && u >= 0 && L.ok[u];
          if (!in) continue;
          const int32_t s = ms[i];
          const bool car = s < 0;
          const int64_t li = -1 - (int64_t)s;
          pv[i] = car ? old.p32[li] : (sp32 ? sp32[s] : 0);
          sv[i] = (car && mean) ? old.slot[li] : 0;
#pragma unroll
          for (int l = 0; l < NFP; ++l)
            fv[l][i] = car ? old.fan[(int64_t)l * cap + li] : sfan[(int64_t)l * sfan_ld + s];
        }
#pragma unroll
        for (int i = 0; i < LU_IT; ++i) {
          if (e0 + i >= M) break;
          const bool ok = okv[i];
          const bool carried = ms[i] < 0;
          km |= (ok ? 0u : 1u) << i;
          fm |= ((mean && ok && carried) ? 1u : 0u) << i;
          am |= ((mean && !ok && !carried) ? 1u : 0u) << i;
        }
      }
      const uint64_t c = (uint64_t)__popc(km) | ((uint64_t)__popc(fm) << 21) | ((uint64_t)__popc(am) << 42);
      uint64_t tot;
      const uint64_t x = block_excl_scan<uint64_t, LU_NT>(c, s_w, &tot);
      const int wv = threadIdx.x / ALTO_WAVE;
      if (wv < 3) {
        const uint64_t tq = (tot >> (21 * wv)) & F21;
        if (lane_id() == 0) lb64_publish(st + wv, tile, 3, tq);
        const uint64_t exq = lb64_resolve_wave(st + wv, tile, 3, tq, status);
        if (lane_id() == 0) {
          s_ex[wv] = (int64_t)exq;
          if (tile == ntiles - 1) {
            const int64_t T = (int64_t)(exq + tq);
            if (wv == 0) {
              if (T > cap) raise_status(status, ALTO_E_CAPACITY);
              if (ctl->emitted > max_emit) raise_status(status, ALTO_E_CAPACITY);   // the emitted set's limit
              if (fpc.in)
                for (int m = fpc.lo; m <= fpc.hi; ++m)
                  if (fpc.in[m] != fpc.nodes[m]) raise_status(status, ALTO_E_FANOUT);
              ctl->live = T > cap ? cap : T;   // read by the next step only
              if (!mean) stream_poison(ctl, status);
            } else {
              __hip_atomic_store(wv == 1 ? &ctl->ftot : &ctl->atot, T, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
          }
        }
      }
      __syncthreads();
      const int64_t k0 = s_ex[0] + (int64_t)(x & F21);
      int64_t r0 = k0, r1 = s_ex[1] + (int64_t)((x >> 21) & F21), r2 = s_ex[2] + (int64_t)((x >> 42) & F21);
#pragma unroll
      for (int i = 0; i < LU_IT; ++i) {
        const int32_t s = ms[i];
        if ((km >> i) & 1u) {
          const int64_t ki = r0++;
          const bool fits = ki < cap;
          if (fits) {
            nw.key[ki] = kk[i];
            nw.p32[ki] = pv[i];
#pragma unroll
            for (int l = 0; l < NFP; ++l) nw.fan[(int64_t)l * cap + ki] = fv[l][i];
            if (mean) nw.slot[ki] = s < 0 ? sv[i] : 0;   // a step element's slot: k_arena_slots
          }
          if (mean && s >= 0) alist[r2++] = fits ? ((ki << 32) | (int64_t)(uint32_t)s) : -1;
        } else if ((fm >> i) & 1u) {
          fslot[r1++] = sv[i];
        }
      }
      // fans of the other levels, one level at a time
      for (int l = NFP; l < nf; ++l) {
        int32_t f[LU_IT];
#pragma unroll
        for (int i = 0; i < LU_IT; ++i) {
          const int32_t s = ms[i];
          f[i] = ((km >> i) & 1u) ? (s < 0 ? old.fan[(int64_t)l * cap + (-1 - (int64_t)s)]
                                           : sfan[(int64_t)l * sfan_ld + s])
                                  : 0;
        }
        int64_t ki = k0;
#pragma unroll
        for (int i = 0; i < LU_IT; ++i) {
          if (!((km >> i) & 1u)) continue;
          if (ki < cap) nw.fan[(int64_t)l * cap + ki] = f[i];
          ++ki;
        }
      }
      __syncthreads();   // s_ex and the ticket are reused by the next tile
    }
    if (cj.tok && idle <= 0)
      concat_chunks_wave<MergedSrc>(cj.chunks, *cj.nlong, cj.chunks_s, *cj.nshort, cj.src, cj.tok, cj.cap_tokens,
                                    (int64_t)blockIdx.x * (LU_NT / ALTO_WAVE) + threadIdx.x / ALTO_WAVE,
                                    (int64_t)gridDim.x * (LU_NT / ALTO_WAVE));
  }
}

// MEAN, after the live-set update (and the mean gather): the means of the emitted
// groups of several chunks (mean_combine_chunks); the arena slots of the kept step elements
// (the slots freed this step first, in scan order, then the top of the free-slot
// stack), their rows copied in (one wave per row), the freed slots not reused
// pushed onto the stack. The stack top is read from top[par] and written to
// top[par ^ 1] (blocks read it while the first one writes); that thread also
// ends the step (every error of the step is known from the totals by then).
__global__ __launch_bounds__(256) void k_arena_slots(StreamCtl* ctl, int64_t cap, const int64_t* __restrict__ alist,
                                                     const int32_t* __restrict__ fslot, int32_t* stack, LiveSet nw,
                                                     const float* __restrict__ spf, int dim, int v4, float* arena,
                                                     int par, const Chunk* __restrict__ chunks, const int64_t* nchunks,
                                                     const double* __restrict__ part, float* mean, int64_t cap_groups,
                                                     int32_t* status) {
  // the emitted groups of several chunks first (their chunks' partial sums)
  if (mean) mean_combine_chunks(chunks, *nchunks, part, dim, mean, cap_groups, blockIdx.x, gridDim.x);
  const int64_t A = ctl->atot, F = ctl->ftot, top = ctl->top[par];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    // the stack after the step; too few free slots, or more than the capacity
    // (the slots past either end are neither taken nor written)
    int64_t t = top - A + F;
    if (t < 0 || t > cap) {
      raise_status(status, ALTO_E_CAPACITY);
      t = t < 0 ? 0 : cap;
    }
    ctl->top[par ^ 1] = t;
    stream_poison(ctl, status);
  }
  const int lane = lane_id();
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / ALTO_WAVE;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / ALTO_WAVE;
  for (int64_t a = wave; a < A; a += nwaves) {   // wave-uniform
    const int64_t v = alist[a];
    if (v < 0) continue;   // its element did not fit the live set (reported)
    int64_t slot = -1;
    if (a < F) {
      slot = fslot[a];
    } else {
      const int64_t p = top - 1 - (a - F);
      if (p >= 0 && p < cap) slot = stack[p];
    }
    if (slot < 0 || slot >= cap) continue;   // past the stack (reported above)
    const int64_t ki = v >> 32, row = v & 0xFFFFFFFFll;
    if (lane == 0) nw.slot[ki] = (int32_t)slot;
    if (v4) {
      const float4* src = reinterpret_cast<const float4*>(spf + row * dim);
      float4* dst = reinterpret_cast<float4*>(arena + slot * (int64_t)dim);
      for (int c = lane; c < dim / 4; c += ALTO_WAVE) dst[c] = src[c];
    } else {
      const float* src = spf + row * dim;
      float* dst = arena + slot * (int64_t)dim;
      for (int c = lane; c < dim; c += ALTO_WAVE) dst[c] = src[c];
    }
  }
  for (int64_t f = A + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; f < F; f += (int64_t)gridDim.x * blockDim.x) {
    const int64_t p = top + (f - A);
    if (p >= 0 && p < cap) stack[p] = fslot[f];
  }
}

// Group records for in-order release: the level-La prefix of every group of the
// merged run.
__global__ void k_rel_keys(LevelNodes L, const int64_t* Gp, const uint64_t* __restrict__ mkey, int shiftLa,
                           uint64_t* rkey) {
  const int64_t G = *Gp;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < G; u += (int64_t)gridDim.x * blockDim.x)
    rkey[u] = key_prefix(mkey[L.start[u]], shiftLa);
}

// In-order release (Section 3.2: the parallelised stream is put back in its
// original order). Over the group records sorted by key, the first record of each
// parent's run walks the run in child order from the parent's release position and
// releases complete children until the first missing or incomplete one; the
// completion flags of the run's groups become their release flags. One thread per
// parent, so a parent's position has one writer per step.
// ridx null: the records are already in key order within each parent (the merged
// run's own order, when the route level is above the aggregation level).
__global__ void k_release(LevelNodes L, const int64_t* Gp, const uint64_t* __restrict__ rsk,
                          const uint32_t* __restrict__ ridx, int cbits, uint64_t cmask, uint64_t* pht, int32_t* pcur,
                          int64_t htcap, int32_t* status) {
  const int64_t R = *Gp;
  bool full = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < R; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t P = rsk[i] >> cbits;
    if (i > 0 && (rsk[i - 1] >> cbits) == P) continue;   // not the first record of its parent
    int64_t h = (int64_t)(mix64(P ^ 0x5851F42D4C957F2Dull) & (uint64_t)(htcap - 1));
    int64_t slot = -1;
    for (int64_t probe = 0; probe < htcap; ++probe) {
      const uint64_t v = pht[h];   // a slot changes once, from empty; the CAS settles a stale empty
      if (v == P) {
        slot = h;
        break;
      }
      if (v == HT_EMPTY) {
        const uint64_t old = atomicCAS((unsigned long long*)&pht[h], (unsigned long long)HT_EMPTY, (unsigned long long)P);
        if (old == HT_EMPTY || old == P) {
          slot = h;
          break;
        }
      }
      h = (h + 1) & (htcap - 1);
    }
    if (slot < 0) full = true;
    int64_t cur = slot >= 0 ? pcur[slot] : -1;   // table full: nothing is released
    bool open = slot >= 0;
    for (int64_t j = i; j < R && (rsk[j] >> cbits) == P; ++j) {
      const int64_t u = ridx ? (int64_t)ridx[j] : j;
      const bool rel = open && L.ok[u] && (int64_t)(rsk[j] & cmask) == cur;
      if (rel) ++cur;
      else open = false;
      L.ok[u] = rel ? 1 : 0;
    }
    if (slot >= 0) pcur[slot] = (int32_t)cur;
  }
  if (full) raise_status(status, ALTO_E_CAPACITY);
}

// pending groups of the live set
__global__ void k_pend_flags(KeyGeom g, int La, const StreamCtl* ctl, int64_t cap, const uint64_t* __restrict__ key,
                             int32_t* flag, int64_t* len1) {
  int64_t Lc = ctl->live;
  Lc = Lc < 0 ? 0 : (Lc > cap ? cap : Lc);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e <= Lc; e += (int64_t)gridDim.x * blockDim.x) {
    if (e == Lc) flag[e] = 0;
    else flag[e] = (e == 0 || key_prefix(key[e], g.shift[La]) != key_prefix(key[e - 1], g.shift[La])) ? 1 : 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *len1 = Lc + 1;
}

__global__ void k_pend_write(KeyGeom g, int La, const StreamCtl* ctl, int64_t cap, const uint64_t* __restrict__ key,
                             const int32_t* __restrict__ scan, GroupOut out, int32_t* status) {
  int64_t Lc = ctl->live;
  Lc = Lc < 0 ? 0 : (Lc > cap ? cap : Lc);
  const int64_t P = scan[Lc];
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < Lc; e += (int64_t)gridDim.x * blockDim.x) {
    const bool start = (e == 0) || key_prefix(key[e], g.shift[La]) != key_prefix(key[e - 1], g.shift[La]);
    if (!start) continue;
    const int64_t id = scan[e];
    int64_t end = e + 1;
    while (end < Lc && key_prefix(key[end], g.shift[La]) == key_prefix(key[e], g.shift[La])) ++end;
    if (id < out.cap_groups) {
      if (out.pend_key) out.pend_key[id] = key_prefix(key[e], g.shift[La]);
      if (out.pend_count) out.pend_count[id] = end - e;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    out.counts[0] = out.counts[1] = out.counts[2] = 0;
    out.counts[3] = P;
    if (P > out.cap_groups) raise_status(status, ALTO_E_CAPACITY);
  }
}

}  // namespace

struct alto_stream {
  KeyGeom g;
  RouteGeom rg;
  alto_agg agg;
  int Lr, D;
  int64_t cap, max_groups, htcap;
  StreamCtl* ctl;
  LiveSet live[2];
  int cur;
  float* arena;
  int32_t* stack;
  uint64_t* ht;
  uint64_t* pht;   // in-order release: parent prefixes
  int32_t* pcur;   // in-order release: next child to release per parent
  int32_t* pflag;
  int32_t* ppart;
  int64_t* plen;
  // overlapped steps (alto_stream_step_overlap): the workspace of the next step,
  // per workspace the end of its step, the routing-done words (device, one per
  // workspace) and the last sequence number
  int wslot;
  bool ev_made;
  bool ev_used[2];
  hipEvent_t ev_done[2];
  uint64_t* rflag;
  uint64_t rseq;
};

namespace {

int64_t ht_capacity(int64_t max_groups) {
  int64_t c = 1024;
  while (c < 2 * max_groups) c <<= 1;
  return c;
}

void carve_state(const KeyGeom& g, const alto_agg& agg, int64_t cap, int64_t max_groups, WsCarver& c, alto_stream* s) {
  const int nf = g.depth - 1;
  s->ctl = c.take<StreamCtl>(1);
  for (int k = 0; k < 2; ++k) {
    s->live[k].key = c.take<uint64_t>(cap);
    s->live[k].p32 = c.take<int32_t>(cap);
    s->live[k].fan = c.take<int32_t>((int64_t)nf * cap);
    s->live[k].slot = agg.op == ALTO_MEAN_F32 ? c.take<int32_t>(cap) : nullptr;
  }
  if (agg.op == ALTO_MEAN_F32) {
    s->arena = c.take<float>(cap * (int64_t)agg.dim);
    s->stack = c.take<int32_t>(cap);
  } else {
    s->arena = nullptr;
    s->stack = nullptr;
  }
  s->htcap = ht_capacity(max_groups);
  s->ht = c.take<uint64_t>(s->htcap);
  if (agg.release == ALTO_RELEASE_IN_ORDER && agg.level >= 2) {   // parents <= groups
    s->pht = c.take<uint64_t>(s->htcap);
    s->pcur = c.take<int32_t>(s->htcap);
  } else {
    s->pht = nullptr;
    s->pcur = nullptr;
  }
  s->pflag = c.take<int32_t>(cap + 1);
  s->ppart = c.take<int32_t>(SCAN_MAX_BLOCKS + 1);
  s->plen = c.take<int64_t>(4);
  s->rflag = c.take<uint64_t>(2 * ROUTE_FLAG_STRIDE);
}

bool layout_valid(const alto_layout* l) {
  if (!l || l->depth < 2 || l->depth > ALTO_MAX_LEVELS) return false;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) {
    if (l->bits[i] < 1 || l->bits[i] > 32) return false;
    total += l->bits[i];
  }
  return total <= 63;
}

bool stream_args_ok(const alto_layout* l, const alto_agg* a, int64_t cap, int64_t max_groups) {
  if (!layout_valid(l) || !a) return false;
  if (a->level < 1 || a->level > l->depth - 1 || a->mask_level != 0) return false;
  if (a->op != ALTO_CONCAT_I32 && a->op != ALTO_MEAN_F32) return false;
  if (a->op == ALTO_MEAN_F32 && (a->dim < 1 || a->dim > (1 << 20))) return false;
  if (a->release != ALTO_RELEASE_COMPLETE && a->release != ALTO_RELEASE_IN_ORDER) return false;
  if (cap < 1 || cap > (int64_t)(1 << 30) || max_groups < 1 || max_groups > ((int64_t)1 << 40)) return false;
  return true;
}

GroupOut dev_out(const alto_groups* o) {
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
  g.mask_key = nullptr;
  g.mask = nullptr;
  g.pend_key = o->pend_key;
  g.pend_count = o->pend_count;
  g.counts = o->counts;
  return g;
}

}  // namespace

extern "C" {

size_t alto_stream_state_bytes(const alto_layout* layout, const alto_agg* agg, int64_t max_live_leaves,
                               int64_t max_groups) {
  if (!stream_args_ok(layout, agg, max_live_leaves, max_groups)) return 0;
  KeyGeom g = make_geom(layout);
  WsCarver c{nullptr, (size_t)-1, 0, true};
  alto_stream s;
  carve_state(g, *agg, max_live_leaves, max_groups, c, &s);
  return c.off;
}

int alto_stream_create(const alto_layout* layout, int32_t route_level, int32_t num_dest, const alto_agg* agg,
                       int64_t max_live_leaves, int64_t max_groups, void* state, size_t state_bytes,
                       hipStream_t stream, alto_stream** out) {
  if (!out || !state || !stream_args_ok(layout, agg, max_live_leaves, max_groups)) return ALTO_E_ARG;
  if (route_level < 1 || route_level > agg->level || num_dest < 1 || num_dest > (1 << 24)) return ALTO_E_ARG;
  alto_stream* s = new alto_stream;
  s->g = make_geom(layout);
  s->rg = make_route(s->g, route_level, num_dest);
  s->agg = *agg;
  s->Lr = route_level;
  s->D = num_dest;
  s->cap = max_live_leaves;
  s->max_groups = max_groups;
  s->cur = 0;
  s->wslot = 0;
  s->ev_made = false;
  s->ev_used[0] = s->ev_used[1] = false;
  s->rseq = fresh_fp_key();   // random base of the routing sequence numbers
  WsCarver c{(char*)state, state_bytes, 0, true};
  carve_state(s->g, *agg, max_live_leaves, max_groups, c, s);
  if (!c.ok) {
    delete s;
    return ALTO_E_ARG;
  }
  k_stream_init<<<grid_for(s->htcap > s->cap ? s->htcap : s->cap, 256), 256, 0, stream>>>(s->ctl, s->stack, s->cap,
                                                                                         s->ht, s->htcap, s->pht,
                                                                                         s->pcur);
  if (hipGetLastError() != hipSuccess) {
    delete s;
    return ALTO_E_HIP;
  }
  *out = s;
  return ALTO_OK;
}

}  // extern "C"

namespace {

// One step; with rslot >= 0, the routing runs on route_st and the rest on st after
// it (the merge waits for routing-done word rslot), and the merge writes the
// caller's perm and dest.
int stream_step(alto_stream* s, const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* payload_i32,
                const float* payload_f32, int64_t n, const int64_t* n_dev, int32_t* perm, int64_t* dest_offsets,
                int32_t* dest, alto_groups* emitted, int32_t* status, void* ws, size_t ws_bytes,
                hipStream_t route_st, hipStream_t st, int rslot) {
  // n: the step's count (n_dev null) or its bound (the count is *n_dev on the device)
  if (!s || !status || !emitted || !emitted->counts || n < 0 || n > (int64_t)INT32_MAX / 2 ||
      emitted->cap_groups < 0 || emitted->cap_tokens < 0)
    return ALTO_E_ARG;
  const alto_agg& agg = s->agg;
  const bool mean = agg.op == ALTO_MEAN_F32;
  if (n > 0 && (!keys || !fan || fan_ld < n || !ws || (!mean && !payload_i32) || (mean && !payload_f32)))
    return ALTO_E_ARG;
  const KeyGeom& g = s->g;
  const int d = g.depth, La = agg.level;
  GroupOut o = dev_out(emitted);
  s->g.fkey = fresh_fp_key();   // a fresh fingerprint key for every step
  if (n == 0) {
    k_stream_begin<<<1, 1, 0, st>>>(s->ctl, status);   // otherwise the merge reports a poisoned handle
    empty_outputs(o, dest_offsets, s->D, st);
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  ProfScope ps_total(PH_TOTAL, st);
  const int64_t ntot = s->cap + n;
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  alto_agg plan_agg = agg;
  AggBufs b;
  plan_buffers(g, ntot, s->rg, &plan_agg, s->Lr, c, b);
  if (!c.ok) return ALTO_E_ARG;
  // 1. route the step on its own
  // (destination offsets: written by the merge, from the step's sorted keys)
  const bool split = rslot >= 0;
  int rc = route_run(g, s->rg, keys, n, b, split ? nullptr : perm, dest_offsets, split ? nullptr : dest, fan, fan_ld,
                     La, d - 1, status, split ? route_st : st, true, false, false, n_dev);
  if (rc) return rc;
  uint64_t* rflag = nullptr;
  const uint64_t rseq = split ? ++s->rseq : 0;
  if (split) {
    rflag = s->rflag + rslot * ROUTE_FLAG_STRIDE;
    k_route_signal<<<1, 64, 0, route_st>>>(rflag, rseq);
  }
  prof_begin(PH_SEGMENT, st);
  const uint32_t* sperm = b.perm_used;
  LiveSet& old = s->live[s->cur];
  LiveSet& nw = s->live[s->cur ^ 1];
  uint64_t* mkey = b.tmp_keys;
  int32_t* msrc = reinterpret_cast<int32_t*>(b.tmp_vals);
  const int64_t* Mp = &s->ctl->merged;
  // look-back words, after the segmentation pass's in the sort's status words:
  // the group scan's, then the live-set update's; tickets after the pass's
  const int64_t seg_words = (cdiv(ntot, SEG_TILE) * SEG_LB_STRIDE + 1) & ~(int64_t)1;
  const int64_t g_words = cdiv(ntot + 1, GROUP_SCAN_TILE) * GROUP_SCAN_WORDS;
  const int64_t l_words = cdiv(ntot, LU_TILE) * 3;
  if (seg_words + 2 * (g_words + l_words) > (int64_t)b.os_ntiles * 2 * SORT_BUCKETS) return ALTO_E_ARG;   // never
  uint64_t* gst = reinterpret_cast<uint64_t*>(b.os_status + seg_words);
  uint64_t* lst = gst + g_words;
  SegJob j;
  memset(&j, 0, sizeof(j));
  j.keys = mkey;
  j.idx = nullptr;
  j.n_dev = Mp;
  j.n_max = ntot;
  j.elem_level = d;
  j.lo = La;
  j.fan = fan;
  j.fan_ld = fan_ld;
  j.fan_base = 1;
  j.src = msrc;
  j.fan2 = old.fan;
  j.fan2_ld = s->cap;
  j.check_dup = 1;
  for (int m = 0; m <= ALTO_MAX_LEVELS; ++m) j.lv[m] = b.lv[m];
  j.nnodes = b.nnodes;
  j.lb_status = b.os_status;
  j.lb_ctr = b.os_ctr;
  j.lb_tiles = b.os_ntiles * 2 * SORT_BUCKETS / SEG_LB_STRIDE;   // the sort's status words, free by now
  j.fp_nodes = b.fp_nodes;
  j.status = status;
  j.no_prep = 1;   // done by the merge
  j.gw = b.gw;
  // the group kernel evaluates the group level's completion (with in-order release,
  // the release kernels read it before the scan)
  j.fold_lo = s->pht ? 0 : 1;
  j.prefetch = 1;   // mkey holds ntot = n_max keys
  if (j.fold_lo) {
    // the pass records each group's first key for the group kernel, in the step's
    // sorted-key buffer (free once the merge has read it)
    b.lv[La].nkey = b.sk;
    j.lv[La].nkey = b.sk;
  }
  // 2. merge with the live set (also: late fragments, a poisoned handle, the step's
  // destination offsets, the clearing of the step's look-back words)
  // (with the routing on another stream at most one block per CU: the merge's
  // blocks wait for the routing, whose kernels need room on the CUs, e.g. the
  // one-workgroup sort's 1,024 threads and up to 107 KB of LDS)
  k_merge<<<grid_for(ntot, 256, split ? 256 : 4096), 256, 0, st>>>(
      g, s->rg, s->ctl, s->cap, old, b.sk, sperm, n, La, d - 1, mkey, msrc, b.fp_in, n_dev, g.shift[La], s->ht,
      s->htcap, dest_offsets, j, gst, lst, b.os_ctr + 1, split ? perm : nullptr, split ? dest : nullptr, rflag, rseq,
      status);
  // 3. nodes and completion over the merged run
  rc = seg_run(g, j, st);
  if (rc) return rc;
  bool words_clear = true;
  if (s->pht && s->Lr < La) {
    // in-order release, a parent's children in one destination: the merged run
    // already lists them in key order
    const int64_t* Gp = b.nnodes + La;
    k_rel_keys<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, mkey, g.shift[La], b.rkey);
    k_release<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, b.rkey, nullptr, g.shift[La - 1] - g.shift[La],
                                                   (uint64_t)g.tagmask[La], s->pht, s->pcur, s->htcap, status);
    ALTO_LAUNCH_CHECK();
  } else if (s->pht) {
    // in-order release, siblings in several destinations: group records by key (the
    // step's sort buffers are free after the merge), then each parent's run from
    // its release position
    const int64_t* Gp = b.nnodes + La;
    k_rel_keys<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, mkey, g.shift[La], b.rkey);
    SortBufs rb;
    memset(&rb, 0, sizeof(rb));
    rb.in_keys = b.rkey;
    rb.tmp_keys = b.sk;
    rb.tmp_vals = b.perm;
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
    rc = sort_pairs(rb, ntot, Gp, none, g.total - g.shift[La], false, st);
    if (rc) return rc;
    words_clear = false;   // the sort used them
    k_release<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, b.rsk, b.ridx, g.shift[La - 1] - g.shift[La],
                                                   (uint64_t)g.tagmask[La], s->pht, s->pcur, s->htcap, status);
    ALTO_LAUNCH_CHECK();
  }
  prof_end(PH_SEGMENT, st);
  // 4. emitted groups (payload over all of each group's leaves, in key order); their
  // record kernel also compares the fan fingerprints and fills the emitted set
  MergedSrc src{msrc, payload_i32, fan, fan_ld, payload_f32, old.p32, old.fan, s->cap, old.slot, s->arena, s->cap,
                agg.dim};
  GroupsExtra ex;
  memset(&ex, 0, sizeof(ex));
  ex.fp_in = b.fp_in;
  ex.fp_nodes = b.fp_nodes;
  ex.flo = La;
  ex.fhi = d - 1;
  ex.xlo = 1;
  ex.xhi = 0;
  ex.gst = gst;
  ex.gctr = b.os_ctr + 1;
  ex.cleared = words_clear ? 1 : 0;
  if (!words_clear) {
    ex.xst = lst;
    ex.xctr = b.os_ctr + 2;
    ex.xlen = Mp;
    ex.xtile = LU_TILE;
    ex.xper = 3;
  }
  ex.ht = s->ht;
  ex.htcap = s->htcap;
  ex.emit_count = &s->ctl->emitted;
  ex.defer_concat = mean ? 0 : 1;   // the live-set update copies the tokens
  ex.defer_combine = mean ? 1 : 0;  // the arena-slot kernel combines the chunks
  FpCheck fpc{nullptr, nullptr, 0, -1};
  if (j.fold_lo) {
    // the group kernel adds the group level's node terms: the comparison waits for
    // the live-set update
    fpc = FpCheck{b.fp_in, b.fp_nodes, La, d - 1};
    ex.fp_in = nullptr;
    ex.fold = 1;
    ex.fold_leafy = La + 1 == d ? 1 : 0;
    ex.fold_level = La;
    ex.fold_es = g.shift[La] - g.shift[d];
    ex.fold_keys = mkey;
    ex.fold_fp = b.fp_nodes;
  }
  rc = groups_run<MergedSrc>(g, s->rg, agg, src, mkey, ntot, b, nullptr, o, status, st, &ex);
  if (rc) return rc;
  // 5. survivors become the new live set
  int32_t* fslot = b.em;
  int64_t* alist = b.tokc;
  {
    const int nf = d - 1;
    ConcatJob cj;
    memset(&cj, 0, sizeof(cj));
    if (!mean && o.tok) {
      cj.chunks = b.chunks;
      cj.nlong = b.scal + 1;
      cj.chunks_s = b.chunks + b.short_base;
      cj.nshort = b.scal + 3;
      cj.long_cap = b.short_base;
      cj.short_cap = ntot + 1;
      cj.src = src;
      cj.tok = o.tok;
      cj.cap_tokens = o.cap_tokens;
    }
#define ALTO_LU_CASE(P)                                                                                          \
  k_live_update<P><<<grid_for(ntot, LU_TILE, 1024), LU_NT, 0, st>>>(g, b.lv[La], b.gw, mkey, msrc, s->ctl, s->cap, \
                                                                   old, nw, payload_i32, fan, fan_ld, mean ? 1 : 0, \
                                                                   fslot, alist, lst, b.os_ctr + 2, cj, fpc,      \
                                                                   s->max_groups, ntot, status)
    if (nf <= 1) ALTO_LU_CASE(1);
    else if (nf == 2) ALTO_LU_CASE(2);
    else ALTO_LU_CASE(3);
#undef ALTO_LU_CASE
  }
  if (mean) {
    const bool v4 = agg.dim % 4 == 0 && ((reinterpret_cast<uintptr_t>(payload_f32) | reinterpret_cast<uintptr_t>(s->arena)) & 15) == 0;
    k_arena_slots<<<grid_for(n * ALTO_WAVE, 256), 256, 0, st>>>(s->ctl, s->cap, alist, fslot, s->stack, nw,
                                                                 payload_f32, agg.dim, v4 ? 1 : 0, s->arena, s->cur,
                                                                 b.chunks, b.scal + 1, b.part, o.mean, o.cap_groups,
                                                                 status);
  }
  ALTO_LAUNCH_CHECK();
  s->cur ^= 1;
  return ALTO_OK;
}

}  // namespace

extern "C" {

int alto_stream_step_dev(alto_stream* s, const uint64_t* keys, const int32_t* fan, int64_t fan_ld,
                         const int32_t* payload_i32, const float* payload_f32, int64_t n, const int64_t* n_dev,
                         int32_t* perm, int64_t* dest_offsets, int32_t* dest, alto_groups* emitted, int32_t* status,
                         void* ws, size_t ws_bytes, hipStream_t st) {
  return stream_step(s, keys, fan, fan_ld, payload_i32, payload_f32, n, n_dev, perm, dest_offsets, dest, emitted,
                     status, ws, ws_bytes, st, st, -1);
}

int alto_stream_step_overlap(alto_stream* s, const uint64_t* keys, const int32_t* fan, int64_t fan_ld,
                             const int32_t* payload_i32, const float* payload_f32, int64_t n, const int64_t* n_dev,
                             int32_t* perm, int64_t* dest_offsets, int32_t* dest, alto_groups* emitted,
                             int32_t* status, void* ws0, void* ws1, size_t ws_bytes, hipStream_t route_stream,
                             hipStream_t st) {
  if (!s || !ws0 || !ws1 || ws0 == ws1) return ALTO_E_ARG;
  if (!s->ev_made) {
    for (int k = 0; k < 2; ++k)
      if (hipEventCreateWithFlags(&s->ev_done[k], hipEventDisableTiming) != hipSuccess) return ALTO_E_HIP;
    s->ev_made = true;
  }
  const int k = s->wslot;
  // the step two calls back used this workspace: its end on st comes first
  if (s->ev_used[k] && hipStreamWaitEvent(route_stream, s->ev_done[k], 0) != hipSuccess) return ALTO_E_HIP;
  const int rc = stream_step(s, keys, fan, fan_ld, payload_i32, payload_f32, n, n_dev, perm, dest_offsets, dest,
                             emitted, status, k ? ws1 : ws0, ws_bytes, route_stream, st, k);
  if (rc) return rc;
  if (hipEventRecord(s->ev_done[k], st) != hipSuccess) return ALTO_E_HIP;
  s->ev_used[k] = true;
  s->wslot = k ^ 1;
  return ALTO_OK;
}

int alto_stream_step(alto_stream* s, const uint64_t* keys, const int32_t* fan, int64_t fan_ld,
                     const int32_t* payload_i32, const float* payload_f32, int64_t n, int32_t* perm,
                     int64_t* dest_offsets, int32_t* dest, alto_groups* emitted, int32_t* status, void* ws,
                     size_t ws_bytes, hipStream_t st) {
  return alto_stream_step_dev(s, keys, fan, fan_ld, payload_i32, payload_f32, n, nullptr, perm, dest_offsets, dest,
                              emitted, status, ws, ws_bytes, st);
}

int alto_stream_pending(alto_stream* s, alto_groups* out, int32_t* status, hipStream_t st) {
  if (!s || !out || !out->counts || !status || out->cap_groups < 0) return ALTO_E_ARG;
  GroupOut o = dev_out(out);
  const LiveSet& L = s->live[s->cur];
  k_stream_begin<<<1, 1, 0, st>>>(s->ctl, status);
  k_pend_flags<<<grid_for(s->cap + 1, 256), 256, 0, st>>>(s->g, s->agg.level, s->ctl, s->cap, L.key, s->pflag, s->plen);
  int rc = scan_exclusive<int32_t>(s->pflag, s->pflag, s->cap + 1, s->plen, s->ppart, nullptr, st);
  if (rc) return rc;
  k_pend_write<<<grid_for(s->cap, 256), 256, 0, st>>>(s->g, s->agg.level, s->ctl, s->cap, L.key, s->pflag, o, status);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

int alto_stream_destroy(alto_stream* s) {
  if (s && s->ev_made) {
    for (int k = 0; k < 2; ++k) (void)hipEventDestroy(s->ev_done[k]);
  }
  if (!s) return ALTO_E_ARG;
  delete s;
  return ALTO_OK;
}

}  // extern "C"
