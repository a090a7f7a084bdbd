// Batch routing and aggregation (internal).
#pragma once
#include "alto_internal.h"
#include "segment.h"
#include "sort.h"

#define GROUP_SCAN_TILE 1024   // groups per tile of the group kernel (k_groups)
#define GROUP_SCAN_WORDS 5     // its look-back words per tile
#define MEAN_CHUNK_ROWS 4096
#define MEAN_SMALL_ROWS 256    // groups of at most this many rows: one chunk, gathered by one wave

// One unit of gather work: rows [begin, begin+len) of the sorted fragments, the
// k-th of nch chunks of emitted group e.
struct Chunk {
  int64_t e;       // emitted group index
  int64_t out;     // concat: tok offset of the chunk's first row
  int64_t part;    // mean: first partial-sum slot of the group (-1 if one chunk)
  int32_t begin;   // first sorted position
  int32_t len;
  int32_t k;
  int32_t nch;
  int32_t count;   // leaves of the group
  int32_t pad;
};

// Device copy of the caller's alto_groups.
struct GroupOut {
  int64_t cap_groups, cap_tokens, cap_mask;
  uint64_t* key;
  int32_t* dest;
  int64_t* count;
  int32_t* first_i32;
  int32_t* fan_up;
  int64_t* tok_off;
  int32_t* tok;
  float* mean;
  uint64_t* mask_key;
  uint8_t* mask;
  uint64_t* pend_key;
  int64_t* pend_count;
  int64_t* counts;
};

// Where the fragments of the sorted element array come from. A batch reads every
// row through perm; a stream step reads either the step's inputs (row >= 0) or
// the carried live leaves (row = -1 - live index).
struct BatchSrc {
  const uint32_t* perm;
  const int32_t* p32;
  const int32_t* fan;
  int64_t fan_ld;
  const float* pf;
  int dim;
  int64_t n;
  int32_t* status;
  // perm is a permutation of 0..n-1 unless the input had duplicate keys: with direct
  // placement a position is then left at DP_UNPLACED, reported here as DUPLICATE
  // (the gathers read every position of the complete groups, i.e. all of them); the
  // row is kept in bounds either way
  __device__ int64_t row(int64_t e) const {
    const uint32_t r = perm[e];
    if (r < (uint64_t)n) return (int64_t)r;
    raise_status(status, ALTO_E_DUPLICATE);
    return 0;
  }
  __device__ int32_t p32_of(int64_t r) const { return p32 ? p32[r] : 0; }
  __device__ int32_t fan_of(int m, int64_t r) const { return fan[(int64_t)(m - 1) * fan_ld + r]; }
  __device__ const float* pay_of(int64_t r) const { return pf + r * (int64_t)dim; }
};

struct MergedSrc {
  const int32_t* src;     // merged element -> step index, or -1 - live index
  const int32_t* sp32;
  const int32_t* sfan;
  int64_t sfan_ld;
  const float* spf;
  const int32_t* lp32;
  const int32_t* lfan;
  int64_t lfan_ld;
  const int32_t* lslot;
  const float* arena;
  int64_t arena_rows;
  int dim;
  __device__ int64_t row(int64_t e) const { return src[e]; }
  __device__ int32_t p32_of(int64_t r) const { return r >= 0 ? (sp32 ? sp32[r] : 0) : lp32[-1 - r]; }
  __device__ int32_t fan_of(int m, int64_t r) const {
    return r >= 0 ? sfan[(int64_t)(m - 1) * sfan_ld + r] : lfan[(int64_t)(m - 1) * lfan_ld + (-1 - r)];
  }
  __device__ const float* pay_of(int64_t r) const {
    if (r >= 0) return spf + r * (int64_t)dim;
    int64_t s = lslot[-1 - r];
    s = (s < 0 || s >= arena_rows) ? 0 : s;   // a corrupt slot after a data error stays in bounds
    return arena + s * (int64_t)dim;
  }
};

// Per-block record of the input-order pass.
struct PrepPartial {
  uint64_t kor, kand;
  uint32_t dor, dand;
  uint32_t flags;   // 1 layout, 2 fan, 4 flow set full
  uint32_t pad;
  uint64_t fp[ALTO_MAX_LEVELS];
};

struct AggBufs {
  PrepPartial* prep_part;   // per-block records of the input-order pass
  int32_t fx_lo, fx_hi;     // count levels checked exactly per flow instead of by fingerprint (fx_lo > fx_hi: none)
  FlowBufs fl;          // flows of the route level (packed sort); hcap == 0 when unused
  uint32_t* os_status;  // sort passes: [2][tiles][256] tile status words
  uint32_t* os_ctr;     // [SORT_MAX_PASSES] tile tickets
  uint32_t* os_hist;    // [SORT_MAX_PASSES][256] digit counts / bases
  int64_t os_ntiles;
  SortCtl* ctl;
  SortCtl* rctl;
  uint64_t* fp_in;
  uint64_t* fp_nodes;
  int64_t* nnodes;
  int64_t* scal;        // [8] device scalars: 1 = chunks of long groups, 2 = block ticket, 3 = short groups
  uint64_t* tmp_keys;
  uint32_t* tmp_vals;
  uint64_t* sk;
  uint32_t* perm;
  uint32_t* perm_used;  // perm buffer the sort wrote (caller's or ours)
  int32_t* scan_i32;
  int64_t* scan_i64;
  LevelNodes lv[ALTO_MAX_LEVELS + 1];
  int32_t* carry_fan;
  uint64_t* rkey;
  uint64_t* rsk;
  uint32_t* ridx;
  int32_t* em;          // [n+1] scratch of the stream's live-set update (freed arena slots)
  int64_t* tokc;        // [n+1] the same (arena slots to fill)
  Chunk* chunks;        // long-group chunks from 0, short-group chunks from short_base
  int64_t short_base;
  double* part;
  uint2* gw;            // [cdiv(n_max, SEG_IT)] group-level boundary words of the segmentation pass (streams)
};

void agg_levels(const KeyGeom& g, int La, int Lm, int Lr, int* Lt, int* Lseg);
// flow_cap: flows of the route level ranked for the packed sort (more flows fall back
// to the general sort)
void plan_buffers(const KeyGeom& g, int64_t n_max, const RouteGeom& rg, const alto_agg* agg, int Lr, WsCarver& c,
                  AggBufs& b, int64_t flow_cap = FLOW_CAP);
// allow_dp: a batch aggregation may use direct placement (FlowBufs.dp)
int route_run(const KeyGeom& g, const RouteGeom& rg, const uint64_t* keys, int64_t n, AggBufs& b, int32_t* perm_out,
              int64_t* dest_offsets, int32_t* dest, const int32_t* fan, int64_t fan_ld, int flo, int fhi,
              int32_t* status, hipStream_t st, bool offsets_later = false, bool exact_flow_levels = false,
              bool allow_dp = false, const int64_t* n_dev = nullptr);
// Work folded into the kernels of groups_run (fewer launches per call):
//  - the comparison of the fan fingerprints, in the group kernel (fp_in null:
//    none; levels flo..fhi, those in xlo..xhi, which the flow set checked exactly,
//    only when ctl reports that the flow set overflowed);
//  - the group kernel's look-back words at gst and its ticket at *gctr (null: the
//    sort's status words and first ticket); cleared = the caller's earlier kernel
//    cleared them (cdiv(n_max + 1, GROUP_SCAN_TILE) * GROUP_SCAN_WORDS words),
//    else a kernel before it does, and also clears another look-back region
//    (xst null: none) of cdiv(*xlen, xtile) * xper words and its ticket *xctr, for
//    a scan that runs after the groups;
//  - the emitted set (ht null: none): the group kernel inserts the key of every
//    emitted group into an insert-only open-addressing set of htcap (a power of
//    two) slots, counting new keys in *emit_count; a full table raises
//    ALTO_E_CAPACITY (the caller compares the count with its own limit later);
//  - concat / multi-chunk means left to the caller (defer_concat, defer_combine).
struct GroupsExtra {
  const uint64_t* fp_in;
  const uint64_t* fp_nodes;
  int32_t flo, fhi, xlo, xhi;
  const SortCtl* ctl;
  uint64_t* gst;
  uint32_t* gctr;
  int32_t cleared;
  uint64_t* xst;
  uint32_t* xctr;
  const int64_t* xlen;
  int64_t xtile, xper;
  uint64_t* ht;
  int64_t htcap;
  int64_t* emit_count;
  // the gathers the caller runs itself later (concat_chunks / mean_combine_chunks)
  int32_t defer_concat, defer_combine;
  // the gathers on another HIP stream (gather_st, after an event recorded on the
  // call's stream; null: the call's stream)
  hipStream_t gather_st;
  // the group kernel evaluates the completion of the group-level nodes itself (the
  // segmentation launched no k_seg_nodes for that level): children are elements
  // (fold_leafy) or next-level nodes; fingerprint terms of fold_level into fold_fp
  // from the elements' keys (prefix shift fold_es)
  int32_t fold, fold_leafy, fold_level, fold_es;
  const uint64_t* fold_keys;
  uint64_t* fold_fp;
};

#define EMIT_EMPTY (~0ull)

// Concatenation of the chunks of the long groups (chunks[0, NB)) and the short
// ones (chunks_s[0, NS)), chunk c0 and every cstride-th after it in that order (a
// block each): every row of a chunk copies its int32 payload to the chunk's token
// range.
template <typename Src>
__device__ inline void concat_chunks(const Chunk* __restrict__ chunks, int64_t NB, const Chunk* __restrict__ chunks_s,
                                     int64_t NS, const Src& src, int32_t* tok, int64_t cap_tokens, int64_t c0,
                                     int64_t cstride) {
  for (int64_t c = c0; c < NB + NS; c += cstride) {
    const Chunk ch = c < NB ? chunks[c] : chunks_s[c - NB];
    for (int r = threadIdx.x; r < ch.len; r += blockDim.x) {
      const int64_t o = ch.out + r;
      if (o < cap_tokens) tok[o] = src.p32_of(src.row(ch.begin + r));
    }
  }
}

// The same with one wave per chunk (wave wid of nw), for chunks of a few rows.
template <typename Src>
__device__ inline void concat_chunks_wave(const Chunk* __restrict__ chunks, int64_t NB,
                                          const Chunk* __restrict__ chunks_s, int64_t NS, const Src& src, int32_t* tok,
                                          int64_t cap_tokens, int64_t wid, int64_t nw) {
  const int lane = lane_id();
  for (int64_t c = wid; c < NB + NS; c += nw) {
    const Chunk ch = c < NB ? chunks[c] : chunks_s[c - NB];
    for (int r = lane; r < ch.len; r += ALTO_WAVE) {
      const int64_t o = ch.out + r;
      if (o < cap_tokens) tok[o] = src.p32_of(src.row(ch.begin + r));
    }
  }
}

// The mean of every group of several chunks from its chunks' partial sums (chunk
// order), long-group chunks [c0, NC) step cstride, a block of 256 threads each: SUBS chunk
// subsets x COLS columns; each thread sums every SUBS-th chunk, then the subsets are
// added in subset order. Every thread of the block calls it (it holds barriers).
__device__ inline void mean_combine_chunks(const Chunk* __restrict__ chunks, int64_t NC,
                                           const double* __restrict__ part, int dim, float* mean,
                                           int64_t cap_groups, int64_t c0, int64_t cstride) {
  constexpr int COLS = 64, SUBS = 256 / COLS;
  __shared__ double red[SUBS][COLS];
  const int col_l = threadIdx.x % COLS, sidx = threadIdx.x / COLS;
  for (int64_t c = c0; c < NC; c += cstride) {
    const Chunk ch = chunks[c];
    if (ch.k != 0 || ch.nch <= 1 || ch.e >= cap_groups) continue;   // uniform per block
    for (int col0 = 0; col0 < dim; col0 += COLS) {
      const int x = col0 + col_l;
      double sum = 0.0;
      if (x < dim) {
#pragma unroll 4
        for (int t = sidx; t < ch.nch; t += SUBS) sum += part[(ch.part + t) * (int64_t)dim + x];
      }
      red[sidx][col_l] = sum;
      __syncthreads();
      if (sidx == 0 && x < dim) {
        double tot = 0.0;
#pragma unroll
        for (int q = 0; q < SUBS; ++q) tot += red[q][col_l];
        mean[ch.e * (int64_t)dim + x] = (float)(tot / (double)ch.count);
      }
      __syncthreads();
    }
  }
}

// Inserts a group key into the emitted set: 1 = new, 0 = present, -1 = table full.
// Each probe is one compare-and-swap (no load first: one round trip per slot).
__device__ inline int emitted_insert(uint64_t gk, uint64_t* ht, int64_t htcap) {
  int64_t h = (int64_t)(mix64(gk) & (uint64_t)(htcap - 1));
  for (int64_t p = 0; p < htcap; ++p) {
    const uint64_t old = atomicCAS((unsigned long long*)&ht[h], (unsigned long long)EMIT_EMPTY, (unsigned long long)gk);
    if (old == EMIT_EMPTY) return 1;
    if (old == gk) return 0;
    h = (h + 1) & (htcap - 1);
  }
  return -1;
}

// Whether a group key is in the emitted set.
__device__ inline bool emitted_has(uint64_t gk, const uint64_t* ht, int64_t htcap) {
  int64_t h = (int64_t)(mix64(gk) & (uint64_t)(htcap - 1));
  for (int64_t p = 0; p < htcap; ++p) {
    const uint64_t v = ht[h];
    if (v == gk) return true;
    if (v == EMIT_EMPTY) return false;
    h = (h + 1) & (htcap - 1);
  }
  return false;
}

// Groups, chunk lists, counts and payload gathers over an element array already
// segmented at level La (nodes in b.lv[La]); elements sorted by (dest, key).
template <typename Src>
int groups_run(const KeyGeom& g, const RouteGeom& rg, const alto_agg& agg, const Src& src, const uint64_t* sk,
               int64_t n_max, AggBufs& b, const int64_t* Mp, const GroupOut& out, int32_t* status, hipStream_t st,
               const GroupsExtra* ex = nullptr);
int aggregate_run(const KeyGeom& g, const RouteGeom& rg, int Lr, const alto_agg& agg, const uint64_t* keys,
                  const int32_t* fan, int64_t fan_ld, const int32_t* p32, const float* pf, int64_t n, AggBufs& b,
                  int32_t* perm_out, int64_t* dest_offsets, int32_t* dest, const GroupOut& out, int32_t* status,
                  hipStream_t st, const int64_t* n_dev = nullptr, hipStream_t gather_st = nullptr);
void empty_outputs(const GroupOut& out, int64_t* dest_offsets, int num_dest, hipStream_t st);
void zero_offsets(int64_t* dest_offsets, int num_dest, hipStream_t st);
