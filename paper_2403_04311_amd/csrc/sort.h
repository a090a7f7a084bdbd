// Radix sort and scan launchers (internal).
#pragma once
#include "alto_internal.h"

#define SORT_NT 512
#define SORT_IT 8
#define SORT_TILE (SORT_NT * SORT_IT)
#ifndef SORT_OS_IT
#define SORT_OS_IT 16   // items per thread of a look-back pass
#endif
#define SORT_OS_TILE (SORT_NT * SORT_OS_IT)
#define SORT_RADIX 8
#define SORT_BUCKETS 256
#define SORT_MAX_PASSES 12
#define SCAN_MAX_BLOCKS 1023
#define SORT_SMALL_MAX 8192
#define FLOW_CAP 8192          // flows sort in one workgroup (<= SORT_SMALL_MAX)
#define FLOW_DIRECT_BITS 12   // flow prefixes varying within this many bits: direct rank table
#define FLOW_EXACT_LEVELS 3   // count levels up to the route level checked exactly per flow

enum { SORT_BUF_INPUT = 0, SORT_BUF_TMP = 1, SORT_BUF_FINAL = 2 };
enum { SORT_GENERAL = 0, SORT_PACKED = 1 };

struct SortPass {
  int32_t active, src, dst, from_dest, lo;
};

struct SortPlan {
  int32_t npass;
  int32_t first;         // slot of the first pass (packed passes end at the host's last packed slot)
  int32_t idle;          // the multi-block path does nothing (sorted in one workgroup)
  int32_t direct;        // packed by child rank, passes over the child-rank bits only; the last
                         // pass puts each element at its final position (see FlowBufs.dp)
  SortPass pass[SORT_MAX_PASSES];
};

// Device control block of one sort.
struct SortCtl {
  uint64_t key_or, key_and;
  uint32_t dest_or, dest_and;
  int32_t mode;          // SORT_GENERAL: (key, index) pairs; SORT_PACKED: one word per element
  int32_t ib;            // packed: bits of the input index (low bits)
  int32_t sbits;         // packed: key bits below the route level (middle bits)
  int32_t rbits;         // packed: bits of the flow rank (high bits)
  int32_t flow_overflow; // the flow set filled up
  int32_t dlo, dbits;    // packed: rank = drank[(prefix >> dlo) & (2^dbits - 1)]; dbits < 0: hashed table
  int32_t cmode;         // packed by child rank: fbase[rank] + child tag replaces (rank, child tag)
  int32_t dp;            // direct placement chosen for this call (FlowBufs.dp)
  int64_t ctotal;        // child ranks in use (sum of the flows' declared child counts)
  int64_t nflows;        // distinct flows inserted
  int64_t nflows_c;      // the same, clamped to the flow capacity
  int64_t hist_len;      // histogram entries the scan covers (0 when idle)
  int64_t ct_mask;       // packed: slots - 1 of the compact rank table
  SortPlan plan;
};

// Distinct route-level prefixes ("flows") of one batch and their rank in
// (destination, prefix) order; used by the packed mode.
struct FlowBufs {
  uint64_t fkey;         // the call's fan fingerprint key (KeyGeom.fkey)
  uint64_t* ht_key;      // [hcap] open-addressing set of prefixes, ~0 = empty
  uint32_t* ht_rank;     // [hcap] rank of the prefix held in the slot
  uint64_t* ct_key;      // [hcap] compact rank table (power of two >= 2 x flows), ~0 = empty
  uint32_t* ct_rank;     // [hcap]
  uint16_t* drank;       // [1 << FLOW_DIRECT_BITS] rank by the varying bits of the prefix
  uint32_t* fdest;       // [fcap] destination of each ranked flow
  int32_t rank_dest;     // fdest holds each flow's rank instead (the counting sweep then
                         // writes every element's flow rank where it writes destinations)
  // child ranks: a flow's children (the nodes one level below the route level) are
  // numbered consecutively from fbase[rank], using the flow's declared child count
  uint32_t* ht_fan;      // [hcap] declared child count of the flow in the slot (the first carrier's; 0 = unset)
  uint32_t* ht_anc;      // [FLOW_EXACT_LEVELS][hcap] counts of the other exactly checked levels (0 = unset)
  int32_t x_route;       // the last exactly checked level is the route level (its counts are in ht_fan)
  uint32_t* fbase;       // [fcap + 1] first child rank of each ranked flow
  uint64_t* ctab;        // [ctab_cap] child rank -> key bits above the child level's suffix
  int64_t ctab_cap;
  int32_t cshift;        // key bits below the child level
  uint32_t cmask;        // tag mask of the child level
  int32_t child_ok;      // the route level's declared child counts are read by the input pass
  int64_t hcap;          // power of two, 0 = flows not used
  int32_t shift;         // bits below the route level
  int32_t ib;            // bits of the largest input index
  uint64_t* flow_key;    // [fcap] compacted prefixes
  uint32_t* flow_slot;   // [fcap]
  uint64_t* flow_sorted; // [fcap] prefixes in (destination, prefix) order
  uint32_t* flow_order;  // [fcap]
  uint64_t* ftmp_keys;   // [fcap] sort scratch
  uint32_t* ftmp_vals;
  SortCtl* fctl;
  int64_t fcap;
  // Direct placement (a batch whose groups are the flows and whose leaves lie one
  // level below the flows' children). A leaf whose tag is its parent's declared
  // count - 1 is a "marker"; the input pass lists them. When every child rank has
  // exactly one marker and the children's declared counts add up to the number of
  // elements, every child and flow is complete (given no duplicate keys) and the
  // sorted position of a leaf is cbase[child rank] + leaf tag: the sort then orders
  // the child-rank bits only and its last pass writes each element's input index
  // there. The permutation is first filled with DP_UNPLACED, so a key given twice
  // (two elements at one position) leaves another position holding it; whoever
  // reads the permutation reports that as DUPLICATE.
  int32_t dp;            // host: the call may use it (markers are collected)
  int32_t dp_level;      // the child level (depth - 1): level of the fingerprint of child counts
  uint64_t* mk_key;      // [mk_cap] keys of the markers: block b of the input pass lists its
  uint32_t* mk_fan;      //   markers at [b * mk_per, (b + 1) * mk_per); and their declared counts
  uint32_t* mk_cnt;      // [mk_blocks] markers seen by each block (may exceed mk_per: then no
                         //   direct placement)
  int64_t mk_cap;
  int32_t mk_per;        // per block (set with the input pass's grid)
  int32_t mk_blocks;     // blocks of the input pass
  uint32_t* cfan;        // [ctab_cap] declared leaf count of each child rank (from its marker)
  uint32_t* cmk;         // [ctab_cap] markers of each child rank
  uint32_t* cbase;       // [ctab_cap + 1] first sorted position of each child rank
  uint64_t* dp_part;     // [3 * (DP_MAX_BLOCKS + 1)] per-block sums, flags and fingerprints
  uint64_t* fp_child;    // fingerprint sum of the child level over nodes (set when direct)
};

#define DP_UNPLACED 0xFFFFFFFFu   // a position of the permutation no element was placed at

#define DP_CHUNK 4096          // child ranks per block of the direct-placement scan
#define PREP_BLOCKS_MAX 512    // blocks of the input pass at most (marker regions)
#define DP_MAX_BLOCKS 1024     // ctab_cap <= DP_CHUNK * DP_MAX_BLOCKS

// A routing call's preparation, done by the one-workgroup sort before it sorts
// (ctl null: none), so that a small call launches one kernel instead of four:
// reset of the control block and the fingerprint sums, the count check of a
// device-side count, each element's destination, the layout and declared-count
// checks, and the fragment side of the fan fingerprint of levels flo..fhi.
struct SmallPrep {
  SortCtl* ctl;
  uint64_t* fp_in;            // [ALTO_MAX_LEVELS + 1]
  uint64_t* fp_nodes;         // [ALTO_MAX_LEVELS + 1] cleared
  const int32_t* fan;         // level-major declared counts (null: no level checked)
  int64_t fan_ld;
  int32_t flo, fhi;
  int32_t* dest;              // nullable
  int32_t* status;
  KeyGeom g;
};

struct SortBufs {
  const uint64_t* in_keys;   // input keys; values are the input indices
  uint64_t* tmp_keys;
  uint32_t* tmp_vals;
  uint64_t* out_keys;        // sorted keys
  uint32_t* out_vals;        // input index of each sorted key
  SortCtl* ctl;
  FlowBufs fl;               // hcap == 0: general mode only
  // multi-block passes (n_max > SORT_SMALL_MAX)
  uint32_t* os_status;       // [2][os_ntiles][256] tile status words, two alternating regions
  uint32_t* os_ctr;          // [SORT_MAX_PASSES] tile tickets
  uint32_t* os_hist;         // [SORT_MAX_PASSES][256] global digit counts, then bases
  int64_t os_ntiles;         // >= sort_tiles(n_max)
  int32_t* status;           // raised to ALTO_E_INTERNAL if a look-back wait gives up (may be null)
  int32_t* dest_out;         // with flows: destination of every input element, written by the
                             // counting sweep (input order); null: not wanted
  SmallPrep prep;            // n_max <= SORT_SMALL_MAX only
};

int sort_tiles(int64_t n_max);   // tiles of SORT_OS_TILE elements (look-back passes)
int sort_max_key_windows(int key_bits);
int sort_max_dest_windows(const RouteGeom& rg);
int bits_for(int64_t v);     // bits needed to hold values 0..v

// Sorts n (= *n_dev if n_dev, else n_max) keys by (destination, key), stably.
// key_bits bounds the width of the keys. If ctl_has_reduction, ctl already holds
// the OR/AND of keys and destinations (see sort_reduce_launch). With b.fl.hcap > 0
// the flow set must have been filled (flow_insert in the input pass); the sort
// then ranks the flows and runs in packed mode when the packing fits. Returns
// ALTO_E_ARG if n_max needs multi-block passes and the os_* buffers are missing.
int sort_pairs(const SortBufs& b, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, int key_bits,
               bool ctl_has_reduction, hipStream_t st);
void sort_reduce_launch(const uint64_t* keys, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, SortCtl* ctl,
                        hipStream_t st);

// Exclusive scan of len (= *len_dev if len_dev, else len_max) elements; in may
// equal out. part needs SCAN_MAX_BLOCKS + 1 entries; part[nb] and *total (if
// non-null) receive the sum.
template <typename T>
int scan_exclusive(const T* in, T* out, int64_t len_max, const int64_t* len_dev, T* part, T* total, hipStream_t st);

// Insert of a route-level prefix into the flow set (called from the input pass);
// returns the prefix's slot, or -1 when the set overflowed.
__device__ inline int64_t flow_insert(const FlowBufs& fl, uint64_t p, bool* overflow) {
  const uint64_t mask = (uint64_t)fl.hcap - 1;
  uint64_t h = mix64(p ^ 0xD6E8FEB86659FD93ull) & mask;
  for (int probe = 0; probe < 256; ++probe) {
    // a plain (cached) read is enough: a slot changes once, from empty to a key,
    // and the compare-and-swap settles a stale empty
    const uint64_t v = fl.ht_key[h];
    if (v == p) return (int64_t)h;
    if (v == ~0ull) {
      const uint64_t old = atomicCAS((unsigned long long*)&fl.ht_key[h], ~0ull, (unsigned long long)p);
      if (old == ~0ull || old == p) return (int64_t)h;
    }
    h = (h + 1) & mask;
  }
  *overflow = true;
  return -1;
}
