// Segmentation of sorted fragments into ancestry nodes and the completion cascade
// (internal).
#pragma once
#include "alto_internal.h"
#include "sort.h"

#define SEG_NT 512
#define SEG_IT 8                       // consecutive elements per thread (a small merged run still spreads over several blocks)
#define SEG_TILE (SEG_NT * SEG_IT)
#define SEG_LB_STRIDE ALTO_MAX_LEVELS  // look-back words per tile (one per level)
#define NODE_GRID 512

// Arrays describing the nodes of one level, in element order.
struct LevelNodes {
  int32_t* start;   // [N+1] first element of each node; start[N] = number of elements
  int32_t* fc;      // [N+1] id of the first child node (next level); fc[N] = child count
  int32_t* par;     // [N] id of the parent node (previous level)
  int32_t* nfan;    // [N] declared child count (from the node's first element)
  uint8_t* ok;      // [N] 1 = the node's whole subtree is present
  uint8_t* bad;     // [N] set when some child is incomplete
  uint64_t* nkey;   // [N] nullable: key of each node's first element (written by the pass)
};

// One segmentation run over elements sorted so that every node of the levels
// [lo, elem_level-1] is a contiguous run. Elements are either fragments
// (elem_level = depth; their fans are read through idx from the caller's level-
// major fan array) or node records of level elem_level (fans from rec_fan, ok flags
// from elem_ok).
struct SegJob {
  const uint64_t* keys;     // sorted element keys (prefix of level elem_level)
  const uint32_t* idx;      // element -> row in the fan source
  const int64_t* n_dev;     // number of elements (device), or null: n_host
  int64_t n_host;
  int64_t n_max;
  int32_t elem_level;
  int32_t lo;               // segmented levels: lo .. elem_level-1
  const int32_t* fan;       // fan source, level-major: level m at fan[(m - fan_base) * fan_ld + row]
  int64_t fan_ld;
  int32_t fan_base;
  const int32_t* src;       // stream steps: element -> step row (>= 0) or -1 - live row;
  const int32_t* fan2;      // the live rows' fans (same level base), used when src is set
  int64_t fan2_ld;
  const uint8_t* elem_ok;   // records: ok flag per row (null for fragments)
  int32_t chain_check;      // records: compare adjacent carriers' fans (exact)
  int32_t check_dup;        // fragments: equal adjacent keys are duplicates
  // carried levels (fragments only): fans of levels [carry_lo, lo-1] are copied
  // from each level-lo node's first element into carry_fan[(m-carry_lo)*carry_ld + node]
  int32_t carry_lo;
  int32_t* carry_fan;
  int64_t carry_ld;
  LevelNodes lv[ALTO_MAX_LEVELS + 1];   // indexed by level
  int64_t* nnodes;          // device [ALTO_MAX_LEVELS + 1]: node count per level
  uint32_t* lb_status;      // [lb_tiles * SEG_LB_STRIDE] look-back words (cleared by seg_run)
  uint32_t* lb_ctr;         // [1] tile tickets
  int64_t lb_tiles;         // >= seg_tiles(n_max)
  uint64_t* fp_nodes;       // device [ALTO_MAX_LEVELS + 1]: fingerprint sums over nodes (fragments)
  int32_t* status;
  int64_t* dest_offsets;    // fragments sorted by (dest, key): start of each destination (nullable)
  RouteGeom rg;
  const SortCtl* skip_ctl;  // nullable: every kernel returns at once when skip_ctl->dp (the sort
                            // placed the elements directly and set the group level itself)
  int32_t no_prep;          // the caller's previous kernel did seg_prep_device (one launch less)
  int32_t prefetch;         // keys holds n_max elements: the pass may load a tile's keys before
                            // it knows the count
  int32_t fold_lo;          // the completion of the level-lo nodes is evaluated by the caller's
                            // group kernel (no k_seg_nodes launch for level lo)
  uint2* gw;                // nullable, [cdiv(n_max, SEG_IT)]: for each run of SEG_IT elements from
                            // element r * SEG_IT, x = level-lo boundaries before the run, y = its
                            // boundary bits (bit i: element r * SEG_IT + i starts a level-lo node),
                            // so the level-lo node of element r * SEG_IT + i is
                            // x + popcount(y & (2^(i+1) - 1)) - 1
};

// What k_seg_prep does, for a kernel that runs before the segmentation pass and
// knows the element count (n elements): clears the look-back words and the ticket,
// and with no element writes the empty node counts. t0/stride: the calling
// thread's grid-stride position.
__device__ inline void seg_prep_device(const SegJob& j, int64_t n, int64_t t0, int64_t stride) {
  const int64_t len = cdiv(n, SEG_TILE) * SEG_LB_STRIDE;
  for (int64_t i = t0; i < len; i += stride) j.lb_status[i] = 0;
  if (t0 == 0) {
    *j.lb_ctr = 0;
    if (n == 0) {
      for (int m = j.lo; m < j.elem_level; ++m) {
        j.nnodes[m] = 0;
        j.lv[m].start[0] = 0;
        if (m + 1 < j.elem_level) j.lv[m].fc[0] = 0;
      }
      if (j.dest_offsets)
        for (uint32_t x = 0; x <= j.rg.num_dest; ++x) j.dest_offsets[x] = 0;
    }
  }
}

int seg_tiles(int64_t n_max);   // tiles of SEG_TILE elements
int seg_run(const KeyGeom& g, SegJob& job, hipStream_t st);
