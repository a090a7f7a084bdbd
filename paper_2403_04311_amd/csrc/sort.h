// Radix sort and scan launchers (internal).
#pragma once
#include "alto_internal.h"

#define SORT_NT 256
#define SORT_IT 16
#define SORT_TILE (SORT_NT * SORT_IT)
#define SORT_RADIX 8
#define SORT_BUCKETS 256
#define SORT_MAX_PASSES 12
#define SCAN_MAX_BLOCKS 1023
#define SORT_SMALL_MAX 4096

enum { SORT_BUF_INPUT = 0, SORT_BUF_TMP = 1, SORT_BUF_FINAL = 2 };

struct SortPass {
  int32_t active, src, dst, from_dest, lo;
};

struct SortPlan {
  int32_t npass;
  SortPass pass[SORT_MAX_PASSES];
};

// Device control block of one sort.
struct SortCtl {
  uint64_t key_or, key_and;
  uint32_t dest_or, dest_and;
  SortPlan plan;
};

struct SortBufs {
  const uint64_t* in_keys;   // input keys; values are the input indices
  uint64_t* tmp_keys;
  uint32_t* tmp_vals;
  uint64_t* out_keys;        // sorted keys
  uint32_t* out_vals;        // input index of each sorted key
  uint32_t* hist;            // [256 * sort_hist_blocks(n_max)]
  uint32_t* scan_part;       // [SCAN_MAX_BLOCKS + 1]
  SortCtl* ctl;
};

int sort_hist_blocks(int64_t n_max);
int sort_max_key_windows(int key_bits);
int sort_max_dest_windows(const RouteGeom& rg);

// Sorts n (= *n_dev if n_dev, else n_max) keys by (destination, key), stably.
// key_bits bounds the width of the keys. If ctl_has_reduction, ctl already holds
// the OR/AND of keys and destinations (see sort_reduce_launch).
int sort_pairs(const SortBufs& b, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, int key_bits,
               bool ctl_has_reduction, hipStream_t st);
void sort_reduce_launch(const uint64_t* keys, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, SortCtl* ctl,
                        hipStream_t st);

// Exclusive scan of len (= *len_dev if len_dev, else len_max) elements; in may
// equal out. part needs SCAN_MAX_BLOCKS + 1 entries; part[nb] and *total (if
// non-null) receive the sum.
template <typename T>
int scan_exclusive(const T* in, T* out, int64_t len_max, const int64_t* len_dev, T* part, T* total, hipStream_t st);
