// Optional per-phase timing with HIP events on the caller's stream (diagnostics).
#pragma once
#include "alto_internal.h"

enum {
  PH_PREP = 0,     // input-order pass: layout, routing hash, fan checks
  PH_SORT = 1,     // radix sort by (destination, key) and destination offsets
  PH_SEGMENT = 2,  // node segmentation and completion cascade
  PH_GROUPS = 3,   // group records, scans, chunk lists
  PH_GATHER = 4,   // payload gathers (concat / mean, with combine)
  PH_MEAN = 5,     // the mean gather kernel alone
  PH_TOTAL = 6,    // whole entry point
  PH_COUNT = 7
};

void prof_begin(int phase, hipStream_t st);
void prof_end(int phase, hipStream_t st);

struct ProfScope {
  int ph;
  hipStream_t st;
  ProfScope(int p, hipStream_t s) : ph(p), st(s) { prof_begin(ph, st); }
  ~ProfScope() { prof_end(ph, st); }
};
