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

constexpr uint64_t HT_EMPTY = ~0ull;

struct StreamCtl {
  int32_t error;     // data error of an earlier step (the handle is poisoned)
  int32_t pad;
  int64_t live;      // carried leaves
  int64_t top;       // free slots on the stack (MEAN)
  int64_t emitted;   // keys in the emitted set
  int64_t merged;    // live + step, this step
  int64_t merged1;   // merged + 1 (scan length)
  int64_t pad2[2];
};

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
    ctl->top = stack ? cap : 0;
    ctl->emitted = 0;
    ctl->merged = 0;
    ctl->merged1 = 1;
  }
}

__global__ void k_stream_begin(const StreamCtl* ctl, int32_t* status) {
  if (threadIdx.x == 0 && blockIdx.x == 0 && ctl->error) raise_status(status, ctl->error);
}

__global__ void k_stream_end(StreamCtl* ctl, const int32_t* status) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    const int32_t s = *status;
    if (s != 0 && ctl->error == 0) ctl->error = s;
  }
}

// Fragments of groups that were already emitted are late.
__global__ void k_late(const uint64_t* __restrict__ keys, int64_t n, int shiftLa, const uint64_t* __restrict__ ht,
                       int64_t htcap, int32_t* status) {
  bool late = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t gk = key_prefix(keys[i], shiftLa);
    int64_t h = (int64_t)(mix64(gk) & (uint64_t)(htcap - 1));
    for (int64_t p = 0; p < htcap; ++p) {
      const uint64_t v = ht[h];
      if (v == gk) {
        late = true;
        break;
      }
      if (v == HT_EMPTY) break;
      h = (h + 1) & (htcap - 1);
    }
  }
  if (late) raise_status(status, ALTO_E_LATE);
}

// Merge path: every element finds its place by binary search in the other run.
// Live elements go before equal step keys (which are duplicates, reported later).
// Also adds the live leaves' terms of the fan fingerprint.
__global__ __launch_bounds__(256) void k_merge(KeyGeom g, RouteGeom rg, StreamCtl* ctl, int64_t cap, LiveSet live,
                                               const uint64_t* __restrict__ sk, const uint32_t* __restrict__ sperm,
                                               int64_t n, int flo, int fhi, uint64_t* mkey, int32_t* msrc,
                                               uint64_t* fp_in) {
  int64_t Lc = ctl->live;
  Lc = Lc < 0 ? 0 : (Lc > cap ? cap : Lc);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctl->merged = Lc + n;
    ctl->merged1 = Lc + n + 1;
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
      const uint64_t k = live.key[t];
      int64_t lo = 0, hi = n;   // number of step keys < k
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (dk_less(rg, sk[mid], k)) lo = mid + 1; else hi = mid;
      }
      mkey[t + lo] = k;
      msrc[t + lo] = (int32_t)(-1 - t);
#pragma unroll
      for (int q = 0; q < ALTO_MAX_LEVELS; ++q)
        if (q < nl)
          fp[q] += fan_term(flo + q, key_prefix(k, sh[q]), (uint32_t)live.fan[(int64_t)(flo + q - 1) * cap + t]);
    } else {
      const int64_t j = t - Lc;
      const uint64_t k = sk[j];
      int64_t lo = 0, hi = Lc;  // number of live keys <= k
      while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (!dk_less(rg, k, live.key[mid])) lo = mid + 1; else hi = mid;
      }
      mkey[j + lo] = k;
      msrc[j + lo] = (int32_t)sperm[j];
    }
  }
#pragma unroll
  for (int q = 0; q < ALTO_MAX_LEVELS; ++q) {
    if (q < nl) {
      const uint64_t v = wave_sum(fp[q]);
      if (lane_id() == 0 && v) atomicAdd((unsigned long long*)&fp_in[flo + q], (unsigned long long)v);
    }
  }
}

// Per merged element: survives (its group is not emitted), frees its arena slot
// (emitted live leaf), or needs a slot (surviving step leaf).
// Per merged element: kept (its group is not released), arena slot freed (MEAN: a
// released group's carried element), slot needed (MEAN: a kept group's new element).
// One thread per element; its group is the last node starting at or before it (the
// nodes of level La cover the merged elements in order), found by binary search.
__global__ void k_keep(LevelNodes L, const int64_t* Gp, const int32_t* __restrict__ msrc, const StreamCtl* ctl,
                       int32_t* keep, int64_t* freef, int64_t* allocf, int mean) {
  const int64_t G = *Gp;
  const int64_t M = ctl->merged;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < M; e += (int64_t)gridDim.x * blockDim.x) {
    int64_t lo = 0, hi = G - 1;
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (L.start[mid] <= e) lo = mid;
      else hi = mid - 1;
    }
    const bool ok = G > 0 && L.ok[lo];
    const bool live_elem = msrc[e] < 0;
    keep[e] = ok ? 0 : 1;
    freef[e] = (mean && ok && live_elem) ? 1 : 0;
    allocf[e] = (mean && !ok && !live_elem) ? 1 : 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    keep[M] = 0;
    freef[M] = 0;
    allocf[M] = 0;
  }
}

__global__ void k_free_slots(const StreamCtl* ctl, int64_t cap, const int32_t* __restrict__ msrc,
                             const int64_t* __restrict__ freef_scan, LiveSet old, int32_t* stack, int32_t* status) {
  const int64_t M = ctl->merged, top = ctl->top;
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < M; e += (int64_t)gridDim.x * blockDim.x) {
    if (freef_scan[e + 1] != freef_scan[e]) {
      const int64_t pos = top + freef_scan[e];
      const int32_t i = -1 - msrc[e];
      if (pos >= 0 && pos < cap && i >= 0 && i < cap) stack[pos] = old.slot[i];
      else bad = true;
    }
  }
  if (bad) raise_status(status, ALTO_E_CAPACITY);
}

__device__ inline int64_t alloc_pos(const StreamCtl* ctl, const int64_t* freef_scan, const int64_t* allocf_scan,
                                    int64_t e) {
  const int64_t M = ctl->merged;
  return ctl->top + freef_scan[M] - allocf_scan[M] + allocf_scan[e];
}

__global__ void k_live_write(KeyGeom g, const StreamCtl* ctl, int64_t cap, const uint64_t* __restrict__ mkey,
                             const int32_t* __restrict__ msrc, const int32_t* __restrict__ keep_scan,
                             const int64_t* __restrict__ freef_scan, const int64_t* __restrict__ allocf_scan,
                             LiveSet old, LiveSet nw, const int32_t* __restrict__ sp32, const int32_t* __restrict__ sfan,
                             int64_t sfan_ld, const int32_t* stack, int mean, int32_t* status) {
  const int64_t M = ctl->merged;
  const int nf = g.depth - 1;
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < M; e += (int64_t)gridDim.x * blockDim.x) {
    if (keep_scan[e + 1] == keep_scan[e]) continue;
    const int64_t ki = keep_scan[e];
    if (ki >= cap) {
      bad = true;
      continue;
    }
    const int32_t s = msrc[e];
    nw.key[ki] = mkey[e];
    if (s < 0) {
      const int64_t i = -1 - (int64_t)s;
      nw.p32[ki] = old.p32[i];
      for (int l = 0; l < nf; ++l) nw.fan[(int64_t)l * cap + ki] = old.fan[(int64_t)l * cap + i];
      if (mean) nw.slot[ki] = old.slot[i];
    } else {
      nw.p32[ki] = sp32 ? sp32[s] : 0;
      for (int l = 0; l < nf; ++l) nw.fan[(int64_t)l * cap + ki] = sfan[(int64_t)l * sfan_ld + s];
      if (mean) {
        const int64_t pos = alloc_pos(ctl, freef_scan, allocf_scan, e);
        if (pos >= 0 && pos < cap) nw.slot[ki] = stack[pos];
        else {
          nw.slot[ki] = 0;
          bad = true;
        }
      }
    }
  }
  if (bad) raise_status(status, ALTO_E_CAPACITY);
}

// Rows of surviving step leaves go to their arena slots (one wave per row).
__global__ void k_arena_copy(const StreamCtl* ctl, int64_t cap, const int32_t* __restrict__ msrc,
                             const int64_t* __restrict__ freef_scan, const int64_t* __restrict__ allocf_scan,
                             const int32_t* stack, const float* __restrict__ spf, int dim, float* arena) {
  const int64_t M = ctl->merged;
  const int lane = lane_id();
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / ALTO_WAVE;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) / ALTO_WAVE;
  for (int64_t e = wave; e < M; e += nwaves) {
    if (allocf_scan[e + 1] == allocf_scan[e]) continue;
    const int64_t pos = alloc_pos(ctl, freef_scan, allocf_scan, e);
    if (pos < 0 || pos >= cap) continue;
    const int64_t slot = stack[pos];
    if (slot < 0 || slot >= cap) continue;
    const float* src = spf + (int64_t)msrc[e] * dim;
    float* dst = arena + slot * (int64_t)dim;
    for (int c = lane; c < dim; c += ALTO_WAVE) dst[c] = src[c];
  }
}

__global__ void k_stream_finish(StreamCtl* ctl, int64_t cap, const int32_t* keep_scan, const int64_t* freef_scan,
                                const int64_t* allocf_scan, int mean, int32_t* status) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int64_t M = ctl->merged;
  const int64_t K = keep_scan[M];
  if (K > cap) raise_status(status, ALTO_E_CAPACITY);
  ctl->live = K > cap ? cap : K;
  if (mean) {
    int64_t t = ctl->top + freef_scan[M] - allocf_scan[M];
    if (t < 0 || t > cap) {
      raise_status(status, ALTO_E_CAPACITY);
      t = t < 0 ? 0 : cap;
    }
    ctl->top = t;
  }
}

// Remember the emitted groups.
__global__ void k_emit_insert(KeyGeom g, int La, LevelNodes L, const int64_t* Gp, const uint64_t* __restrict__ mkey,
                              uint64_t* ht, int64_t htcap, int64_t max_groups, StreamCtl* ctl, int32_t* status) {
  const int64_t G = *Gp;
  bool full = false;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < G; u += (int64_t)gridDim.x * blockDim.x) {
    if (!L.ok[u]) continue;
    const uint64_t gk = key_prefix(mkey[L.start[u]], g.shift[La]);
    int64_t h = (int64_t)(mix64(gk) & (uint64_t)(htcap - 1));
    bool done = false;
    for (int64_t p = 0; p < htcap && !done; ++p) {
      const uint64_t v = ht[h];
      if (v == gk) {
        done = true;
      } else if (v == HT_EMPTY) {
        const uint64_t old = atomicCAS((unsigned long long*)&ht[h], (unsigned long long)HT_EMPTY, (unsigned long long)gk);
        if (old == HT_EMPTY || old == gk) {
          done = true;
          if (old == HT_EMPTY) {
            const int64_t c = atomicAdd((unsigned long long*)&ctl->emitted, 1ull);
            if (c + 1 > max_groups) full = true;
          }
        } else {
          h = (h + 1) & (htcap - 1);
        }
      } else {
        h = (h + 1) & (htcap - 1);
      }
    }
    if (!done) full = true;
  }
  if (full) raise_status(status, ALTO_E_CAPACITY);
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

int alto_stream_step(alto_stream* s, const uint64_t* keys, const int32_t* fan, int64_t fan_ld,
                     const int32_t* payload_i32, const float* payload_f32, int64_t n, int32_t* perm,
                     int64_t* dest_offsets, int32_t* dest, alto_groups* emitted, int32_t* status, void* ws,
                     size_t ws_bytes, hipStream_t st) {
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
  k_stream_begin<<<1, 1, 0, st>>>(s->ctl, status);
  if (n == 0) {
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
  int rc = route_run(g, s->rg, keys, n, b, perm, dest_offsets, dest, fan, fan_ld, La, d - 1, status, st);
  if (rc) return rc;
  prof_begin(PH_SEGMENT, st);
  const uint32_t* sperm = b.perm_used;
  k_late<<<grid_for(n, 256), 256, 0, st>>>(keys, n, g.shift[La], s->ht, s->htcap, status);
  // 2. merge with the live set
  LiveSet& old = s->live[s->cur];
  LiveSet& nw = s->live[s->cur ^ 1];
  uint64_t* mkey = b.tmp_keys;
  int32_t* msrc = reinterpret_cast<int32_t*>(b.tmp_vals);
  const int64_t* Mp = &s->ctl->merged;
  k_merge<<<grid_for(ntot, 256), 256, 0, st>>>(g, s->rg, s->ctl, s->cap, old, b.sk, sperm, n, La, d - 1, mkey, msrc,
                                               b.fp_in);
  // 3. nodes and completion over the merged run
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
  rc = seg_run(g, j, st);
  if (rc) return rc;
  fp_compare_launch(b.fp_in, b.fp_nodes, La, d - 1, status, st);
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
    k_release<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, b.rsk, b.ridx, g.shift[La - 1] - g.shift[La],
                                                   (uint64_t)g.tagmask[La], s->pht, s->pcur, s->htcap, status);
    ALTO_LAUNCH_CHECK();
  }
  prof_end(PH_SEGMENT, st);
  // 4. emitted groups (payload over all of each group's leaves, in key order)
  MergedSrc src{msrc, payload_i32, fan, fan_ld, payload_f32, old.p32, old.fan, s->cap, old.slot, s->arena, s->cap,
                agg.dim};
  rc = groups_run<MergedSrc>(g, s->rg, agg, src, mkey, ntot, b, nullptr, o, status, st);
  if (rc) return rc;
  // 5. survivors become the new live set
  const int64_t* Gp = b.nnodes + La;
  int32_t* keep = b.em;
  int64_t* freef = b.tokc;
  int64_t* allocf = b.nch;
  const int64_t* M1 = &s->ctl->merged1;
  k_keep<<<grid_for(ntot, 256), 256, 0, st>>>(b.lv[La], Gp, msrc, s->ctl, keep, freef, allocf, mean ? 1 : 0);
  rc = scan_exclusive<int32_t>(keep, keep, ntot + 1, M1, b.scan_i32, nullptr, st);
  if (!rc && mean) rc = scan_exclusive<int64_t>(freef, freef, ntot + 1, M1, b.scan_i64, nullptr, st);
  if (!rc && mean) rc = scan_exclusive<int64_t>(allocf, allocf, ntot + 1, M1, b.scan_i64, nullptr, st);
  if (rc) return rc;
  if (mean) k_free_slots<<<grid_for(ntot, 256), 256, 0, st>>>(s->ctl, s->cap, msrc, freef, old, s->stack, status);
  k_live_write<<<grid_for(ntot, 256), 256, 0, st>>>(g, s->ctl, s->cap, mkey, msrc, keep, freef, allocf, old, nw,
                                                    payload_i32, fan, fan_ld, s->stack, mean ? 1 : 0, status);
  if (mean)
    k_arena_copy<<<grid_for(ntot * ALTO_WAVE, 256), 256, 0, st>>>(s->ctl, s->cap, msrc, freef, allocf, s->stack,
                                                                  payload_f32, agg.dim, s->arena);
  k_emit_insert<<<grid_for(ntot, 256), 256, 0, st>>>(g, La, b.lv[La], Gp, mkey, s->ht, s->htcap, s->max_groups, s->ctl,
                                                     status);
  k_stream_finish<<<1, 1, 0, st>>>(s->ctl, s->cap, keep, freef, allocf, mean ? 1 : 0, status);
  k_stream_end<<<1, 1, 0, st>>>(s->ctl, status);
  ALTO_LAUNCH_CHECK();
  s->cur ^= 1;
  return ALTO_OK;
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
  if (!s) return ALTO_E_ARG;
  delete s;
  return ALTO_OK;
}

}  // extern "C"
