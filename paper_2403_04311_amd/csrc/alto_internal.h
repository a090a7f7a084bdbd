// Internal declarations of libalto: device helpers shared by the kernels and the
// host launchers. gfx950 (CDNA4) only: 64-lane wavefronts, 160 KB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/alto.h"

#define ALTO_WAVE 64
#define ALTO_MAX_LEVELS 16

// ---------------------------------------------------------------------------
// key layout, precomputed on the host and passed by value to kernels
// ---------------------------------------------------------------------------
struct KeyGeom {
  int32_t depth;
  int32_t total;                      // sum of bits
  int32_t shift[ALTO_MAX_LEVELS + 1]; // shift[l] = bits below level l (l = 1..depth), shift[0] = total
  uint32_t tagmask[ALTO_MAX_LEVELS + 1];  // tagmask[l] = 2^bits[l-1] - 1
  uint64_t fkey;                      // key of the fan fingerprint, drawn afresh for every call
};

__host__ __device__ inline uint64_t key_prefix(uint64_t k, int sh) { return sh >= 64 ? 0ull : (k >> sh); }

__host__ __device__ inline uint32_t key_tag(const KeyGeom& g, uint64_t k, int level) {
  return (uint32_t)(key_prefix(k, g.shift[level]) & (uint64_t)g.tagmask[level]);
}

// SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014).
__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Destination of a tag prefix: hash, then Lemire's multiply-shift range reduction.
__host__ __device__ inline uint32_t dest_of_prefix(uint64_t p, uint32_t num_dest) {
  return (uint32_t)(((mix64(p) >> 32) * (uint64_t)num_dest) >> 32);
}

struct RouteGeom {
  int32_t shift;      // bits below the route level (64 = route everything to one place)
  uint32_t num_dest;
};

__host__ __device__ inline uint32_t dest_of_key(const RouteGeom& r, uint64_t k) {
  return r.shift >= 64 ? 0u : dest_of_prefix(k >> r.shift, r.num_dest);
}

// Term of the additive multiset fingerprint used to check that all carriers of a
// node declare the same child count (sums of a random-looking function over a
// multiset, Clarke et al., "Incremental multiset hash functions", ASIACRYPT 2003).
// Keyed: the node is hashed with the call's key first, so which (node, count)
// pairs collide depends on a key the input cannot know; the count and level are
// then mixed into that hash.
__host__ __device__ inline uint64_t fan_term(uint64_t key, int level, uint64_t node, uint32_t fan) {
  return mix64(mix64(node ^ key) ^ (((uint64_t)fan << 8) | (uint64_t)level));
}

// ---------------------------------------------------------------------------
// status word: the highest-priority error wins
// ---------------------------------------------------------------------------
__host__ __device__ inline int status_priority(int code) {
  switch (code) {
    case ALTO_E_INTERNAL: return 6;
    case ALTO_E_LAYOUT: return 5;
    case ALTO_E_LATE: return 4;
    case ALTO_E_FANOUT: return 3;
    case ALTO_E_DUPLICATE: return 2;
    case ALTO_E_CAPACITY: return 1;
    default: return 0;
  }
}

__device__ inline void raise_status(int32_t* st, int code) {
  int cur = __hip_atomic_load(st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  while (status_priority(code) > status_priority(cur)) {
    int old = atomicCAS(st, cur, code);
    if (old == cur) break;
    cur = old;
  }
}

// Element count of a call whose count may be on the device (n_dev, written by
// earlier work on the stream, e.g. a previous stage's emitted count): n_max bounds
// every buffer; a device count outside [0, n_max] is clamped (and reported as
// CAPACITY by the call's first kernel).
__device__ inline int64_t dev_n(const int64_t* n_dev, int64_t n_max) {
  if (!n_dev) return n_max;
  const int64_t v = *n_dev;
  return v < 0 ? 0 : (v > n_max ? n_max : v);
}

// ---------------------------------------------------------------------------
// wave / block primitives
// ---------------------------------------------------------------------------
__device__ inline int lane_id() { return threadIdx.x & (ALTO_WAVE - 1); }

__device__ inline uint64_t lanemask_lt() { return (1ull << lane_id()) - 1ull; }

template <typename T>
__device__ inline T wave_incl_scan(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < ALTO_WAVE; o <<= 1) {
    T u = __shfl_up(v, o, ALTO_WAVE);
    if (lane >= o) v += u;
  }
  return v;
}

template <typename T>
__device__ inline T wave_sum(T v) {
#pragma unroll
  for (int o = ALTO_WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, ALTO_WAVE);
  return v;
}

// Exclusive scan over a block of NT threads; returns the exclusive prefix of v and
// writes the block total to *total. `sh` holds NT / 64 entries.
template <typename T, int NT>
__device__ inline T block_excl_scan(T v, T* sh, T* total) {
  constexpr int NW = NT / ALTO_WAVE;
  const int lane = lane_id(), w = threadIdx.x / ALTO_WAVE;
  T inc = wave_incl_scan(v);
  if (lane == ALTO_WAVE - 1) sh[w] = inc;
  __syncthreads();
  T off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    T s = sh[i];
    if (i < w) off += s;
    tot += s;
  }
  __syncthreads();
  *total = tot;
  return off + inc - v;
}

// ---------------------------------------------------------------------------
// decoupled look-back over tiles processed in ticket order
// ---------------------------------------------------------------------------
// A tile publishes its count, then finds the exclusive prefix of all earlier tiles
// by walking back over their words, one per round trip: a count is added and
// passed, an inclusive prefix ends the walk (tile 0 publishes one at once). A tile
// only waits on tiles whose tickets were taken before its own, by blocks that are
// running, so the walk ends; the wait for an unpublished word is still bounded,
// and on giving up the status word gets ALTO_E_INTERNAL and the kernel goes on.
// Word: 0 = not yet published, bit 31 = inclusive prefix in bits 0-30, bit 30 =
// the tile's own count in bits 0-29 (counts < 2^30, prefixes < 2^31).
#define LB_INC (1u << 31)
#define LB_AGG (1u << 30)
#define LB_SPIN_LIMIT (1 << 22)

__device__ inline void lb_publish(uint32_t* st, int64_t tile, int64_t stride, uint32_t count) {
  __hip_atomic_store(&st[tile * stride], (tile == 0 ? LB_INC : LB_AGG) | count, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline uint32_t lb_resolve(uint32_t* st, int64_t tile, int64_t stride, uint32_t count, int32_t* status) {
  if (tile == 0) return 0;
  uint32_t excl = 0;
  for (int64_t t = tile - 1;; --t) {
    uint32_t u = __hip_atomic_load(&st[t * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int spin = 0;
    while (u == 0) {
      if (++spin > LB_SPIN_LIMIT) {
        if (status) raise_status(status, ALTO_E_INTERNAL);
        u = LB_INC;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      u = __hip_atomic_load(&st[t * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    excl += (u & LB_INC) ? (u & ~LB_INC) : (u & (LB_AGG - 1u));
    if (u & LB_INC) break;
  }
  __hip_atomic_store(&st[tile * stride], LB_INC | (excl + count), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return excl;
}

// The same with 64-bit words (bit 63 = inclusive prefix, bit 62 = count, 62-bit
// values), for sums that may exceed 2^30 per tile.
#define LB64_INC (1ull << 63)
#define LB64_AGG (1ull << 62)

__device__ inline void lb64_publish(uint64_t* st, int64_t tile, int64_t stride, uint64_t count) {
  __hip_atomic_store(&st[tile * stride], (tile == 0 ? LB64_INC : LB64_AGG) | count, __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline uint64_t lb64_resolve(uint64_t* st, int64_t tile, int64_t stride, uint64_t count, int32_t* status) {
  if (tile == 0) return 0;
  uint64_t excl = 0;
  for (int64_t t = tile - 1;; --t) {
    uint64_t u = __hip_atomic_load(&st[t * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int spin = 0;
    while (u == 0) {
      if (++spin > LB_SPIN_LIMIT) {
        if (status) raise_status(status, ALTO_E_INTERNAL);
        u = LB64_INC;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
      u = __hip_atomic_load(&st[t * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    excl += u & (LB64_AGG - 1ull);
    if (u & LB64_INC) break;
  }
  __hip_atomic_store(&st[tile * stride], LB64_INC | (excl + count), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return excl;
}

// The same look-back by a whole wave: its lanes read the words of up to 64
// earlier tiles at once, so a tile far from the last inclusive prefix waits for
// one round trip per 64 tiles instead of one per tile. All 64 lanes call it;
// the count was published before (lb64_publish).
__device__ inline uint64_t lb64_resolve_wave(uint64_t* st, int64_t tile, int64_t stride, uint64_t count,
                                             int32_t* status) {
  const int lane = lane_id();
  uint64_t excl = 0;
  for (int64_t t = tile - 1; t >= 0; t -= ALTO_WAVE) {
    const int64_t tt = t - lane;
    uint64_t u = LB64_INC;   // before tile 0: nothing to add
    if (tt >= 0) {
      u = __hip_atomic_load(&st[tt * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      int spin = 0;
      while (u == 0) {
        if (++spin > LB_SPIN_LIMIT) {
          if (status) raise_status(status, ALTO_E_INTERNAL);
          u = LB64_INC;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        u = __hip_atomic_load(&st[tt * stride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    const uint64_t inc = __ballot((u & LB64_INC) != 0ull);
    const int first = inc ? __builtin_ctzll(inc) : ALTO_WAVE - 1;   // the nearest inclusive prefix
    excl += wave_sum(lane <= first ? (u & (LB64_AGG - 1ull)) : 0ull);
    if (inc) break;   // uniform
  }
  if (lane == 0) __hip_atomic_store(&st[tile * stride], LB64_INC | (excl + count), __ATOMIC_RELAXED,
                                    __HIP_MEMORY_SCOPE_AGENT);
  return excl;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
#define ALTO_LAUNCH_CHECK()                                  \
  do {                                                        \
    if (hipGetLastError() != hipSuccess) return ALTO_E_HIP;   \
  } while (0)

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Blocks for a grid-stride loop over n items with nt threads per block, at most cap.
inline int grid_for(int64_t n, int nt, int cap = 4096) {
  const int64_t b = cdiv(n < 1 ? 1 : n, nt);
  return (int)(b < cap ? b : cap);
}

// Bump allocator over a caller workspace; every buffer is 256-byte aligned.
struct WsCarver {
  char* base;
  size_t cap;
  size_t off;
  bool ok;
  template <typename T>
  T* take(int64_t count) {
    size_t bytes = ((size_t)(count < 1 ? 1 : count) * sizeof(T) + 255) & ~(size_t)255;
    if (off + bytes > cap) { ok = false; return nullptr; }
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += bytes;
    return p;
  }
};

// Geometry helpers (host). make_geom draws a fresh fingerprint key (fresh_fp_key).
KeyGeom make_geom(const alto_layout* l);
uint64_t fresh_fp_key();
RouteGeom make_route(const KeyGeom& g, int route_level, int num_dest);
