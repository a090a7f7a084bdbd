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

namespace {

constexpr int NT = SORT_NT;
constexpr int IT = SORT_IT;
constexpr int TILE = SORT_TILE;
constexpr int NW = NT / ALTO_WAVE;

__device__ inline int64_t load_n(int64_t n_host, const int64_t* n_dev) { return n_dev ? *n_dev : n_host; }

__global__ void k_sort_init(SortCtl* ctl) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    ctl->key_or = 0;
    ctl->key_and = ~0ull;
    ctl->dest_or = 0;
    ctl->dest_and = ~0u;
  }
}

// OR / AND of keys and destinations (which bits vary).
__global__ __launch_bounds__(256) void k_sort_reduce(const uint64_t* __restrict__ keys, int64_t n_host,
                                                     const int64_t* n_dev, RouteGeom rg, SortCtl* ctl) {
  const int64_t n = load_n(n_host, n_dev);
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u;
  // waves with no element skip the atomics (they would only add contention)
  const int64_t wave0 = (int64_t)blockIdx.x * blockDim.x + (threadIdx.x & ~(ALTO_WAVE - 1));
  if (wave0 >= n) return;
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
  if (lane_id() == 0) {
    atomicOr((unsigned long long*)&ctl->key_or, (unsigned long long)kor);
    atomicAnd((unsigned long long*)&ctl->key_and, (unsigned long long)kand);
    atomicOr(&ctl->dest_or, dor);
    atomicAnd(&ctl->dest_and, dand);
  }
}

// Greedy cover of the varying bits with 8-bit windows (optimal for fixed-width
// interval cover), key windows first, then destination windows; then the buffer
// ping-pong so that the last pass lands in the final buffers.
__global__ void k_sort_plan(SortCtl* ctl, int max_key_windows, int max_dest_windows) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  SortPlan p;
  int np = 0;
  uint64_t vk = ctl->key_or ^ ctl->key_and;
  while (vk && np < max_key_windows) {
    int lo = __builtin_ctzll(vk);
    p.pass[np].from_dest = 0;
    p.pass[np].lo = lo;
    ++np;
    vk = (lo + SORT_RADIX >= 64) ? 0ull : (vk & ~((1ull << (lo + SORT_RADIX)) - 1ull));
  }
  uint32_t vd = ctl->dest_or ^ ctl->dest_and;
  int nk = np;
  while (vd && np < nk + max_dest_windows) {
    int lo = __builtin_ctz(vd);
    p.pass[np].from_dest = 1;
    p.pass[np].lo = lo;
    ++np;
    vd = (lo + SORT_RADIX >= 32) ? 0u : (vd & ~((1u << (lo + SORT_RADIX)) - 1u));
  }
  for (int k = 0; k < np; ++k) {
    p.pass[k].active = 1;
    p.pass[k].dst = ((np - 1 - k) % 2 == 0) ? SORT_BUF_FINAL : SORT_BUF_TMP;
    p.pass[k].src = (k == 0) ? SORT_BUF_INPUT : p.pass[k - 1].dst;
  }
  for (int k = np; k < SORT_MAX_PASSES; ++k) {
    p.pass[k].active = 0;
    p.pass[k].src = p.pass[k].dst = 0;
    p.pass[k].from_dest = p.pass[k].lo = 0;
  }
  p.npass = np;
  ctl->plan = p;
}

__device__ inline uint32_t digit_of(const SortPass& ps, const RouteGeom& rg, uint64_t k) {
  uint64_t src = ps.from_dest ? (uint64_t)dest_of_key(rg, k) : k;
  return (uint32_t)((src >> ps.lo) & (SORT_BUCKETS - 1));
}

struct SrcPtrs {
  const uint64_t* keys;
  const uint32_t* vals;   // nullptr: value = index
};

__device__ inline SrcPtrs pick_src(int sel, const SortBufs& b) {
  if (sel == SORT_BUF_INPUT) return {b.in_keys, nullptr};
  if (sel == SORT_BUF_TMP) return {b.tmp_keys, b.tmp_vals};
  return {b.out_keys, b.out_vals};
}

// Stable in-wave ranking of one row of 64 digits: returns the rank of this lane
// among the valid lanes holding the same digit, and the lane mask of those peers.
__device__ inline uint64_t match_digit(uint32_t dig, bool valid) {
  uint64_t peers = __ballot(valid);
#pragma unroll
  for (int b = 0; b < SORT_RADIX; ++b) {
    bool bit = (dig >> b) & 1u;
    uint64_t m = __ballot(bit);
    peers &= bit ? m : ~m;
  }
  return peers;
}

__global__ __launch_bounds__(NT) void k_sort_upsweep(SortBufs b, int64_t n_host, const int64_t* n_dev, int slot,
                                                     RouteGeom rg, int nblocks) {
  const SortPass ps = b.ctl->plan.pass[slot];
  if (!ps.active) return;
  const int64_t n = load_n(n_host, n_dev);
  __shared__ uint32_t s_cnt[NW][SORT_BUCKETS];
  for (int i = threadIdx.x; i < NW * SORT_BUCKETS; i += NT) (&s_cnt[0][0])[i] = 0;
  __syncthreads();
  const SrcPtrs src = pick_src(ps.src, b);
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  const int64_t tile0 = (int64_t)blockIdx.x * TILE;
#pragma unroll 4
  for (int j = 0; j < IT; ++j) {
    int64_t gi = tile0 + (int64_t)w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    bool valid = gi < n;
    uint32_t dig = valid ? digit_of(ps, rg, src.keys[gi]) : 0u;
    uint64_t peers = match_digit(dig, valid);
    if (valid && lane == __ffsll((unsigned long long)peers) - 1) s_cnt[w][dig] += (uint32_t)__popcll(peers);
  }
  __syncthreads();
  for (int d = threadIdx.x; d < SORT_BUCKETS; d += NT) {
    uint32_t c = 0;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) c += s_cnt[ww][d];
    b.hist[(int64_t)d * nblocks + blockIdx.x] = c;
  }
}

__global__ __launch_bounds__(NT) void k_sort_downsweep(SortBufs b, int64_t n_host, const int64_t* n_dev, int slot,
                                                       RouteGeom rg, int nblocks) {
  const SortPass ps = b.ctl->plan.pass[slot];
  if (!ps.active) return;
  const int64_t n = load_n(n_host, n_dev);
  const int64_t tile0 = (int64_t)blockIdx.x * TILE;
  if (tile0 >= n) return;
  __shared__ uint32_t s_cnt[NW][SORT_BUCKETS];
  __shared__ uint32_t s_base[SORT_BUCKETS];
  __shared__ uint32_t s_gbase[SORT_BUCKETS];
  __shared__ uint32_t s_wsum[NT / ALTO_WAVE];
  __shared__ uint64_t s_key[TILE];
  __shared__ uint32_t s_val[TILE];
  __shared__ uint8_t s_dig[TILE];
  for (int i = threadIdx.x; i < NW * SORT_BUCKETS; i += NT) (&s_cnt[0][0])[i] = 0;
  for (int d = threadIdx.x; d < SORT_BUCKETS; d += NT) s_gbase[d] = b.hist[(int64_t)d * nblocks + blockIdx.x];
  __syncthreads();
  const SrcPtrs src = pick_src(ps.src, b);
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  uint64_t key[IT];
  uint32_t val[IT], dig[IT], off[IT];
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    int64_t gi = tile0 + (int64_t)w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    bool valid = gi < n;
    key[j] = valid ? src.keys[gi] : 0ull;
    val[j] = valid ? (src.vals ? src.vals[gi] : (uint32_t)gi) : 0u;
    dig[j] = valid ? digit_of(ps, rg, key[j]) : 0u;
  }
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    int64_t gi = tile0 + (int64_t)w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    bool valid = gi < n;
    uint64_t peers = match_digit(dig[j], valid);
    int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
    uint32_t old = 0;
    if (valid && lane == leader) {
      old = s_cnt[w][dig[j]];
      s_cnt[w][dig[j]] = old + (uint32_t)__popcll(peers);
    }
    old = __shfl(old, leader);
    off[j] = old + (uint32_t)__popcll(peers & lanemask_lt());
  }
  __syncthreads();
  // per digit: exclusive prefix over waves, then exclusive scan over digits
  uint32_t tot = 0;
  const int d = threadIdx.x;   // NT == SORT_BUCKETS
  {
    uint32_t run = 0;
#pragma unroll
    for (int ww = 0; ww < NW; ++ww) {
      uint32_t c = s_cnt[ww][d];
      s_cnt[ww][d] = run;
      run += c;
    }
    uint32_t btot;
    uint32_t ex = block_excl_scan<uint32_t, NT>(run, s_wsum, &btot);
    s_base[d] = ex;
    tot = btot;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < IT; ++j) {
    int64_t gi = tile0 + (int64_t)w * (IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    if (gi < n) {
      uint32_t pos = s_base[dig[j]] + s_cnt[w][dig[j]] + off[j];
      s_key[pos] = key[j];
      s_val[pos] = val[j];
      s_dig[pos] = (uint8_t)dig[j];
    }
  }
  __syncthreads();
  uint64_t* dk = (ps.dst == SORT_BUF_TMP) ? b.tmp_keys : b.out_keys;
  uint32_t* dv = (ps.dst == SORT_BUF_TMP) ? b.tmp_vals : b.out_vals;
  for (uint32_t e = threadIdx.x; e < tot; e += NT) {
    uint32_t dg = s_dig[e];
    uint64_t g = (uint64_t)s_gbase[dg] + (e - s_base[dg]);
    dk[g] = s_key[e];
    dv[g] = s_val[e];
  }
}

__global__ void k_sort_identity(SortBufs b, int64_t n_host, const int64_t* n_dev) {
  if (b.ctl->plan.npass != 0) return;
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
constexpr int SM_IT = SORT_SMALL_MAX / SM_NT;
constexpr int SM_NW = SM_NT / ALTO_WAVE;

__global__ __launch_bounds__(SM_NT) void k_sort_small(SortBufs b, int64_t n_host, const int64_t* n_dev, RouteGeom rg,
                                                      int max_key_windows, int max_dest_windows) {
  __shared__ uint64_t s_key[SORT_SMALL_MAX];
  __shared__ uint32_t s_val[SORT_SMALL_MAX];
  __shared__ uint16_t s_cnt[SM_NW][SORT_BUCKETS];
  __shared__ uint32_t s_base[SORT_BUCKETS];
  __shared__ uint32_t s_wsum[SM_NW];
  __shared__ uint64_t s_or[SM_NW], s_and[SM_NW];
  __shared__ uint32_t s_dor[SM_NW], s_dand[SM_NW];
  __shared__ int s_np;
  __shared__ int s_lo[SORT_MAX_PASSES], s_fd[SORT_MAX_PASSES];
  const int64_t n = load_n(n_host, n_dev);
  const int w = threadIdx.x / ALTO_WAVE, lane = lane_id();
  uint64_t kor = 0, kand = ~0ull;
  uint32_t dor = 0, dand = ~0u;
  for (int j = 0; j < SM_IT; ++j) {
    const int e = w * (SM_IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
    if (e < n) {
      const uint64_t k = b.in_keys[e];
      s_key[e] = k;
      s_val[e] = (uint32_t)e;
      kor |= k;
      kand &= k;
      const uint32_t d = dest_of_key(rg, k);
      dor |= d;
      dand &= d;
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
    uint32_t vd = da ^ dc;
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
    uint64_t key[SM_IT];
    uint32_t val[SM_IT], dig[SM_IT], off[SM_IT];
#pragma unroll
    for (int j = 0; j < SM_IT; ++j) {
      const int e = w * (SM_IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      const bool valid = e < n;
      key[j] = valid ? s_key[e] : 0ull;
      val[j] = valid ? s_val[e] : 0u;
      dig[j] = valid ? digit_of(ps, rg, key[j]) : 0u;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SM_IT; ++j) {
      const int e = w * (SM_IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      const bool valid = e < n;
      const uint64_t peers = match_digit(dig[j], valid);
      const int leader = valid ? (__ffsll((unsigned long long)peers) - 1) : lane;
      uint32_t old = 0;
      if (valid && lane == leader) {
        old = s_cnt[w][dig[j]];
        s_cnt[w][dig[j]] = (uint16_t)(old + (uint32_t)__popcll(peers));
      }
      old = __shfl(old, leader);
      off[j] = old + (uint32_t)__popcll(peers & lanemask_lt());
    }
    __syncthreads();
    if (threadIdx.x < SORT_BUCKETS) {
      const int d = threadIdx.x;
      uint32_t run = 0;
      for (int ww = 0; ww < SM_NW; ++ww) {
        const uint32_t c = s_cnt[ww][d];
        s_cnt[ww][d] = (uint16_t)run;
        run += c;
      }
      s_base[d] = run;
    }
    __syncthreads();
    {
      // every thread of the block takes part (the scan holds barriers)
      uint32_t tot;
      const uint32_t v = threadIdx.x < SORT_BUCKETS ? s_base[threadIdx.x] : 0u;
      const uint32_t ex = block_excl_scan<uint32_t, SM_NT>(v, s_wsum, &tot);
      if (threadIdx.x < SORT_BUCKETS) s_base[threadIdx.x] = ex;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SM_IT; ++j) {
      const int e = w * (SM_IT * ALTO_WAVE) + j * ALTO_WAVE + lane;
      if (e < n) {
        const uint32_t pos = s_base[dig[j]] + (uint32_t)s_cnt[w][dig[j]] + off[j];
        s_key[pos] = key[j];
        s_val[pos] = val[j];
      }
    }
    __syncthreads();
  }
  for (int e = threadIdx.x; e < n; e += SM_NT) {
    b.out_keys[e] = s_key[e];
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

int sort_hist_blocks(int64_t n_max) { return (int)(n_max < 1 ? 1 : cdiv(n_max, SORT_TILE)); }

int sort_max_key_windows(int key_bits) { return (int)cdiv(key_bits, SORT_RADIX); }

int sort_max_dest_windows(const RouteGeom& rg) {
  if (rg.shift >= 64 || rg.num_dest <= 1) return 0;
  int bits = 0;
  while (bits < 32 && ((uint64_t)1 << bits) < rg.num_dest) ++bits;
  return (int)cdiv(bits, SORT_RADIX);
}

int sort_pairs(const SortBufs& b, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, int key_bits,
               bool ctl_has_reduction, hipStream_t st) {
  if (n_max <= SORT_SMALL_MAX) {
    k_sort_small<<<1, 1024, 0, st>>>(b, n_max, n_dev, rg, sort_max_key_windows(key_bits), sort_max_dest_windows(rg));
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  const int nblocks = sort_hist_blocks(n_max);
  const int grid_r = (int)(n_max < 1 ? 1 : (cdiv(n_max, 256 * 8) < 2048 ? cdiv(n_max, 256 * 8) : 2048));
  if (!ctl_has_reduction) {
    k_sort_init<<<1, 1, 0, st>>>(b.ctl);
    k_sort_reduce<<<grid_r, 256, 0, st>>>(b.in_keys, n_max, n_dev, rg, b.ctl);
  }
  const int mk = sort_max_key_windows(key_bits), md = sort_max_dest_windows(rg);
  k_sort_plan<<<1, 1, 0, st>>>(b.ctl, mk, md);
  ALTO_LAUNCH_CHECK();
  for (int slot = 0; slot < mk + md; ++slot) {
    k_sort_upsweep<<<nblocks, NT, 0, st>>>(b, n_max, n_dev, slot, rg, nblocks);
    int rc = scan_exclusive<uint32_t>(b.hist, b.hist, (int64_t)SORT_BUCKETS * nblocks, nullptr, b.scan_part,
                                      nullptr, st);
    if (rc) return rc;
    k_sort_downsweep<<<nblocks, NT, 0, st>>>(b, n_max, n_dev, slot, rg, nblocks);
  }
  k_sort_identity<<<grid_r, 256, 0, st>>>(b, n_max, n_dev);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

void sort_reduce_launch(const uint64_t* keys, int64_t n_max, const int64_t* n_dev, const RouteGeom& rg, SortCtl* ctl,
                        hipStream_t st) {
  const int grid_r = (int)(n_max < 1 ? 1 : (cdiv(n_max, 256 * 8) < 2048 ? cdiv(n_max, 256 * 8) : 2048));
  k_sort_init<<<1, 1, 0, st>>>(ctl);
  k_sort_reduce<<<grid_r, 256, 0, st>>>(keys, n_max, n_dev, rg, ctl);
}
