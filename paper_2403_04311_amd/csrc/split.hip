// split_text at a pmap entry (Section 3.2, the split_text operator; Section 4.2:
// entering a pmap pushes a level onto every fragment's tag stack). The fragments
// are tokens, leaves whose parent is one stream element and whose leaf tag is the
// token's index in it. A parent's tokens are cut at a delimiter token into
// segments (maximal runs of the other tokens); every placed token gets a key one
// level deeper, (parent, segment, index in segment), and the declared child counts
// of the two new levels. A parent is split only when all of its declared tokens
// are present, since a missing token could be a delimiter.
//
// Steps: the keys are sorted the way alto_route sorts them, with the parents as the
// flows of the route level and one destination (the parents are ranked in prefix
// order and (rank, position, index) words sort in a few passes over the bits that
// vary); this puts each parent's tokens next to each other in index order. A marking pass over LDS tiles of the sorted order checks
// the keys and decides per token, with two reads, whether its parent is complete:
// a run of distinct indices below P that holds index 0 at its start and index P-1
// P-1 places later holds every index. It flags segment starts and ends; one
// exclusive scan of (placed tokens, segment starts) gives every placed token its
// output row and its segment number; the first and last position of each segment
// are scattered per segment; an emit pass writes the new fragments in sorted order
// (which is new-key order), every access coalesced. The sorted order is never
// scattered back to the input order: the caller gets the input index of each new
// fragment instead, as alto_route's perm.
#include "aggregate.h"
#include "sort.h"

#include <limits.h>
#include <string.h>

namespace {

#define SPLIT_NT 256
#define SPLIT_FLOW_CAP (1 << 16)   // parents ranked for the packed sort (more: general sort)
#define SPLIT_IT 4
#define SPLIT_TILE (SPLIT_NT * SPLIT_IT)

enum : uint8_t {
  SF_PLACED = 1,      // complete parent, not a delimiter
  SF_START = 2,       // first token of a segment
  SF_END = 4,         // last token of a segment
  SF_DELIM = 8,       // delimiter of a complete parent
  SF_INCOMPLETE = 16  // token of an incomplete parent
};

struct SplitBufs {
  AggBufs ab;          // the routing sort: ab.sk sorted keys, ab.perm input index of each
  uint8_t* sflag;      // [n] SF_* of each sorted position
  int32_t* stok;       // [n] token of each sorted position
  int32_t* sfan;       // [n] declared token count of its parent
  int2* tf;            // [n] (token, parent's declared count) in input order, one gather per token
  int64_t* cpl;        // [n + 1] (placed tokens << 32) | segment starts, before each sorted position
  int64_t* part;       // [SCAN_MAX_BLOCKS + 1] scan partials
  uint32_t* cinc;      // [n + 1] tokens of incomplete parents before each sorted position
  uint32_t* part32;    // [SCAN_MAX_BLOCKS + 1]
  uint32_t* sbeg;      // [n] sorted position of each segment's first token
  uint32_t* send;      // [n] ... and of its last
};

void plan_split(const KeyGeom& g, int64_t n_max, WsCarver& c, SplitBufs& b) {
  const int64_t n = n_max < 1 ? 1 : n_max;
  const RouteGeom rg = make_route(g, g.depth - 1, 1);
  plan_buffers(g, n, rg, nullptr, g.depth - 1, c, b.ab, SPLIT_FLOW_CAP);
  b.sflag = c.take<uint8_t>(n);
  b.stok = c.take<int32_t>(n);
  b.sfan = c.take<int32_t>(n);
  b.tf = c.take<int2>(n);
  b.cpl = c.take<int64_t>(n + 1);
  b.part = c.take<int64_t>(SCAN_MAX_BLOCKS + 1);
  b.cinc = c.take<uint32_t>(n + 1);
  b.part32 = c.take<uint32_t>(SCAN_MAX_BLOCKS + 1);
  b.sbeg = c.take<uint32_t>(n);
  b.send = c.take<uint32_t>(n);
}


__global__ void k_split_init(int64_t* counts, int64_t* cpl_end, uint32_t* cinc_end) {
  if (threadIdx.x < 4) counts[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    *cpl_end = 0;
    *cinc_end = 0;
  }
}

__device__ inline void block_add4(uint64_t v[4], uint64_t (*s)[SPLIT_NT / ALTO_WAVE], int64_t* counts) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const uint64_t w = wave_sum(v[q]);
    if (lane_id() == 0) s[q][threadIdx.x / ALTO_WAVE] = w;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    uint64_t t = 0;
    for (int w = 0; w < SPLIT_NT / ALTO_WAVE; ++w) t += s[threadIdx.x][w];
    if (t) atomicAdd((unsigned long long*)&counts[threadIdx.x], (unsigned long long)t);
  }
}

// Token and declared count side by side: the marking pass then fetches one cache
// line per token instead of two (its reads are in sorted order, scattered over the
// input).
__global__ __launch_bounds__(256) void k_split_pair(const int32_t* __restrict__ tok, const int32_t* __restrict__ pfan,
                                                    int64_t n, int2* __restrict__ tf) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    tf[i] = make_int2(tok[i], pfan[i]);
}

// Marking pass, one tile of SPLIT_TILE sorted positions per block iteration. The
// tile and one position on either side are staged in LDS: key, token, and the
// parent's declared token count (gathered together from input order). Tiles go to the
// XCDs in contiguous ranges (workgroups are dealt to the 8 XCDs in turn): the
// gathers of neighbouring parents then share one L2.
__global__ __launch_bounds__(SPLIT_NT) void k_split_mark(const uint64_t* __restrict__ skey,
                                                         const uint32_t* __restrict__ sidx,
                                                         const int2* __restrict__ tf, int64_t n, int total,
                                                         int tbits, int32_t delim, uint8_t* __restrict__ sflag,
                                                         int32_t* __restrict__ stok, int32_t* __restrict__ sfan,
                                                         int64_t* __restrict__ cpl, uint32_t* __restrict__ cinc,
                                                         int64_t* counts,
                                                         int32_t* status) {
  __shared__ uint64_t s_key[SPLIT_TILE + 2];
  __shared__ int32_t s_tok[SPLIT_TILE + 2];
  __shared__ int32_t s_fan[SPLIT_TILE + 2];
  __shared__ uint64_t s_red[4][SPLIT_NT / ALTO_WAVE];
  const uint64_t tmask = ((uint64_t)1 << tbits) - 1;
  bool bad_layout = false, bad_fan = false, dup = false;
  uint64_t cnt[4] = {0, 0, 0, 0};   // placed, delimiters, incomplete, segments
  const int64_t ntiles = cdiv(n, SPLIT_TILE);
  const int64_t lb = (gridDim.x % 8 == 0) ? (int64_t)(blockIdx.x % 8) * (gridDim.x / 8) + blockIdx.x / 8
                                          : (int64_t)blockIdx.x;
  for (int64_t tile = lb; tile < ntiles; tile += gridDim.x) {
    const int64_t t0 = tile * SPLIT_TILE;
    __syncthreads();
    for (int q = threadIdx.x; q < SPLIT_TILE + 2; q += SPLIT_NT) {
      const int64_t j = t0 - 1 + q;
      if (j >= 0 && j < n) {
        const int2 v = tf[sidx[j]];
        s_key[q] = skey[j];
        s_tok[q] = v.x;
        s_fan[q] = v.y;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < SPLIT_IT; ++u) {
      const int q = 1 + u * SPLIT_NT + threadIdx.x;
      const int64_t j = t0 - 1 + q;
      if (j >= n) continue;
      const uint64_t k = s_key[q];
      const uint64_t par = k >> tbits;
      const int64_t idx = (int64_t)(k & tmask);
      const int64_t P = s_fan[q];
      const int32_t tk = s_tok[q];
      const bool is_delim = tk == delim;
      bad_layout |= (k >> total) != 0;
      bad_fan |= P < 1 || idx >= P;
      const bool has_prev = j > 0 && (s_key[q - 1] >> tbits) == par;
      if (has_prev) {
        bad_fan |= s_fan[q - 1] != P;
        dup |= s_key[q - 1] == k;
      }
      // complete: the run starting at j - idx holds index 0 first and index P-1 last
      bool complete = false;
      const int64_t s = j - idx;
      if (P >= 1 && idx < P && s >= 0 && s + P - 1 < n) {
        const uint64_t base = par << tbits;
        complete = skey[s] == base && skey[s + P - 1] == (base | (uint64_t)(P - 1));
      }
      uint8_t f;
      if (!complete) {
        f = SF_INCOMPLETE;
        ++cnt[2];
      } else if (is_delim) {
        f = SF_DELIM;
        ++cnt[1];
      } else {
        f = SF_PLACED;
        ++cnt[0];
        if (idx == 0 || s_tok[q - 1] == delim) {
          f |= SF_START;
          ++cnt[3];
        }
        if (idx == P - 1 || s_tok[q + 1] == delim) f |= SF_END;
      }
      sflag[j] = f;
      stok[j] = tk;
      sfan[j] = (int32_t)P;
      cpl[j] = ((int64_t)((f & SF_PLACED) ? 1 : 0) << 32) | ((f & SF_START) ? 1 : 0);
      if (cinc) cinc[j] = (f & SF_INCOMPLETE) ? 1u : 0u;
    }
  }
  if (bad_layout) raise_status(status, ALTO_E_LAYOUT);
  if (bad_fan) raise_status(status, ALTO_E_FANOUT);
  if (dup) raise_status(status, ALTO_E_DUPLICATE);
  block_add4(cnt, s_red, counts);
}

// Sorted position of each segment's first and last token.
__global__ __launch_bounds__(256) void k_split_bounds(const uint8_t* __restrict__ sflag,
                                                      const int64_t* __restrict__ cpl, int64_t n,
                                                      uint32_t* __restrict__ sbeg, uint32_t* __restrict__ send) {
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint8_t f = sflag[j];
    if (!(f & (SF_START | SF_END))) continue;
    const uint32_t c = (uint32_t)cpl[j];
    if (f & SF_START) sbeg[c] = (uint32_t)j;
    if (f & SF_END) {
      const int64_t g = (int64_t)c + ((f & SF_START) ? 1 : 0) - 1;
      if (g >= 0) send[g] = (uint32_t)j;
    }
  }
}

// The new fragments, in sorted order: key, declared counts, token, input index;
// the input indices of the tokens of incomplete parents. The indices read are
// clamped into their arrays: on inputs with errors the flags may be inconsistent,
// and the outputs are then undefined but every access stays in bounds.
__global__ __launch_bounds__(256) void k_split_emit(const uint64_t* __restrict__ skey,
                                                    const uint32_t* __restrict__ sidx,
                                                    const uint8_t* __restrict__ sflag,
                                                    const int32_t* __restrict__ stok,
                                                    const int32_t* __restrict__ sfan,
                                                    const int64_t* __restrict__ cpl,
                                                    const uint32_t* __restrict__ cinc,
                                                    const uint32_t* __restrict__ sbeg,
                                                    const uint32_t* __restrict__ send,
                                                    const int32_t* __restrict__ fan, int64_t fan_ld, int dfan,
                                                    int64_t n, int tbits, int seg_bits, int tok_bits,
                                                    uint64_t* __restrict__ out_keys, int32_t* __restrict__ out_fan,
                                                    int64_t out_ld, int32_t* __restrict__ out_tok,
                                                    int32_t* __restrict__ out_idx, int32_t* __restrict__ rest_idx,
                                                    int32_t* status) {
  const uint64_t tmask = ((uint64_t)1 << tbits) - 1;
  const int64_t tot = cpl[n];
  const int64_t nseg_all = tot & 0xffffffffll, nplaced = tot >> 32;
  bool cap = false;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x) {
    const uint8_t f = sflag[j];
    if (f & SF_INCOMPLETE) {
      if (rest_idx) rest_idx[cinc[j]] = (int32_t)sidx[j];
      continue;
    }
    if (!(f & SF_PLACED) || nseg_all == 0) continue;
    const int64_t cj = cpl[j];
    int64_t r = cj >> 32;
    r = r >= nplaced ? nplaced - 1 : r;
    const uint32_t i = sidx[j];
    const uint64_t k = skey[j];
    const int64_t idx = (int64_t)(k & tmask);
    int64_t s = j - idx;
    s = s < 0 ? 0 : s;
    int64_t e = s + (int64_t)sfan[j];
    e = e > n ? n : (e < s ? s : e);
    int64_t g = (cj & 0xffffffffll) + ((f & SF_START) ? 1 : 0) - 1;
    g = g < 0 ? 0 : (g >= nseg_all ? nseg_all - 1 : g);
    const int64_t cs = cpl[s] & 0xffffffffll;
    const int64_t c = g - cs;
    const int64_t nseg = (cpl[e] & 0xffffffffll) - cs;
    const int64_t b0 = sbeg[g];
    const int64_t t = j - b0;
    const int64_t len = (int64_t)send[g] - b0 + 1;
    cap |= c < 0 || t < 0 || c >= ((int64_t)1 << seg_bits) || t >= ((int64_t)1 << tok_bits);
    out_keys[r] = ((k >> tbits) << (seg_bits + tok_bits)) | (((uint64_t)c & (((uint64_t)1 << seg_bits) - 1)) << tok_bits) |
                  ((uint64_t)t & (((uint64_t)1 << tok_bits) - 1));
    for (int l = 0; l < dfan - 1; ++l) out_fan[(int64_t)l * out_ld + r] = fan[(int64_t)l * fan_ld + i];
    out_fan[(int64_t)(dfan - 1) * out_ld + r] = (int32_t)nseg;
    out_fan[(int64_t)dfan * out_ld + r] = (int32_t)len;
    if (out_tok) out_tok[r] = stok[j];
    if (out_idx) out_idx[r] = (int32_t)i;
  }
  if (cap) raise_status(status, ALTO_E_CAPACITY);
}

bool split_layout_ok(const alto_layout* l, int seg_bits, int tok_bits) {
  if (!l || l->depth < 2 || l->depth > ALTO_MAX_LEVELS - 1) return false;
  if (seg_bits < 1 || seg_bits > 32 || tok_bits < 1 || tok_bits > 32) return false;
  int total = 0;
  for (int i = 0; i < l->depth; ++i) {
    if (l->bits[i] < 1 || l->bits[i] > 32) return false;
    total += l->bits[i];
  }
  return total <= 63 && total - l->bits[l->depth - 1] + seg_bits + tok_bits <= 63;
}

const int64_t SPLIT_N_LIMIT = (int64_t)INT_MAX - 1;

}  // namespace

extern "C" {

size_t alto_split_workspace_bytes(const alto_layout* layout, int64_t n_max) {
  if (!split_layout_ok(layout, 1, 1) || n_max < 0 || n_max > SPLIT_N_LIMIT) return 0;
  WsCarver c{nullptr, (size_t)-1, 0, true};
  SplitBufs b;
  plan_split(make_geom(layout), n_max, c, b);
  return c.off;
}

int alto_split(const uint64_t* keys, const int32_t* fan, int64_t fan_ld, const int32_t* tokens, int64_t n,
               const alto_layout* layout, int32_t delim, int32_t seg_bits, int32_t tok_bits, uint64_t* out_keys,
               int32_t* out_fan, int64_t out_fan_ld, int32_t* out_tokens, int32_t* out_idx, int32_t* rest_idx,
               int64_t* counts, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!split_layout_ok(layout, seg_bits, tok_bits) || n < 0 || n > SPLIT_N_LIMIT || !counts || !status || !ws)
    return ALTO_E_ARG;
  if (n > 0 && (!keys || !fan || !tokens || !out_keys || !out_fan || fan_ld < n || out_fan_ld < n))
    return ALTO_E_ARG;
  const KeyGeom g = make_geom(layout);
  const int d = layout->depth;
  WsCarver c{(char*)ws, ws_bytes, 0, true};
  SplitBufs b;
  plan_split(g, n, c, b);
  if (!c.ok) return ALTO_E_ARG;
  k_split_init<<<1, 64, 0, stream>>>(counts, b.cpl + n, b.cinc + n);
  if (n == 0) {
    ALTO_LAUNCH_CHECK();
    return ALTO_OK;
  }
  const RouteGeom rg = make_route(g, d - 1, 1);
  // duplicates are reported by k_split_mark (the routing sort's own offset pass is skipped)
  int rc = route_run(g, rg, keys, n, b.ab, nullptr, nullptr, nullptr, nullptr, 0, 1, 0, status, stream, true);
  if (rc) return rc;
  const uint64_t* skey = b.ab.sk;
  const uint32_t* sidx = b.ab.perm;
  const int tbits = layout->bits[d - 1];
  const int mgrid = (int)(cdiv(n, SPLIT_TILE) < 2048 ? cdiv(n, SPLIT_TILE) : 2048);
  k_split_pair<<<grid_for(n, 256), 256, 0, stream>>>(tokens, fan + (int64_t)(d - 2) * fan_ld, n, b.tf);
  k_split_mark<<<mgrid, SPLIT_NT, 0, stream>>>(skey, sidx, b.tf, n, g.total,
                                               tbits, delim, b.sflag, b.stok, b.sfan, b.cpl, rest_idx ? b.cinc : nullptr,
                                               counts, status);
  rc = scan_exclusive<int64_t>(b.cpl, b.cpl, n + 1, nullptr, b.part, nullptr, stream);
  if (!rc && rest_idx) rc = scan_exclusive<uint32_t>(b.cinc, b.cinc, n + 1, nullptr, b.part32, nullptr, stream);
  if (rc) return rc;
  k_split_bounds<<<grid_for(n, 256), 256, 0, stream>>>(b.sflag, b.cpl, n, b.sbeg, b.send);
  k_split_emit<<<grid_for(n, 256), 256, 0, stream>>>(skey, sidx, b.sflag, b.stok, b.sfan, b.cpl, b.cinc, b.sbeg, b.send, fan,
                                               fan_ld, d - 1, n, tbits, seg_bits, tok_bits, out_keys, out_fan,
                                               out_fan_ld, out_tokens, out_idx, rest_idx, status);
  ALTO_LAUNCH_CHECK();
  return ALTO_OK;
}

}  // extern "C"
