/*
 * alto.h -- C ABI of libalto: batched routing and re-aggregation of fragments that
 * carry nested ancestry, on AMD Instinct MI355X (gfx950).
 *
 * Model (paper, Sections 4.1-4.3). Every fragment carries a stack of ancestry
 * tags, one per level of pmap nesting (Section 4.2): level 1 is the request, level
 * d the fragment itself, and levels >= 2 hold the index of the element in its
 * parent's stream. Fragments with the same tags go to the same instance, picked by
 * hashing the tags, like ECMP (Section 4.3). A parallelised stream is put back in
 * its original order before sequential consumers see it (Sections 3.2 and 4.1). A
 * pmap exit pops a level and aggregates what the call produced (Section 4.3;
 * the aggregate operator of Section 3.3). The extent of a generated stream is known
 * only at its end (Section 3.1), so every node declares its child count, and a group
 * is released only when its whole subtree has arrived.
 *
 * Conventions for every entry point:
 *  - Array arguments are DEVICE pointers owned by the caller. The library never
 *    allocates device memory; temporary memory comes from a caller workspace sized
 *    by alto_workspace_bytes() (alto_aggregate_noalloc instead uses a fixed array
 *    of the library's own, see there). Struct arguments (alto_layout, alto_agg,
 *    alto_groups) are HOST pointers to structs whose array members are device
 *    pointers.
 *  - Calls only enqueue work on the given stream and return without synchronising.
 *  - The return value reports host-detectable problems only: ALTO_E_ARG for bad
 *    arguments (nothing is enqueued), ALTO_E_HIP for a failed launch.
 *  - Data-dependent problems are written to the device word *status, which the
 *    caller sets to 0 beforehand and reads after its own synchronisation. When
 *    several problems are present the one reported is, in decreasing priority:
 *    INTERNAL, LAYOUT, LATE, FANOUT, DUPLICATE, CAPACITY. After a data error the outputs are
 *    undefined and a stream handle is poisoned; writes always stay inside the
 *    buffers and capacities given.
 *  - Level-major arrays: element (l, i) of a [levels][n] array lives at
 *    [l * ld + i] with ld >= n, so that loads across fragments are coalesced.
 *  - n < 2^31.
 *
 * Orders. perm lists input indices by (destination, key). Packed keys order
 * fragments exactly as their tag tuples, i.e. in original stream order. Groups,
 * pending groups and mask nodes at a level >= route_level lie within one
 * destination and are listed by (destination, key); mask nodes above the route
 * level span destinations and are listed by key.
 */
#ifndef ALTO_H
#define ALTO_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ALTO_OK = 0,
  ALTO_E_ARG = 1,        /* bad argument (host check; nothing enqueued) */
  ALTO_E_LAYOUT = 2,     /* a tag >= 2^bits[level] or < 0, or a key wider than the layout */
  ALTO_E_DUPLICATE = 3,  /* the same full key twice (within a batch, or across stream steps) */
  ALTO_E_FANOUT = 4,     /* declared child count < 1, child index >= declared count,
                            or two carriers of one node declaring different counts */
  ALTO_E_LATE = 5,       /* stream: fragment of a group that was already emitted */
  ALTO_E_CAPACITY = 6,   /* an output or state capacity is too small; the sizes
                            needed are written to counts[] */
  ALTO_E_HIP = 7,        /* a HIP launch failed */
  ALTO_E_INTERNAL = 8    /* a bounded device-side wait gave up (not expected in
                            operation; outputs are invalid) */
} alto_status;

/* Key layout: depth d in [2, 16] levels; bits[l-1] >= 1 bits for level l, level 1
 * most significant; sum(bits) <= 63 so keys are also valid non-negative int64. */
typedef struct {
  int32_t depth;
  uint8_t bits[16];
} alto_layout;

enum { ALTO_CONCAT_I32 = 0, ALTO_MEAN_F32 = 1 };
enum { ALTO_RELEASE_COMPLETE = 0, ALTO_RELEASE_IN_ORDER = 1 };

/* Aggregation at a pmap exit: level = La in [1, d-1] (groups are the level-La
 * nodes); op = ALTO_CONCAT_I32 (list the int32 payloads of a group's leaves in key
 * order) or ALTO_MEAN_F32 (flat mean of the float32 rows of all leaves, float64
 * accumulation, one rounding to float32); dim = row width for MEAN (1 for
 * CONCAT); mask_level = Lm in [1, d-1], or 0 for no completion mask.
 * release (streams): ALTO_RELEASE_COMPLETE emits a group in the step that completes
 * it; ALTO_RELEASE_IN_ORDER puts the pmap's output stream back in its original
 * order (Section 3.2): the children of one parent (the level-(La-1) node) leave in
 * child-index order, a complete group waiting in the carried state until all of its
 * earlier siblings have left (with La = 1 the two coincide). Batches take
 * ALTO_RELEASE_COMPLETE only. */
typedef struct {
  int32_t level;
  int32_t op;
  int32_t dim;
  int32_t mask_level;
  int32_t release;
} alto_agg;

/* Outputs of an aggregation. Any array pointer may be NULL to skip that output;
 * counts must not be NULL. Capacities bound every write. */
typedef struct {
  int64_t cap_groups;   /* rows of key/dest/count/first_i32/fan_up/mean/pend_* */
  int64_t cap_tokens;   /* entries of tok */
  int64_t cap_mask;     /* entries of mask_key/mask */
  uint64_t *key;        /* [cap_groups] emitted (complete) group keys: the level-La prefix
                           (key >> bits below La) */
  int32_t *dest;        /* [cap_groups] destination of each emitted group */
  int64_t *count;       /* [cap_groups] leaves per emitted group */
  int32_t *first_i32;   /* [cap_groups] int32 payload of the group's first leaf in key order */
  int32_t *fan_up;      /* [(La-1) * cap_groups] declared child counts of levels 1..La-1 of
                           the group's ancestors, level-major with ld = cap_groups
                           (feeds a following aggregation stage) */
  int64_t *tok_off;     /* CONCAT: [cap_groups + 1] offsets into tok */
  int32_t *tok;         /* CONCAT: [cap_tokens] */
  float *mean;          /* MEAN: [cap_groups][dim] */
  uint64_t *mask_key;   /* [cap_mask] level-Lm nodes present in the batch */
  uint8_t *mask;        /* [cap_mask] 1 = the node's whole subtree is present */
  uint64_t *pend_key;   /* [cap_groups] incomplete level-La groups (not emitted) */
  int64_t *pend_count;  /* [cap_groups] leaves present per pending group */
  int64_t *counts;      /* device [4]: emitted groups, tokens, mask nodes, pending groups
                           (always written, also on ALTO_E_CAPACITY) */
} alto_groups;

/* Workspace bytes needed by alto_pack_keys / alto_route / alto_aggregate for up to
 * n_max fragments with this layout, destination count and aggregation (agg may be
 * NULL for routing only). Returns 0 for invalid arguments. */
size_t alto_workspace_bytes(const alto_layout *layout, int64_t n_max, int32_t num_dest,
                            const alto_agg *agg);

/* Key construction (Section 4.2: the tag stack of a fragment). Packs path (int32
 * [depth][path_ld], level-major, tag of level l at row l-1) into keys[n]
 * (uint64), level 1 in the most significant bits. A tag outside [0, 2^bits) sets
 * ALTO_E_LAYOUT. */
int alto_pack_keys(const int32_t *path, int64_t path_ld, int64_t n, const alto_layout *layout,
                   uint64_t *keys, int32_t *status, hipStream_t stream);

/* Routing by ancestry (Section 4.3) and order reconstitution (Sections 3.2, 4.1).
 * dest[i] = ((mix64(keys[i] >> bits below route_level) >> 32) * num_dest) >> 32 with
 * mix64 the SplitMix64 output function; route_level in [1, depth], num_dest in
 * [1, 2^24]. perm[n] (int32): input indices by (dest, key). dest_offsets[num_dest+1]
 * (int64): start of each destination's segment of perm; dest_offsets[num_dest] = n.
 * dest (nullable): per input fragment. Errors: LAYOUT, DUPLICATE. */
int alto_route(const uint64_t *keys, int64_t n, const alto_layout *layout, int32_t route_level,
               int32_t num_dest, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
               int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* Routing plus aggregation of one batch at a pmap exit (Sections 3.3 and 4.3).
 * fan: int32 [(depth-1)][fan_ld]; row l-1 holds each fragment's level-l ancestor's
 * declared child count. Rows of levels min(La, Lm)..depth-1 are read (checked:
 * >= 1, > the child index under it, equal on all carriers); rows 1..La-1 of the
 * group's first leaf are copied to fan_up. payload_i32 [n] is needed for CONCAT
 * and for first_i32; payload_f32 [n][dim] for MEAN. route_level = 0 sends every
 * fragment to destination 0 (num_dest must be 1); otherwise route_level must be in
 * [1, La] so that a group never spans destinations (a stateful consumer sees all
 * elements of its stream, Section 4.1). perm/dest_offsets/dest are as in
 * alto_route (perm and dest_offsets nullable here). A group is complete when every
 * node of its subtree has as many complete children as it declares (leaves are
 * complete on arrival); complete groups are emitted, the others listed as pending.
 * Errors: LAYOUT, FANOUT, DUPLICATE, CAPACITY. */
int alto_aggregate(const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                   const int32_t *payload_i32, const float *payload_f32, int64_t n,
                   const alto_layout *layout, const alto_agg *agg, int32_t route_level,
                   int32_t num_dest, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
                   alto_groups *out, int32_t *status, void *ws, size_t ws_bytes,
                   hipStream_t stream);

/* alto_aggregate with a count held in device memory (Section 4.2: a pmap exit
 * pops a level, so one stage's records are the next stage's fragments; reading the
 * count on the device lets a caller chain stages without a host synchronisation).
 * n_dev: device int64, read by the call's kernels in stream order (so it may be
 * written by earlier work on the same stream, e.g. counts[0] of a previous call);
 * n_max: a host bound on it that sizes every array argument (fan_ld >= n_max,
 * perm/dest/payloads of n_max entries) and the workspace (alto_workspace_bytes
 * with n_max). A count outside [0, n_max] is clamped and reported as CAPACITY.
 * With n_dev NULL this is alto_aggregate with n = n_max. Otherwise as
 * alto_aggregate (the radix sort then does not use its packed-word mode, whose
 * index width the host fixes). */
int alto_aggregate_dev(const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                       const int32_t *payload_i32, const float *payload_f32, int64_t n_max,
                       const int64_t *n_dev, const alto_layout *layout, const alto_agg *agg,
                       int32_t route_level, int32_t num_dest, int32_t *perm, int64_t *dest_offsets,
                       int32_t *dest, alto_groups *out, int32_t *status, void *ws, size_t ws_bytes,
                       hipStream_t stream);

/* alto_aggregate with the payload gathers (the concatenation, or the mean rows and
 * their combination) on gather_stream and everything before them (routing, order,
 * completion, group records) on `stream`; gather_stream waits for the records
 * through an event the call records on `stream`. A caller with several batches
 * runs the routing of the next batch beside this batch's gathers (the gathers are
 * bandwidth bound, the routing mostly latency bound): give each batch in flight
 * its own workspace, perm and `out`, and make `stream` wait for gather_stream (an
 * event) before a batch reuses them. The inputs are read on both streams. `out`'s
 * counts and records are written on `stream`, tok or mean on gather_stream. As
 * alto_aggregate otherwise; gather_stream == stream is alto_aggregate. */
int alto_aggregate_overlap(const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                           const int32_t *payload_i32, const float *payload_f32, int64_t n,
                           const alto_layout *layout, const alto_agg *agg, int32_t route_level,
                           int32_t num_dest, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
                           alto_groups *out, int32_t *status, void *ws, size_t ws_bytes,
                           hipStream_t stream, hipStream_t gather_stream);

/* ---- alto_aggregate without a workspace argument ----
 * For callers that cannot allocate device memory at the time of the call (code
 * under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, outputs, orders and errors as alto_aggregate, without ws and
 * ws_bytes: the workspace is a fixed array of ALTO_NOALLOC_SCRATCH_BYTES in the
 * library's own device memory, one per GPU, held from the first call on that GPU
 * until the process ends. Calls with alto_workspace_bytes(layout, n, num_dest,
 * agg) > ALTO_NOALLOC_SCRATCH_BYTES return ALTO_E_ARG (nothing is enqueued); that
 * is about 600k fragments for a six-level layout with a 128-float mean and a
 * completion mask, 1.1M for a five-level one with a 768-float mean. The call
 * allocates nothing. Every call on one GPU
 * shares that GPU's array, and it keeps what the last call left there: calls on
 * one GPU that overlap in time (different streams, or different host threads)
 * race on it and give undefined outputs; serialise them. ALTO_E_HIP if the
 * array's device address cannot be obtained. */
#define ALTO_NOALLOC_SCRATCH_BYTES (128ull << 20)
int alto_aggregate_noalloc(const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                           const int32_t *payload_i32, const float *payload_f32, int64_t n,
                           const alto_layout *layout, const alto_agg *agg, int32_t route_level,
                           int32_t num_dest, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
                           alto_groups *out, int32_t *status, hipStream_t stream);

/* ---- streams: partial groups carried across steps (Section 3.1: outputs stream
 * before their inputs are complete; Section 4.2: aggregation at pmap exit) ---- */

typedef struct alto_stream alto_stream; /* opaque host handle; state memory is the caller's */

/* Device state bytes for a stream that holds at most max_live_leaves arrived
 * leaves of not-yet-emitted groups and sees at most max_groups distinct level-La
 * groups over its lifetime (emitted groups are remembered to detect late
 * fragments; with in-order release, so are the parents' release positions).
 * Returns 0 for invalid arguments. */
size_t alto_stream_state_bytes(const alto_layout *layout, const alto_agg *agg,
                               int64_t max_live_leaves, int64_t max_groups);

/* Creates a handle over caller-owned device memory `state` (state_bytes from
 * alto_stream_state_bytes with the same limits) and clears it on `stream`.
 * route_level must be in [1, La]; mask_level must be 0. */
int alto_stream_create(const alto_layout *layout, int32_t route_level, int32_t num_dest,
                       const alto_agg *agg, int64_t max_live_leaves, int64_t max_groups,
                       void *state, size_t state_bytes, hipStream_t stream, alto_stream **out);

/* One step: routes the step's n fragments on their own (perm, dest_offsets, dest as
 * in alto_route, all nullable), merges them into the carried state, and emits the
 * groups this step releases (see alto_agg.release), each once, with its payload
 * computed over all of its leaves in key order (count, key, dest, first_i32,
 * fan_up, tok_off/tok or mean); groups not released are listed in pend_key/pend_count.
 * Emitted groups per step are at most n; emitted tokens at most max_live_leaves + n.
 * Workspace: alto_workspace_bytes(layout, max_live_leaves + n_max, num_dest, agg)
 * with n_max >= n (the step is merged with the carried leaves).
 * Errors: LAYOUT, LATE, FANOUT, DUPLICATE, CAPACITY (state full or outputs too
 * small). A data error poisons the handle: every later step reports it again. */
int alto_stream_step(alto_stream *s, const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                     const int32_t *payload_i32, const float *payload_f32, int64_t n,
                     int32_t *perm, int64_t *dest_offsets, int32_t *dest, alto_groups *emitted,
                     int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* alto_stream_step with the step's count in device memory (n_dev, read in stream
 * order; n_max bounds it and sizes the arrays, the workspace and the emitted
 * capacities as n does for alto_stream_step). Chaining two streams: stage B's
 * keys, fan, payload_i32 and n_dev are stage A's emitted key, fan_up, first_i32
 * and counts[0] (emitted groups per step are at most the step's count, so stage A's
 * bound serves as stage B's n_max). A count outside [0, n_max] is clamped and
 * reported as CAPACITY. */
int alto_stream_step_dev(alto_stream *s, const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                         const int32_t *payload_i32, const float *payload_f32, int64_t n_max,
                         const int64_t *n_dev, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
                         alto_groups *emitted, int32_t *status, void *ws, size_t ws_bytes,
                         hipStream_t stream);

/* alto_stream_step_dev with the step's routing (its sort, the checks of its keys and
 * counts, the fragment side of the fan fingerprint) on route_stream and the rest
 * (merge, completion, emission, carried state) on `stream` after it, so that the
 * routing of the next step runs beside this step's merge and emission (Section 3.1:
 * partial outputs are streamed; the routing of a step does not depend on the
 * carried state). Steps use ws0 and ws1 alternately (each sized as for
 * alto_stream_step_dev, ws0 != ws1); route_stream first waits until the step two
 * calls back, which used the same workspace, has ended on `stream` (events held by
 * the handle, created at the first call). The merge's first kernel waits on the
 * device for the routing: a one-thread kernel on route_stream, after the routing
 * and whatever the caller enqueued there before, stores the step's sequence number
 * in a word of the handle's state, and the merge's blocks that hold elements (at
 * most 256, one per CU, so that the routing finds room beside them) poll it
 * before they read the routing's outputs. The wait is bounded (seconds; then ALTO_E_INTERNAL in `status`), so
 * route_stream must not wait for work that the caller enqueues on `stream` after
 * this call. The inputs (keys, fan, payloads, n_dev) are read on route_stream,
 * and on `stream` only after the routing's word (by kernels that follow the
 * merge's wait): they must be ready on route_stream; a producer on another stream
 * needs only route_stream to wait for it. perm, dest, dest_offsets and `emitted`
 * are written on `stream`; the routing of the next call may already
 * run when this call returns, so consecutive calls must not share input buffers
 * that the caller rewrites in between. Errors as for alto_stream_step_dev; ALTO_E_ARG
 * when ws0 or ws1 is null or they are equal. */
int alto_stream_step_overlap(alto_stream *s, const uint64_t *keys, const int32_t *fan, int64_t fan_ld,
                             const int32_t *payload_i32, const float *payload_f32, int64_t n_max,
                             const int64_t *n_dev, int32_t *perm, int64_t *dest_offsets, int32_t *dest,
                             alto_groups *emitted, int32_t *status, void *ws0, void *ws1, size_t ws_bytes,
                             hipStream_t route_stream, hipStream_t stream);

/* Lists the groups that have arrived leaves but were never released (incomplete,
 * or complete and waiting for an earlier sibling), by (dest, key):
 * pend_key, pend_count and counts[3] of `out`; other members are ignored. */
int alto_stream_pending(alto_stream *s, alto_groups *out, int32_t *status, hipStream_t stream);

/* Frees the host handle (the caller frees the state memory). */
int alto_stream_destroy(alto_stream *s);

/* ---- pcombine: combining the outputs of two parallel branches by ancestry
 * (Section 3.2, the pcombine operator; Section 4.2: the runtime associates objects
 * that share ancestry) ---- */

/* Workspace bytes for alto_join with up to n_left_max left objects. */
size_t alto_join_workspace_bytes(const alto_layout *layout, int64_t n_left_max);

/* Pairs every right fragment with the left object of its level-`level` ancestor.
 * left[n_left] (uint64): one object per level-`level` node, given by the node's
 * prefix (key >> bits below `level`, the format of alto_groups.key); right_keys
 * [n_right] (uint64): full keys of `layout`. level in [1, depth].
 * match[n_right] (int32): index into left of the fragment's object, -1 if none.
 * hits[n_left] (int32, nullable): right fragments paired with each left object.
 * counts: device int64[2]: paired right fragments, left objects with a pair.
 * All arrays are caller-owned device memory; enqueues on `stream`, no sync.
 * Errors: LAYOUT (a right key or left prefix wider than its levels), DUPLICATE
 * (two left objects for one node; match is then undefined). */
int alto_join(const uint64_t *left, int64_t n_left, const uint64_t *right_keys, int64_t n_right,
              const alto_layout *layout, int32_t level, int32_t *match, int32_t *hits, int64_t *counts,
              int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* ---- load-aware routing (Section 4.3: the destination of a new flow of tags may
 * be chosen by load instead of by hashing; Section 5: replicas chosen by queue
 * length) ---- */

typedef struct alto_router alto_router; /* opaque host handle; flow table in caller memory */

/* Device state bytes for a router that remembers up to max_flows flows. */
size_t alto_router_state_bytes(int64_t max_flows);

/* Creates a router over caller-owned device memory `state` and clears it on
 * `stream`. A flow is a distinct level-`route_level` prefix (route_level in [1,
 * depth]); num_dest in [1, 4096]. */
int alto_router_create(const alto_layout *layout, int32_t route_level, int32_t num_dest, int64_t max_flows,
                       void *state, size_t state_bytes, hipStream_t stream, alto_router **out);

/* Frees the host handle (the caller frees the state memory). */
int alto_router_destroy(alto_router *r);

/* Workspace bytes for alto_route_load with up to n_max fragments (layout and
 * route_level as given to alto_router_create). */
size_t alto_route_load_workspace_bytes(const alto_layout *layout, int32_t route_level, int64_t n_max,
                                       int32_t num_dest);

/* Routes one batch. load: device int64[num_dest], the destinations' queue lengths,
 * updated in place (the caller subtracts what a destination has consumed between
 * calls). A flow seen in an earlier call keeps its destination, and its fragments
 * are added to that queue first; then the batch's new flows, in ascending prefix
 * order, each go to the shortest queue (the lowest index among equal ones), which
 * grows by the flow's fragments in the batch. perm (int32 [n], nullable): input
 * indices in (destination, key) order; dest_offsets (int64 [num_dest + 1],
 * nullable); dest (int32 [n], nullable): per input fragment. counts: device
 * int64[2]: new flows assigned, flows seen before. Errors: LAYOUT, DUPLICATE,
 * CAPACITY (the new flows do not fit in max_flows). On any error, including one
 * already in *status on entry, neither load nor the flow table changes and the
 * outputs are undefined. Calls on one router must not overlap. */
int alto_route_load(alto_router *r, const uint64_t *keys, int64_t n, int64_t *load, int32_t *perm,
                    int64_t *dest_offsets, int32_t *dest, int64_t *counts, int32_t *status, void *ws,
                    size_t ws_bytes, hipStream_t stream);

/* ---- split_text at a pmap entry (Section 3.2, the split_text operator; Section
 * 4.2: entering a pmap pushes a level onto the tag stack) ---- */

/* Workspace bytes for alto_split with up to n_max tokens. */
size_t alto_split_workspace_bytes(const alto_layout *layout, int64_t n_max);

/* Splits token streams at a delimiter. keys[n] (uint64, `layout` of depth d in
 * [2, 15]): tokens, leaves whose level-(d-1) node (the parent) is one stream
 * element and whose leaf tag is the token's index in it. fan: int32 [(d-1)][fan_ld]
 * as in alto_aggregate; row d-2 holds the parent's declared token count.
 * tokens[n] (int32): token ids; tokens equal to `delim` separate segments. A
 * parent whose declared tokens are all present is cut into segments, the maximal
 * runs of non-delimiter tokens in index order (no empty segments); a parent with a
 * token missing is not cut (the missing token could be a delimiter).
 * The new fragments leave as a batch in ascending new-key order, rows
 * 0..counts[0]-1 of: out_keys (uint64): (parent prefix << (seg_bits + tok_bits)) |
 * (segment index << tok_bits) | index in segment, a key of the layout
 * bits[0..d-2] + (seg_bits, tok_bits), seg_bits and tok_bits in [1, 32];
 * out_fan: int32 [d][out_fan_ld], rows 0..d-3 copied from fan, row d-2 the
 * parent's segment count, row d-1 the segment's token count; out_tokens (int32,
 * nullable): the token; out_idx (int32, nullable): its input index (to move other
 * payload columns). rest_idx (int32, nullable): input indices of the tokens of
 * incomplete parents, in key order, counts[2] of them (to be offered again with
 * the rest of their stream). Delimiters are dropped. Every output array holds n
 * entries (out_fan_ld >= n). counts: device int64[4]: placed tokens, delimiters of
 * complete parents, tokens of incomplete parents, segments. Arrays are
 * caller-owned device memory; enqueues on `stream`, no sync. Errors: LAYOUT (a key
 * wider than the layout), FANOUT (a declared count < 1, an index >= it, carriers
 * of one parent disagreeing), DUPLICATE (a token key twice), CAPACITY (a segment
 * index or an index in a segment that does not fit its bits); outputs are
 * undefined on any error. */
int alto_split(const uint64_t *keys, const int32_t *fan, int64_t fan_ld, const int32_t *tokens, int64_t n,
               const alto_layout *layout, int32_t delim, int32_t seg_bits, int32_t tok_bits,
               uint64_t *out_keys, int32_t *out_fan, int64_t out_fan_ld, int32_t *out_tokens,
               int32_t *out_idx, int32_t *rest_idx, int64_t *counts, int32_t *status, void *ws,
               size_t ws_bytes, hipStream_t stream);

/* ---- diagnostics: per-phase timing with HIP events on the caller's stream ----
 * Phases: 0 input-order pass (layout check, routing hash, fan checks), 1 radix sort
 * and destination offsets, 2 node segmentation and completion, 3 group records and
 * chunk lists, 4 payload gathers, 5 the mean gather kernel alone, 6 whole call.
 * alto_profile_begin creates a pool of max_records event pairs; while it is active,
 * every entry point records one pair per phase it runs (until the pool is used
 * up). alto_profile_end waits for the recorded events, writes the summed
 * milliseconds and the number of records per phase (arrays of nphase entries),
 * and destroys the pool. Host-side only; not thread-safe. */
int alto_profile_begin(int32_t max_records);

/* Selects the phases recorded by the next alto_profile_begin (bit p = phase p;
 * default: all). Fewer event pairs per call disturb the timed calls less. Not
 * while a pool is active (ALTO_E_ARG). */
int alto_profile_phases(uint32_t mask);

/* Diagnostics: reads `bytes` (a multiple of 16, 16-byte aligned) of device memory
 * once with a plain streaming kernel; the attainable read bandwidth that the kernels
 * above are compared with. out: device uint64[ALTO_READ_PROBE_WORDS]; entry b gets
 * the XOR of the 32-bit words read by block b (unused entries 0), so the XOR of all
 * entries is the XOR of all words read. */
enum { ALTO_READ_PROBE_WORDS = 16384 };
int alto_read_probe(const void *p, int64_t bytes, uint64_t *out, hipStream_t stream);
int alto_profile_end(float *ms, int32_t *calls, int32_t nphase);

#ifdef __cplusplus
}
#endif

#endif /* ALTO_H */
