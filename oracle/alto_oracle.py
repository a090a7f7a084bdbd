"""CPU oracle for nested-ancestry routing and aggregation.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this module. It is a plain, slow, single-threaded
numpy definition of what the GPU path computes, and it shares no code with it.

Model (paper, Section 4.2 "Nested Ancestry" and Section 4.3 "Routing with
Ancestry"): every fragment carries a stack of ancestry tags, one per level of
pmap nesting. Level 1 is the request, level ``d`` the fragment itself. A pmap
entry pushes a tag (the element's index in its parent's stream); a pmap exit pops
one and aggregates the outputs generated under the same parent. All elements that
share the same tags are routed to the same instance (Section 4.3, like ECMP but on
tags). A stream that is parallelised must be put back in its original order for
sequential consumers (Section 3.2, pmap; Section 4.1). The size of a generated
stream is unknown until its end (Section 3.1), so every node declares its child
count and a group is complete only when its whole subtree has arrived.

Readings where the paper is silent (each is listed in the design notes):

* Keys: tags are packed most-significant level first into one uint64, ``bits[l-1]``
  bits for level ``l``; numeric key order is then the lexicographic path order,
  the original stream order.
* Routing hash: ``dest = ((mix64(prefix) >> 32) * D) >> 32`` where ``mix64`` is the
  SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014) and the range
  reduction is Lemire's multiply-shift (2019).
* ``perm`` lists input indices ordered by (dest, key). Groups, pending groups and
  mask nodes at a level ``L >= Lr`` are ordered by (dest, key); mask nodes above the
  route level (``L < Lr``) span destinations and are ordered by key.
* Completion is the recursive definition: a leaf is complete on arrival; a node
  at level ``l`` is complete when the number of its complete children equals its
  declared child count ``fan[l]``.
* MEAN pools all leaves of a group (flat mean), accumulated in float64 and
  rounded once to float32. CONCAT lists the payloads of a group's leaves in key
  order. FIRST is the payload of the group's first leaf in key order.
* Error priority in a batch: layout, then fan-out, then duplicate, then capacity.
  In a stream: layout, late, fan-out, duplicate, capacity.
* Release order of a stream (Section 3.2, pmap: as items finish, the stream is put
  back in its original order and sent on): by default a group leaves in the step
  that completes it; in order, the groups under one parent (the level above the
  aggregation level) leave in child-index order, a complete group waiting for all
  of its earlier siblings. Groups of different parents do not wait for each other.
* split_text at a pmap entry (Section 3.2; Section 4.2 pushes a level): a parent's
  tokens are cut at a delimiter token into maximal runs of other tokens; only a
  parent whose declared tokens have all arrived is cut (a missing token could be a
  delimiter). The new fragments leave as a batch in new-key order; the tokens of
  incomplete parents are listed in key order for a later attempt.
* Load-aware routing (Section 4.3: a new flow of tags may be sent by load rather
  than by hash; Section 5: replicas chosen by queue length): a flow is a distinct
  route-level prefix and keeps its first destination. Per batch the fragments of
  known flows join their queues first, then new flows in ascending prefix order take
  the shortest queue (lowest index among ties), which grows by the flow's fragments.

Parity is pinned against brute force, closed forms and textbook routines in
``tests/test_oracle_*.py``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

OK, E_ARG, E_LAYOUT, E_DUPLICATE, E_FANOUT, E_LATE, E_CAPACITY = 0, 1, 2, 3, 4, 5, 6
CONCAT, MEAN = "concat", "mean"

U64 = np.uint64


class OracleError(Exception):
    def __init__(self, code: int, what: str = ""):
        super().__init__(f"code {code}: {what}")
        self.code = code


# ---------------------------------------------------------------------------
# keys (nested ancestry tags packed into one integer)
# ---------------------------------------------------------------------------

def shift_below(bits: Sequence[int], level: int) -> int:
    """Number of key bits that belong to levels deeper than ``level`` (1-based)."""
    return int(sum(bits[level:]))


def prefix(keys: np.ndarray, bits: Sequence[int], level: int) -> np.ndarray:
    """The tags of levels 1..level, as an integer (key with deeper levels dropped)."""
    return keys >> U64(shift_below(bits, level))


def tag(keys: np.ndarray, bits: Sequence[int], level: int) -> np.ndarray:
    """The level-``level`` tag of each key."""
    return prefix(keys, bits, level) & U64((1 << bits[level - 1]) - 1)


def check_layout(bits: Sequence[int]):
    if not (2 <= len(bits) <= 16) or any(b < 1 for b in bits) or sum(bits) > 63:
        raise OracleError(E_ARG, "layout")


def pack_keys(path: np.ndarray, bits: Sequence[int]) -> np.ndarray:
    """Pack int32 tags ``path[l-1][i]`` into uint64 keys, level 1 most significant."""
    check_layout(bits)
    path = np.asarray(path)
    d = len(bits)
    if path.ndim != 2 or path.shape[0] != d:
        raise OracleError(E_ARG, "path shape")
    keys = np.zeros(path.shape[1], dtype=U64)
    for level in range(1, d + 1):
        t = path[level - 1].astype(np.int64)
        if t.size and (t.min() < 0 or t.max() >= (1 << bits[level - 1])):
            raise OracleError(E_LAYOUT, f"tag at level {level} does not fit")
        keys |= t.astype(U64) << U64(shift_below(bits, level))
    return keys


# ---------------------------------------------------------------------------
# routing (Section 4.3)
# ---------------------------------------------------------------------------

def mix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64 output function: two xor-shift-multiply rounds and a final xor-shift."""
    with np.errstate(over="ignore"):
        z = np.asarray(x, dtype=U64).copy()
        z = (z ^ (z >> U64(30))) * U64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> U64(27))) * U64(0x94D049BB133111EB)
        return z ^ (z >> U64(31))


def dest_of(prefixes: np.ndarray, num_dest: int) -> np.ndarray:
    """Destination of a tag prefix: hash, then multiply-shift range reduction."""
    h = mix64(prefixes) >> U64(32)
    with np.errstate(over="ignore"):
        return ((h * U64(num_dest)) >> U64(32)).astype(np.int32)


def route_dest(keys: np.ndarray, bits: Sequence[int], route_level: int, num_dest: int):
    if route_level == 0:
        return np.zeros(len(keys), dtype=np.int32)
    return dest_of(prefix(keys, bits, route_level), num_dest)


def _check_keys_fit(keys: np.ndarray, bits: Sequence[int]):
    if len(keys) and int(keys.max()) >> int(sum(bits)) != 0:
        raise OracleError(E_LAYOUT, "key wider than the layout")


@dataclass
class Route:
    perm: np.ndarray          # int32 [n], input indices in (dest, key) order
    dest_offsets: np.ndarray  # int64 [D+1]
    dest: np.ndarray          # int32 [n], input order


def route(keys: np.ndarray, bits: Sequence[int], route_level: int, num_dest: int) -> Route:
    """Hash-partition fragments by their level-``route_level`` prefix, then order
    each destination's fragments by key (the original stream order)."""
    check_layout(bits)
    keys = np.asarray(keys, dtype=U64)
    if not (1 <= route_level <= len(bits)) or num_dest < 1:
        raise OracleError(E_ARG, "route level / destinations")
    _check_keys_fit(keys, bits)
    if len(np.unique(keys)) != len(keys):
        raise OracleError(E_DUPLICATE, "same key twice")
    dest = route_dest(keys, bits, route_level, num_dest)
    perm = np.lexsort((keys, dest)).astype(np.int32)
    counts = np.bincount(dest, minlength=num_dest).astype(np.int64)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    return Route(perm, offs, dest)


# ---------------------------------------------------------------------------
# completion (Section 3.1 end-of-output; pmap exit in Section 4.2)
# ---------------------------------------------------------------------------

def node_fans(keys: np.ndarray, fan: np.ndarray, bits: Sequence[int], level: int):
    """Distinct level-``level`` nodes among the keys and the child count each declares.

    Raises FANOUT when the carriers of one node disagree."""
    p = prefix(keys, bits, level)
    nodes, inv = np.unique(p, return_inverse=True)
    f = fan[level - 1].astype(np.int64)
    lo = np.full(len(nodes), np.iinfo(np.int64).max)
    hi = np.full(len(nodes), np.iinfo(np.int64).min)
    np.minimum.at(lo, inv, f)
    np.maximum.at(hi, inv, f)
    if (lo != hi).any():
        raise OracleError(E_FANOUT, f"carriers disagree at level {level}")
    return nodes, lo


def check_fanout(keys, fan, bits, lo_level: int):
    """Declared child counts of levels lo_level..d-1: at least 1, larger than every
    child index under the node, and identical on every carrier."""
    d = len(bits)
    for level in range(lo_level, d):
        f = fan[level - 1].astype(np.int64)
        if f.size and f.min() < 1:
            raise OracleError(E_FANOUT, f"child count < 1 at level {level}")
        if f.size and (tag(keys, bits, level + 1).astype(np.int64) >= f).any():
            raise OracleError(E_FANOUT, f"child index >= child count at level {level}")
        node_fans(keys, fan, bits, level)


def completion(keys, fan, bits, lo_level: int) -> Dict[int, tuple]:
    """For each level from d-1 down to ``lo_level``: (nodes, complete flags).

    A leaf is complete; a node is complete when its complete children number
    exactly its declared child count."""
    d = len(bits)
    out = {}
    child_nodes = np.unique(keys)
    child_complete = np.ones(len(child_nodes), dtype=bool)
    for level in range(d - 1, lo_level - 1, -1):
        nodes, declared = node_fans(keys, fan, bits, level)
        parent_of_child = child_nodes >> U64(bits[level])
        idx = np.searchsorted(nodes, parent_of_child)
        ncomplete = np.bincount(idx, weights=child_complete.astype(np.float64),
                                minlength=len(nodes)).astype(np.int64)
        complete = ncomplete == declared
        out[level] = (nodes, complete)
        child_nodes, child_complete = nodes, complete
    return out


# ---------------------------------------------------------------------------
# aggregation at pmap exit (Section 3.3 aggregate operator, Section 4.3)
# ---------------------------------------------------------------------------

@dataclass
class Groups:
    key: np.ndarray                  # uint64 [G] emitted (complete) groups
    dest: np.ndarray                 # int32 [G]
    count: np.ndarray                # int64 [G] leaves per group
    first_i32: Optional[np.ndarray]  # int32 [G]
    fan_up: np.ndarray               # int32 [La-1][G]
    tok_off: Optional[np.ndarray]    # int64 [G+1]   (concat)
    tok: Optional[np.ndarray]        # int32 [sum]   (concat)
    mean: Optional[np.ndarray]       # float32 [G][dim] (mean)
    mask_key: Optional[np.ndarray]   # uint64 [M]
    mask: Optional[np.ndarray]       # uint8 [M]
    pend_key: np.ndarray             # uint64 [P] incomplete groups
    pend_count: np.ndarray           # int64 [P]


def _order_by_dest_key(keys_at_level: np.ndarray, dests: np.ndarray) -> np.ndarray:
    return np.lexsort((keys_at_level, dests))


def _group_payloads(members: List[np.ndarray], op: str, dim: int, payload_i32, payload_f32):
    """Payload of each group over its leaves (``members[g]``, input indices in key order)."""
    tok_off = tok = mean = None
    if op == CONCAT:
        tok_off = np.concatenate([[0], np.cumsum([len(m) for m in members])]).astype(np.int64)
        tok = (np.concatenate([payload_i32[m] for m in members]) if members
               else np.zeros(0)).astype(np.int32)
    else:
        mean = np.zeros((len(members), dim), dtype=np.float32)
        budget = max(1, (1 << 24) // max(dim, 1))          # rows per float64 batch
        gi = 0
        while gi < len(members):
            gj, rows = gi, 0
            while gj < len(members) and (gj == gi or rows + len(members[gj]) <= budget):
                rows += len(members[gj])
                gj += 1
            part = members[gi:gj]
            x = np.asarray(payload_f32[np.concatenate(part)], dtype=np.float64)
            starts = np.concatenate([[0], np.cumsum([len(m) for m in part])[:-1]]).astype(np.int64)
            sums = np.add.reduceat(x, starts, axis=0)
            cnt = np.array([len(m) for m in part], dtype=np.float64)
            mean[gi:gj] = (sums / cnt[:, None]).astype(np.float32)
            gi = gj
    return tok_off, tok, mean


def group_mean(rows) -> np.ndarray:
    """The pooled vector of one group from all of its leaves' rows: their float64
    sum divided by their count, rounded once to float32 (the aggregate operator of
    Section 3.3 read as a flat mean over the group's leaves). ``aggregate`` computes
    the same for every group of a batch; this form takes one group's rows at a time,
    so a check of a very large batch never holds more than one group in float64."""
    x = np.asarray(rows, dtype=np.float32)
    if x.ndim != 2 or len(x) == 0:
        raise OracleError(E_ARG, "rows of one non-empty group")
    return (x.sum(axis=0, dtype=np.float64) / np.float64(len(x))).astype(np.float32)


def aggregate(keys, fan, bits, agg_level: int, op: str, dim: int = 1, mask_level: int = 0,
              route_level: int = 0, num_dest: int = 1, payload_i32=None, payload_f32=None,
              cap_groups: Optional[int] = None, cap_tokens: Optional[int] = None,
              cap_mask: Optional[int] = None):
    """Route a batch and aggregate it at ``agg_level``.

    Returns ``(Route, Groups)``. Raises ``OracleError`` with the status code the
    GPU path must report."""
    check_layout(bits)
    d = len(bits)
    keys = np.asarray(keys, dtype=U64)
    n = len(keys)
    La, Lm, Lr = agg_level, mask_level, route_level
    if not (1 <= La <= d - 1) or not (Lm == 0 or 1 <= Lm <= d - 1):
        raise OracleError(E_ARG, "levels")
    if not (0 <= Lr <= La) or num_dest < 1 or (Lr == 0 and num_dest != 1):
        raise OracleError(E_ARG, "route level must not exceed the aggregation level")
    if op not in (CONCAT, MEAN) or (op == MEAN and (payload_f32 is None or dim < 1)):
        raise OracleError(E_ARG, "op")
    if op == CONCAT and payload_i32 is None:
        raise OracleError(E_ARG, "concat needs int32 payload")
    fan = np.asarray(fan)
    lo = min(La, Lm) if Lm else La
    _check_keys_fit(keys, bits)
    check_fanout(keys, fan, bits, lo)
    if len(np.unique(keys)) != n:
        raise OracleError(E_DUPLICATE, "same key twice")

    dest = route_dest(keys, bits, Lr, num_dest)
    perm = np.lexsort((keys, dest)).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(np.bincount(dest, minlength=num_dest))]).astype(np.int64)
    rt = Route(perm, offs, dest)

    comp = completion(keys, fan, bits, lo)
    gnodes, gcomplete = comp[La]                       # ascending group keys
    # leaves of each group, in key order
    by_key = np.argsort(keys, kind="stable")
    gk_sorted = prefix(keys, bits, La)[by_key]
    gstart = np.searchsorted(gk_sorted, gnodes, side="left")
    gend = np.searchsorted(gk_sorted, gnodes, side="right")
    gdest = route_dest(gnodes << U64(shift_below(bits, La)), bits, Lr, num_dest)
    order = _order_by_dest_key(gnodes, gdest)
    emit = [int(g) for g in order if gcomplete[g]]
    pend = [int(g) for g in order if not gcomplete[g]]
    members = [by_key[gstart[g]:gend[g]] for g in emit]
    first = np.array([m[0] for m in members], dtype=np.int64)
    fan_up = (np.stack([fan[l - 1][first] for l in range(1, La)]).astype(np.int32)
              if La > 1 else np.zeros((0, len(emit)), np.int32))
    first_i32 = payload_i32[first].astype(np.int32) if payload_i32 is not None else None
    tok_off, tok, mean = _group_payloads(members, op, dim, payload_i32, payload_f32)
    mask_key = mask = None
    if Lm:
        mnodes, mcomplete = comp[Lm]
        if Lm >= Lr:
            md = route_dest(mnodes << U64(shift_below(bits, Lm)), bits, Lr, num_dest)
            o = _order_by_dest_key(mnodes, md)
        else:
            o = np.argsort(mnodes, kind="stable")
        mask_key, mask = mnodes[o], mcomplete[o].astype(np.uint8)
    gcount = (gend - gstart).astype(np.int64)
    g = Groups(gnodes[emit], gdest[emit], gcount[emit], first_i32, fan_up, tok_off, tok, mean,
               mask_key, mask, gnodes[pend], gcount[pend])
    need = (len(emit), 0 if tok is None else len(tok), 0 if mask is None else len(mask), len(pend))
    if ((cap_groups is not None and (need[0] > cap_groups or need[3] > cap_groups))
            or (cap_tokens is not None and need[1] > cap_tokens)
            or (cap_mask is not None and need[2] > cap_mask)):
        err = OracleError(E_CAPACITY, "output capacity")
        err.need = need
        raise err
    return rt, g


# ---------------------------------------------------------------------------
# streams: partial groups carried between steps
# ---------------------------------------------------------------------------

@dataclass
class StepResult:
    route: Route
    groups: Groups       # emitted this step (mask and pending unused)


RELEASE_COMPLETE, RELEASE_IN_ORDER = "complete", "in_order"


class Stream:
    """Feed a stream in steps. Each step is routed on its own; leaves of groups that
    are not released are carried; a group is emitted once, in the step that releases
    it, with its payload computed over all of its leaves in key order.

    release="complete": a group is released in the step that completes it.
    release="in_order": the children of one parent (level agg_level - 1) are released
    in child-index order: child c leaves once children 0..c are all complete (the
    pmap exit of Section 3.2 puts the parallelised stream back in its original
    order). With agg_level 1 there is no parent and the two coincide."""

    def __init__(self, bits, route_level: int, num_dest: int, agg_level: int, op: str,
                 dim: int = 1, release: str = RELEASE_COMPLETE):
        check_layout(bits)
        d = len(bits)
        if not (1 <= agg_level <= d - 1) or not (1 <= route_level <= agg_level) or num_dest < 1:
            raise OracleError(E_ARG, "levels")
        if release not in (RELEASE_COMPLETE, RELEASE_IN_ORDER):
            raise OracleError(E_ARG, "release order")
        self.release = release
        self.cursor = {}                                       # parent prefix -> next child to release
        self.bits, self.Lr, self.D, self.La, self.op, self.dim = tuple(bits), route_level, num_dest, agg_level, op, dim
        self.d = d
        self.keys = np.zeros(0, U64)                           # arrived leaves of live groups
        self.fan = np.zeros((d - 1, 0), np.int32)
        self.p32 = np.zeros(0, np.int32)
        self.pf = np.zeros((0, dim), np.float32) if op == MEAN else None
        self.emitted = set()
        self.error = OK

    def step(self, keys, fan, payload_i32=None, payload_f32=None) -> StepResult:
        if self.error:
            raise OracleError(self.error, "stream poisoned")
        try:
            return self._step(keys, fan, payload_i32, payload_f32)
        except OracleError as e:
            if e.code != E_ARG:
                self.error = e.code
            raise

    def _step(self, keys, fan, payload_i32, payload_f32) -> StepResult:
        bits, La = self.bits, self.La
        keys = np.asarray(keys, dtype=U64)
        fan = np.asarray(fan).astype(np.int32)
        n = len(keys)
        if payload_i32 is None:
            payload_i32 = np.zeros(n, np.int32)
        _check_keys_fit(keys, bits)
        gk = prefix(keys, bits, La)
        if any(int(k) in self.emitted for k in np.unique(gk)):
            raise OracleError(E_LATE, "fragment of an emitted group")
        all_keys = np.concatenate([self.keys, keys])
        all_fan = np.concatenate([self.fan, fan], axis=1)
        check_fanout(all_keys, all_fan, bits, La)
        if len(np.unique(all_keys)) != len(all_keys):
            raise OracleError(E_DUPLICATE, "same key twice")
        rt = route(keys, bits, self.Lr, self.D)
        all_p32 = np.concatenate([self.p32, np.asarray(payload_i32, np.int32)])
        all_pf = None
        if self.op == MEAN:
            all_pf = np.concatenate([self.pf, np.asarray(payload_f32, np.float32).reshape(n, self.dim)])
        live_gk = prefix(all_keys, bits, La)
        if self.release == RELEASE_IN_ORDER and La >= 2:
            # completion of every live group (a complete group may wait for earlier
            # siblings across steps), then each parent's children in child order
            comp = completion(all_keys, all_fan, bits, La)
            gnodes, gcomplete = comp[La]
            complete = set(int(x) for x in gnodes[gcomplete])
            cb = bits[La - 1]
            released = []
            for parent in sorted(set(int(x) >> cb for x in gnodes)):
                c = self.cursor.get(parent, 0)
                while ((parent << cb) | c) in complete:
                    released.append((parent << cb) | c)
                    c += 1
                self.cursor[parent] = c
            done = np.array(sorted(released), dtype=U64)
        else:
            # completion of the groups this step touched, over all their arrived leaves
            touched = np.unique(gk)
            sel = np.isin(live_gk, touched)
            comp = completion(all_keys[sel], all_fan[:, sel], bits, La)
            gnodes, gcomplete = comp[La]
            done = gnodes[gcomplete]
        in_done = np.isin(live_gk, done)
        if len(done):
            _, g = aggregate(all_keys[in_done], all_fan[:, in_done], bits, La, self.op, self.dim, 0,
                             self.Lr, self.D, all_p32[in_done],
                             None if all_pf is None else all_pf[in_done])
        else:
            g = _empty_groups(La, self.op, self.dim)
        for k in done:
            self.emitted.add(int(k))
        keep = ~in_done
        self.keys, self.fan, self.p32 = all_keys[keep], all_fan[:, keep], all_p32[keep]
        if self.op == MEAN:
            self.pf = all_pf[keep]
        return StepResult(rt, g)

    def pending(self):
        """Groups with arrived leaves that never completed: (keys, counts), (dest, key) order."""
        gk = prefix(self.keys, self.bits, self.La)
        nodes, cnt = np.unique(gk, return_counts=True)
        dest = route_dest(nodes << U64(shift_below(self.bits, self.La)), self.bits, self.Lr, self.D)
        o = _order_by_dest_key(nodes, dest)
        return nodes[o], cnt[o].astype(np.int64)


def _empty_groups(La, op, dim):
    z64 = np.zeros(0, U64)
    return Groups(z64, np.zeros(0, np.int32), np.zeros(0, np.int64), np.zeros(0, np.int32),
                  np.zeros((La - 1, 0), np.int32),
                  np.zeros(1, np.int64) if op == CONCAT else None,
                  np.zeros(0, np.int32) if op == CONCAT else None,
                  np.zeros((0, dim), np.float32) if op == MEAN else None,
                  None, None, z64, np.zeros(0, np.int64))


# ---------------------------------------------------------------------------
# pcombine: join of two branches by ancestry
# ---------------------------------------------------------------------------

@dataclass
class Join:
    match: np.ndarray      # int32 [n_right]: left index with the same level-Lj prefix, or -1
    hits: np.ndarray       # int32 [n_left]: right elements matched to each left object
    counts: np.ndarray     # int64 [2]: matched right elements, left objects with a match


def join(left_prefixes, right_keys, bits, level: int) -> Join:
    """Section 3.2 (pcombine) and Section 4.2: objects produced by two parallel branches
    under the same ancestry are combined. Left: one object per level-``level`` node,
    given by its prefix (``key >> bits below level``, as the group keys of
    ``aggregate``); right: fragments with full keys of layout ``bits``. Each right
    element is paired with the left object whose prefix is its own level-``level``
    prefix, or none (-1). A prefix held by two left objects is a DUPLICATE error;
    a right key or left prefix wider than the layout is a LAYOUT error."""
    check_layout(bits)
    d = len(bits)
    if not (1 <= level <= d):
        raise OracleError(E_ARG, "join level")
    left = np.asarray(left_prefixes, dtype=U64)
    right = np.asarray(right_keys, dtype=U64)
    _check_keys_fit(right, bits)
    lbits = sum(bits[:level])
    if len(left) and int(left.max()) >> lbits:
        raise OracleError(E_LAYOUT, "left prefix wider than its levels")
    index = {}
    for i, p in enumerate(left.tolist()):
        if p in index:
            raise OracleError(E_DUPLICATE, "two left objects for one node")
        index[p] = i
    rp = prefix(right, bits, level)
    match = np.array([index.get(int(p), -1) for p in rp.tolist()], dtype=np.int32)
    hits = np.zeros(len(left), np.int32)
    for m in match.tolist():
        if m >= 0:
            hits[m] += 1
    counts = np.array([int((match >= 0).sum()), int((hits > 0).sum())], np.int64)
    return Join(match, hits, counts)


# ---------------------------------------------------------------------------
# split_text: pmap entry, one more level of ancestry
# ---------------------------------------------------------------------------

SPLIT_NONE = np.uint64(0xFFFFFFFFFFFFFFFF)


@dataclass
class Split:
    keys: np.ndarray     # uint64 [n]: keys of layout bits_in[:-1] + (seg_bits, tok_bits), or SPLIT_NONE
    fan: np.ndarray      # int32 [d][n]: declared child counts of levels 1..d of the new layout
    counts: np.ndarray   # int64 [4]: tokens placed, delimiters, tokens of incomplete parents, segments
    order: np.ndarray    # int64 [placed]: input indices of the placed tokens, by new key
    rest: np.ndarray     # int64 [incomplete]: input indices of the tokens of incomplete parents, by key


def split_text(keys, fan, tokens, bits_in, delim: int, seg_bits: int, tok_bits: int) -> Split:
    """Section 3.2 (split_text) and Section 4.2 (pmap entry pushes a level). The
    fragments are tokens: leaves of layout ``bits_in`` whose parent (level d-1) is one
    stream element, e.g. one language-model output, and whose leaf tag is the token's
    index in that stream. Each parent's tokens are split at ``delim`` tokens into
    segments (maximal runs of other tokens; the delimiters are separators and are not
    placed, empty segments do not exist). A placed token gets the key (parent, segment
    index, index in segment) in the layout ``bits_in[:-1] + (seg_bits, tok_bits)`` and
    the declared child counts of the new levels: segments of its parent, tokens of its
    segment (the counts of the levels above are copied). A parent is split only when
    all of its declared tokens are present (the segment boundaries depend on every
    token); its tokens are otherwise left unplaced (SPLIT_NONE), like delimiters.
    The new fragments leave the entry as a batch in new-key order (``order``); the
    tokens of incomplete parents are listed in key order (``rest``), to be offered
    again with the rest of their stream.
    Errors, by priority: LAYOUT (a key wider than bits_in), FANOUT (a declared count
    < 1, a token index >= it, carriers of one parent disagreeing), DUPLICATE (a token
    key twice), CAPACITY (a segment index or an index in a segment that does not fit
    its bits)."""
    bits_in = tuple(bits_in)
    check_layout(bits_in)
    d = len(bits_in)
    if d < 2 or seg_bits < 1 or tok_bits < 1 or seg_bits > 32 or tok_bits > 32:
        raise OracleError(E_ARG, "split layout")
    bits_out = bits_in[:-1] + (seg_bits, tok_bits)
    check_layout(bits_out)
    keys = np.asarray(keys, dtype=U64)
    fan = np.asarray(fan).astype(np.int64).reshape(d - 1, len(keys))
    tokens = np.asarray(tokens).astype(np.int64)
    n = len(keys)
    _check_keys_fit(keys, bits_in)
    par = prefix(keys, bits_in, d - 1)
    idx = tag(keys, bits_in, d)
    pfan = fan[d - 2]
    if n and (pfan.min() < 1 or (idx >= pfan).any()):
        raise OracleError(E_FANOUT, "token index outside its parent's declared count")
    declared = {}
    for p, f in zip(par.tolist(), pfan.tolist()):
        if declared.setdefault(p, f) != f:
            raise OracleError(E_FANOUT, "carriers of one parent disagree")
    if len(np.unique(keys)) != n:
        raise OracleError(E_DUPLICATE, "same token twice")
    out_keys = np.full(n, SPLIT_NONE, dtype=U64)
    out_fan = np.zeros((d, n), np.int32)
    placed = delims = incomplete = segments = 0
    rest = []
    rows = {}
    for i, p in enumerate(par.tolist()):
        rows.setdefault(p, []).append(i)
    for p, members in rows.items():
        if len(members) != declared[p]:
            incomplete += len(members)
            rest.extend(members)
            continue
        members.sort(key=lambda i: int(idx[i]))
        segs, cur = [], []
        for i in members:
            if tokens[i] == delim:
                delims += 1
                if cur:
                    segs.append(cur)
                cur = []
            else:
                cur.append(i)
        if cur:
            segs.append(cur)
        segments += len(segs)
        for c, seg in enumerate(segs):
            for t, i in enumerate(seg):
                if c >= (1 << seg_bits) or t >= (1 << tok_bits):
                    raise OracleError(E_CAPACITY, "segment or index does not fit its bits")
                out_keys[i] = (U64(p) << U64(seg_bits + tok_bits)) | (U64(c) << U64(tok_bits)) | U64(t)
                out_fan[: d - 2, i] = fan[: d - 2, i]
                out_fan[d - 2, i] = len(segs)
                out_fan[d - 1, i] = len(seg)
                placed += 1
    placed_idx = np.nonzero(out_keys != SPLIT_NONE)[0]
    order = placed_idx[np.argsort(out_keys[placed_idx], kind="stable")]
    rest = np.array(sorted(rest, key=lambda i: int(keys[i])), dtype=np.int64)
    return Split(out_keys, out_fan, np.array([placed, delims, incomplete, segments], np.int64),
                 order.astype(np.int64), rest)


# ---------------------------------------------------------------------------
# load-aware routing (Section 4.3: a new flow of tags may go where the load is
# lowest instead of where a hash sends it; Section 5: replicas chosen by queue length)
# ---------------------------------------------------------------------------

@dataclass
class LoadRoute:
    perm: np.ndarray          # int32 [n], input indices in (dest, key) order
    dest_offsets: np.ndarray  # int64 [D+1]
    dest: np.ndarray          # int32 [n], input order
    load: np.ndarray          # int64 [D], queue lengths after the batch
    counts: np.ndarray        # int64 [2]: new flows assigned, flows seen before


class LoadRouter:
    """Sticky least-loaded routing of flows (distinct level-``route_level`` prefixes).

    A flow keeps the destination it was first given, so all fragments with the same
    tags reach the same instance (Section 4.3). Per batch: the fragments of flows
    seen before join their destination's queue first; then the new flows, in
    ascending prefix order, each go to the destination with the shortest queue
    (ties: the lowest index), whose queue then grows by the flow's fragments in the
    batch. Queue lengths are the caller's (``load``): routing adds every fragment it
    sends, the caller subtracts what a destination has consumed. At most
    ``max_flows`` flows are remembered; a batch whose new flows do not fit raises
    CAPACITY and changes nothing."""

    def __init__(self, bits, route_level: int, num_dest: int, max_flows: int):
        check_layout(bits)
        if not (1 <= route_level <= len(bits)) or num_dest < 1 or max_flows < 1:
            raise OracleError(E_ARG, "load router")
        self.bits, self.Lr, self.D, self.max_flows = tuple(bits), route_level, num_dest, max_flows
        self.table: Dict[int, int] = {}

    def route(self, keys, load, with_perm: bool = True) -> LoadRoute:
        """``with_perm=False`` leaves perm empty (large batches in tests)."""
        keys = np.asarray(keys, dtype=U64)
        load = np.array(load, dtype=np.int64).copy()
        if load.shape != (self.D,) or (load < 0).any():
            raise OracleError(E_ARG, "load")
        n = len(keys)
        _check_keys_fit(keys, self.bits)
        if len(np.unique(keys)) != n:
            raise OracleError(E_DUPLICATE, "same key twice")
        flows, inverse, sizes = np.unique(prefix(keys, self.bits, self.Lr), return_inverse=True,
                                          return_counts=True)
        flows, sizes = flows.tolist(), sizes.tolist()           # ascending prefix order
        new = [k for k, f in enumerate(flows) if f not in self.table]
        if len(self.table) + len(new) > self.max_flows:
            raise OracleError(E_CAPACITY, "flow table full")
        known = 0
        for f, c in zip(flows, sizes):
            if f in self.table:
                load[self.table[f]] += c
                known += 1
        for k in new:
            d = int(np.argmin(load))          # first minimum: the lowest index among ties
            self.table[flows[k]] = d
            load[d] += sizes[k]
        dest = np.array([self.table[f] for f in flows], dtype=np.int32)[inverse].astype(np.int32)
        perm = np.lexsort((keys, dest)).astype(np.int32) if with_perm else np.zeros(0, np.int32)
        offs = np.concatenate([[0], np.cumsum(np.bincount(dest, minlength=self.D))]).astype(np.int64)
        return LoadRoute(perm, offs, dest, load, np.array([len(new), known], np.int64))
