"""Brute-force semantic model for tiny trees (test helper, pure Python).

It works on tag tuples and on the true tree the generator drew, so it defines
completion independently of the oracle's count cascade: a node is complete when
every leaf the true tree has under it has arrived (Section 3.1: a stream's extent
is known only at its end; pmap exit aggregates what its call produced).
Orders come from Python tuple comparison, never from packed keys.
"""
from fractions import Fraction


def leaves_of(path):
    """Tag tuples of the fragments, in array order."""
    d, n = len(path), len(path[0])
    return [tuple(int(path[l][i]) for l in range(d)) for i in range(n)]


def true_fans(path, fan):
    """node tuple -> declared child count, from a complete (undropped) tree."""
    d = len(path)
    out = {}
    for i in range(len(path[0])):
        t = tuple(int(path[l][i]) for l in range(d))
        for level in range(1, d):
            out[t[:level]] = int(fan[level - 1][i])
    return out


def complete_nodes(true_leaves, arrived, level):
    """Level-``level`` node tuples that have arrived leaves, with completeness:
    complete iff all true leaves below it have arrived."""
    arrived = set(arrived)
    present = {t[:level] for t in arrived}
    below = {}
    for t in true_leaves:
        below.setdefault(t[:level], []).append(t)
    return {p: all(t in arrived for t in below[p]) for p in present}


def batch_expect(true_leaves, arrived_leaves, payload_i32, payload_f32, agg_level, mask_level,
                 dest_fn, route_level):
    """Expected outputs of a single batch.

    ``arrived_leaves[i]`` is the tag tuple of input fragment i; payload arrays are in
    input order. ``dest_fn(prefix_tuple)`` maps a route-level prefix to a destination.
    """
    idx = {t: i for i, t in enumerate(arrived_leaves)}
    comp = complete_nodes(true_leaves, arrived_leaves, agg_level)

    def gdest(g):
        return dest_fn(g[:route_level]) if route_level else 0

    groups = sorted(comp, key=lambda g: (gdest(g), g))
    emitted, pending = [], []
    for g in groups:
        members = sorted(t for t in arrived_leaves if t[:agg_level] == g)
        rec = {"key": g, "dest": gdest(g), "count": len(members),
               "members": [idx[t] for t in members]}
        if payload_i32 is not None:
            rec["tok"] = [int(payload_i32[idx[t]]) for t in members]
            rec["first"] = int(payload_i32[idx[members[0]]])
        if payload_f32 is not None:
            dim = len(payload_f32[0])
            rec["mean"] = [sum((Fraction(float(payload_f32[idx[t]][c])) for t in members),
                               Fraction(0)) / len(members) for c in range(dim)]
        (emitted if comp[g] else pending).append(rec)
    mask = None
    if mask_level:
        mc = complete_nodes(true_leaves, arrived_leaves, mask_level)
        if mask_level >= route_level:
            mk = sorted(mc, key=lambda m: (dest_fn(m[:route_level]) if route_level else 0, m))
        else:
            mk = sorted(mc)
        mask = [(m, mc[m]) for m in mk]
    perm = sorted(range(len(arrived_leaves)),
                  key=lambda i: (dest_fn(arrived_leaves[i][:route_level]) if route_level else 0,
                                 arrived_leaves[i]))
    return {"emitted": emitted, "pending": pending, "mask": mask, "perm": perm}


def stream_emission_steps(true_leaves, arrival, step_of_arrival, agg_level):
    """Group tuple -> step in which it completes (its last true leaf arrives), for the
    groups whose leaves all arrive; other groups are absent."""
    last = {}
    arrived_set = set(arrival)
    for t, s in zip(arrival, step_of_arrival):
        g = t[:agg_level]
        last[g] = max(last.get(g, -1), s)
    out = {}
    for g, s in last.items():
        if all(t in arrived_set for t in true_leaves if t[:agg_level] == g):
            out[g] = s
    return out


def stream_release_steps_in_order(true_leaves, arrival, step_of_arrival, agg_level):
    """Group tuple -> step in which it leaves when each parent's children leave in
    child-index order: the latest completion step among children 0..c of its parent,
    if all of them complete; absent otherwise. With no parent level, completion."""
    comp = stream_emission_steps(true_leaves, arrival, step_of_arrival, agg_level)
    if agg_level < 2:
        return comp
    out = {}
    for g in {t[:agg_level] for t in true_leaves}:
        sibs = [g[:-1] + (k,) for k in range(g[-1] + 1)]
        if all(s in comp for s in sibs):
            out[g] = max(comp[s] for s in sibs)
    return out
