"""Pins of the CPU oracle against things other than itself: published hash outputs,
closed forms, textbook routines and a brute-force model on tiny trees."""
import functools
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import alto_oracle as O
from paper_2403_04311_amd import workloads as W
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- hash

def test_mix64_matches_published_splitmix64_outputs():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "splitmix64_seed0.txt"))
            if l.strip() and not l.startswith("#")]
    states = np.array([int(r[1], 16) for r in rows], dtype=np.uint64)
    want = [int(r[2], 16) for r in rows]
    got = [int(v) for v in O.mix64(states)]
    assert got == want


def test_dest_power_of_two_is_top_bits_of_hash():
    rng = np.random.default_rng(0)
    p = rng.integers(0, 2**62, size=10000, dtype=np.int64).astype(np.uint64)
    h = O.mix64(p)
    for k in range(0, 12):
        d = O.dest_of(p, 1 << k)
        if k == 0:
            assert (d == 0).all()
        else:
            assert np.array_equal(d.astype(np.uint64), h >> np.uint64(64 - k))


@pytest.mark.parametrize("D", [3, 7, 64, 256, 1000])
def test_dest_range_and_balance(D):
    p = np.arange(200000, dtype=np.uint64)
    d = O.dest_of(p, D)
    assert d.min() >= 0 and d.max() < D
    c = np.bincount(d, minlength=D)
    exp = len(p) / D
    chi2 = ((c - exp) ** 2 / exp).sum()
    assert chi2 < D + 6 * np.sqrt(2 * D)   # loose: a biased reduction fails by far


def test_dest_lemire_bound_small_cases():
    # Lemire's reduction maps the 32-bit hash x to floor(x * D / 2^32): check against
    # exact rational arithmetic.
    rng = np.random.default_rng(1)
    p = rng.integers(0, 2**40, size=500).astype(np.uint64)
    x = [int(v) >> 32 for v in O.mix64(p)]
    for D in (5, 12, 255):
        got = O.dest_of(p, D)
        want = [int(Fraction(xi * D, 2**32)) for xi in x]
        assert list(got) == want


# ---------------------------------------------------------------- keys

def test_pack_literal():
    keys = O.pack_keys(np.array([[1, 0], [5, 7]]), (2, 3))
    assert list(keys) == [0b01101, 0b00111]


def test_pack_preserves_lexicographic_path_order():
    path, fan = W.random_tree(3, 4, 12, (3, 4, 5), (31, 2, 3, 3))
    [path], _ = W.permute([path], 4)
    keys = O.pack_keys(path, (31, 2, 3, 3))
    tuples = brute.leaves_of(path)
    assert list(np.argsort(keys, kind="stable")) == sorted(range(len(tuples)), key=lambda i: tuples[i])
    for level in range(1, 5):
        assert list(O.tag(keys, (31, 2, 3, 3), level)) == [t[level - 1] for t in tuples]


def test_pack_rejects_tags_that_do_not_fit():
    with pytest.raises(O.OracleError) as e:
        O.pack_keys(np.array([[0], [8]]), (2, 3))
    assert e.value.code == O.E_LAYOUT
    with pytest.raises(O.OracleError) as e:
        O.pack_keys(np.array([[-1], [0]]), (2, 3))
    assert e.value.code == O.E_LAYOUT
    with pytest.raises(O.OracleError) as e:
        O.pack_keys(np.array([[0], [0]]), (40, 24))
    assert e.value.code == O.E_ARG


# ---------------------------------------------------------------- route

@pytest.mark.parametrize("D,Lr", [(1, 1), (3, 1), (8, 2), (256, 3), (5, 4)])
def test_route_matches_brute_force_sort(D, Lr):
    bits = (31, 2, 3, 4)
    path, fan = W.random_tree(10 + D, 4, 20, (4, 8, 16), bits)
    [path], _ = W.permute([path], D)
    keys = O.pack_keys(path, bits)
    r = O.route(keys, bits, Lr, D)
    tuples = brute.leaves_of(path)

    @functools.lru_cache(maxsize=None)
    def dfn(t):
        v = 0
        for level, tg in enumerate(t):
            v = (v << bits[level]) | tg
        return int(O.dest_of(np.array([v], np.uint64), D)[0])

    want = sorted(range(len(tuples)), key=lambda i: (dfn(tuples[i][:Lr]), tuples[i]))
    assert list(r.perm) == want
    assert list(r.dest) == [dfn(t[:Lr]) for t in tuples]
    assert list(r.dest_offsets) == [0] + list(np.cumsum([sum(1 for t in tuples if dfn(t[:Lr]) == d)
                                                         for d in range(D)]))


def test_route_invariants_and_duplicate():
    keys = np.array([5, 9, 1, 7], dtype=np.uint64)
    r = O.route(keys, (4, 4), 2, 3)
    assert sorted(r.perm) == [0, 1, 2, 3]
    with pytest.raises(O.OracleError) as e:
        O.route(np.array([5, 9, 5], np.uint64), (4, 4), 2, 3)
    assert e.value.code == O.E_DUPLICATE
    with pytest.raises(O.OracleError) as e:
        O.route(np.array([5, 300], np.uint64), (4, 4), 2, 3)
    assert e.value.code == O.E_LAYOUT


# ---------------------------------------------------------------- aggregate vs brute force

def _dest_fn(bits, D):
    def f(prefix_tuple):
        v = 0
        for level, tg in enumerate(prefix_tuple):
            v = (v << bits[level]) | tg
        return int(O.dest_of(np.array([v], np.uint64), D)[0])
    return f


def _tuple_of(k, bits, level):
    """Tag tuple of a level-``level`` prefix value (inverse of _key_of)."""
    out = []
    for l in range(level, 0, -1):
        out.append(k & ((1 << bits[l - 1]) - 1))
        k >>= bits[l - 1]
    return tuple(reversed(out))


def _key_of(t, bits):
    v = 0
    for level, tg in enumerate(t):
        v = (v << bits[level]) | tg
    return v


CASES = [
    # depth, bits, max_fan per level, La, Lm, Lr, D, drop
    (2, (8, 4), (5,), 1, 0, 1, 3, 0.0),
    (3, (10, 3, 3), (4, 5), 2, 1, 1, 4, 0.2),
    (4, (31, 2, 3, 4), (4, 8, 16), 3, 0, 1, 8, 0.0),
    (4, (31, 2, 3, 4), (3, 3, 3), 2, 3, 2, 5, 0.15),
    (5, (6, 3, 2, 3, 5), (3, 3, 3, 6), 4, 2, 4, 16, 0.1),
    (5, (6, 3, 2, 3, 5), (3, 2, 3, 4), 3, 1, 2, 7, 0.05),
    (4, (5, 3, 3, 3), (3, 3, 4), 1, 2, 0, 1, 0.1),
    (6, (3, 3, 3, 3, 3, 4), (2, 3, 2, 3, 5), 4, 2, 4, 256, 0.08),
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("op", ["concat", "mean"])
def test_aggregate_matches_brute_force(case, op):
    depth, bits, mf, La, Lm, Lr, D, drop = CASES[case]
    for rep in range(3):
        seed = 1000 * case + rep
        path, fan = W.random_tree(seed, depth, 3 + rep, mf, bits)
        true_leaves = brute.leaves_of(path)
        if drop:
            path, fan, _ = W.drop_leaves(path, fan, drop, seed + 1)
        rng = np.random.default_rng(seed + 2)
        n = path.shape[1]
        p32 = rng.integers(-1000, 1000, size=n).astype(np.int32)
        pf = (rng.integers(-64, 64, size=(n, 3)) / 16.0).astype(np.float32)   # dyadic: exact
        (path, fan, p32, pf_t), _ = W.permute([path, fan, p32, pf.T], seed + 3)
        pf = np.ascontiguousarray(pf_t.T)
        keys = O.pack_keys(path, bits)
        rt, g = O.aggregate(keys, fan, bits, La, op, 3, Lm, Lr, D, p32, pf if op == "mean" else None)
        arrived = brute.leaves_of(path)
        exp = brute.batch_expect(true_leaves, arrived, p32, pf if op == "mean" else None, La, Lm,
                                 _dest_fn(bits, D), Lr)
        assert list(rt.perm) == exp["perm"]
        em = exp["emitted"]
        assert [int(k) for k in g.key] == [_key_of(r["key"], bits) for r in em]
        assert list(g.dest) == [r["dest"] for r in em]
        assert list(g.count) == [r["count"] for r in em]
        assert list(g.first_i32) == [r["first"] for r in em]
        tf = brute.true_fans(path, fan)
        for level in range(1, La):
            assert list(g.fan_up[level - 1]) == [tf[r["key"][:level]] for r in em]
        assert [int(k) for k in g.pend_key] == [_key_of(r["key"], bits) for r in exp["pending"]]
        assert list(g.pend_count) == [r["count"] for r in exp["pending"]]
        if op == "concat":
            assert list(g.tok) == [t for r in em for t in r["tok"]]
            assert list(g.tok_off) == [0] + list(np.cumsum([r["count"] for r in em]))
        else:
            want = np.array([[float(v) for v in r["mean"]] for r in em], np.float64).reshape(-1, 3)
            assert np.array_equal(g.mean, want.astype(np.float32))
        if Lm:
            assert [int(k) for k in g.mask_key] == [_key_of(m, bits) for m, _ in exp["mask"]]
            assert list(g.mask) == [int(c) for _, c in exp["mask"]]


def test_single_batch_concat_reproduces_depth_first_payload_order():
    # Closed form: with every leaf present, all groups are complete, and the groups'
    # token lists in key order concatenate to the pre-shuffle (depth-first) payloads.
    bits = (31, 2, 3, 4)
    path, fan = W.random_tree(77, 4, 40, (4, 8, 16), bits, dense_roots=True)
    dfs_tok = np.arange(path.shape[1], dtype=np.int32) * 3 + 1
    (sp, sf, st), _ = W.permute([path, fan, dfs_tok], 78)
    keys = O.pack_keys(sp, bits)
    _, g = O.aggregate(keys, sf, bits, 3, "concat", 1, 0, 1, 8, st)
    assert len(g.pend_key) == 0
    o = np.argsort(g.key)
    toks = np.concatenate([g.tok[g.tok_off[i]:g.tok_off[i + 1]] for i in o])
    assert np.array_equal(toks, dfs_tok)


def test_mean_is_textbook_group_mean():
    bits = (31, 3, 2, 3, 8)
    path, fan = W.random_tree(5, 5, 6, (8, 3, 5, 20), bits)
    rng = np.random.default_rng(6)
    x = rng.standard_normal((path.shape[1], 16)).astype(np.float32)
    (sp, sf, xt), _ = W.permute([path, fan, x.T], 7)
    x = np.ascontiguousarray(xt.T)
    keys = O.pack_keys(sp, bits)
    _, g = O.aggregate(keys, sf, bits, 4, "mean", 16, 0, 2, 32, None, x)
    gk = O.prefix(keys, bits, 4)
    for i, k in enumerate(g.key):
        rows = x[gk == k].astype(np.float64)
        assert np.allclose(g.mean[i], rows.mean(axis=0).astype(np.float32), rtol=0, atol=1e-7)


def test_mean_float64_batches_match_exact_rational_means():
    # The oracle sums a group's rows in float64 batches of at most 2^24 / dim rows
    # (a group larger than that takes a batch of its own). At dim 2^20 a batch holds
    # 16 rows, so these group sizes put groups exactly at, just over and far over the
    # budget, runs of small groups that fill a batch exactly, and single rows. Rows
    # are multiples of 1/16 in [-4, 4): every float64 sum is exact, so each mean must
    # equal the exact rational mean (integer sum over 16 x count) rounded once to
    # float64 and then to float32 (the aggregate operator of Section 3.3, flat mean).
    dim = 1 << 20
    assert (1 << 24) // dim == 16
    sizes = [3, 13, 16, 17, 1, 1, 14, 35, 2, 9, 16, 15, 1]
    bits = (2, 5, 7)
    rows = []
    for g, s in enumerate(sizes):
        rows += [(0, g, c) for c in range(s)]
    path = np.array(rows, dtype=np.int64).T
    fan = np.stack([np.ones(len(rows), np.int32) * len(sizes),
                    np.array([sizes[g] for _, g, _ in rows], np.int32)])
    rng = np.random.default_rng(11)
    ints = (np.frombuffer(rng.bytes(len(rows) * dim), np.int8) >> 1).reshape(len(rows), dim)   # [-64, 64)
    (sp, sf, order), _ = W.permute([path, fan, np.arange(len(rows))], 12)
    x = ints[order].astype(np.float32)
    x *= np.float32(1.0 / 16.0)
    keys = O.pack_keys(sp, bits)
    _, g = O.aggregate(keys, sf, bits, 2, "mean", dim, payload_f32=x)
    assert [int(k) for k in g.key] == list(range(len(sizes)))
    assert list(g.count) == sizes
    start = 0
    for gi, s in enumerate(sizes):
        isum = ints[start:start + s].sum(axis=0, dtype=np.int64)       # rows in generation order
        want = (isum.astype(np.float64) / np.float64(16 * s)).astype(np.float32)
        assert np.array_equal(g.mean[gi], want), gi
        start += s


def test_arrival_permutation_invariance():
    bits = (6, 3, 2, 3, 5)
    path, fan = W.random_tree(9, 5, 4, (3, 3, 3, 6), bits)
    path, fan, _ = W.drop_leaves(path, fan, 0.1, 10)
    p32 = np.arange(path.shape[1], dtype=np.int32)
    ref = None
    for s in range(5):
        (sp, sf, st), _ = W.permute([path, fan, p32], 100 + s)
        keys = O.pack_keys(sp, bits)
        rt, g = O.aggregate(keys, sf, bits, 3, "concat", 1, 2, 2, 7, st)
        out = (list(g.key), list(g.tok), list(g.mask_key), list(g.mask), list(keys[rt.perm]))
        if ref is None:
            ref = out
        assert out == ref


# ---------------------------------------------------------------- error paths

def _small():
    bits = (4, 3, 3)
    path, fan = W.random_tree(21, 3, 3, (4, 5), bits)
    return bits, path.copy(), fan.copy()


def test_fanout_errors():
    bits, path, fan = _small()
    keys = O.pack_keys(path, bits)
    O.aggregate(keys, fan, bits, 2, "concat", payload_i32=np.zeros(len(keys), np.int32))
    f2 = fan.copy()
    f2[1, 0] += 1                                   # one carrier disagrees
    with pytest.raises(O.OracleError) as e:
        O.aggregate(keys, f2, bits, 2, "concat", payload_i32=np.zeros(len(keys), np.int32))
    assert e.value.code == O.E_FANOUT
    f3 = fan.copy()
    f3[1, :] = np.maximum(f3[1, :] - 1, 0)          # child index >= declared count
    with pytest.raises(O.OracleError) as e:
        O.aggregate(keys, f3, bits, 2, "concat", payload_i32=np.zeros(len(keys), np.int32))
    assert e.value.code == O.E_FANOUT
    # levels above the aggregation level are not read
    f4 = fan.copy()
    f4[0, 0] = -5
    O.aggregate(keys, f4, bits, 2, "concat", payload_i32=np.zeros(len(keys), np.int32))
    with pytest.raises(O.OracleError) as e:
        O.aggregate(keys, f4, bits, 2, "concat", 1, 1, payload_i32=np.zeros(len(keys), np.int32))
    assert e.value.code == O.E_FANOUT


def test_error_priority():
    bits, path, fan = _small()
    keys = O.pack_keys(path, bits)
    dup = np.concatenate([keys, keys[:1]])
    fdup = np.concatenate([fan, fan[:, :1]], axis=1)
    z = np.zeros(len(dup), np.int32)
    with pytest.raises(O.OracleError) as e:
        O.aggregate(dup, fdup, bits, 2, "concat", payload_i32=z)
    assert e.value.code == O.E_DUPLICATE
    fbad = fdup.copy()
    fbad[1, 0] += 3
    with pytest.raises(O.OracleError) as e:
        O.aggregate(dup, fbad, bits, 2, "concat", payload_i32=z)
    assert e.value.code == O.E_FANOUT
    wide = dup.copy()
    wide[1] = np.uint64(1 << 20)
    with pytest.raises(O.OracleError) as e:
        O.aggregate(wide, fbad, bits, 2, "concat", payload_i32=z)
    assert e.value.code == O.E_LAYOUT


def test_argument_errors():
    bits, path, fan = _small()
    keys = O.pack_keys(path, bits)
    z = np.zeros(len(keys), np.int32)
    for kw in [dict(agg_level=3), dict(agg_level=1, route_level=2, num_dest=4),
               dict(agg_level=2, route_level=0, num_dest=4)]:
        with pytest.raises(O.OracleError) as e:
            O.aggregate(keys, fan, bits, op="concat", payload_i32=z, **kw)
        assert e.value.code == O.E_ARG


def test_capacity_reports_needs():
    bits, path, fan = _small()
    keys = O.pack_keys(path, bits)
    z = np.zeros(len(keys), np.int32)
    _, g = O.aggregate(keys, fan, bits, 2, "concat", payload_i32=z)
    with pytest.raises(O.OracleError) as e:
        O.aggregate(keys, fan, bits, 2, "concat", payload_i32=z, cap_tokens=len(keys) - 1)
    assert e.value.code == O.E_CAPACITY and e.value.need[1] == len(keys)


def test_empty_batch():
    bits = (4, 3, 3)
    keys = np.zeros(0, np.uint64)
    rt, g = O.aggregate(keys, np.zeros((2, 0), np.int32), bits, 2, "concat", 1, 1, 1, 4,
                        np.zeros(0, np.int32))
    assert len(rt.perm) == 0 and list(rt.dest_offsets) == [0] * 5
    assert len(g.key) == 0 and len(g.tok) == 0 and list(g.tok_off) == [0] and len(g.mask) == 0


# ---------------------------------------------------------------- streams

def _run_stream(bits, Lr, D, La, op, path, fan, p32, cuts):
    s = O.Stream(bits, Lr, D, La, op, 1)
    keys = O.pack_keys(path, bits)
    out = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        r = s.step(keys[a:b], fan[:, a:b], p32[a:b], None)
        out.append(r)
    return s, out


def test_stream_brute_force_all_orders_and_cuts():
    # Every arrival order of tiny trees (sampled above 6 leaves), cut into steps at
    # random points: each group is emitted exactly once, in the step holding its
    # last leaf, with the same tokens whatever the order; nothing stays pending.
    bits = (4, 2, 2, 3)
    La, Lr, D = 2, 1, 3
    checked = 0
    for seed in range(40):
        roots = 1 + seed % 2
        path, fan = W.random_tree(300 + seed, 4, roots, (2, 2, 2), bits)
        n = path.shape[1]
        if n > 8:
            continue
        true_leaves = brute.leaves_of(path)
        p32 = np.arange(n, dtype=np.int32) + 100
        batch = brute.batch_expect(true_leaves, true_leaves, p32, None, La, 0,
                                   _dest_fn(bits, D), Lr)
        tok_of = {r["key"]: r["tok"] for r in batch["emitted"]}
        rng = np.random.default_rng(seed)
        if n <= 6:
            orders = [list(o) for o in itertools.permutations(range(n))]
        else:
            orders = [list(rng.permutation(n)) for _ in range(150)]
        for oi, order in enumerate(orders):
            ncut = 1 + oi % min(n, 4)
            cuts = [0] + sorted(rng.choice(np.arange(1, n), size=ncut - 1, replace=False).tolist()) + [n]
            sp, sf, st = path[:, order], fan[:, order], p32[order]
            s, res = _run_stream(bits, Lr, D, La, "concat", sp, sf, st, cuts)
            arrival = brute.leaves_of(sp)
            step_of = np.searchsorted(cuts, np.arange(n), side="right") - 1
            want = brute.stream_emission_steps(true_leaves, arrival, step_of, La)
            seen = {}
            for si, r in enumerate(res):
                for j, k in enumerate(r.groups.key):
                    gt = _tuple_of(int(k), bits, La)
                    assert gt not in seen            # emitted exactly once
                    seen[gt] = si
                    toks = list(r.groups.tok[r.groups.tok_off[j]:r.groups.tok_off[j + 1]])
                    assert toks == tok_of[gt]         # arrival-order invariant content
            assert seen == want
            assert len(s.pending()[0]) == 0
            checked += 1
    assert checked > 3000


def test_stream_mean_brute_force_all_orders_and_cuts():
    # The MEAN variant of the test above: carried rows must follow their leaves from
    # step to step (Section 3.1: outputs stream before the input is complete). Every
    # arrival order of tiny trees (sampled above 6 leaves), cut into steps at random
    # points: each group is emitted once, in the step of its last leaf, and its mean
    # is exactly the mean of all of its leaves' rows (dyadic rows: exact sums),
    # whatever the order and the cuts.
    bits = (4, 2, 2, 3)
    La, Lr, D, dim = 2, 1, 3, 2
    checked = 0
    for seed in range(40):
        roots = 1 + seed % 2
        path, fan = W.random_tree(300 + seed, 4, roots, (2, 2, 2), bits)
        n = path.shape[1]
        if n > 8 or n < 3:
            continue
        true_leaves = brute.leaves_of(path)
        rng = np.random.default_rng(seed + 7)
        pf = (rng.integers(-64, 64, size=(n, dim)) / 16.0).astype(np.float32)
        batch = brute.batch_expect(true_leaves, true_leaves, None, pf, La, 0, _dest_fn(bits, D), Lr)
        mean_of = {r["key"]: np.array([float(v) for v in r["mean"]], np.float64).astype(np.float32)
                   for r in batch["emitted"]}
        if n <= 6:
            orders = [list(o) for o in itertools.permutations(range(n))]
        else:
            orders = [list(rng.permutation(n)) for _ in range(150)]
        for oi, order in enumerate(orders):
            ncut = 1 + oi % min(n, 4)
            cuts = [0] + sorted(rng.choice(np.arange(1, n), size=ncut - 1, replace=False).tolist()) + [n]
            sp, sf, spf = path[:, order], fan[:, order], pf[order]
            s = O.Stream(bits, Lr, D, La, "mean", dim)
            keys = O.pack_keys(sp, bits)
            arrival = brute.leaves_of(sp)
            step_of = np.searchsorted(cuts, np.arange(n), side="right") - 1
            want = brute.stream_emission_steps(true_leaves, arrival, step_of, La)
            seen = {}
            for si, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
                r = s.step(keys[a:b], sf[:, a:b], None, spf[a:b])
                assert r.groups.mean.shape == (len(r.groups.key), dim)
                for j, k in enumerate(r.groups.key):
                    gt = _tuple_of(int(k), bits, La)
                    assert gt not in seen
                    seen[gt] = si
                    assert np.array_equal(r.groups.mean[j], mean_of[gt]), (seed, order, cuts, gt)
            assert seen == want
            assert len(s.pending()[0]) == 0 and len(s.keys) == 0 and s.pf.shape == (0, dim)
            checked += 1
    assert checked > 2000


def test_stream_late_and_duplicate():
    bits = (4, 3, 3)
    path, fan = W.random_tree(31, 3, 2, (3, 4), bits)
    keys = O.pack_keys(path, bits)
    z = np.zeros(len(keys), np.int32)
    s = O.Stream(bits, 1, 4, 2, "concat")
    s.step(keys, fan, z)
    with pytest.raises(O.OracleError) as e:
        s.step(keys[:1], fan[:, :1], z[:1])
    assert e.value.code == O.E_LATE
    with pytest.raises(O.OracleError) as e:               # poisoned
        s.step(keys[:0], fan[:, :0], z[:0])
    assert e.value.code == O.E_LATE
    # duplicate across steps of a group that is still open
    keep = O.prefix(keys, bits, 2) == O.prefix(keys[:1], bits, 2)[0]
    s = O.Stream(bits, 1, 4, 2, "concat")
    if keep.sum() >= 2:
        first = np.nonzero(keep)[0][:1]
        s.step(keys[first], fan[:, first], z[first])
        with pytest.raises(O.OracleError) as e:
            s.step(keys[first], fan[:, first], z[first])
        assert e.value.code == O.E_DUPLICATE


def test_token_stream_emission_step_closed_form():
    # Tokens of a generator arrive in order, so a sentence is emitted in the step of
    # its last token: floor(arrival index of the last token / step).
    w = W.token_stream(generators=16, sentences=8, step=256)
    path, fan, tok = w.path.numpy(), w.fan.numpy(), w.payload_i32.numpy()
    keys = O.pack_keys(path, w.bits)
    s = O.Stream(w.bits, w.route_level, w.num_dest, w.agg_level, "concat")
    got = {}
    for si, a in enumerate(range(0, w.n, w.step)):
        b = min(a + w.step, w.n)
        r = s.step(keys[a:b], fan[:, a:b], tok[a:b])
        for k in r.groups.key:
            got[int(k)] = si
    gk = O.prefix(keys, w.bits, 2)
    want = {}
    for i, k in enumerate(gk):
        want[int(k)] = i // w.step
    assert got == want
    assert len(s.pending()[0]) == 0


def test_stream_in_order_release_brute_force():
    # Children of one parent leave in child-index order: a group leaves in the step
    # where it and all of its earlier siblings are complete (brute force on tag
    # tuples and the arrival schedule), exactly once, with the same content whatever
    # the arrival order; with a leaf missing, that group and its later siblings never
    # leave and are pending, complete or not.
    bits = (4, 2, 2, 3)
    Lr, D = 1, 3
    checked = 0
    for seed in range(60):
        La = 2 + seed % 2
        path, fan = W.random_tree(500 + seed, 4, 1 + seed % 2, (2, 3, 2), bits)
        n = path.shape[1]
        if n > 9 or n < 3:
            continue
        true_leaves = brute.leaves_of(path)
        drop = seed % 3 == 0
        keep_idx = np.arange(n)
        if drop:
            keep_idx = np.delete(keep_idx, seed % n)
        p32 = np.arange(n, dtype=np.int32) + 100
        batch = brute.batch_expect(true_leaves, true_leaves, p32, None, La, 0, _dest_fn(bits, D), Lr)
        tok_of = {r["key"]: r["tok"] for r in batch["emitted"]}
        rng = np.random.default_rng(seed)
        m = len(keep_idx)
        for oi in range(60):
            order = keep_idx[rng.permutation(m)]
            ncut = 1 + oi % min(m, 4)
            cuts = [0] + sorted(rng.choice(np.arange(1, m), size=ncut - 1, replace=False).tolist()) + [m]
            sp, sf, st = path[:, order], fan[:, order], p32[order]
            s = O.Stream(bits, Lr, D, La, "concat", 1, release="in_order")
            keys = O.pack_keys(sp, bits)
            seen = {}
            for si, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
                r = s.step(keys[a:b], sf[:, a:b], st[a:b], None)
                for j, k in enumerate(r.groups.key):
                    gt = _tuple_of(int(k), bits, La)
                    assert gt not in seen
                    seen[gt] = si
                    assert list(r.groups.tok[r.groups.tok_off[j]:r.groups.tok_off[j + 1]]) == tok_of[gt]
            arrival = brute.leaves_of(sp)
            step_of = np.searchsorted(cuts, np.arange(m), side="right") - 1
            want = brute.stream_release_steps_in_order(true_leaves, arrival, step_of, La)
            assert seen == want
            pend = {_tuple_of(int(k), bits, La) for k in s.pending()[0]}
            assert pend == {t[:La] for t in arrival} - set(want)
            if drop:
                assert true_leaves[seed % n][:La] not in seen   # its group never completes
            checked += 1
    assert checked > 1500


def test_in_order_release_token_stream_matches_completion():
    # Tokens of a generator arrive in order, so its sentences also complete in order:
    # in-order release changes nothing (floor(last token's arrival index / step)).
    w = W.token_stream(generators=16, sentences=8, step=256)
    path, fan, tok = w.path.numpy(), w.fan.numpy(), w.payload_i32.numpy()
    keys = O.pack_keys(path, w.bits)
    s = O.Stream(w.bits, w.route_level, w.num_dest, w.agg_level, "concat", release="in_order")
    got = {}
    for si, a in enumerate(range(0, w.n, w.step)):
        b = min(a + w.step, w.n)
        r = s.step(keys[a:b], fan[:, a:b], tok[a:b])
        for k in r.groups.key:
            got[int(k)] = si
    gk = O.prefix(keys, w.bits, 2)
    assert got == {int(k): i // w.step for i, k in enumerate(gk)}


def test_in_order_release_argument():
    with pytest.raises(O.OracleError) as e:
        O.Stream((4, 3, 3), 1, 4, 2, "concat", release="sorted")
    assert e.value.code == O.E_ARG


# ---------------------------------------------------------------- pcombine join

def test_join_matches_tuple_brute_force():
    # Each right fragment is paired with the left object of its level-Lj ancestor
    # (tuple comparison on the tag paths, no packed keys), or with none.
    bits = (5, 3, 3, 4)
    for seed in range(30):
        path, fan = W.random_tree(700 + seed, 4, 6, (4, 5, 9), bits)
        rng = np.random.default_rng(seed)
        Lj = 1 + seed % 3
        leaves = brute.leaves_of(path)
        nodes = sorted({t[:Lj] for t in leaves})
        chosen = [nodes[i] for i in rng.permutation(len(nodes))[: max(1, int(0.7 * len(nodes)))]]
        chosen.append(tuple(list(nodes[0][:-1]) + [(1 << bits[Lj - 1]) - 1]))   # a node without fragments
        chosen = list(dict.fromkeys(chosen))
        left = np.array([_key_of(t + (0,) * (len(bits) - Lj), bits) >> O.shift_below(bits, Lj)
                         for t in chosen], dtype=np.uint64)
        sel = rng.random(len(leaves)) < 0.8
        right = O.pack_keys(path[:, sel], bits)
        rleaves = [t for t, s in zip(leaves, sel) if s]
        j = O.join(left, right, bits, Lj)
        pos = {t: i for i, t in enumerate(chosen)}
        want = [pos.get(t[:Lj], -1) for t in rleaves]
        assert j.match.tolist() == want
        assert j.hits.tolist() == [sum(1 for w in want if w == i) for i in range(len(chosen))]
        assert j.counts.tolist() == [sum(1 for w in want if w >= 0), sum(1 for i in range(len(chosen)) if i in want)]
        assert j.hits[-1] == 0 or chosen[-1] in {t[:Lj] for t in rleaves}


def test_join_errors_and_empty():
    bits = (5, 3, 3, 4)
    path, fan = W.random_tree(9, 4, 3, (3, 3, 3), bits)
    keys = O.pack_keys(path, bits)
    left = np.unique(O.prefix(keys, bits, 2))
    with pytest.raises(O.OracleError) as e:
        O.join(np.concatenate([left, left[:1]]), keys, bits, 2)
    assert e.value.code == O.E_DUPLICATE
    with pytest.raises(O.OracleError) as e:
        O.join(np.array([1 << 8], np.uint64), keys, bits, 2)          # 9 bits for 8 bits of levels 1-2
    assert e.value.code == O.E_LAYOUT
    with pytest.raises(O.OracleError) as e:
        O.join(left, np.array([1 << 15], np.uint64), bits, 2)
    assert e.value.code == O.E_LAYOUT
    j = O.join(left, keys[:0], bits, 2)
    assert len(j.match) == 0 and j.hits.tolist() == [0] * len(left) and j.counts.tolist() == [0, 0]
    j = O.join(left[:0], keys, bits, 2)
    assert (j.match == -1).all() and j.counts.tolist() == [0, 0]


# ---------------------------------------------------------------- split_text (pmap entry)

def _text_case(seed, parents, max_len, delim, p_delim, drop=0.0):
    """Parents (level 2 of a (bits 6, 8, 10) layout) each holding a token stream;
    returns keys, fan, tokens (shuffled) and the streams as Python lists."""
    rng = np.random.default_rng(seed)
    streams = {}
    for q in range(parents):
        L = int(rng.integers(1, max_len + 1))
        toks = [int(delim) if rng.random() < p_delim else int(rng.integers(0, 1000)) for _ in range(L)]
        streams[(int(rng.integers(0, 64)), q)] = toks
    rows = [(r, q, i, t, len(toks)) for (r, q), toks in streams.items() for i, t in enumerate(toks)]
    if drop:
        rows = [x for x in rows if rng.random() >= drop]
    rows = [rows[i] for i in rng.permutation(len(rows))]
    path = np.array([[x[0] for x in rows], [x[1] for x in rows], [x[2] for x in rows]], np.int32)
    fan = np.array([[1] * len(rows), [x[4] for x in rows]], np.int32)
    # level-1 declared counts must agree per node: the number of parents under each root
    roots = {}
    for (r, q) in streams:
        roots[r] = roots.get(r, 0) + 1
    fan[0] = [roots[x[0]] for x in rows]
    return path, fan, np.array([x[3] for x in rows], np.int32), streams


def test_split_text_matches_list_splitting():
    # Segments are the maximal runs of non-delimiter tokens of each complete parent,
    # in token order (plain list splitting); keys decode to (parent, segment, index)
    # and carry the new declared counts.
    bits = (6, 8, 10)
    for seed in range(40):
        delim = 7
        path, fan, tok, streams = _text_case(900 + seed, 12, 40, delim, 0.2, drop=0.05 if seed % 4 == 0 else 0.0)
        keys = O.pack_keys(path, bits)
        sp = O.split_text(keys, fan, tok, bits, delim, 6, 8)
        present = {}
        for i in range(len(keys)):
            present.setdefault((int(path[0, i]), int(path[1, i])), set()).add(int(path[2, i]))
        want_segments = 0
        for i in range(len(keys)):
            par = (int(path[0, i]), int(path[1, i]))
            toks = streams[par]
            complete = len(present[par]) == len(toks)
            segs, cur = [], []
            for j, t in enumerate(toks):
                if t == delim:
                    if cur:
                        segs.append(cur)
                    cur = []
                else:
                    cur.append(j)
            if cur:
                segs.append(cur)
            where = {j: (c, k) for c, sg in enumerate(segs) for k, j in enumerate(sg)}
            j = int(path[2, i])
            if not complete or j not in where:
                assert sp.keys[i] == O.SPLIT_NONE
                assert (sp.fan[:, i] == 0).all()
                continue
            c, k = where[j]
            assert _tuple_of(int(sp.keys[i]), (6, 8, 6, 8), 4) == par + (c, k)
            assert sp.fan[:, i].tolist() == [int(fan[0, i]), len(segs), len(segs[c])]
        for par, toks in streams.items():
            if par in present and len(present[par]) == len(toks):
                want_segments += sum(1 for x in "".join("d" if t == delim else "x" for t in toks).split("d") if x)
        n_inc = sum(len(v) for p, v in present.items() if len(v) != len(streams[p]))
        n_del = sum(1 for i in range(len(keys)) if tok[i] == delim
                    and len(present[(int(path[0, i]), int(path[1, i]))]) == len(streams[(int(path[0, i]), int(path[1, i]))]))
        assert sp.counts.tolist() == [int((sp.keys != O.SPLIT_NONE).sum()), n_del, n_inc, want_segments]
        # the batch leaves in (parent, segment, index) order; the rest in (parent, position) order
        tup = {}
        for i in range(len(keys)):
            par = (int(path[0, i]), int(path[1, i]))
            if sp.keys[i] != O.SPLIT_NONE:
                tup[i] = _tuple_of(int(sp.keys[i]), (6, 8, 6, 8), 4)
        assert sp.order.tolist() == sorted(tup, key=lambda i: tup[i])
        inc = [i for i in range(len(keys)) if len(present[(int(path[0, i]), int(path[1, i]))])
               != len(streams[(int(path[0, i]), int(path[1, i]))])]
        assert sp.rest.tolist() == sorted(inc, key=lambda i: (int(path[0, i]), int(path[1, i]), int(path[2, i])))


def test_split_text_round_trip_through_concat():
    # Concatenating the split tokens per segment (level 3 of the new layout) gives the
    # segments of each parent's stream, in order.
    bits = (6, 8, 10)
    path, fan, tok, streams = _text_case(77, 20, 60, 3, 0.15)
    keys = O.pack_keys(path, bits)
    sp = O.split_text(keys, fan, tok, bits, 3, 6, 8)
    keep = sp.keys != O.SPLIT_NONE
    rt, g = O.aggregate(sp.keys[keep], sp.fan[:, keep], (6, 8, 6, 8), 3, "concat", 1, 0, 0, 1, tok[keep])
    assert len(g.pend_key) == 0
    got = {}
    for j, k in enumerate(g.key):
        par = _tuple_of(int(k), (6, 8, 6, 8), 3)[:2]
        got.setdefault(par, []).append(list(g.tok[g.tok_off[j]:g.tok_off[j + 1]]))
    for par, toks in streams.items():
        segs, cur = [], []
        for t in toks:
            if t == 3:
                if cur:
                    segs.append(cur)
                cur = []
            else:
                cur.append(t)
        if cur:
            segs.append(cur)
        assert got.get(par, []) == segs


def test_split_text_errors():
    bits = (6, 8, 10)
    path, fan, tok, _ = _text_case(5, 6, 30, 9, 0.1)
    keys = O.pack_keys(path, bits)
    for kind, code in [("dup", O.E_DUPLICATE), ("fan", O.E_FANOUT), ("idx", O.E_FANOUT), ("layout", O.E_LAYOUT),
                       ("capacity", O.E_CAPACITY)]:
        k, f, t = keys.copy(), fan.copy(), tok.copy()
        sb, tb = 6, 8
        if kind == "dup":
            k, f, t = np.concatenate([k, k[:1]]), np.concatenate([f, f[:, :1]], axis=1), np.concatenate([t, t[:1]])
        elif kind == "fan":
            f[1, 0] += 1
        elif kind == "idx":
            f[1] = np.where(O.prefix(k, bits, 2) == O.prefix(k[:1], bits, 2)[0], 1, f[1])
        elif kind == "layout":
            k[0] = np.uint64(1 << 24)
        else:
            tb = 1                                            # segments longer than 2 tokens
        with pytest.raises(O.OracleError) as e:
            O.split_text(k, f, t, bits, 9, sb, tb)
        assert e.value.code == code, kind


# ---------------------------------------------------------------- load-aware routing

def _keys2(pairs):
    """Keys of layout (4, 4) from (flow, leaf) pairs."""
    return np.array([(f << 4) | c for f, c in pairs], dtype=np.uint64)


def test_load_router_worked_example():
    # Two destinations, flows at level 1. Batch 1 from empty queues: flow 1 (two
    # fragments) takes destination 0, flow 3 the then shorter queue 1. Batch 2, the
    # caller reports queues [5, 0]: flow 3 is known, its 7 fragments join queue 1
    # (-> [5, 7]); new flow 2 (3 fragments) takes queue 0 (-> [8, 7]); new flow 4 takes
    # queue 1 (-> [8, 8]).
    r = O.LoadRouter((4, 4), 1, 2, 16)
    a = r.route(_keys2([(3, 0), (1, 0), (1, 1)]), [0, 0])
    assert a.dest.tolist() == [1, 0, 0] and a.load.tolist() == [2, 1] and a.counts.tolist() == [2, 0]
    assert a.perm.tolist() == [1, 2, 0] and a.dest_offsets.tolist() == [0, 2, 3]
    b = r.route(_keys2([(4, 0)] + [(3, c) for c in range(1, 8)] + [(2, 0), (2, 1), (2, 2)]), [5, 0])
    assert b.dest.tolist() == [1] + [1] * 7 + [0, 0, 0]
    assert b.load.tolist() == [8, 8] and b.counts.tolist() == [2, 1]
    assert b.perm.tolist() == [8, 9, 10] + list(range(1, 8)) + [0]


def test_load_router_equal_flows_go_round_robin():
    # F new flows of m fragments each on D empty queues: flow k (prefix order) lands
    # on queue k mod D; queues end at m * ceil or floor of F / D.
    for D, F, m in [(4, 10, 3), (7, 7, 1), (3, 20, 5), (16, 5, 2)]:
        r = O.LoadRouter((8, 4), 1, D, 64)
        rng = np.random.default_rng(D * 100 + F)
        flows = np.sort(rng.choice(256, F, replace=False))
        keys = _keys_fl(flows, m)
        out = r.route(keys[rng.permutation(len(keys))], np.zeros(D, np.int64))
        for k, f in enumerate(flows):
            assert r.table[int(f)] == k % D
        assert out.load.tolist() == [m * (F // D + (1 if d < F % D else 0)) for d in range(D)]


def _keys_fl(flows, m):
    return np.array([(int(f) << 4) | c for f in flows for c in range(m)], dtype=np.uint64)


def test_load_router_sticky_balanced_and_ordered():
    # Over random batches: a flow's destination never changes; after the first batch
    # from empty queues the longest queue is within one flow of the mean (the bound
    # of greedy list scheduling); queue growth equals the batch size; perm is the
    # (destination, key) order.
    bits = (6, 5, 4)
    for seed in range(12):
        rng = np.random.default_rng(4000 + seed)
        D = int(rng.integers(1, 9))
        r = O.LoadRouter(bits, 2, D, 4096)
        load = np.zeros(D, np.int64)
        seen = {}
        for step in range(4):
            path, fan = W.random_tree(4100 + seed * 10 + step, 3, int(rng.integers(1, 30)), (12, 9), bits)
            keys = O.pack_keys(path, bits)
            keys = keys[rng.permutation(len(keys))]
            out = r.route(keys, load)
            flows = O.prefix(keys, bits, 2)
            sizes = {}
            for f, d in zip(flows.tolist(), out.dest.tolist()):
                assert seen.setdefault(f, d) == d
                sizes[f] = sizes.get(f, 0) + 1
            assert int(out.load.sum() - load.sum()) == len(keys)
            if step == 0:
                assert out.load.max() <= len(keys) / D + max(sizes.values())
            want = sorted(range(len(keys)), key=lambda i: (int(out.dest[i]), int(keys[i])))
            assert out.perm.tolist() == want
            assert out.dest_offsets.tolist() == [0] + np.cumsum(np.bincount(out.dest, minlength=D)).tolist()
            # a replica drains part of its queue between batches
            load = out.load - rng.integers(0, out.load + 1)


def test_load_router_errors():
    r = O.LoadRouter((4, 4), 1, 2, 2)
    with pytest.raises(O.OracleError) as e:
        r.route(_keys2([(1, 0), (1, 0)]), [0, 0])
    assert e.value.code == O.E_DUPLICATE
    with pytest.raises(O.OracleError) as e:
        r.route(np.array([1 << 9], np.uint64), [0, 0])
    assert e.value.code == O.E_LAYOUT
    r.route(_keys2([(1, 0)]), [0, 0])
    with pytest.raises(O.OracleError) as e:
        r.route(_keys2([(2, 0), (3, 0)]), [0, 0])       # two new flows, one slot left
    assert e.value.code == O.E_CAPACITY
    assert r.table == {1: 0}                             # nothing changed
    out = r.route(_keys2([(2, 0), (1, 1)]), [0, 0])
    assert out.counts.tolist() == [1, 1] and r.table == {1: 0, 2: 1}


def test_group_mean_of_one_group_matches_aggregate_and_exact_means():
    # group_mean (one group's rows at a time) against aggregate's means of the same
    # groups (pinned above against the brute-force model) and, for dyadic rows,
    # against the exact rational mean rounded once.
    bits = (31, 3, 2, 3, 8)
    path, fan = W.random_tree(15, 5, 5, (6, 3, 5, 30), bits)
    rng = np.random.default_rng(16)
    x = rng.standard_normal((path.shape[1], 24)).astype(np.float32)
    (sp, sf, xt), _ = W.permute([path, fan, x.T], 17)
    x = np.ascontiguousarray(xt.T)
    keys = O.pack_keys(sp, bits)
    _, g = O.aggregate(keys, sf, bits, 3, "mean", 24, 0, 2, 32, None, x)
    gk = O.prefix(keys, bits, 3)
    for i, k in enumerate(g.key):
        rows = x[gk == k]
        assert np.array_equal(O.group_mean(rows[::-1]), g.mean[i]) or \
            np.abs(O.group_mean(rows[::-1]) - g.mean[i]).max() <= 1e-6 * np.abs(g.mean[i]).max()
    ints = rng.integers(-64, 64, size=(37, 5))
    want = np.array([float(Fraction(int(c), 16 * 37)) for c in ints.sum(axis=0)]).astype(np.float32)
    assert np.array_equal(O.group_mean((ints / 16.0).astype(np.float32)), want)
    with pytest.raises(O.OracleError):
        O.group_mean(np.zeros((0, 3), np.float32))
