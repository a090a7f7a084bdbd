"""Declared child counts that disagree among a node's carriers, at the levels the
GPU checks with the keyed additive fingerprint rather than exactly per flow: the
levels below the route level in the 5-level FacTool layout (31,3,2,3,8), and
the leaves' parent level in the 6-level Zipf layout (3,12,12,12,12,12), through
the multi-workgroup sort (general and direct-placement paths). Each planting is
checked by the oracle (exact: FANOUT) and run twice on the GPU; every call draws
its own fingerprint key, so both must report FANOUT.

Plantings: one carrier one above the others; one carrier one below (still above
its own child tag); a power of two of carriers of one node (a multiplicity that a
modular sum could cancel); two nodes whose carriers swap each other's counts."""
import numpy as np
import pytest

from oracle import alto_oracle as O
from paper_2403_04311_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

FACTOOL = (31, 3, 2, 3, 8)
ZIPF = (3, 12, 12, 12, 12, 12)


def _nodes(keys, bits, level):
    """Level-`level` node of every fragment, and the fragments of each node."""
    pre = O.prefix(keys, bits, level)
    uniq, inv, counts = np.unique(pre, return_inverse=True, return_counts=True)
    return inv, counts


def _plant(keys, fan, bits, level, kind, rng):
    """A copy of fan with one disagreement at `level` (row level - 1)."""
    fan = fan.copy()
    row = level - 1
    inv, counts = _nodes(keys, bits, level)
    child = O.tag(keys, bits, level + 1).astype(np.int64)
    declared = fan[row].astype(np.int64)
    if kind == "up":
        u = rng.choice(np.nonzero(counts >= 2)[0])
        c = rng.choice(np.nonzero(inv == u)[0])
        fan[row, c] += 1
    elif kind == "down":
        # a carrier whose own child tag stays below the lowered count
        ok = (declared >= 3) & (child <= declared - 2)
        cand = np.nonzero(ok & (counts[inv] >= 2))[0]
        c = rng.choice(cand)
        fan[row, c] -= 1
    elif kind == "pow2":
        u = rng.choice(np.nonzero(counts >= 8)[0])
        cs = rng.choice(np.nonzero(inv == u)[0], size=4, replace=False)
        fan[row, cs] += 1
    elif kind == "swap":
        many = np.nonzero(counts >= 2)[0]
        for _ in range(1000):
            a, b = rng.choice(many, size=2, replace=False)
            ca, cb = np.nonzero(inv == a)[0], np.nonzero(inv == b)[0]
            fa, fb = int(declared[ca[0]]), int(declared[cb[0]])
            if fa == fb:
                continue
            lo = min(fa, fb)
            xa, xb = ca[child[ca] < lo], cb[child[cb] < lo]
            if len(xa) and len(xb):
                fan[row, xa[0]] = fb
                fan[row, xb[0]] = fa
                break
        else:
            raise AssertionError("no pair of nodes to swap")
    else:
        raise ValueError(kind)
    return fan


def _check(keys, fan, bits, La, Lm, Lr, D, level, kinds, seed):
    rng = np.random.default_rng(seed)
    p32 = rng.integers(0, 1 << 30, size=len(keys)).astype(np.int32)
    for kind in kinds:
        bad = _plant(keys, fan, bits, level, kind, rng)
        code, _, _ = U.oracle_aggregate(keys, bad, bits, La, "concat", 1, Lm, Lr, D, p32)
        assert code == O.E_FANOUT, kind
        for rep in range(2):
            res = U.run_aggregate(keys, bad, bits, La, "concat", 1, Lm, Lr, D, p32)
            assert res["status"] == O.E_FANOUT, (kind, rep, res["status"])
    # the unplanted batch is clean
    code, _, _ = U.oracle_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    res = U.run_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert res["status"] == code


KINDS = ["up", "down", "pow2", "swap"]


@pytest.mark.parametrize("La,level", [(4, 4), (3, 3), (3, 4)])
def test_fanout_factool_layout_fingerprinted_levels(La, level):
    # counts are checked from the aggregation level down; route level 2
    path, fan = W.random_tree(700 + level, 5, 40, (8, 4, 8, 60), FACTOOL)
    (path, fan), _ = W.permute([path, fan], 710 + level)
    keys = O.pack_keys(path, FACTOOL)
    assert len(keys) > 8192   # the multi-workgroup sort with its flow set
    _check(keys, fan, FACTOOL, La, 0, 2, 32, level, KINDS, 720 + level)


@pytest.mark.parametrize("drop", [0.0, 0.01])
def test_fanout_zipf_layout_leaf_parent_level(drop):
    # one root, one level-2 and one level-3 node (the 2^26-fragment shape): complete
    # batches take direct placement, a batch with dropped leaves the general path
    path, fan = W.random_tree(730, 6, 1, (1, 1, 150, 30, 40), ZIPF, dense_roots=True)
    if drop:
        path, fan, _ = W.drop_leaves(path, fan, drop, 731)
    (path, fan), _ = W.permute([path, fan], 732)
    keys = O.pack_keys(path, ZIPF)
    assert len(keys) > 8192
    _check(keys, fan, ZIPF, 4, 2, 4, 256, 5, KINDS, 733)
