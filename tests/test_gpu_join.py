"""GPU parity of alto_join (pcombine by ancestry) against the oracle, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def run_join(left, right, bits, level):
    dl = U.to_dev(left.astype(np.uint64).view(np.int64)) if len(left) else torch.empty(1, dtype=torch.int64,
                                                                                        device="cuda")
    dr = U.to_dev(right.astype(np.uint64).view(np.int64)) if len(right) else torch.empty(1, dtype=torch.int64,
                                                                                          device="cuda")
    m, h, c, st = alto.join(dl, dr, bits, level, n_left=len(left), n_right=len(right))
    torch.cuda.synchronize()
    return (int(st.item()), m[:len(right)].cpu().numpy(), h[:len(left)].cpu().numpy(), c.cpu().numpy())


def _case(seed, bits, mf, roots, Lj, frac_left=0.7, frac_right=0.8, extra_left=0):
    depth = len(bits)
    path, fan = W.random_tree(seed, depth, roots, mf, bits)
    keys = O.pack_keys(path, bits)
    rng = np.random.default_rng(seed)
    nodes = np.unique(O.prefix(keys, bits, Lj))
    left = nodes[rng.permutation(len(nodes))[: max(1, int(frac_left * len(nodes)))]]
    if extra_left:   # objects of nodes that have no fragment
        top = np.uint64((1 << sum(bits[:Lj])) - 1)
        left = np.concatenate([left, top - np.arange(extra_left, dtype=np.uint64)])
        left = np.unique(left)[rng.permutation(len(np.unique(left)))]
    right = keys[rng.random(len(keys)) < frac_right]
    right = right[rng.permutation(len(right))]
    return left, right


CASES = [
    # bits, max_fan, roots, level
    ((5, 3, 3, 4), (4, 5, 9), 6, 1),
    ((5, 3, 3, 4), (4, 5, 9), 6, 2),
    ((5, 3, 3, 4), (4, 5, 9), 6, 4),
    ((31, 3, 2, 3, 8), (4, 3, 5, 40), 300, 3),      # more left objects than one workgroup sorts
    ((20, 12, 12), (2000, 40), 8, 2),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_join_parity(case):
    bits, mf, roots, Lj = CASES[case]
    left, right = _case(800 + case, bits, mf, roots, Lj, extra_left=3)
    j = O.join(left, right, bits, Lj)
    st, m, h, c = run_join(left, right, bits, Lj)
    assert st == O.OK
    assert np.array_equal(m, j.match)
    assert np.array_equal(h, j.hits)
    assert np.array_equal(c, j.counts)


def test_join_factool_search_queries():
    """Search-query objects (level 3 of the FacTool-shaped tree, e.g. query embeddings)
    joined with every sentence below them (908,008 fragments)."""
    w = W.factool_batch("cpu")
    keys = O.pack_keys(w.path.numpy(), w.bits)
    rng = np.random.default_rng(5)
    left = np.unique(O.prefix(keys, w.bits, 3))
    left = left[rng.permutation(len(left))]
    j = O.join(left, keys, w.bits, 3)
    st, m, h, c = run_join(left, keys, w.bits, 3)
    assert st == O.OK and c[0] == len(keys) and c[1] == len(left)
    assert np.array_equal(m, j.match)
    assert np.array_equal(h, j.hits)


@pytest.mark.parametrize("kind", ["dup", "layout_left", "layout_right", "empty_right", "empty_left"])
def test_join_errors_and_empty(kind):
    bits = (5, 3, 3, 4)
    left, right = _case(21, bits, (3, 3, 3), 3, 2)
    if kind == "dup":
        left = np.concatenate([left, left[:1]])
    elif kind == "layout_left":
        left = np.concatenate([left, np.array([1 << 8], np.uint64)])
    elif kind == "layout_right":
        right = np.concatenate([right, np.array([1 << 15], np.uint64)])
    elif kind == "empty_right":
        right = right[:0]
    else:
        left = left[:0]
    try:
        j = O.join(left, right, bits, 2)
        code = O.OK
    except O.OracleError as e:
        code, j = e.code, None
    st, m, h, c = run_join(left, right, bits, 2)
    assert st == code
    if j is not None:
        assert np.array_equal(m, j.match) and np.array_equal(h, j.hits) and np.array_equal(c, j.counts)
