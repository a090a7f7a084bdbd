"""GPU parity of load-aware routing (alto_router_*, alto_route_load) against the
oracle, through the C ABI, over several batches with queues drained in between."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def gpu_route(rt, keys, load):
    """keys: numpy uint64; load: numpy int64 (copied to the device, updated there)."""
    n = len(keys)
    dk = U.to_dev(keys.astype(np.uint64).view(np.int64)) if n else torch.empty(1, dtype=torch.int64, device="cuda")
    dl = U.to_dev(np.asarray(load, np.int64))
    perm, offs, dest, counts, st = rt.route(dk, dl, n=n)
    torch.cuda.synchronize()
    return {"status": int(st.item()), "perm": perm[:n].cpu().numpy(), "offs": offs.cpu().numpy(),
            "dest": dest[:n].cpu().numpy(), "load": dl.cpu().numpy(), "counts": counts.cpu().numpy()}


def same(g, o):
    assert g["status"] == O.OK
    assert np.array_equal(g["dest"], o.dest)
    assert np.array_equal(g["load"], o.load)
    assert np.array_equal(g["counts"], o.counts)
    assert np.array_equal(g["offs"], o.dest_offsets)
    if len(o.perm):
        assert np.array_equal(g["perm"], o.perm)


def test_load_route_worked_example():
    rt = alto.LoadRouter((4, 4), 1, 2, 16, 64)
    orc = O.LoadRouter((4, 4), 1, 2, 16)
    for keys, load in [([(3, 0), (1, 0), (1, 1)], [0, 0]),
                       ([(4, 0)] + [(3, c) for c in range(1, 8)] + [(2, 0), (2, 1), (2, 2)], [5, 0])]:
        k = np.array([(f << 4) | c for f, c in keys], np.uint64)
        same(gpu_route(rt, k, load), orc.route(k, load))


CASES = [
    # seed, bits, route level, D, max_fan, roots, batches
    (1, (6, 5, 4), 2, 5, (12, 9), 20, 4),
    (2, (31, 3, 2, 3, 8), 2, 32, (6, 3, 5, 40), 60, 3),        # multi-block sorts
    (3, (20, 12, 8), 2, 1, (300, 30), 40, 3),                   # one destination
    (4, (20, 12, 8), 2, 4096, (300, 30), 50, 3),                # most destinations, > 2,048 new flows
    (5, (16, 10, 6), 1, 7, (50, 20), 3000, 2),                  # 3,000 level-1 flows per batch
    (6, (8, 8, 8), 3, 64, (8, 8), 100, 3),                      # flows are the leaves
    (7, (20, 12, 8), 2, 48, (400, 30), 60, 2),                  # > 8,192 flows: general sort, table lookups
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_load_route_parity_over_batches(case):
    # one tree's leaves, shuffled and cut into consecutive batches: flows recur
    # across batches (known flows) and keep appearing (new flows)
    seed, bits, Lr, D, mf, roots, batches = CASES[case]
    rng = np.random.default_rng(5000 + seed)
    rt = alto.LoadRouter(bits, Lr, D, 1 << 16, 1 << 20)
    orc = O.LoadRouter(bits, Lr, D, 1 << 16)
    path, fan = W.random_tree(5100 + seed, len(bits), roots, mf, bits)
    keys = O.pack_keys(path, bits)
    keys = keys[rng.permutation(len(keys))]
    load = np.zeros(D, np.int64)
    for part in np.array_split(keys, batches):
        o = orc.route(part, load)
        same(gpu_route(rt, part, load), o)
        load = o.load - rng.integers(0, o.load + 1)
    assert len(orc.table) > 0


def test_load_route_empty_and_errors():
    bits = (6, 5, 4)
    rt = alto.LoadRouter(bits, 2, 3, 40, 4096)
    orc = O.LoadRouter(bits, 2, 3, 40)
    g = gpu_route(rt, np.zeros(0, np.uint64), [1, 2, 3])
    assert g["status"] == O.OK and g["load"].tolist() == [1, 2, 3] and g["offs"].tolist() == [0, 0, 0, 0]
    path, fan = W.random_tree(77, 3, 4, (5, 6), bits)
    keys = O.pack_keys(path, bits)
    first = keys[O.prefix(keys, bits, 1) == O.prefix(keys[:1], bits, 1)[0]]
    same(gpu_route(rt, first, [0, 0, 0]), orc.route(first, [0, 0, 0]))
    # each error leaves queues and table as they were: the next call still agrees
    dup = np.concatenate([keys, keys[:1]])
    wide = keys.copy()
    wide[3] |= np.uint64(1 << 20)
    for bad, code in [(dup, O.E_DUPLICATE), (wide, O.E_LAYOUT)]:
        with pytest.raises(O.OracleError) as e:
            orc.route(bad, [4, 4, 4])
        g = gpu_route(rt, bad, [4, 4, 4])
        assert e.value.code == code and g["status"] == code and g["load"].tolist() == [4, 4, 4]
    many = O.pack_keys(W.random_tree(78, 3, 50, (5, 6), bits)[0], bits)   # more than 40 flows
    with pytest.raises(O.OracleError) as e:
        orc.route(many, [0, 0, 0])
    g = gpu_route(rt, many, [0, 0, 0])
    assert e.value.code == O.E_CAPACITY and g["status"] == O.E_CAPACITY and g["load"].tolist() == [0, 0, 0]
    same(gpu_route(rt, keys, [2, 0, 1]), orc.route(keys, [2, 0, 1]))


def test_load_route_rejects_bad_arguments():
    import ctypes as C
    lib = alto.load()
    L = alto.layout((6, 5, 4))
    st = torch.empty(int(lib.alto_router_state_bytes(8)), dtype=torch.uint8, device="cuda")
    h = C.c_void_p()
    for Lr, D, mf in [(0, 2, 8), (4, 2, 8), (1, 0, 8), (1, 4097, 8), (1, 2, 0)]:
        assert lib.alto_router_create(C.byref(L), Lr, D, mf, st.data_ptr(), st.numel(), None, C.byref(h)) == 1
    assert lib.alto_router_create(C.byref(L), 1, 2, 1 << 20, st.data_ptr(), st.numel(), None, C.byref(h)) == 1
    assert lib.alto_route_load_workspace_bytes(C.byref(L), 1, 16, 0) == 0
    assert lib.alto_route_load_workspace_bytes(C.byref(L), 4, 16, 2) == 0
    assert lib.alto_route_load_workspace_bytes(C.byref(L), 1, 16, 2) > 0
    assert lib.alto_router_state_bytes(0) == 0


def test_load_route_zipf_tree_full_size():
    """All 2^26 fragments of the Zipf depth-6 tree, flows at level 4 (1,452 of them)
    to 256 destinations from empty queues, in the launch configuration the benchmark
    times: destinations and queues against the oracle, perm by its defining order."""
    w = W.zipf_tree("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    del w
    torch.cuda.empty_cache()
    bits = (3, 12, 12, 12, 12, 12)
    n = keys.numel()
    rt = alto.LoadRouter(bits, 4, 256, 1 << 16, n)
    load = torch.zeros(256, dtype=torch.int64, device="cuda")
    perm, offs, dest, counts, st2 = rt.route(keys, load)
    torch.cuda.synchronize()
    assert int(st.item()) == O.OK and int(st2.item()) == O.OK
    keys_np = keys.cpu().numpy().view(np.uint64)
    o = O.LoadRouter(bits, 4, 256, 1 << 16).route(keys_np, np.zeros(256, np.int64), with_perm=False)
    assert np.array_equal(dest.cpu().numpy(), o.dest)
    assert np.array_equal(load.cpu().numpy(), o.load)
    assert np.array_equal(offs.cpu().numpy(), o.dest_offsets)
    assert counts.cpu().tolist() == o.counts.tolist()
    # perm: a permutation, destinations ascending, keys ascending within each
    p = perm.long()
    assert int(torch.bincount(p, minlength=n).max()) == 1
    ks = keys[p]
    same_d = dest[p][1:] == dest[p][:-1]
    assert bool((dest[p][1:] >= dest[p][:-1]).all())
    assert bool((ks[1:] > ks[:-1])[same_d].all())


def test_load_route_factool_stream_steps():
    """A FacTool-shaped tree (1,024 queries, ~0.9M fragments, shuffled arrival) streamed
    in 4,096-fragment steps, routed by claim (level 2) to 32 destinations, each
    destination draining 128 fragments per step: destinations, queues, perm and counts
    of every step against the oracle."""
    rng = np.random.default_rng(W.SEED_BASE + 2)
    roots = W.distinct_ids(rng, 1024)
    path, _ = W.expand_tree(W.factool_fans(rng, roots), roots)   # the FacTool-shaped tree, no payload
    (path,), _ = W.permute([path], 77)
    bits = (31, 3, 2, 3, 8)
    keys = O.pack_keys(path, bits)
    step, D = 4096, 32
    rt = alto.LoadRouter(bits, 2, D, 1 << 16, step)
    orc = O.LoadRouter(bits, 2, D, 1 << 16)
    load = np.zeros(D, np.int64)
    for s in range(0, len(keys), step):
        part = keys[s:s + step]
        o = orc.route(part, load)
        same(gpu_route(rt, part, load), o)
        load = np.maximum(o.load - 128, 0)
    assert len(orc.table) > 1000
