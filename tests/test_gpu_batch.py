"""GPU parity of the batch path (alto_pack_keys, alto_route, alto_aggregate) against
the CPU oracle, through the C ABI."""
import numpy as np
import pytest

from oracle import alto_oracle as O
from paper_2403_04311_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _case(seed, depth, bits, mf, roots, drop=0.0, dim=3):
    path, fan = W.random_tree(seed, depth, roots, mf, bits)
    if drop:
        path, fan, _ = W.drop_leaves(path, fan, drop, seed + 1)
    rng = np.random.default_rng(seed + 2)
    n = path.shape[1]
    p32 = rng.integers(-(2**31), 2**31 - 1, size=n).astype(np.int32)
    pf = rng.standard_normal((n, dim)).astype(np.float32)
    (path, fan, p32, pft), _ = W.permute([path, fan, p32, pf.T], seed + 3)
    return path, fan, p32, np.ascontiguousarray(pft.T)


CASES = [
    # depth, bits, max_fan, roots, La, Lm, Lr, D, drop, dim
    (2, (8, 4), (5,), 7, 1, 0, 1, 3, 0.0, 4),
    (3, (10, 3, 3), (4, 5), 30, 2, 1, 1, 4, 0.2, 5),
    (4, (31, 2, 3, 4), (4, 8, 16), 64, 3, 0, 1, 8, 0.0, 8),
    (4, (31, 2, 3, 4), (3, 3, 3), 50, 2, 3, 2, 5, 0.15, 16),
    (5, (6, 3, 2, 3, 5), (3, 3, 3, 6), 40, 4, 2, 4, 16, 0.1, 128),
    (5, (6, 3, 2, 3, 5), (3, 2, 3, 4), 40, 3, 1, 2, 7, 0.05, 1),
    (4, (5, 3, 3, 3), (3, 3, 4), 20, 1, 2, 0, 1, 0.1, 12),
    (6, (3, 3, 3, 3, 3, 4), (2, 3, 2, 3, 5), 6, 4, 2, 4, 256, 0.08, 64),
    (3, (20, 12, 12), (40, 3000), 3, 2, 0, 2, 64, 0.01, 768),      # groups span many chunks
    (4, (31, 8, 8, 10), (200, 1, 1000), 2, 1, 3, 1, 1000, 0.0, 4),  # one giant group per root
    # mask above the route level with more than one workgroup's worth of fragments
    (5, (6, 3, 2, 3, 8), (4, 3, 5, 60), 20, 4, 2, 3, 64, 0.02, 8),
    (6, (3, 12, 12, 12, 12, 12), (3, 4, 30, 60, 40), 2, 4, 2, 4, 256, 0.0, 128),
    # groups are the flows (mean gathered beside segmentation), incomplete groups and
    # a mask above them
    (5, (6, 3, 2, 3, 8), (4, 3, 5, 60), 40, 3, 1, 3, 64, 0.03, 16),
]


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("op", ["concat", "mean"])
def test_aggregate_parity(case, op):
    depth, bits, mf, roots, La, Lm, Lr, D, drop, dim = CASES[case]
    path, fan, p32, pf = _case(100 + case, depth, bits, mf, roots, drop, dim)
    keys = O.pack_keys(path, bits)
    code, rt, g = U.oracle_aggregate(keys, fan, bits, La, op, dim, Lm, Lr, D, p32,
                                     pf if op == "mean" else None)
    assert code == O.OK
    res = U.run_aggregate(keys, fan, bits, La, op, dim, Lm, Lr, D, p32, pf if op == "mean" else None)
    assert res["status"] == O.OK
    U.compare(res, rt, g, op, Lm, La)


@pytest.mark.parametrize("drop,Lr,seed", [(0.0, 4, 113), (0.01, 4, 113), (0.01, 3, 117)])
def test_mean_dim128_groups_of_several_chunks(drop, Lr, seed):
    # The 2^26-fragment workload's layout and launch (128-d rows, mean at level 4,
    # mask at level 2, 256 destinations) at a size the oracle finishes quickly, with
    # level-4 groups longer than one 4,096-row gather chunk (partial sums per chunk,
    # combined in chunk order) and, with drop > 0, incomplete groups and masks.
    bits = (3, 12, 12, 12, 12, 12)
    path, fan, p32, pf = _case(seed, 6, bits, (2, 2, 3, 200, 60), 2, drop, 128)
    keys = O.pack_keys(path, bits)
    _, cnt = np.unique(O.prefix(keys, bits, 4), return_counts=True)
    assert (cnt > 4096).sum() >= 2 and (cnt <= 256).sum() + ((cnt > 256) & (cnt <= 4096)).sum() >= 1
    code, rt, g = U.oracle_aggregate(keys, fan, bits, 4, "mean", 128, 2, Lr, 256, p32, pf)
    assert code == O.OK
    if drop:
        assert len(g.pend_key) > 0 and (g.mask == 0).any()
    res = U.run_aggregate(keys, fan, bits, 4, "mean", 128, 2, Lr, 256, p32, pf)
    assert res["status"] == O.OK
    U.compare(res, rt, g, "mean", 2, 4)


def test_pack_parity_and_layout_error():
    bits = (31, 2, 3, 4)
    path, fan, _, _ = _case(5, 4, bits, (4, 8, 16), 64)
    k, st = U.pack_gpu(path, bits)
    assert st == O.OK
    assert np.array_equal(k.cpu().numpy().view(np.uint64), O.pack_keys(path, bits))
    bad = path.copy()
    bad[2, 7] = 8
    _, st = U.pack_gpu(bad, bits)
    assert st == O.E_LAYOUT
    bad = path.copy()
    bad[0, 3] = -1
    _, st = U.pack_gpu(bad, bits)
    assert st == O.E_LAYOUT


@pytest.mark.parametrize("D,Lr", [(1, 1), (3, 2), (256, 3), (1000, 4), (1 << 20, 2)])
def test_route_parity(D, Lr):
    import torch
    from paper_2403_04311_amd import alto
    bits = (31, 2, 3, 4)
    path, fan, _, _ = _case(40 + D, 4, bits, (4, 8, 16), 300)
    keys = O.pack_keys(path, bits)
    rt = O.route(keys, bits, Lr, D)
    perm, offs, dest, st = alto.route(U.to_dev(keys.view(np.int64)), bits, Lr, D)
    torch.cuda.synchronize()
    assert int(st.item()) == O.OK
    assert np.array_equal(perm.cpu().numpy(), rt.perm)
    assert np.array_equal(offs.cpu().numpy(), rt.dest_offsets)
    assert np.array_equal(dest.cpu().numpy(), rt.dest)


@pytest.mark.parametrize("op", ["concat", "mean"])
def test_general_mode_sort(op):
    """More distinct route prefixes than the flow set holds: the sort falls back to
    (key, index) pairs with destination windows (no packed words)."""
    bits = (17, 2, 2, 3)
    path, fan, p32, pf = _case(321, 4, bits, (2, 2, 3), 40000, 0.01, 8)
    keys = O.pack_keys(path, bits)
    assert len(np.unique(O.prefix(keys, bits, 1))) > 32768
    code, rt, g = U.oracle_aggregate(keys, fan, bits, 2, op, 8, 0, 1, 1000, p32, pf if op == "mean" else None)
    assert code == O.OK
    res = U.run_aggregate(keys, fan, bits, 2, op, 8, 0, 1, 1000, p32, pf if op == "mean" else None)
    assert res["status"] == O.OK
    U.compare(res, rt, g, op, 0, 2)


def test_child_index_error_with_child_ranks():
    """A child tag equal to its node's declared count in a batch that the sort packs
    by child ranks over several workgroups: the FANOUT error is reported (the order is
    undefined then, and the rank table is still read within bounds)."""
    bits = (5, 5, 8, 8)
    path, fan, p32, _ = _case(91, 4, bits, (6, 40, 60), 20)
    keys = O.pack_keys(path, bits)
    assert len(keys) > 8192
    fan = fan.copy()
    i = int(np.argmax(O.tag(keys, bits, 3)))
    sel = O.prefix(keys, bits, 2) == O.prefix(keys[i:i + 1], bits, 2)[0]
    fan[1, sel] = int(O.tag(keys[i:i + 1], bits, 3)[0])     # child index == declared count
    La, Lm, Lr, D = 2, 0, 2, 16
    code, _, _ = U.oracle_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert code == O.E_FANOUT
    res = U.run_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert res["status"] == code


def test_route_duplicate_and_layout():
    import torch
    from paper_2403_04311_amd import alto
    keys = np.array([5, 9, 1, 7, 9], np.uint64)
    _, _, _, st = alto.route(U.to_dev(keys.view(np.int64)), (4, 4), 2, 3)
    torch.cuda.synchronize()
    assert int(st.item()) == O.E_DUPLICATE
    keys = np.array([5, 300, 1], np.uint64)
    _, _, _, st = alto.route(U.to_dev(keys.view(np.int64)), (4, 4), 2, 3)
    torch.cuda.synchronize()
    assert int(st.item()) == O.E_LAYOUT


def test_tiny_tree_full():
    w = W.tiny_tree("cpu")
    path, fan, tok = w.path.numpy(), w.fan.numpy(), w.payload_i32.numpy()
    keys = O.pack_keys(path, w.bits)
    code, rt, g = U.oracle_aggregate(keys, fan, w.bits, w.agg_level, w.op, 1, 0, w.route_level,
                                     w.num_dest, tok)
    assert code == O.OK
    res = U.run_aggregate(keys, fan, w.bits, w.agg_level, w.op, 1, 0, w.route_level, w.num_dest, tok)
    assert res["status"] == O.OK
    U.compare(res, rt, g, w.op, 0, w.agg_level)


def _error_inputs():
    bits = (6, 3, 4)
    path, fan, p32, _ = _case(77, 3, bits, (5, 9), 20)
    return bits, path, fan, p32


@pytest.mark.parametrize("kind", ["dup", "fan_disagree", "child_index", "fan_zero", "layout",
                                  "dup_and_fan", "capacity_tokens", "capacity_groups", "mask_above"])
def test_error_paths(kind):
    bits, path, fan, p32 = _error_inputs()
    keys = O.pack_keys(path, bits)
    La, Lm, Lr, D = 2, 0, 1, 5
    caps = None
    if kind == "dup":
        keys = np.concatenate([keys, keys[3:4]])
        fan = np.concatenate([fan, fan[:, 3:4]], axis=1)
        p32 = np.concatenate([p32, p32[:1]])
    elif kind == "fan_disagree":
        fan = fan.copy()
        fan[1, 11] += 1
    elif kind == "child_index":
        fan = fan.copy()
        i = int(np.argmax(O.tag(keys, bits, 3)))
        sel = O.prefix(keys, bits, 2) == O.prefix(keys[i:i + 1], bits, 2)[0]
        fan[1, sel] = int(O.tag(keys[i:i + 1], bits, 3)[0])     # child index == declared count
    elif kind == "fan_zero":
        fan = fan.copy()
        fan[1, :] = np.where(O.prefix(keys, bits, 2) == O.prefix(keys[:1], bits, 2)[0], 0, fan[1])
    elif kind == "layout":
        keys = keys.copy()
        keys[5] = np.uint64(1 << 13)
    elif kind == "dup_and_fan":
        keys = np.concatenate([keys, keys[3:4]])
        fan = np.concatenate([fan, fan[:, 3:4]], axis=1)
        p32 = np.concatenate([p32, p32[:1]])
        fan[1, 0] += 2
    elif kind == "capacity_tokens":
        caps = (len(keys), len(keys) - 1, 0)
    elif kind == "capacity_groups":
        caps = (3, len(keys), 0)
    elif kind == "mask_above":
        # disagreement only visible across destinations, on a level above the route level
        La, Lm, Lr, D = 2, 1, 2, 7
        fan = fan.copy()
        r0 = O.prefix(keys, bits, 1)
        first_root = r0 == r0[0]
        idx = np.nonzero(first_root)[0]
        g2 = O.prefix(keys[idx], bits, 2)
        other = idx[g2 != g2[0]]
        if len(other):
            fan[0, other] += 1
    code, _, _ = U.oracle_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    if kind.startswith("capacity"):
        code = O.E_CAPACITY
    res = U.run_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32, caps=caps)
    assert code != O.OK
    assert res["status"] == code, (kind, res["status"], code)
    if kind == "capacity_tokens":
        assert res["counts"][1] == len(keys)


@pytest.mark.parametrize("n", [0, 1, 2])
def test_tiny_batches(n):
    bits = (4, 3, 3)
    path, fan, p32, pf = _case(9, 3, bits, (3, 4), 5, dim=4)
    path, fan, p32, pf = path[:, :n], fan[:, :n], p32[:n], pf[:n]
    keys = O.pack_keys(path, bits)
    for op in ("concat", "mean"):
        code, rt, g = U.oracle_aggregate(keys, fan, bits, 2, op, 4, 1, 1, 3, p32,
                                         pf if op == "mean" else None)
        res = U.run_aggregate(keys, fan, bits, 2, op, 4, 1, 1, 3, p32, pf if op == "mean" else None)
        assert res["status"] == code == O.OK
        if n == 0:
            assert res["counts"] == (0, 0, 0, 0)
        else:
            U.compare(res, rt, g, op, 1, 2)


def test_determinism_and_permutation_invariance_of_means():
    bits = (6, 3, 2, 3, 8)
    path, fan, p32, pf = _case(55, 5, bits, (4, 3, 5, 200), 8, dim=64)
    keys = O.pack_keys(path, bits)
    a = U.run_aggregate(keys, fan, bits, 3, "mean", 64, 0, 2, 9, p32, pf)
    b = U.run_aggregate(keys, fan, bits, 3, "mean", 64, 0, 2, 9, p32, pf)
    assert np.array_equal(a["mean"], b["mean"])
    (path2, fan2, p322, pft2), _ = W.permute([path, fan, p32, pf.T], 999)
    keys2 = O.pack_keys(path2, bits)
    c = U.run_aggregate(keys2, fan2, bits, 3, "mean", 64, 0, 2, 9, p322, np.ascontiguousarray(pft2.T))
    assert np.array_equal(a["mean"], c["mean"])          # sums follow key order, not arrival
    assert np.array_equal(a["key"], c["key"])


def _flow_case():
    bits = (6, 3, 2, 3, 8)
    path, fan, p32, _ = _case(61, 5, bits, (4, 3, 5, 60), 40)
    keys = O.pack_keys(path, bits)
    assert len(keys) > 8192           # multi-workgroup sort: the input pass keeps a flow set
    return bits, keys, fan, p32


def _carriers(keys, bits, level, min_count=2):
    """Fragments of the first level-`level` node that has at least min_count of them."""
    pre = O.prefix(keys, bits, level)
    vals, counts = np.unique(pre, return_counts=True)
    v = vals[np.argmax(counts >= min_count)]
    return np.nonzero(pre == v)[0]


@pytest.mark.parametrize("kind", ["valid", "route_level", "above_same_flow", "above_across_flows"])
def test_flow_level_count_checks(kind):
    """Declared counts of the route level and the levels above it are compared per
    flow in the input pass; disagreements between flows are caught on the node
    records. Route level 3, mean at level 4, mask at level 2 (levels 2..4 read)."""
    bits, keys, fan, p32 = _flow_case()
    La, Lm, Lr, D = 4, 2, 3, 64
    fan = fan.copy()
    if kind == "route_level":
        c = _carriers(keys, bits, 3)
        fan[2, c[-1]] += 1                       # one carrier of a level-3 node
    elif kind == "above_same_flow":
        c = _carriers(keys, bits, 3)
        fan[1, c[0]] += 1                        # its level-2 count, one carrier
    elif kind == "above_across_flows":
        pre2 = O.prefix(keys, bits, 2)
        pre3 = O.prefix(keys, bits, 3)
        # a level-2 node with several level-3 children: change all carriers of one child
        v2 = next(v for v in np.unique(pre2) if len(np.unique(pre3[pre2 == v])) > 1)
        child = np.unique(pre3[pre2 == v2])[1]
        fan[1, pre3 == child] += 1
    code, rt, g = U.oracle_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert code == (O.OK if kind == "valid" else O.E_FANOUT)
    res = U.run_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert res["status"] == code, (kind, res["status"], code)
    if kind == "valid":
        U.compare(res, rt, g, "concat", Lm, La)


@pytest.mark.parametrize("bad", [False, True])
def test_flow_set_overflow_count_check(bad):
    """More route prefixes than the flow set holds, with the route level's counts
    read: the per-flow check is incomplete, so those counts join the fingerprint."""
    bits = (17, 2, 2, 3)
    path, fan, p32, _ = _case(322, 4, bits, (2, 2, 3), 40000)
    keys = O.pack_keys(path, bits)
    assert len(np.unique(O.prefix(keys, bits, 1))) > 32768
    La, Lm, Lr, D = 1, 0, 1, 1000
    if bad:
        fan = fan.copy()
        c = _carriers(keys, bits, 1)
        fan[0, c[-1]] += 1
    code, rt, g = U.oracle_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert code == (O.E_FANOUT if bad else O.OK)
    res = U.run_aggregate(keys, fan, bits, La, "concat", 1, Lm, Lr, D, p32)
    assert res["status"] == code
    if not bad:
        U.compare(res, rt, g, "concat", Lm, La)


def test_two_stage_batches_pipelined_on_two_hip_streams_match_one_stream():
    """The FacTool-shaped batch's two stages with stage B of a batch on a second HIP
    stream beside stage A of the next (stage A's records in one of two buffers, events
    between the stages), over four batches: the outputs of every batch are the same
    bits as with both stages on one stream."""
    import torch
    from paper_2403_04311_amd import alto
    w = W.factool_batch("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, dim = w.n, w.dim
    sb = W.FACTOOL_CLAIM_STAGE
    ws = alto.new_workspace(alto.workspace_bytes(w.bits, n, 32, 4, "mean", dim))
    stA, stB = alto.new_status(), alto.new_status()
    gAs = [alto.new_groups(n // 4 + 1024, 4, "mean", dim), alto.new_groups(n // 4 + 1024, 4, "mean", dim)]
    alto.aggregate(keys, w.fan, w.bits, 4, "mean", dim, 0, 2, 32, w.payload_i32, w.payload_f32, ws=ws,
                   out=gAs[0], status=stA, n=n)
    torch.cuda.synchronize()
    E = int(gAs[0].counts[0])
    assert int(stA.item()) == 0 and E > 0
    wsB = alto.new_workspace(alto.workspace_bytes(sb["bits"], E, 32, 2, "concat"))
    gB = alto.new_groups(E, 2, "concat", cap_tokens=E)

    def snap_a(g):
        return [g.counts.clone(), g.key[:E].clone(), g.mean[:E].clone(), g.first_i32[:E].clone()]

    def snap_b(g):
        return [g.counts.clone(), g.key.clone(), g.tok_off.clone(), g.tok.clone()]

    def stage_a(g, stream):
        alto.aggregate(keys, w.fan, w.bits, 4, "mean", dim, 0, 2, 32, w.payload_i32, w.payload_f32, ws=ws,
                       out=g, status=stA, n=n, stream=stream)

    def stage_b(g, stream):
        alto.aggregate(g.key, g.fan_up.view(3, -1)[:, :E], sb["bits"], 2, "concat", 1, 0, 2, 32, g.first_i32,
                       None, ws=wsB, out=gB, status=stB, n=E, stream=stream)
    main = torch.cuda.current_stream()
    seq = []
    for b in range(4):
        stage_a(gAs[0], main)
        sa = snap_a(gAs[0])
        stage_b(gAs[0], main)
        seq.append((sa, snap_b(gB)))
    side = torch.cuda.Stream()
    side.wait_stream(main)
    a_done = [torch.cuda.Event(), torch.cuda.Event()]
    b_done = [torch.cuda.Event(), torch.cuda.Event()]
    par = []
    for b in range(4):
        k = b & 1
        if b >= 2:
            main.wait_event(b_done[k])
        stage_a(gAs[k], main)
        sa = snap_a(gAs[k])
        a_done[k].record(main)
        side.wait_event(a_done[k])
        with torch.cuda.stream(side):
            stage_b(gAs[k], side)
            par.append((sa, snap_b(gB)))
        b_done[k].record(side)
    main.wait_stream(side)
    torch.cuda.synchronize()
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    for (a0, b0), (a1, b1) in zip(seq, par):
        for x, y in zip(a0 + b0, a1 + b1):
            assert torch.equal(x, y)
