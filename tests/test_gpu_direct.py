"""GPU parity of batches that the sort can place directly: groups are the route
level's flows and leaves lie one level below their children (the 2^26-fragment
workload's shape: one root, one level-2 and one level-3 node, so the flows'
prefixes differ in the level-4 tag only). Complete batches, and the data errors
whose detection direct placement changes: a key given twice (a position of the
sorted order left empty) and a leaf declaring another count than its siblings
(the child level's fingerprint), alone and together (FANOUT wins), against the
oracle's status."""
import numpy as np
import pytest

from oracle import alto_oracle as O
from paper_2403_04311_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

BITS = (3, 12, 12, 12, 12, 12)


def _tree(seed, f4=150, f5=30, f6=40, dim=8):
    path, fan = W.random_tree(seed, 6, 1, (1, 1, f4, f5, f6), BITS, dense_roots=True)
    rng = np.random.default_rng(seed + 1)
    n = path.shape[1]
    pf = rng.standard_normal((n, dim)).astype(np.float32)
    p32 = rng.integers(0, 1 << 30, size=n).astype(np.int32)
    (path, fan, p32, pft), _ = W.permute([path, fan, p32, pf.T], seed + 2)
    return path, fan, p32, np.ascontiguousarray(pft.T)


def _eligible(keys, fan):
    # complete batch, more than one workgroup's sort, flows varying in the level-4 tag
    n = len(keys)
    assert n > 8192
    assert len(np.unique(O.prefix(keys, BITS, 3))) == 1
    comp = O.completion(keys, fan, BITS, 4)
    assert comp[4][1].all() and comp[5][1].all()


@pytest.mark.parametrize("seed,op,Lm", [(500, "mean", 2), (501, "concat", 0), (502, "mean", 4), (503, "concat", 3)])
def test_direct_placement_complete_batches(seed, op, Lm):
    path, fan, p32, pf = _tree(seed)
    keys = O.pack_keys(path, BITS)
    _eligible(keys, fan)
    dim = pf.shape[1] if op == "mean" else 1
    code, rt, g = U.oracle_aggregate(keys, fan, BITS, 4, op, dim, Lm, 4, 256, p32, pf if op == "mean" else None)
    assert code == O.OK
    res = U.run_aggregate(keys, fan, BITS, 4, op, dim, Lm, 4, 256, p32, pf if op == "mean" else None)
    assert res["status"] == O.OK
    U.compare(res, rt, g, op, Lm, 4)


def _leaf_cols(keys, fan):
    """Per fragment: level-5 prefix, leaf tag, declared leaf count."""
    return O.prefix(keys, BITS, 5), O.tag(keys, BITS, 6).astype(np.int64), fan[4].astype(np.int64)


@pytest.mark.parametrize("case", ["duplicate", "fanout", "both"])
def test_direct_placement_errors_match_oracle(case):
    path, fan, p32, pf = _tree(510)
    keys = O.pack_keys(path, BITS)
    _eligible(keys, fan)
    node, tag, cnt = _leaf_cols(keys, fan)
    # two non-marker leaves of one level-5 node with at least 3 leaves
    nodes, nc = np.unique(node, return_counts=True)
    big = nodes[np.argmax(nc)]
    idx = np.nonzero((node == big) & (tag != cnt - 1))[0]
    assert len(idx) >= 2
    keys, fan = keys.copy(), fan.copy()
    if case in ("duplicate", "both"):
        keys[idx[0]] = keys[idx[1]]                  # a key twice, another tag missing
    if case in ("fanout", "both"):
        other = np.nonzero((node != big) & (tag != cnt - 1))[0][0]
        fan[4, other] += 1                           # one carrier disagrees (still > its tag)
    want = {"duplicate": O.E_DUPLICATE, "fanout": O.E_FANOUT, "both": O.E_FANOUT}[case]
    code, _, _ = U.oracle_aggregate(keys, fan, BITS, 4, "mean", 8, 2, 4, 256, p32, pf)
    assert code == want
    for rep in range(2):   # the second call finds the first one's workspace contents
        res = U.run_aggregate(keys, fan, BITS, 4, "mean", 8, 2, 4, 256, p32, pf)
        assert res["status"] == want, rep


def test_direct_placement_not_taken_when_a_marker_is_missing():
    # the marker of one node replaced by a duplicate of a sibling: that node has no
    # marker, so the sort takes the ordinary path, which finds the duplicate
    path, fan, p32, pf = _tree(520)
    keys = O.pack_keys(path, BITS)
    _eligible(keys, fan)
    node, tag, cnt = _leaf_cols(keys, fan)
    m = np.nonzero((tag == cnt - 1) & (cnt >= 2))[0][0]
    sib = np.nonzero((node == node[m]) & (tag != cnt - 1))[0][0]
    keys = keys.copy()
    keys[m] = keys[sib]
    code, _, _ = U.oracle_aggregate(keys, fan, BITS, 4, "mean", 8, 2, 4, 256, p32, pf)
    assert code == O.E_DUPLICATE
    res = U.run_aggregate(keys, fan, BITS, 4, "mean", 8, 2, 4, 256, p32, pf)
    assert res["status"] == O.E_DUPLICATE


@pytest.mark.parametrize("seed,op,Lm,drop", [(540, "mean", 2, 0.0), (541, "mean", 0, 0.01), (542, "concat", 3, 0.0)])
def test_gathers_on_a_second_stream_match_one_stream(seed, op, Lm, drop):
    """alto_aggregate_overlap: the gathers of a batch on a second HIP stream beside the
    next batch's routing (two sets of workspace and outputs, events between them), over
    four batches in a row: every output equals alto_aggregate on one stream (direct
    placement for the complete batches, the general path with dropped leaves)."""
    import torch
    from paper_2403_04311_amd import alto
    path, fan, p32, pf = _tree(seed)
    if drop:
        keep = np.random.default_rng(seed + 9).random(path.shape[1]) >= drop
        path, fan, p32, pf = path[:, keep], fan[:, keep], p32[keep], pf[keep]
    keys = O.pack_keys(path, BITS)
    n = len(keys)
    dim = pf.shape[1] if op == "mean" else 1
    tk = U.to_dev(keys.view(np.int64))
    tf = U.to_dev(fan.astype(np.int32))
    t32 = U.to_dev(p32)
    tpf = U.to_dev(pf) if op == "mean" else None

    def outs():
        return (alto.new_workspace(alto.workspace_bytes(BITS, n, 256, 4, op, dim, Lm)),
                torch.empty(n, dtype=torch.int32, device="cuda"), torch.empty(257, dtype=torch.int64, device="cuda"),
                torch.empty(n, dtype=torch.int32, device="cuda"),
                alto.new_groups(n, 4, op, dim, cap_tokens=n if op == "concat" else 0, cap_mask=n if Lm else 0))

    def snapshot(o):
        ws, perm, offs, dest, g = o
        E, T, M, P = [int(x) for x in g.counts.cpu()]
        r = [perm.cpu(), offs.cpu(), dest.cpu(), g.counts.cpu(), g.key[:E].cpu(), g.count[:E].cpu()]
        if op == "mean":
            r.append(g.mean[:E].cpu())
        else:
            r += [g.tok_off[:E + 1].cpu(), g.tok[:T].cpu()]
        if Lm:
            r += [g.mask_key[:M].cpu(), g.mask[:M].cpu()]
        return r
    ref = outs()
    st = alto.new_status()
    alto.aggregate(tk, tf, BITS, 4, op, dim, Lm, 4, 256, t32, tpf, ws=ref[0], perm=ref[1], dest_offsets=ref[2],
                   dest=ref[3], out=ref[4], status=st, n=n)
    torch.cuda.synchronize()
    want_status = int(st.item())
    want = snapshot(ref)
    sets = [outs(), outs()]
    main = torch.cuda.current_stream()
    gather = torch.cuda.Stream()
    gather.wait_stream(main)
    done = [torch.cuda.Event(), torch.cuda.Event()]
    got = []
    for b in range(4):
        k = b & 1
        if b >= 2:
            main.wait_event(done[k])
            main.synchronize()   # the previous batch of this set is compared before it is overwritten
            got.append(snapshot(sets[k]))
        ws, perm, offs, dest, g = sets[k]
        alto.aggregate(tk, tf, BITS, 4, op, dim, Lm, 4, 256, t32, tpf, ws=ws, perm=perm, dest_offsets=offs,
                       dest=dest, out=g, status=st, n=n, stream=main, gather_stream=gather)
        done[k].record(gather)
    main.wait_stream(gather)
    torch.cuda.synchronize()
    got += [snapshot(sets[0]), snapshot(sets[1])]
    assert int(st.item()) == want_status == O.OK
    assert len(got) == 4
    for r in got:
        for a, b in zip(want, r):
            assert torch.equal(a, b)
