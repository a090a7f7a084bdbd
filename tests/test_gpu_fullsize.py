"""Parity at the full workload sizes, in the launch configuration the benchmark
times. Outputs the oracle can compute one by one are compared element by element;
the rest through properties that fix them uniquely (a permutation ordered by
(dest, key) is unique when keys are unique) and closed forms (in a stream a group
is emitted in the step holding its last leaf)."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def log(msg):
    print(f"[fullsize] {msg}", flush=True)


def _group_rows(gk):
    """Input rows of every group (ascending group key): (groups, order, starts, counts)
    with the rows of group i at order[starts[i]:starts[i] + counts[i]]."""
    order = np.argsort(gk, kind="stable")
    groups, starts, counts = np.unique(gk[order], return_index=True, return_counts=True)
    return groups, order, starts, counts


def _oracle_means(payload, rows_of, idx):
    """The oracle's pooled vector of each listed group, one group at a time (rows
    gathered from the device-resident payload with torch indexing)."""
    out = []
    for i in idx:
        r = torch.from_numpy(rows_of(i)).cuda()
        out.append(O.group_mean(payload.index_select(0, r).cpu().numpy()))
    return np.stack(out) if out else np.zeros((0, payload.shape[1]), np.float32)


def _zipf_call(w, keys, n):
    perm = torch.empty(n, dtype=torch.int32, device="cuda")
    offs = torch.empty(w.num_dest + 1, dtype=torch.int64, device="cuda")
    dest = torch.empty(n, dtype=torch.int32, device="cuda")
    out = alto.new_groups(1 << 16, w.agg_level, "mean", w.dim, cap_mask=1 << 16, with_first=False)
    _, _, _, out, st = alto.aggregate(keys, w.fan, w.bits, w.agg_level, "mean", w.dim, w.mask_level,
                                      w.route_level, w.num_dest, None, w.payload_f32, perm=perm,
                                      dest_offsets=offs, dest=dest, out=out, n=n)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return perm, offs, dest, out


def test_zipf_64M_mean_mask():
    log("config: zipf depth-6, 2^26 fragments, 128-d mean at level 4, mask at level 2")
    w = W.zipf_tree("cuda")
    n = w.n
    keys, st = alto.pack_keys(w.path, w.bits)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    hkeys = O.pack_keys(w.path.cpu().numpy(), w.bits)
    assert np.array_equal(keys.cpu().numpy().view(np.uint64), hkeys)
    w.path = None
    perm, offs, dest, out = _zipf_call(w, keys, n)
    log("gpu done; checking routing")
    odest = O.route_dest(hkeys, w.bits, w.route_level, w.num_dest)
    assert np.array_equal(dest.cpu().numpy(), odest)
    assert np.array_equal(offs.cpu().numpy(),
                          np.concatenate([[0], np.cumsum(np.bincount(odest, minlength=w.num_dest))]))
    p = perm.cpu().numpy()
    assert (np.bincount(p, minlength=n) == 1).all()                      # a permutation
    d, k = odest[p], hkeys[p]
    assert ((d[1:] > d[:-1]) | ((d[1:] == d[:-1]) & (k[1:] > k[:-1]))).all()   # strictly by (dest, key)
    del p, d, k
    log("checking groups")
    E, T, M, P = [int(x) for x in out.counts.cpu()]
    gk = O.prefix(hkeys, w.bits, w.agg_level)
    nodes, order, starts, cnt = _group_rows(gk)
    gd = O.route_dest(nodes << np.uint64(O.shift_below(w.bits, w.agg_level)), w.bits, w.route_level,
                      w.num_dest)
    o = np.lexsort((nodes, gd))
    assert (E, P) == (len(nodes), 0)
    assert np.array_equal(out.key[:E].cpu().numpy().view(np.uint64), nodes[o])
    assert np.array_equal(out.count[:E].cpu().numpy(), cnt[o])
    assert np.array_equal(out.dest[:E].cpu().numpy(), gd[o])
    m2 = np.unique(O.prefix(hkeys, w.bits, w.mask_level))
    assert M == len(m2)
    assert np.array_equal(out.mask_key[:M].cpu().numpy().view(np.uint64), m2)
    assert (out.mask[:M].cpu().numpy() == 1).all()
    log(f"checking all {E} means against the oracle")
    rows_of = lambda i: order[starts[o[i]]:starts[o[i]] + cnt[o[i]]]
    U.assert_mean_close(out.mean[:E].cpu().numpy(), _oracle_means(w.payload_f32, rows_of, range(E)))
    # the same batch without its last arrival: one leaf missing leaves its
    # level-5 node, its group and every ancestor incomplete
    log("again without the last fragment in arrival order")
    perm, offs, dest, out = _zipf_call(w, keys, n - 1)
    miss = int(gk[n - 1])
    gi = int(np.searchsorted(nodes, np.uint64(miss)))
    E2, _, M2, P2 = [int(x) for x in out.counts.cpu()]
    keep = o[nodes[o] != np.uint64(miss)]
    assert (E2, P2, M2) == (E - 1, 1, M)
    assert np.array_equal(out.key[:E2].cpu().numpy().view(np.uint64), nodes[keep])
    assert np.array_equal(out.count[:E2].cpu().numpy(), cnt[keep])
    assert out.pend_key[:1].cpu().numpy().view(np.uint64)[0] == miss
    assert int(out.pend_count[0]) == int(cnt[gi]) - 1
    mk = O.prefix(hkeys[n - 1:n], w.bits, w.mask_level)[0]
    mask = out.mask[:M2].cpu().numpy()
    assert np.array_equal(out.mask_key[:M2].cpu().numpy().view(np.uint64), m2)
    assert list(mask) == [0 if k == mk else 1 for k in m2]
    pos = {int(x): j for j, x in enumerate(nodes[o])}
    rng = np.random.default_rng(5)
    picks = rng.choice(E2, size=min(E2, 24), replace=False)
    got = out.mean[:E2].cpu().numpy()[picks]
    U.assert_mean_close(got, _oracle_means(w.payload_f32, rows_of, [pos[int(nodes[keep][j])] for j in picks]))
    p = perm[:n - 1].cpu().numpy()
    assert np.array_equal(np.sort(p), np.arange(n - 1))
    d, k = odest[p], hkeys[p]
    assert ((d[1:] > d[:-1]) | ((d[1:] == d[:-1]) & (k[1:] > k[:-1]))).all()


def test_factool_batch_two_stages():
    log("config: FacTool depth-5, 1,024 queries, 768-d mean per doc, then doc-id concat per claim")
    w = W.factool_batch("cuda")
    path, fan, docid = w.path.cpu().numpy(), w.fan.cpu().numpy(), w.payload_i32.cpu().numpy()
    keys = O.pack_keys(path, w.bits)
    pf = w.payload_f32.cpu().numpy()
    code, rt, g = U.oracle_aggregate(keys, fan, w.bits, 4, "mean", 768, 0, 2, 32, docid, pf)
    assert code == O.OK
    res = U.run_aggregate(keys, fan, w.bits, 4, "mean", 768, 0, 2, 32, docid, pf)
    assert res["status"] == O.OK
    U.compare(res, rt, g, "mean", 0, 4)
    sb = W.FACTOOL_CLAIM_STAGE
    kB, fB, pB = res["key"], res["fan_up"], res["first_i32"]
    code, rtB, gB = U.oracle_aggregate(kB, fB, sb["bits"], 2, "concat", 1, 0, 2, 32, pB)
    assert code == O.OK
    resB = U.run_aggregate(kB, fB, sb["bits"], 2, "concat", 1, 0, 2, 32, pB)
    assert resB["status"] == O.OK
    U.compare(resB, rtB, gB, "concat", 0, 2)


def test_factool_stream_10000_steps():
    log("config: FacTool windowed stream, 10,000 steps x 4,096 fragments, two stages chained on the device")
    w = W.factool_stream("cuda")
    log(f"generated: window {w.info['window']:.0f}, long-lived fraction {w.info['calibrated_frac']:.3f}")
    step, steps = w.step, w.info["steps"]
    ring = w.payload_f32
    ring_rows = ring.shape[0]
    keys_d, st = alto.pack_keys(w.path, w.bits)
    torch.cuda.synchronize()
    hkeys = O.pack_keys(w.path.cpu().numpy(), w.bits)
    hfan = w.fan.cpu().numpy()
    hdoc = w.payload_i32.cpu().numpy()
    assert np.array_equal(keys_d.cpu().numpy().view(np.uint64), hkeys)
    sA = alto.Stream(w.bits, 2, 32, 4, "mean", 768, max_live_leaves=1 << 17, max_groups=1 << 22, step_max=step)
    sbB = W.FACTOOL_CLAIM_STAGE
    sB = alto.Stream(sbB["bits"], 2, 32, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 20,
                     step_max=step)
    # expected: a document is emitted in the step of its last sentence, if all arrived
    gk = O.prefix(hkeys, w.bits, 4)
    stepof = np.arange(w.n) // step
    o = np.argsort(gk, kind="stable")
    docs, first_idx, cnt = np.unique(gk[o], return_index=True, return_counts=True)
    last_step = np.maximum.reduceat(stepof[o], first_idx)
    declared = hfan[3][o][first_idx]
    complete = cnt == declared
    want_step = dict(zip(docs[complete].tolist(), last_step[complete].tolist()))
    full_steps = set(range(0, steps, max(steps // 100, 1)))     # every document and the routing checked
    got_step, got_first, got_count = {}, {}, {}
    step_means = {}
    recB_keys, recB_step = [], []
    claims_got = {}
    gA = alto.new_groups(step, 4, "mean", 768, device="cuda")
    gB = alto.new_groups(step, 2, "concat", 1, cap_tokens=(1 << 16) + step, device="cuda")
    stA, stB = alto.new_status(), alto.new_status()
    perm = torch.empty(step, dtype=torch.int32, device="cuda")
    offs = torch.empty(33, dtype=torch.int64, device="cuda")
    dest = torch.empty(step, dtype=torch.int32, device="cuda")
    checked_route = 0
    for s in range(steps):
        a, b = s * step, (s + 1) * step
        r0 = (s * step) % ring_rows
        stA.zero_()
        full = s in full_steps
        sA.step(keys_d[a:b], w.fan[:, a:b], w.payload_i32[a:b], ring[r0:r0 + step], out=gA, status=stA,
                perm=perm if full else None, dest_offsets=offs if full else None, dest=dest if full else None)
        # stage B takes stage A's records and count on the device (no host read between)
        stB.zero_()
        sB.step(gA.key, gA.fan_up.view(3, -1), gA.first_i32, None, out=gB, status=stB, n=step,
                n_dev=gA.counts[0:1])
        torch.cuda.synchronize()
        assert int(stA.item()) == 0, s
        assert int(stB.item()) == 0, s
        E = int(gA.counts[0])
        if full:
            rt = O.route(hkeys[a:b], w.bits, 2, 32)
            assert np.array_equal(perm.cpu().numpy(), rt.perm), s
            assert np.array_equal(dest.cpu().numpy(), rt.dest), s
            assert np.array_equal(offs.cpu().numpy(), rt.dest_offsets), s
            step_means[s] = (gA.key[:E].cpu().numpy().view(np.uint64).copy(), gA.mean[:E].cpu().numpy())
            checked_route += 1
        ks = gA.key[:E].cpu().numpy().view(np.uint64)
        for kk in ks.tolist():
            got_step[kk] = s
        got_first.update(zip(ks.tolist(), gA.first_i32[:E].cpu().numpy().tolist()))
        got_count.update(zip(ks.tolist(), gA.count[:E].cpu().numpy().tolist()))
        EB, TB = int(gB.counts[0]), int(gB.counts[1])
        kb = gB.key[:EB].cpu().numpy().view(np.uint64)
        toff = gB.tok_off[:EB + 1].cpu().numpy()
        tok = gB.tok[:TB].cpu().numpy()
        for i, kk in enumerate(kb.tolist()):
            claims_got[kk] = (s, tok[toff[i]:toff[i + 1]].tolist())
        if s % 1000 == 0:
            log(f"step {s}: {E} documents, {EB} claims emitted")
    log("checking documents")
    assert got_step == want_step
    doc_first = dict(zip(docs.tolist(), hdoc[o][first_idx].tolist()))
    assert all(got_first[k] == doc_first[k] for k in got_step)
    assert all(got_count[k] == int(c) for k, c in zip(docs[complete].tolist(), cnt[complete].tolist()))
    log(f"checking every document mean of {len(step_means)} steps (routing of those steps: {checked_route})")
    assert len(step_means) >= 100
    ndocs = 0
    for s, (ks, means) in sorted(step_means.items()):
        di = np.searchsorted(docs, ks)
        if len(di) == 0:
            continue
        rows = [o[first_idx[j]:first_idx[j] + cnt[j]] for j in di]
        allrows = np.concatenate(rows)
        x = ring.index_select(0, torch.from_numpy(allrows % ring_rows).cuda()).cpu().numpy()   # one copy per step
        ends = np.cumsum([len(r) for r in rows])
        ref = [O.group_mean(x[e - len(r):e]) for r, e in zip(rows, ends)]
        U.assert_mean_close(means, np.stack(ref))
        ndocs += len(ks)
    log(f"{ndocs} document means checked")
    log("checking claims")
    # a claim is emitted once all its documents were emitted, in the step of the last one
    ck = O.prefix(docs, (31, 3, 2, 3), 2)
    dfan = hfan[:, o][:, first_idx]            # fans of each document's first sentence
    nsq = dfan[1]                               # search queries per claim
    want_claims = {}
    for c in np.unique(ck):
        sel = np.nonzero(ck == c)[0]
        if not complete[sel].all() or len(sel) != int(nsq[sel[0]]) * 5:
            continue
        want_claims[int(c)] = (int(last_step[sel].max()), [doc_first[int(d)] for d in docs[sel]])
    assert claims_got == want_claims
    pend, pst = sA.pending(cap=1 << 17)
    torch.cuda.synchronize()
    P = int(pend.counts[3])
    pk = pend.pend_key[:P].cpu().numpy().view(np.uint64)
    assert set(pk.tolist()) == set(docs[~complete].tolist())
    sA.close()
    sB.close()
