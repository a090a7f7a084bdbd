"""GPU parity of the stream path (alto_stream_*) against the oracle's Stream, step by
step, through the C ABI."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def gpu_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pf, cuts, max_live=4096, max_groups=1 << 16,
              step_max=None, release="complete"):
    """Runs a stream on the GPU; returns per-step dicts of numpy outputs and statuses."""
    step_max = step_max or max(int(np.diff(cuts).max()), 1)
    s = alto.Stream(bits, Lr, D, La, op, dim, max_live_leaves=max_live, max_groups=max_groups,
                    step_max=step_max, release=release)
    dk = U.to_dev(keys.astype(np.uint64).view(np.int64))
    dfan = U.to_dev(fan.astype(np.int32))
    d32 = U.to_dev(p32.astype(np.int32)) if p32 is not None else None
    dpf = U.to_dev(pf.astype(np.float32)) if pf is not None else None
    out = []
    cap_g = step_max
    for a, b in zip(cuts[:-1], cuts[1:]):
        n = b - a
        g = alto.new_groups(cap_g, La, op, dim, cap_tokens=max_live + step_max if op == "concat" else 0,
                            device="cuda", with_first=p32 is not None)
        perm = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
        offs = torch.empty(D + 1, dtype=torch.int64, device="cuda")
        dest = torch.empty(max(n, 1), dtype=torch.int32, device="cuda")
        st = alto.new_status()
        s.step(dk[a:b], dfan[:, a:b], None if d32 is None else d32[a:b], None if dpf is None else dpf[a:b],
               out=g, perm=perm, dest_offsets=offs, dest=dest, status=st, n=n)
        torch.cuda.synchronize()
        E, T, _, _ = [int(x) for x in g.counts.cpu()]
        r = {"status": int(st.item()), "E": E}
        if r["status"] == 0:
            r["perm"] = perm[:n].cpu().numpy()
            r["offs"] = offs.cpu().numpy()
            r["dest"] = dest[:n].cpu().numpy()
            r["key"] = g.key[:E].cpu().numpy().view(np.uint64)
            r["gdest"] = g.dest[:E].cpu().numpy()
            r["count"] = g.count[:E].cpu().numpy()
            if g.first_i32 is not None:
                r["first"] = g.first_i32[:E].cpu().numpy()
            fu = g.fan_up.cpu().numpy()
            r["fan_up"] = (np.stack([fu[(l - 1) * cap_g:(l - 1) * cap_g + E] for l in range(1, La)])
                           if La > 1 else None)
            if op == "concat":
                r["tok_off"] = g.tok_off[:E + 1].cpu().numpy()
                r["tok"] = g.tok[:T].cpu().numpy()
            else:
                r["mean"] = g.mean[:E].cpu().numpy()
        out.append(r)
    pend, pst = s.pending(cap=max_live)
    torch.cuda.synchronize()
    P = int(pend.counts[3])
    pres = {"status": int(pst.item()), "key": pend.pend_key[:P].cpu().numpy().view(np.uint64),
            "count": pend.pend_count[:P].cpu().numpy()}
    s.close()
    return out, pres


def oracle_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pf, cuts, release="complete"):
    s = O.Stream(bits, Lr, D, La, op, dim, release=release)
    res = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        try:
            r = s.step(keys[a:b], fan[:, a:b], None if p32 is None else p32[a:b],
                       None if pf is None else pf[a:b])
            res.append((O.OK, r))
        except O.OracleError as e:
            res.append((e.code, None))
    pend = s.pending() if s.error == 0 else None
    return res, pend


def compare_steps(gpu, ora, op, La):
    (gsteps, gpend), (osteps, opend) = gpu, ora
    assert len(gsteps) == len(osteps)
    for i, (g, (code, o)) in enumerate(zip(gsteps, osteps)):
        assert g["status"] == code, (i, g["status"], code)
        if code != O.OK:
            continue
        assert np.array_equal(g["perm"], o.route.perm), i
        assert np.array_equal(g["offs"], o.route.dest_offsets), i
        assert np.array_equal(g["dest"], o.route.dest), i
        gr = o.groups
        assert np.array_equal(g["key"], gr.key), i
        assert np.array_equal(g["gdest"], gr.dest), i
        assert np.array_equal(g["count"], gr.count), i
        if "first" in g and gr.first_i32 is not None and len(gr.key):
            assert np.array_equal(g["first"], gr.first_i32), i
        if La > 1 and len(gr.key):
            assert np.array_equal(g["fan_up"], gr.fan_up), i
        if op == "concat":
            assert np.array_equal(g["tok_off"], gr.tok_off), i
            assert np.array_equal(g["tok"], gr.tok), i
        else:
            U.assert_mean_close(g["mean"], gr.mean)
    if opend is not None:
        assert gpend["status"] == O.OK
        assert np.array_equal(gpend["key"], opend[0])
        assert np.array_equal(gpend["count"], opend[1])


def _tiny(seed, depth, bits, mf, roots, drop, dim):
    path, fan = W.random_tree(seed, depth, roots, mf, bits)
    if drop:
        path, fan, _ = W.drop_leaves(path, fan, drop, seed + 1)
    rng = np.random.default_rng(seed + 2)
    n = path.shape[1]
    p32 = rng.integers(0, 1 << 30, size=n).astype(np.int32)
    pf = rng.standard_normal((n, dim)).astype(np.float32)
    (path, fan, p32, pft), _ = W.permute([path, fan, p32, pf.T], seed + 3)
    return O.pack_keys(path, bits), fan, p32, np.ascontiguousarray(pft.T)


STREAM_CASES = [
    # depth, bits, max_fan, roots, La, Lr, D, drop, dim, nsteps
    (3, (10, 3, 4), (5, 9), 12, 2, 1, 4, 0.0, 4, 7),
    (4, (31, 2, 3, 4), (4, 8, 16), 30, 3, 2, 9, 0.05, 8, 11),
    (4, (31, 2, 3, 4), (3, 4, 6), 25, 2, 2, 64, 0.0, 16, 5),
    (5, (31, 3, 2, 3, 8), (4, 3, 5, 20), 10, 4, 2, 32, 0.02, 768, 9),
    (5, (31, 3, 2, 3, 8), (3, 3, 5, 10), 10, 3, 1, 7, 0.0, 12, 13),
]


@pytest.mark.parametrize("case", range(len(STREAM_CASES)))
@pytest.mark.parametrize("op", ["concat", "mean"])
def test_stream_parity(case, op):
    depth, bits, mf, roots, La, Lr, D, drop, dim, nsteps = STREAM_CASES[case]
    keys, fan, p32, pf = _tiny(500 + case, depth, bits, mf, roots, drop, dim)
    n = len(keys)
    rng = np.random.default_rng(case)
    cuts = [0] + sorted(rng.choice(np.arange(1, n), size=nsteps - 1, replace=False).tolist()) + [n]
    pfa = pf if op == "mean" else None
    gpu = gpu_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pfa, cuts)
    ora = oracle_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pfa, cuts)
    compare_steps(gpu, ora, op, La)


def test_token_stream_full():
    w = W.token_stream("cpu")
    path, fan, tok = w.path.numpy(), w.fan.numpy(), w.payload_i32.numpy()
    keys = O.pack_keys(path, w.bits)
    cuts = list(range(0, w.n, w.step)) + [w.n]
    gpu = gpu_steps(w.bits, w.route_level, w.num_dest, w.agg_level, "concat", 1, keys, fan, tok, None,
                    cuts, max_live=1 << 14, max_groups=1 << 15, step_max=w.step)
    ora = oracle_steps(w.bits, w.route_level, w.num_dest, w.agg_level, "concat", 1, keys, fan, tok, None,
                       cuts)
    compare_steps(gpu, ora, "concat", w.agg_level)
    # closed form: a sentence is emitted in the step of its last token
    gk = O.prefix(keys, w.bits, 2)
    want = {}
    for i, k in enumerate(gk):
        want[int(k)] = i // w.step
    got = {}
    for si, r in enumerate(gpu[0]):
        for k in r["key"]:
            got[int(k)] = si
    assert got == want


def _windowed_factool(seed, queries, W_frag, step):
    """A small continuous FacTool-shaped stream (same construction as the 10,000-step
    workload, fewer queries)."""
    rng = np.random.default_rng(seed)
    roots = W.distinct_ids(rng, queries)
    fans = W.factool_fans(rng, roots)
    path, fan = W.expand_tree(fans, roots)
    docid = W.doc_ids_per_sentence(rng, fans)
    q = W._leaves_per_root(fans)
    qoff = np.cumsum(q) - q
    pos = np.repeat(qoff, q) + rng.random(path.shape[1]) * W_frag
    order = np.argsort(pos, kind="stable")
    pf = rng.standard_normal((path.shape[1], 768)).astype(np.float32)
    return path[:, order], fan[:, order], docid[order], pf[order]


def gpu_chain(bits, keys, fan, p32, pf, cuts, step_max, max_live, max_groups, release="complete"):
    """The two FacTool stages on the device, step by step, stage B reading stage A's
    emitted count on the device (alto_stream_step_dev): no host read between the
    stages. Returns per-step (stage A dict, stage B dict)."""
    bB = W.FACTOOL_CLAIM_STAGE["bits"]
    sA = alto.Stream(bits, 2, 32, 4, "mean", 768, max_live_leaves=max_live, max_groups=max_groups,
                     step_max=step_max, release=release)
    sB = alto.Stream(bB, 2, 32, 2, "concat", 1, max_live_leaves=max_live, max_groups=max_groups,
                     step_max=step_max, release=release)
    dk = U.to_dev(keys.astype(np.uint64).view(np.int64))
    dfan = U.to_dev(fan.astype(np.int32))
    d32 = U.to_dev(p32.astype(np.int32))
    dpf = U.to_dev(pf.astype(np.float32))
    gA = alto.new_groups(step_max, 4, "mean", 768, device="cuda")
    gB = alto.new_groups(step_max, 2, "concat", 1, cap_tokens=max_live + step_max, device="cuda")
    stA, stB = alto.new_status(), alto.new_status()
    out = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        stA.zero_()
        stB.zero_()
        sA.step(dk[a:b], dfan[:, a:b], d32[a:b], dpf[a:b], out=gA, status=stA, n=b - a)
        sB.step(gA.key, gA.fan_up.view(3, -1), gA.first_i32, None, out=gB, status=stB, n=step_max,
                n_dev=gA.counts[0:1])
        torch.cuda.synchronize()
        E, EB, TB = int(gA.counts[0]), int(gB.counts[0]), int(gB.counts[1])
        out.append(({"status": int(stA.item()), "key": gA.key[:E].cpu().numpy().view(np.uint64),
                     "count": gA.count[:E].cpu().numpy(), "first": gA.first_i32[:E].cpu().numpy(),
                     "mean": gA.mean[:E].cpu().numpy()},
                    {"status": int(stB.item()), "key": gB.key[:EB].cpu().numpy().view(np.uint64),
                     "count": gB.count[:EB].cpu().numpy(), "gdest": gB.dest[:EB].cpu().numpy(),
                     "tok_off": gB.tok_off[:EB + 1].cpu().numpy(), "tok": gB.tok[:TB].cpu().numpy()}))
    sA.close()
    sB.close()
    return out


def compare_chain(got, oA, bB, release):
    """Stage A against the oracle's stream, stage B against the oracle's stream fed
    with stage A's oracle emissions."""
    sB = O.Stream(bB, 2, 32, 2, "concat", 1, release=release)
    assert len(got) == len(oA[0])
    for (ga, gb), (ca, ra) in zip(got, oA[0]):
        assert ca == O.OK and ga["status"] == O.OK and gb["status"] == O.OK
        assert np.array_equal(ga["key"], ra.groups.key)
        assert np.array_equal(ga["count"], ra.groups.count)
        assert np.array_equal(ga["first"], ra.groups.first_i32)
        U.assert_mean_close(ga["mean"], ra.groups.mean)
        rb = sB.step(ra.groups.key, ra.groups.fan_up, ra.groups.first_i32, None)
        assert np.array_equal(gb["key"], rb.groups.key)
        assert np.array_equal(gb["count"], rb.groups.count)
        assert np.array_equal(gb["gdest"], rb.groups.dest)
        assert np.array_equal(gb["tok_off"], rb.groups.tok_off)
        assert np.array_equal(gb["tok"], rb.groups.tok)


def test_factool_stream_two_stages():
    path, fan, docid, pf = _windowed_factool(7, 24, 3000, 256)
    bits = (31, 3, 2, 3, 8)
    keys = O.pack_keys(path, bits)
    n = len(keys)
    cuts = list(range(0, n, 256)) + [n]
    cuts = sorted(set(cuts))
    # stage B consumes stage A's emitted records step by step, on the device
    got = gpu_chain(bits, keys, fan, docid, pf, cuts, 256, 8192, 1 << 14)
    oA = oracle_steps(bits, 2, 32, 4, "mean", 768, keys, fan, docid, pf, cuts)
    compare_chain(got, oA, W.FACTOOL_CLAIM_STAGE["bits"], "complete")
    # and through host-side copies of stage A's records, with per-step routing outputs
    gA = gpu_steps(bits, 2, 32, 4, "mean", 768, keys, fan, docid, pf, cuts, max_live=8192,
                   max_groups=1 << 14, step_max=256)
    compare_steps(gA, oA, "mean", 4)
    bB = W.FACTOOL_CLAIM_STAGE["bits"]
    kB, fB, pB, cB = [], [], [], [0]
    for r in gA[0]:
        kB.append(r["key"])
        fB.append(r["fan_up"])
        pB.append(r["first"])
        cB.append(cB[-1] + len(r["key"]))
    kB = np.concatenate(kB)
    fB = np.concatenate(fB, axis=1)
    pB = np.concatenate(pB)
    gB = gpu_steps(bB, 2, 32, 2, "concat", 1, kB, fB, pB, None, cB, max_live=8192, max_groups=1 << 14,
                   step_max=max(int(np.diff(cB).max()), 1))
    oB = oracle_steps(bB, 2, 32, 2, "concat", 1, kB, fB, pB, None, cB)
    compare_steps(gB, oB, "concat", 2)


@pytest.mark.parametrize("op", ["concat", "mean"])
@pytest.mark.parametrize("drop", [0.0, 0.0002])
def test_stream_long_groups(op, drop):
    """Groups of up to 6,000 leaves carried across steps: long groups (chunks of
    4,096 rows after the first, written by the whole wave; means combined from
    partial sums), next to short ones, element by element against the oracle."""
    bits = (8, 4, 13)
    keys, fan, p32, pf = _tiny(640 + int(drop * 10000), 3, bits, (12, 6000), 2, drop, 8)
    n = len(keys)
    assert n > 4 * 4096
    rng = np.random.default_rng(641)
    cuts = [0] + sorted(rng.choice(np.arange(1, n), size=5, replace=False).tolist()) + [n]
    pfa = pf if op == "mean" else None
    gpu = gpu_steps(bits, 1, 4, 2, op, 8, keys, fan, p32, pfa, cuts, max_live=1 << 16, max_groups=1 << 10)
    ora = oracle_steps(bits, 1, 4, 2, op, 8, keys, fan, p32, pfa, cuts)
    long_emitted = [int((r.groups.count > 4096).sum()) for c, r in ora[0] if c == O.OK]
    assert sum(long_emitted) > 0
    compare_steps(gpu, ora, op, 2)


def _cross_step_case():
    bits = (6, 3, 4)
    path, fan = W.random_tree(41, 3, 6, (4, 9), bits)
    keys = O.pack_keys(path, bits)
    return bits, keys, fan, np.arange(len(keys), dtype=np.int32)


@pytest.mark.parametrize("kind", ["late", "dup_across", "fan_across", "live_capacity", "emit_capacity"])
def test_stream_errors_and_poison(kind):
    bits, keys, fan, p32 = _cross_step_case()
    n = len(keys)
    gk = O.prefix(keys, bits, 2)
    vals, cnt = np.unique(gk, return_counts=True)
    big = vals[np.argmax(cnt)]                      # a group with several leaves
    assert cnt.max() >= 2
    first_group = gk == big
    idx_g = np.nonzero(first_group)[0]
    rest = np.nonzero(~first_group)[0]
    max_live = 4096
    if kind == "late":
        # whole first group, then one of its leaves again, then anything
        order = np.concatenate([idx_g, idx_g[:1], rest])
        cuts = [0, len(idx_g), len(idx_g) + 1, len(order)]
    elif kind == "dup_across":
        # part of a group, then the same leaf again while the group is open
        if len(idx_g) < 2:
            pytest.skip("group too small")
        order = np.concatenate([idx_g[:1], idx_g[:1], idx_g[1:], rest])
        cuts = [0, 1, 2, len(order)]
    elif kind == "fan_across":
        if len(idx_g) < 2:
            pytest.skip("group too small")
        fan = fan.copy()
        fan[1, idx_g[1]] += 1
        order = np.concatenate([idx_g[:1], idx_g[1:], rest])
        cuts = [0, 1, len(idx_g), len(order)]
    elif kind == "live_capacity":
        max_live = 4
        order = np.random.default_rng(3).permutation(n)
        cuts = [0, n // 2, n]
    else:
        # more groups emitted than the stream's max_groups: the live-set update of
        # the step that passes the limit reports it
        max_groups = 2
        order = np.random.default_rng(4).permutation(n)
        cuts = [0, n // 3, 2 * n // 3, n]
    k, f, p = keys[order], fan[:, order], p32[order]
    gpu = gpu_steps(bits, 1, 5, 2, "concat", 1, k, f, p, None, cuts, max_live=max_live,
                    max_groups=max_groups if kind == "emit_capacity" else 1024)
    ora = oracle_steps(bits, 1, 5, 2, "concat", 1, k, f, p, None, cuts)
    codes_g = [r["status"] for r in gpu[0]]
    codes_o = [c for c, _ in ora[0]]
    if kind in ("live_capacity", "emit_capacity"):
        if kind == "emit_capacity":
            # the step whose emissions first take the total past the limit reports it
            assert all(c == O.OK for c in codes_o)
            total = np.cumsum([len(r.groups.key) for _, r in ora[0]])
            assert total[-1] > max_groups
            assert codes_g.index(O.E_CAPACITY) == int(np.argmax(total > max_groups)), (codes_g, total)
        assert O.E_CAPACITY in codes_g
        first = codes_g.index(O.E_CAPACITY)
        assert all(c == O.E_CAPACITY for c in codes_g[first:])       # poisoned
    else:
        assert codes_g == codes_o, (codes_g, codes_o)
        assert codes_o[-1] != O.OK                                    # poisoned after the error


# ---------------------------------------------------------------- in-order release

@pytest.mark.parametrize("case", range(len(STREAM_CASES)))
@pytest.mark.parametrize("op", ["concat", "mean"])
def test_stream_in_order_release_parity(case, op):
    """Children of a parent leave in child-index order (the pmap exit puts its output
    stream back in order); complete groups wait in the carried state."""
    depth, bits, mf, roots, La, Lr, D, drop, dim, nsteps = STREAM_CASES[case]
    keys, fan, p32, pf = _tiny(600 + case, depth, bits, mf, roots, drop, dim)
    n = len(keys)
    rng = np.random.default_rng(100 + case)
    cuts = [0] + sorted(rng.choice(np.arange(1, n), size=nsteps - 1, replace=False).tolist()) + [n]
    pfa = pf if op == "mean" else None
    gpu = gpu_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pfa, cuts, release="in_order")
    ora = oracle_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pfa, cuts, release="in_order")
    compare_steps(gpu, ora, op, La)
    # something was held back at least once (the order differs from completion)
    ora_c = oracle_steps(bits, Lr, D, La, op, dim, keys, fan, p32, pfa, cuts)
    step_of = lambda res: {int(k): i for i, (c, r) in enumerate(res[0]) if c == O.OK for k in r.groups.key}
    assert step_of(ora) != step_of(ora_c)


@pytest.mark.parametrize("Lr", [1, 2])
def test_stream_in_order_release_many_groups(Lr):
    """More groups in one step than one workgroup sorts, with dropped leaves holding
    later siblings back. Route level 2 = aggregation level: siblings sit in several
    destinations and the group records take the multi-block sort; route level 1:
    they are contiguous in the merged run."""
    bits = (10, 8, 4)
    keys, fan, p32, pf = _tiny(71, 3, bits, (60, 3), 400, 0.01, 1)
    n = len(keys)
    cuts = [0, n // 3, n]
    gpu = gpu_steps(bits, Lr, 16, 2, "concat", 1, keys, fan, p32, None, cuts, max_live=1 << 15,
                    max_groups=1 << 15, step_max=n, release="in_order")
    ora = oracle_steps(bits, Lr, 16, 2, "concat", 1, keys, fan, p32, None, cuts, release="in_order")
    assert sum(len(r.groups.key) for c, r in ora[0] if c == O.OK) > 8192
    compare_steps(gpu, ora, "concat", 2)


def test_factool_stream_in_order_two_stages():
    """Documents leave in order within their search query; claims in order within
    their query."""
    path, fan, docid, pf = _windowed_factool(8, 24, 3000, 256)
    bits = (31, 3, 2, 3, 8)
    keys = O.pack_keys(path, bits)
    n = len(keys)
    cuts = sorted(set(list(range(0, n, 256)) + [n]))
    oA = oracle_steps(bits, 2, 32, 4, "mean", 768, keys, fan, docid, pf, cuts, release="in_order")
    got = gpu_chain(bits, keys, fan, docid, pf, cuts, 256, 8192, 1 << 14, release="in_order")
    compare_chain(got, oA, W.FACTOOL_CLAIM_STAGE["bits"], "in_order")
    gA = gpu_steps(bits, 2, 32, 4, "mean", 768, keys, fan, docid, pf, cuts, max_live=8192,
                   max_groups=1 << 14, step_max=256, release="in_order")
    compare_steps(gA, oA, "mean", 4)
    bB = W.FACTOOL_CLAIM_STAGE["bits"]
    kB, fB, pB, cB = [], [], [], [0]
    for r in gA[0]:
        kB.append(r["key"])
        fB.append(r["fan_up"])
        pB.append(r["first"])
        cB.append(cB[-1] + len(r["key"]))
    kB, fB, pB = np.concatenate(kB), np.concatenate(fB, axis=1), np.concatenate(pB)
    gB = gpu_steps(bB, 2, 32, 2, "concat", 1, kB, fB, pB, None, cB, max_live=8192, max_groups=1 << 14,
                   step_max=max(int(np.diff(cB).max()), 1), release="in_order")
    oB = oracle_steps(bB, 2, 32, 2, "concat", 1, kB, fB, pB, None, cB, release="in_order")
    compare_steps(gB, oB, "concat", 2)


def _masked_sum(x, count):
    """Integer sum of the first `count` rows of x (count a device scalar), as int64:
    the same bits give the same sum in any order."""
    n = x.shape[0]
    keep = torch.arange(n, device=x.device) < count
    v = x.reshape(n, -1)
    if v.dtype == torch.float32:
        v = v.view(torch.int32)
    v = v.to(torch.int64)
    return torch.where(keep[:, None], v, torch.zeros_like(v)).sum()


def test_two_stage_stream_pipelined_on_two_hip_streams_matches_sequential():
    """The FacTool-shaped stream's two stages with stage B of step s on a second HIP
    stream beside stage A of step s + 1 (stage A's records double-buffered, events
    between the stages), and each stage's routing on a stream of its own
    (alto_stream_step_overlap): every step's outputs are the same bits as when the
    stages run one after the other on one stream (checksums of the emitted document keys and
    means, and of the claim stage's keys, token offsets and tokens, per step)."""
    from paper_2403_04311_amd import workloads as W
    w = W.factool_stream("cuda", steps=300)
    step, steps = w.step, 300
    ring, ring_rows = w.payload_f32, w.payload_f32.shape[0]
    keys, st = alto.pack_keys(w.path, w.bits)
    sbB = W.FACTOOL_CLAIM_STAGE

    def streams():
        sA = alto.Stream(w.bits, 2, 32, 4, "mean", 768, max_live_leaves=1 << 17, max_groups=1 << 22,
                         step_max=step)
        sB = alto.Stream(sbB["bits"], 2, 32, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 20,
                         step_max=step)
        return sA, sB

    def sums_a(g):
        c = g.counts[0]
        return torch.stack([c, _masked_sum(g.key, c), _masked_sum(g.mean, c)])

    def sums_b(g):
        c, t = g.counts[0], g.counts[1]
        return torch.stack([c, t, _masked_sum(g.key, c), _masked_sum(g.tok_off, c), _masked_sum(g.tok, t)])

    gAs = [alto.new_groups(step, 4, "mean", 768), alto.new_groups(step, 4, "mean", 768)]
    gB = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
    stA, stB = alto.new_status(), alto.new_status()
    # one stream
    sA, sB = streams()
    seq_a, seq_b = [], []
    for s in range(steps):
        a, b = s * step, (s + 1) * step
        r0 = (s * step) % ring_rows
        g = gAs[0]
        sA.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], ring[r0:r0 + step], out=g, status=stA)
        seq_a.append(sums_a(g))
        sB.step(g.key, g.fan_up.view(3, -1), g.first_i32, None, out=gB, status=stB, n=step,
                n_dev=g.counts[0:1])
        seq_b.append(sums_b(gB))
    torch.cuda.synchronize()
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    sA.close()
    sB.close()
    # four streams: stage A's routing (rA) and the rest (main), stage B's routing (rB)
    # and the rest (side)
    sA, sB = streams()
    main = torch.cuda.current_stream()
    side, rA, rB = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    for x in (side, rA, rB):
        x.wait_stream(main)
    a_done = [torch.cuda.Event() for _ in range(2)]
    b_done = [torch.cuda.Event() for _ in range(2)]
    par_a, par_b = [], []
    for s in range(steps):
        k = s & 1
        a, b = s * step, (s + 1) * step
        r0 = (s * step) % ring_rows
        if s >= 2:
            main.wait_event(b_done[k])
        g = gAs[k]
        sA.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], ring[r0:r0 + step], out=g, status=stA, stream=main,
                route_stream=rA)
        par_a.append(sums_a(g))
        a_done[k].record(main)
        # stage B's merge side reads stage A's records only after stage B's routing
        # (on rB, which waits for them) has signalled: side needs no wait of its own
        rB.wait_event(a_done[k])
        with torch.cuda.stream(side):
            sB.step(g.key, g.fan_up.view(3, -1), g.first_i32, None, out=gB, status=stB, n=step,
                    n_dev=g.counts[0:1], stream=side, route_stream=rB)
            par_b.append(sums_b(gB))
        b_done[k].record(side)
    for x in (side, rA, rB):
        main.wait_stream(x)
    torch.cuda.synchronize()
    assert int(stA.item()) == 0 and int(stB.item()) == 0
    sA.close()
    sB.close()
    emitted = int(torch.stack(seq_a)[:, 0].sum())
    assert emitted > 1000
    assert torch.equal(torch.stack(seq_a), torch.stack(par_a))
    assert torch.equal(torch.stack(seq_b), torch.stack(par_b))


def test_overlapped_steps_match_sequential_token_stream():
    """alto_stream_step_overlap (each step's routing on a second HIP stream, beside
    the previous step's merge and emission, two workspaces) gives every step the same
    outputs as alto_stream_step_dev on one stream: the step's perm, dest and
    dest_offsets, the emitted groups (keys, token offsets, tokens) and their counts."""
    from paper_2403_04311_amd import workloads as W
    w = W.token_stream("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, step = w.n, w.step
    nsteps = (n + step - 1) // step

    def run(overlap):
        s = alto.Stream(w.bits, 2, 64, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 16, step_max=step)
        out = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
        status = alto.new_status()
        main = torch.cuda.current_stream()
        route = torch.cuda.Stream()
        route.wait_stream(main)
        res = []
        for i in range(nsteps):
            a, b = i * step, min(n, (i + 1) * step)
            m = b - a
            perm = torch.full((m,), -7, dtype=torch.int32, device="cuda")
            dest = torch.full((m,), -7, dtype=torch.int32, device="cuda")
            offs = torch.full((65,), -7, dtype=torch.int64, device="cuda")
            s.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], None, out=out, status=status, perm=perm,
                   dest=dest, dest_offsets=offs, stream=main, route_stream=route if overlap else None)
            c = out.counts.clone()
            res.append((perm, dest, offs, c, out.key.clone(), out.tok_off.clone(), out.tok.clone()))
        main.wait_stream(route)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        s.close()
        return res
    seq = run(False)
    ovl = run(True)
    total = 0
    for i in range(nsteps):
        (p0, d0, o0, c0, k0, t0, x0), (p1, d1, o1, c1, k1, t1, x1) = seq[i], ovl[i]
        assert torch.equal(p0, p1) and torch.equal(d0, d1) and torch.equal(o0, o1), i
        assert torch.equal(c0, c1), i
        E, T = int(c0[0]), int(c0[1])
        assert torch.equal(k0[:E], k1[:E]) and torch.equal(t0[:E + 1], t1[:E + 1]) and torch.equal(x0[:T], x1[:T]), i
        assert (p0 >= 0).all() and (d0 >= 0).all()
        total += E
    assert total > 10000


@pytest.mark.gpu
@pytest.mark.parametrize("overlap", [False, True])
def test_prepared_steps_match_step(overlap):
    """Stream.prepare (fixed arguments checked once, per-step inputs only) calls the
    same entry point as Stream.step: every step's perm, dest, dest_offsets and
    emitted groups are the same bits, on one stream and with the routing on a
    second one; and it refuses inputs on the wrong device or a step above step_max."""
    from paper_2403_04311_amd import workloads as W
    w = W.token_stream("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, step = w.n, w.step
    nsteps = (n + step - 1) // step

    def run(prepared):
        s = alto.Stream(w.bits, 2, 64, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 16, step_max=step)
        out = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
        status = alto.new_status()
        perm = torch.empty(step, dtype=torch.int32, device="cuda")
        dest = torch.empty(step, dtype=torch.int32, device="cuda")
        offs = torch.empty(65, dtype=torch.int64, device="cuda")
        main = torch.cuda.current_stream()
        route = torch.cuda.Stream() if overlap else None
        if route is not None:
            route.wait_stream(main)
        one = s.prepare(out, status, perm=perm, dest_offsets=offs, dest=dest, stream=main,
                        route_stream=route) if prepared else None
        res = []
        for i in range(nsteps):
            a, b = i * step, min(n, (i + 1) * step)
            m = b - a
            if prepared:
                one(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b])
            else:
                s.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], None, out=out, status=status, perm=perm,
                       dest=dest, dest_offsets=offs, stream=main, route_stream=route)
            c = out.counts.clone()
            res.append((perm[:m].clone(), dest[:m].clone(), offs.clone(), c, out.key.clone(), out.tok_off.clone(),
                        out.tok.clone()))
        if route is not None:
            main.wait_stream(route)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        if prepared:
            with pytest.raises(alto.AltoError):
                one(keys[:step + 1], w.fan[:, :step + 1], w.payload_i32[:step + 1])
            with pytest.raises(alto.AltoError):
                one(keys[:8].cpu(), w.fan[:, :8].cpu(), w.payload_i32[:8].cpu())
        s.close()
        return res
    ref = run(False)
    got = run(True)
    total = 0
    for i in range(nsteps):
        (p0, d0, o0, c0, k0, t0, x0), (p1, d1, o1, c1, k1, t1, x1) = ref[i], got[i]
        assert torch.equal(p0, p1) and torch.equal(d0, d1) and torch.equal(o0, o1), i
        assert torch.equal(c0, c1), i
        E, T = int(c0[0]), int(c0[1])
        assert torch.equal(k0[:E], k1[:E]) and torch.equal(t0[:E + 1], t1[:E + 1]) and torch.equal(x0[:T], x1[:T]), i
        total += E
    assert total > 10000


@pytest.mark.gpu
def test_overlapped_steps_with_empty_steps_match_sequential():
    """alto_stream_step_overlap with empty steps between non-empty ones (a host
    count of 0: nothing is routed and no routing word is signalled for them) keeps
    the workspace alternation and the routing join of the following steps: every
    step's emitted groups are the same bits as on one stream."""
    from paper_2403_04311_amd import workloads as W
    w = W.token_stream("cuda")
    keys, st = alto.pack_keys(w.path, w.bits)
    n, step = w.n, w.step
    nsteps = min((n + step - 1) // step, 40)
    order = []
    for i in range(nsteps):
        order.append(i)
        if i % 3 == 1:
            order.append(None)   # an empty step
            if i % 2 == 1:
                order.append(None)

    def run(overlap):
        s = alto.Stream(w.bits, 2, 64, 2, "concat", 1, max_live_leaves=1 << 16, max_groups=1 << 16, step_max=step)
        out = alto.new_groups(step, 2, "concat", cap_tokens=(1 << 16) + step)
        status = alto.new_status()
        main = torch.cuda.current_stream()
        route = torch.cuda.Stream() if overlap else None
        if route is not None:
            route.wait_stream(main)
        res = []
        for i in order:
            a, b = (0, 0) if i is None else (i * step, min(n, (i + 1) * step))
            s.step(keys[a:b], w.fan[:, a:b], w.payload_i32[a:b], None, out=out, status=status, stream=main,
                   route_stream=route)
            c = out.counts.clone()
            res.append((c, out.key.clone(), out.tok_off.clone(), out.tok.clone()))
        if route is not None:
            main.wait_stream(route)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        s.close()
        return res
    ref, got = run(False), run(True)
    total = 0
    for j in range(len(order)):
        (c0, k0, t0, x0), (c1, k1, t1, x1) = ref[j], got[j]
        assert torch.equal(c0, c1), j
        E, T = int(c0[0]), int(c0[1])
        assert torch.equal(k0[:E], k1[:E]) and torch.equal(t0[:E + 1], t1[:E + 1]) and torch.equal(x0[:T], x1[:T]), j
        total += E
    assert total > 1000
