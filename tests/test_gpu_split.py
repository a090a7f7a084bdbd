"""GPU parity of alto_split (split_text at a pmap entry) against the oracle, through
the C ABI."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def run_split(keys, fan, tok, bits, delim, sb, tb):
    """keys: numpy uint64 or a device int64 tensor. Returns status and the outputs
    cut to their counts."""
    n = len(tok)
    dk = keys if torch.is_tensor(keys) else U.to_dev(keys.astype(np.uint64).view(np.int64))
    if n == 0:
        dk = torch.empty(1, dtype=torch.int64, device="cuda")
        df = torch.ones((len(bits) - 1, 1), dtype=torch.int32, device="cuda")
        dt = torch.empty(1, dtype=torch.int32, device="cuda")
    else:
        df = U.to_dev(np.ascontiguousarray(fan).astype(np.int32))
        dt = U.to_dev(np.asarray(tok).astype(np.int32))
    ok, of, otok, oidx, rest, c, st = alto.split(dk, df, dt, bits, delim, sb, tb, n=n)
    torch.cuda.synchronize()
    c = c.cpu().numpy()
    m, r = int(c[0]), int(c[2])
    return {"status": int(st.item()), "counts": c, "keys": ok[:m].cpu().numpy().view(np.uint64),
            "fan": of[:, :m].cpu().numpy(), "tok": otok[:m].cpu().numpy(), "idx": oidx[:m].cpu().numpy(),
            "rest": rest[:r].cpu().numpy()}


def same(got, want, tok):
    assert got["status"] == O.OK
    assert np.array_equal(got["counts"], want.counts)
    assert np.array_equal(got["idx"], want.order)
    assert np.array_equal(got["keys"], want.keys[want.order])
    assert np.array_equal(got["fan"], want.fan[:, want.order])
    assert np.array_equal(got["tok"], np.asarray(tok)[want.order])
    assert np.array_equal(got["rest"], want.rest)


def check(path, fan, tok, bits, delim, sb, tb):
    keys = O.pack_keys(path, bits)
    want = O.split_text(keys, fan, tok, bits, delim, sb, tb)
    same(run_split(keys, fan, tok, bits, delim, sb, tb), want, tok)
    return want


CASES = [
    # seed, bits, max_fan (last: stream length), roots, p_delim, drop, seg_bits, tok_bits
    (1, (6, 10), (40,), 5, 0.2, 0.0, 6, 8),
    (2, (6, 10), (40,), 5, 0.2, 0.1, 6, 8),
    (3, (5, 3, 12), (4, 900), 20, 0.05, 0.0, 8, 10),           # several tiles, multi-block sort
    (4, (5, 3, 12), (4, 900), 20, 0.05, 0.02, 8, 10),
    (5, (31, 3, 2, 14), (4, 3, 3000), 12, 0.01, 0.0, 6, 12),    # long segments, ragged tail
    (6, (8, 4, 4, 6), (6, 9, 30), 40, 0.5, 0.05, 5, 6),         # many delimiters, short segments
    (7, (20, 9), (300,), 700, 0.1, 0.0, 7, 9),                  # many parents
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_split_parity(case):
    seed, bits, mf, roots, pd, drop, sb, tb = CASES[case]
    path, fan, tok = W.random_text(3100 + seed, len(bits), roots, mf, bits, pd, drop)
    w = check(path, fan, tok, bits, W.DELIM_TOKEN, sb, tb)
    assert w.counts[0] > 0


def test_split_gpu_packed_keys():
    # keys packed on the GPU (alto_pack_keys), the oracle packing its own
    path, fan, tok = W.random_text(3200, 3, 30, (5, 200), (9, 4, 9), 0.1, 0.05)
    keys, st = U.pack_gpu(path, (9, 4, 9))
    assert st == O.OK
    want = O.split_text(O.pack_keys(path, (9, 4, 9)), fan, tok, (9, 4, 9), W.DELIM_TOKEN, 6, 8)
    same(run_split(keys, fan, tok, (9, 4, 9), W.DELIM_TOKEN, 6, 8), want, tok)


@pytest.mark.parametrize("kind", ["empty", "one", "one_delim", "all_delims", "no_delims", "edges", "incomplete"])
def test_split_edge_cases(kind):
    bits = (4, 8)
    if kind == "empty":
        got = run_split(np.zeros(0, np.uint64), np.zeros((1, 0), np.int32), np.zeros(0, np.int32), bits, 7, 4, 4)
        assert got["status"] == O.OK and got["counts"].tolist() == [0, 0, 0, 0]
        return
    streams = {
        "one": [[5]],
        "one_delim": [[7]],
        "all_delims": [[7, 7, 7], [7]],
        "no_delims": [[1, 2, 3, 4], [9]],
        "edges": [[7, 1, 1, 7, 7, 2, 7], [7, 7, 3], [3, 7], [7, 3, 7]],
        "incomplete": [[1, 7, 2], [4, 5, 7, 6]],
    }[kind]
    rows = [(p, i, t, len(s)) for p, s in enumerate(streams) for i, t in enumerate(s)]
    if kind == "incomplete":
        rows = [r for r in rows if not (r[0] == 1 and r[1] == 2)]   # stream 1 misses its delimiter
    rows = [rows[i] for i in np.random.default_rng(1).permutation(len(rows))]
    path = np.array([[r[0] for r in rows], [r[1] for r in rows]], np.int32)
    fan = np.array([[r[3] for r in rows]], np.int32)
    tok = np.array([r[2] for r in rows], np.int32)
    check(path, fan, tok, bits, 7, 4, 4)


@pytest.mark.parametrize("kind", ["dup", "fan_disagree", "index", "zero_fan", "layout", "capacity_seg",
                                  "capacity_tok", "dup_and_capacity"])
def test_split_errors(kind):
    bits = (5, 3, 12)
    path, fan, tok = W.random_text(3300, 3, 10, (3, 200), bits, 0.05)
    keys = O.pack_keys(path, bits)
    sb, tb = 8, 10
    if kind in ("dup", "dup_and_capacity"):
        keys, fan, tok = (np.concatenate([keys, keys[3:4]]), np.concatenate([fan, fan[:, 3:4]], axis=1),
                          np.concatenate([tok, tok[3:4]]))
        if kind == "dup_and_capacity":
            tb = 2
    elif kind == "fan_disagree":
        fan = fan.copy()
        fan[1, 5] += 1
    elif kind == "index":
        fan = fan.copy()
        same = O.prefix(keys, bits, 2) == O.prefix(keys[:1], bits, 2)[0]
        fan[1, same] = 1
    elif kind == "zero_fan":
        fan = fan.copy()
        fan[1, O.prefix(keys, bits, 2) == O.prefix(keys[:1], bits, 2)[0]] = 0
    elif kind == "layout":
        keys = keys.copy()
        keys[2] |= np.uint64(1 << 40)
    elif kind == "capacity_seg":
        sb = 1
    elif kind == "capacity_tok":
        tb = 3
    with pytest.raises(O.OracleError) as e:
        O.split_text(keys, fan, tok, bits, W.DELIM_TOKEN, sb, tb)
    assert run_split(keys, fan, tok, bits, W.DELIM_TOKEN, sb, tb)["status"] == e.value.code, kind


def test_split_rejects_bad_arguments():
    lib = alto.load()
    L = alto.layout((4, 8))
    import ctypes as C
    ws = alto.new_workspace(lib.alto_split_workspace_bytes(C.byref(L), 8), "cuda")
    d = torch.zeros(16, dtype=torch.int64, device="cuda")
    p = d.data_ptr()
    for sb, tb in [(0, 4), (4, 0), (33, 4), (40, 20)]:
        rc = lib.alto_split(p, p, 8, p, 8, C.byref(L), 7, sb, tb, p, p, 8, p, p, p, p, p, ws.data_ptr(),
                            ws.numel(), None)
        assert rc == 1, (sb, tb)
    rc = lib.alto_split(p, p, 4, p, 8, C.byref(L), 7, 4, 4, p, p, 8, p, p, p, p, p, ws.data_ptr(), ws.numel(), None)
    assert rc == 1           # fan_ld < n
    rc = lib.alto_split(p, p, 8, p, 8, C.byref(L), 7, 4, 4, p, p, 8, p, p, p, p, p, ws.data_ptr(), 16, None)
    assert rc == 1           # workspace too small


def test_split_token_streams_against_oracle():
    """The 256 generator streams of the token-stream workload (408,190 positions), in
    the launch configuration the benchmark times, element by element."""
    t = W.token_stream_text("cpu")
    path, fan, tok = t.path.numpy(), t.fan.numpy(), t.tokens.numpy()
    w = check(path, fan, tok, t.bits, t.delim, t.seg_bits, t.tok_bits)
    assert w.counts.tolist() == [t.n - 16384, 16384, 0, 16384]


def test_split_scaled_streams_give_back_their_tree():
    """16,384 generator streams (64x the token-stream workload, 26,210,335 positions):
    the new fragments are exactly the (request, sentence, index) tags the streams
    were written from, with their (sentences, sentence length) counts and tokens, in
    key order; sampled parents are checked against the oracle."""
    t = W.token_stream_text("cuda", generators=16384)
    keys, st = alto.pack_keys(t.path, t.bits)
    ok, of, otok, oidx, rest, c, st2 = alto.split(keys, t.fan, t.tokens, t.bits, t.delim, t.seg_bits, t.tok_bits)
    torch.cuda.synchronize()
    assert int(st.item()) == O.OK and int(st2.item()) == O.OK
    placed = t.tree_path[0] >= 0
    nd = int((~placed).sum())
    m = t.n - nd
    assert c.cpu().tolist() == [m, nd, 0, nd]
    idx = oidx[:m].long()
    assert bool(placed[idx].all())
    assert int(torch.unique(idx).numel()) == m                  # every placed position once
    tp = t.tree_path[:, idx].cpu().numpy()
    k = ok[:m].cpu().numpy().view(np.uint64)
    assert np.array_equal(k, O.pack_keys(tp, (31, 6, 12)))
    assert bool((k[1:] > k[:-1]).all())                         # ascending new keys
    assert torch.equal(of[:, :m], t.tree_fan[:, idx])
    assert torch.equal(otok[:m], t.tokens[idx])
    # sampled parents against the oracle, one at a time
    keys_np = keys.cpu().numpy().view(np.uint64)
    fan_np, tok_np = t.fan.cpu().numpy(), t.tokens.cpu().numpy()
    par = O.prefix(keys_np, t.bits, 1)
    rng = np.random.default_rng(9)
    idx_np = idx.cpu().numpy()
    for p in rng.choice(np.unique(par), 8, replace=False):
        sel = np.nonzero(par == p)[0]
        want = O.split_text(keys_np[sel], fan_np[:, sel], tok_np[sel], t.bits, t.delim, t.seg_bits, t.tok_bits)
        rows = np.nonzero(O.prefix(k, (31, 6, 12), 1) == p)[0]
        assert np.array_equal(idx_np[rows], sel[want.order])
        assert np.array_equal(k[rows], want.keys[want.order])
        assert np.array_equal(of[:, rows].cpu().numpy(), want.fan[:, want.order])
