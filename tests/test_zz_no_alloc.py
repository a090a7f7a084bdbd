"""alto_aggregate_noalloc (workspace in the library's fixed device array) against
alto_aggregate (caller workspace) through the C ABI: two calls in a row on one
GPU, the second with a smaller input, each compared with alto_aggregate on the
same input. The fixed array keeps what the first call left; the second call must
not depend on it."""
import numpy as np
import pytest
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto, workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


def _inputs(seed, roots, drop):
    bits = (3, 12, 12, 12, 12, 12)
    path, fan = W.random_tree(seed, 6, roots, (2, 3, 4, 60, 40), bits)
    if drop:
        path, fan, _ = W.drop_leaves(path, fan, drop, seed + 1)
    rng = np.random.default_rng(seed + 2)
    n = path.shape[1]
    p32 = rng.integers(-(2**31), 2**31 - 1, size=n).astype(np.int32)
    pf = rng.standard_normal((n, 128)).astype(np.float32)
    (path, fan, p32, pft), _ = W.permute([path, fan, p32, pf.T], seed + 3)
    return bits, O.pack_keys(path, bits), fan, p32, np.ascontiguousarray(pft.T)


def _run(fn_noalloc, bits, keys, fan, p32, pf, op):
    n = len(keys)
    dim = 128 if op == "mean" else 1
    dk = U.to_dev(keys.view(np.int64))
    df = U.to_dev(fan.astype(np.int32))
    d32 = U.to_dev(p32)
    dpf = U.to_dev(pf) if op == "mean" else None
    perm = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    offs = torch.full((257,), -7, dtype=torch.int64, device="cuda")
    dest = torch.full((n,), -7, dtype=torch.int32, device="cuda")
    out = alto.new_groups(n, 4, op, dim, cap_tokens=n if op == "concat" else 0, cap_mask=n, device="cuda")
    st = alto.new_status()
    if fn_noalloc:
        alto.aggregate_noalloc(dk, df, bits, 4, op, dim, 2, 4, 256, d32, dpf, perm=perm, dest_offsets=offs,
                               dest=dest, out=out, status=st)
    else:
        alto.aggregate(dk, df, bits, 4, op, dim, 2, 4, 256, d32, dpf, perm=perm, dest_offsets=offs, dest=dest,
                       out=out, status=st)
    torch.cuda.synchronize()
    E, T, M, P = [int(x) for x in out.counts.cpu()]
    r = {"status": int(st.item()), "counts": (E, T, M, P), "perm": perm.cpu().numpy(),
         "offs": offs.cpu().numpy(), "dest": dest.cpu().numpy(),
         "key": out.key[:E].cpu().numpy(), "gdest": out.dest[:E].cpu().numpy(),
         "count": out.count[:E].cpu().numpy(), "first": out.first_i32[:E].cpu().numpy(),
         "fan_up": out.fan_up.view(3, -1)[:, :E].cpu().numpy(),
         "mask_key": out.mask_key[:M].cpu().numpy(), "mask": out.mask[:M].cpu().numpy(),
         "pend_key": out.pend_key[:P].cpu().numpy(), "pend_count": out.pend_count[:P].cpu().numpy()}
    if op == "mean":
        r["mean"] = out.mean[:E].cpu().numpy()
    else:
        r["tok_off"] = out.tok_off[:E + 1].cpu().numpy()
        r["tok"] = out.tok[:T].cpu().numpy()
    return r


@pytest.mark.parametrize("op", ["mean", "concat"])
def test_noalloc_matches_workspace_entry_point_twice(op):
    big = _inputs(41, 3, 0.01)
    small = _inputs(42, 1, 0.02)
    assert len(small[1]) < len(big[1]) and len(big[1]) > 8192     # multi-block sort on the first call
    need = alto.workspace_bytes(big[0], len(big[1]), 256, 4, op, 128 if op == "mean" else 1, 2)
    assert need <= alto.NOALLOC_SCRATCH_BYTES
    print(f"[noalloc] op={op} n={len(big[1])} then n={len(small[1])}", flush=True)
    for bits, keys, fan, p32, pf in (big, small):
        a = _run(True, bits, keys, fan, p32, pf, op)
        b = _run(False, bits, keys, fan, p32, pf, op)
        assert a["status"] == O.OK and b["status"] == O.OK
        assert a["counts"] == b["counts"]
        for k in b:
            if k in ("status", "counts"):
                continue
            if k == "mean":
                U.assert_mean_close(a[k], b[k])
            else:
                assert np.array_equal(a[k], b[k]), k
        # and both against the oracle
        code, rt, g = U.oracle_aggregate(keys, fan, bits, 4, op, 128 if op == "mean" else 1, 2, 4, 256, p32,
                                         pf if op == "mean" else None)
        assert code == O.OK
        assert np.array_equal(a["perm"], rt.perm) and np.array_equal(a["key"].view(np.uint64), g.key)
        if op == "mean":
            U.assert_mean_close(a["mean"], g.mean)
        else:
            assert np.array_equal(a["tok"], g.tok)
