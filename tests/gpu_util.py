"""Helpers for GPU parity tests: run the HIP path through the C ABI and compare
with the CPU oracle."""
import numpy as np
import torch

from oracle import alto_oracle as O
from paper_2403_04311_amd import alto

DEV = "cuda"


def gpu_available() -> bool:
    return torch.cuda.is_available()


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def pack_gpu(path_np, bits):
    path = to_dev(path_np.astype(np.int32))
    keys, st = alto.pack_keys(path, bits)
    torch.cuda.synchronize()
    return keys, int(st.item())


def run_aggregate(keys_np, fan_np, bits, La, op, dim=1, Lm=0, Lr=0, D=1, p32=None, pf=None,
                  caps=None):
    """Runs alto_aggregate on device copies of numpy inputs; returns numpy outputs."""
    n = len(keys_np)
    keys = to_dev(keys_np.astype(np.uint64).view(np.int64))
    fan = to_dev(fan_np.astype(np.int32)) if fan_np.size else torch.zeros((max(len(bits) - 1, 1), 1),
                                                                            dtype=torch.int32, device=DEV)
    t32 = to_dev(p32.astype(np.int32)) if p32 is not None else None
    tf = to_dev(pf.astype(np.float32)) if pf is not None else None
    cg, ct, cm = caps if caps else (n, n if op == "concat" else 0, max(n, 1) if Lm else 0)
    out = alto.new_groups(cg, La, op, dim, cap_tokens=ct, cap_mask=cm, device=DEV,
                          with_first=p32 is not None)
    perm, offs, dest, out, st = alto.aggregate(keys, fan, bits, La, op, dim, Lm, Lr, D, t32, tf,
                                               out=out, n=n)
    torch.cuda.synchronize()
    status = int(st.item())
    counts = out.counts.cpu().numpy()
    E, T, M, P = [int(x) for x in counts]
    res = {"status": status, "counts": (E, T, M, P)}
    if status != O.OK:
        return res
    res["perm"] = perm[:n].cpu().numpy()
    res["dest_offsets"] = offs.cpu().numpy()
    res["dest"] = dest[:n].cpu().numpy()
    res["key"] = out.key[:E].cpu().numpy().view(np.uint64)
    res["gdest"] = out.dest[:E].cpu().numpy()
    res["count"] = out.count[:E].cpu().numpy()
    if out.first_i32 is not None:
        res["first_i32"] = out.first_i32[:E].cpu().numpy()
    fu = out.fan_up.cpu().numpy()
    res["fan_up"] = np.stack([fu[(l - 1) * cg:(l - 1) * cg + E] for l in range(1, La)]) if La > 1 else None
    if op == "concat":
        res["tok_off"] = out.tok_off[:E + 1].cpu().numpy()
        res["tok"] = out.tok[:T].cpu().numpy()
    else:
        res["mean"] = out.mean[:E].cpu().numpy()
    if Lm:
        res["mask_key"] = out.mask_key[:M].cpu().numpy().view(np.uint64)
        res["mask"] = out.mask[:M].cpu().numpy()
    res["pend_key"] = out.pend_key[:P].cpu().numpy().view(np.uint64)
    res["pend_count"] = out.pend_count[:P].cpu().numpy()
    return res


def oracle_aggregate(keys_np, fan_np, bits, La, op, dim=1, Lm=0, Lr=0, D=1, p32=None, pf=None):
    try:
        rt, g = O.aggregate(keys_np, fan_np, bits, La, op, dim, Lm, Lr, D, p32, pf)
        return O.OK, rt, g
    except O.OracleError as e:
        return e.code, None, None


MEAN_RTOL = 1e-5


def assert_mean_close(got, ref):
    """Per pooled vector: max |g - r| <= 1e-5 * max |r|."""
    assert got.shape == ref.shape
    for i in range(len(ref)):
        scale = float(np.abs(ref[i]).max())
        err = float(np.abs(got[i].astype(np.float64) - ref[i].astype(np.float64)).max())
        assert err <= MEAN_RTOL * scale + 1e-30, (i, err, scale)


def compare(res, rt, g, op, Lm, La):
    assert np.array_equal(res["perm"], rt.perm)
    assert np.array_equal(res["dest"], rt.dest)
    assert np.array_equal(res["dest_offsets"], rt.dest_offsets)
    assert np.array_equal(res["key"], g.key)
    assert np.array_equal(res["gdest"], g.dest)
    assert np.array_equal(res["count"], g.count)
    if g.first_i32 is not None and "first_i32" in res:
        assert np.array_equal(res["first_i32"], g.first_i32)
    if La > 1:
        assert np.array_equal(res["fan_up"], g.fan_up)
    assert np.array_equal(res["pend_key"], g.pend_key)
    assert np.array_equal(res["pend_count"], g.pend_count)
    if op == "concat":
        assert np.array_equal(res["tok_off"], g.tok_off)
        assert np.array_equal(res["tok"], g.tok)
    else:
        assert_mean_close(res["mean"], g.mean)
    if Lm:
        assert np.array_equal(res["mask_key"], g.mask_key)
        assert np.array_equal(res["mask"], g.mask)
