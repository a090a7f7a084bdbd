"""Diagnostics entry points through the C ABI: the streaming read probe."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2403_04311_amd import alto

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("words", [4, 1000, 1 << 20, (1 << 22) + 12])
def test_read_probe_reads_every_word(words):
    # XOR of all 32-bit words, read once by the probe
    rng = np.random.default_rng(words)
    a = rng.integers(0, 2**32, size=words, dtype=np.uint32)
    x = torch.from_numpy(a.view(np.int32)).to("cuda")
    out = torch.full((16384,), -1, dtype=torch.int64, device="cuda")   # every entry is written
    lib = alto.load()
    lib.alto_read_probe.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
    rc = lib.alto_read_probe(C.c_void_p(x.data_ptr()), words * 4, C.c_void_p(out.data_ptr()), None)
    assert rc == 0
    torch.cuda.synchronize()
    want = int(np.bitwise_xor.reduce(a))
    got = int(np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint64)))
    assert got & 0xFFFFFFFF == want
    assert lib.alto_read_probe(C.c_void_p(x.data_ptr()), 12, C.c_void_p(out.data_ptr()), None) == 1
