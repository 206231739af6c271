"""The kernels' contract primitives on the GPU (test helper tests/native/libcontract_check.so,
built by __graft_entry__.build()): the branch-free quantised exponential against the contract's
definition floor(detexp32(x) 2^40) for all 2^32 binary32 inputs, and Philox4x32-10's output
words 0 and 1 against the published known-answer vectors and the oracle."""
import ctypes
import os

import pytest
import torch

HELPER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "libcontract_check.so")


@pytest.mark.gpu
def test_quant_detexp32_equals_contract_for_every_float():
    assert os.path.exists(HELPER), "build the test helper first (__graft_entry__.build())"
    lib = ctypes.CDLL(HELPER)
    f = lib.dbl_test_quant_exhaustive
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    dev = torch.device("cuda:0")
    bad = torch.zeros(1, dtype=torch.int64, device=dev)
    first = torch.full((1,), -1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    print("[contract] quant_detexp32 over all 2^32 inputs", flush=True)
    assert f(bad.data_ptr(), first.data_ptr(), stream) == 0
    torch.cuda.synchronize(dev)
    n, u = int(bad.item()), int(first.item()) & 0xffffffff
    assert n == 0, f"{n} inputs differ, first bit pattern {u:#010x}"


@pytest.mark.gpu
def test_kernel_philox_words_0_and_1():
    """The kernels' Philox4x32-10 against the published known-answer vectors (output words 0
    and 1, the ones the draws use) and against the oracle on random counters and keys."""
    import numpy as np

    from oracle import contract as C
    assert os.path.exists(HELPER), "build the test helper first (__graft_entry__.build())"
    lib = ctypes.CDLL(HELPER)
    f = lib.dbl_test_philox01
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    golden = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                          "philox4x32_10_kat.txt")
    kat = [[int(t, 16) for t in line.split()] for line in open(golden)
           if line.strip() and not line.startswith("#")]
    rng = np.random.default_rng(5)
    rand = rng.integers(0, 2**32, size=(1000, 6), dtype=np.uint64)
    rows = np.concatenate([np.array([r[:6] for r in kat], dtype=np.uint64), rand])
    dev = torch.device("cuda:0")
    inp = torch.from_numpy(rows.astype(np.uint32).view(np.int32)).to(dev)
    out = torch.zeros((len(rows), 2), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    assert f(inp.data_ptr(), out.data_ptr(), len(rows), stream) == 0
    torch.cuda.synchronize(dev)
    got = out.cpu().numpy().view(np.uint32)
    for i, r in enumerate(kat):
        assert (int(got[i, 0]), int(got[i, 1])) == (r[6], r[7])
    for i in range(len(kat), len(rows)):
        w = [int(v) for v in rows[i]]
        want = C.philox4x32_10(w[0:4], w[4:6])
        assert (int(got[i, 0]), int(got[i, 1])) == (want[0], want[1])
