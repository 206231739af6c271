"""The sampler's and verifier's branch-free quantised exponential against the determinism
contract's definition, floor(detexp32(x) 2^40), for all 2^32 binary32 inputs (GPU test helper
tests/native/libcontract_check.so, built by __graft_entry__.build())."""
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
