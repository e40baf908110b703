"""The matrix-core rate probe (libutdiag.so) does the work it reports: with
every operand 1.0 each lane's accumulator sum is 16384 per iteration for
both MFMA shapes, and the clock counters advance."""
import ctypes
import os

import pytest
import torch

import paper_2609_23169_amd as ut

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [0, 1])
def test_mfma_rate_probe_accumulates_exactly(shape):
    lib = ctypes.CDLL(os.path.join(os.path.dirname(ut.__file__), "libutdiag.so"))
    f = lib.ut_diag_mfma_rate
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int] * 3 + [ctypes.c_void_p] * 4
    grid, iters = 8, 3
    ones = torch.ones(grid * 256 * 128, dtype=torch.bfloat16, device="cuda")
    out = torch.full((grid * 256,), -1.0, dtype=torch.float32, device="cuda")
    clk = torch.zeros(2, dtype=torch.int64, device="cuda")
    st = f(shape, iters, grid, ones.data_ptr(), out.data_ptr(), clk.data_ptr(),
           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0
    torch.cuda.synchronize()
    assert torch.all(out == 16384.0 * iters)
    c = clk.cpu().tolist()
    assert c[0] > 0 and c[1] > 0
