"""The allocation-free sampling entry point (lede_op_sample_noalloc) against
lede_op_sample, row by row, through the C ABI: two calls in a row on the
same device array, the second with fewer and shorter rows, and a call with a
row stride past the row length.  The draws are integers: bit-exact."""
import ctypes

import numpy as np
import pytest

import lede_inputs as li
from tests.parity import say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _rows(n, V, seed, scale=3.0):
    z = li.normal(seed, 70, n * V, scale, "f32").reshape(n, V)
    return torch.from_numpy(z).to("cuda")


def _reference(z, T, u):
    from paper_2606_03113_amd import op_sample
    return [op_sample(z[r], T, float(u[r])) for r in range(z.shape[0])]


def test_noalloc_sampling_matches_allocating_entry_point():
    from paper_2606_03113_amd import op_sample_noalloc
    for n, V, T, seed in ((20, 32000, 0.6, 1), (5, 1000, 0.05, 2)):
        say("noalloc sampling rows=%d V=%d T=%g" % (n, V, T))
        z = _rows(n, V, seed)
        u = li.uniform01(seed, 71, n)
        got = op_sample_noalloc(z, T, u)
        assert got == _reference(z, T, u)


def test_noalloc_row_stride_and_limits():
    from paper_2606_03113_amd import load, op_sample_noalloc
    from paper_2606_03113_amd.lede import LEDE_E_ARG
    L = load()
    n, V, ld = 32, 1025, 1031
    say("noalloc sampling rows=%d V=%d ld=%d" % (n, V, ld))
    zf = _rows(n, ld, 3)
    u = li.uniform01(3, 72, n)
    out = np.zeros(n, dtype=np.int32)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    up = u.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
    op = out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert L.lede_op_sample_noalloc(zf.data_ptr(), n, ld, V, 0.6, up, op, s) == 0
    assert out.tolist() == _reference(zf[:, :V].contiguous(), 0.6, u)
    # more rows than the static key array holds, a stride below the row length,
    # a bad temperature or uniform: refused before anything runs
    u33 = np.full(33, 0.5, dtype=np.float32)
    assert L.lede_op_sample_noalloc(zf.data_ptr(), 33, ld, V, 0.6, u33.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                    op, s) == LEDE_E_ARG
    assert L.lede_op_sample_noalloc(zf.data_ptr(), n, V - 1, V, 0.6, up, op, s) == LEDE_E_ARG
    assert L.lede_op_sample_noalloc(zf.data_ptr(), n, ld, V, 0.0, up, op, s) == LEDE_E_ARG
    bad = u.copy()
    bad[3] = 1.0
    assert L.lede_op_sample_noalloc(zf.data_ptr(), n, ld, V, 0.6, bad.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                    op, s) == LEDE_E_ARG
    # the array still serves a smaller call afterwards
    z2 = _rows(2, 64, 4)
    u2 = li.uniform01(4, 73, 2)
    assert op_sample_noalloc(z2, 1.0, u2) == _reference(z2, 1.0, u2)
