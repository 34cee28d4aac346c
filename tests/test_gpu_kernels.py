"""Kernel-level parity of the tiled linear kernels (the draft path's vector
kernel and the verify path's matrix-core kernel) against the oracle's fp64
matvec, at small ragged shapes and at the full projection shapes of the
Llama-2-7B / Llama-3-8B / Llama-2-13B / Llama-2-70B configurations."""
import numpy as np
import pytest

import lede_inputs as li
from oracle.model import matvec
from tests.parity import say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _inputs(N, K, M, dtype, seed):
    W = li.normal(seed, 7, N * K, 0.02, dtype).reshape(N, K)
    x = li.normal(seed, 8, M * K, 1.0, dtype).reshape(M, K)
    return W, x


def _dev(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(a).to("cuda")


def _f64(a, dtype):
    return li.bf16_to_f32(a).astype(np.float64) if dtype == "bf16" else a.astype(np.float64)


def _check(N, K, M, dtype, mfma, seed=0, rows=None):
    from paper_2606_03113_amd import op_linear
    say("linear N=%d K=%d M=%d %s %s" % (N, K, M, dtype, "mfma" if mfma else "vec"))
    W, x = _inputs(N, K, M, dtype, seed)
    y = op_linear(_dev(W, dtype), _dev(x, dtype), mfma).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    sel = np.arange(N) if rows is None else rows
    ref = matvec(W[sel], _f64(x, dtype), dtype == "bf16")
    bound = np.abs(_f64(W[sel], dtype)) @ np.abs(_f64(x, dtype)).T  # [rows][M]
    err = np.abs(y[:, sel] - ref)
    tol = 1e-5 * bound.T + 1e-7
    assert np.all(err <= tol), "max err %.3g (tol %.3g)" % (err.max(), tol.max())


# K past the last whole tile: 688 and 1000 (bf16 tiles of 32 columns), 1000
# and 40 (fp32 tiles of 16); the tiles' zero padding meets the rows' padding
RAGGED = [(64, 688), (48, 1000), (16, 40), (256, 11000)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,K", [(16, 32), (48, 96), (64, 1184), (688, 256), (256, 704), (1024, 4096)] + RAGGED)
def test_linear_vec_small(dtype, N, K):
    _check(N, K, 1, dtype, mfma=False)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M", [1, 2, 5, 9, 16])
@pytest.mark.parametrize("N,K", [(16, 32), (48, 96), (64, 1184), (256, 704)] + RAGGED)
def test_linear_mfma_small(dtype, M, N, K):
    _check(N, K, M, dtype, mfma=True)


def test_ragged_k_is_ragged():
    for N, K in RAGGED:
        assert K % 32 or K % 16


FULL = [
    ("7b-qkv", 12288, 4096), ("7b-o", 4096, 4096), ("7b-gateup", 22016, 4096), ("7b-down", 4096, 11008),
    ("7b-head", 32000, 4096), ("8b-qkv", 6144, 4096), ("8b-down", 4096, 14336), ("8b-head", 128256, 4096),
    ("13b-down", 5120, 13824), ("70b-down", 8192, 28672),
]


@pytest.mark.parametrize("name,N,K", FULL, ids=[f[0] for f in FULL])
def test_linear_full_shapes(name, N, K):
    rows = np.random.default_rng(1).choice(N, 256, replace=False)
    _check(N, K, 1, "bf16", mfma=False, rows=np.sort(rows))
    _check(N, K, 5, "bf16", mfma=True, rows=np.sort(rows))


def test_mfma_rows_independent_of_batch():
    """A row's matrix-core result does not depend on the other rows."""
    from paper_2606_03113_amd import op_linear
    W, x = _inputs(512, 4096, 9, "bf16", 3)
    Wd, xd = _dev(W, "bf16"), _dev(x, "bf16")
    y9 = op_linear(Wd, xd, True)
    for m in (0, 4, 8):
        y1 = op_linear(Wd, xd[m:m + 1].contiguous(), True)
        assert torch.equal(y1[0], y9[m])


@pytest.mark.parametrize("n_words,grid", [(4, 1), (1000, 3), (1 << 20, 4096), ((1 << 20) + 12, 257)])
def test_read_probe_reads_every_word(n_words, grid):
    """The bandwidth probe touches every 16-byte chunk exactly once: the XOR
    of its per-block results equals the XOR of all words."""
    from paper_2606_03113_amd import op_read_probe, load
    import ctypes
    words = li.uniform_int(5, 9, n_words, 0, (1 << 31) - 1).view(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to("cuda")
    sink = torch.zeros(grid, dtype=torch.int32, device="cuda")
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert load().lede_op_read_probe(buf.data_ptr(), n_words * 4, sink.data_ptr(), grid, s, None) == 0
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(words)
    assert op_read_probe(buf) > 0


@pytest.mark.parametrize("n_groups,tiles", [(1, 1), (3, 37), (256, 128), (17, 344)])
def test_read_groups_reads_every_word(n_groups, tiles):
    """The group-structured read probe touches every word of its groups once
    (ragged batches included): the XOR of its per-block results equals the
    XOR of all words, and nothing past the groups is read into it."""
    from paper_2606_03113_amd import op_read_groups, load
    import ctypes
    n_words = n_groups * tiles * 256
    words = li.uniform_int(5, 10, n_words + 256, 0, (1 << 31) - 1).view(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to("cuda")
    sink = torch.zeros(n_groups, dtype=torch.int32, device="cuda")
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert load().lede_op_read_groups(buf.data_ptr(), n_groups, tiles, sink.data_ptr(), s, None) == 0
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(words[:n_words])
    assert op_read_groups(buf, n_groups, tiles) > 0
