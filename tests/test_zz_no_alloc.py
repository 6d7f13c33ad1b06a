"""The no-alloc creation entry point (miriam_op_create_noalloc), through the C ABI: ops whose
split-K workspace lives in the library's static device scratch give bitwise the output of the
same ops created with miriam_op_create (same kernels, same reduction order), on two calls in a
row, the second with a smaller input; sizes beyond the scratch are rejected."""
import ctypes

import numpy as np
import pytest
import torch

from gpu_util import RTOL, bits, empty, gpu_available, rand, rel_err, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


def _create(L, desc, noalloc):
    h = ctypes.c_void_p()
    fn = L.load().miriam_op_create_noalloc if noalloc else L.load().miriam_op_create
    rc = fn(ctypes.byref(desc), ctypes.byref(h))
    return rc, h


def _info(L, h):
    info = L.OpInfo()
    L.check(L.load().miriam_op_query(h, ctypes.byref(info)), "miriam_op_query")
    return info


def _run(L, h, T, grid, stream):
    L.check(L.load().miriam_elastic_launch(h, 0, T, grid, 256, stream), "miriam_elastic_launch")


def _pair(L, desc_of, y_ref, y_na):
    """Create the op both ways over separate outputs, run each whole, return both infos."""
    rc, h_ref = _create(L, desc_of(y_ref), False)
    assert rc == 0, L.load().miriam_last_error()
    rc, h_na = _create(L, desc_of(y_na), True)
    assert rc == 0, L.load().miriam_last_error()
    try:
        i_ref, i_na = _info(L, h_ref), _info(L, h_na)
        assert i_ref.ksplit == i_na.ksplit and i_na.ksplit > 1 and i_ref.num_tiles == i_na.num_tiles
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        _run(L, h_ref, i_ref.num_tiles, i_ref.full_grid, st)
        _run(L, h_na, i_na.num_tiles, i_na.full_grid, st)
        # a sharded pass over the no-alloc op as well (the counters return to zero after each pass)
        from oracle import oracle as orc
        for (b, l) in orc.balanced_split(int(i_na.num_tiles), 3):
            L.check(L.load().miriam_elastic_launch(h_na, b, l, 5, 128, st), "miriam_elastic_launch")
        torch.cuda.synchronize()
        return i_na
    finally:
        assert L.load().miriam_op_destroy(h_ref) == 0
        assert L.load().miriam_op_destroy(h_na) == 0


def test_noalloc_skinny_split_k_matches_allocating_create(orc):
    from paper_2307_04339_amd import _lib as L
    from paper_2307_04339_amd import ops
    for (M, N, K) in [(8, 1000, 8192), (4, 300, 2048)]:  # second call smaller
        x, x64 = rand((M, K), "f16", 40 + M)
        w, w64 = rand((N, K), "f16", 41 + M, -0.05, 0.05)
        y_ref, y_na = empty((M, N), "f16"), empty((M, N), "f16")

        def desc_of(y):
            d = L.OpDesc()
            d.kind, d.dtype, d.act = L.OP_GEMM, L.F16, L.ACT_CODE["relu"]
            d.m, d.nn, d.kk = M, N, K
            d.tile, d.ksplit = 5, 4
            d.x, d.wt, d.y = x.data_ptr(), w.data_ptr(), y.data_ptr()
            return d
        _pair(L, desc_of, y_ref, y_na)
        assert bits(y_na) == bits(y_ref)
        assert rel_err(to_f64(y_na), orc.linear(x64, w64, act="relu")) <= RTOL["f16"]


def test_noalloc_conv_split_k_matches_allocating_create(orc):
    from paper_2307_04339_amd import _lib as L
    for (H, C, K) in [(7, 512, 512), (5, 256, 64)]:  # second call smaller
        x, x64 = rand((1, H, H, C), "bf16", 50 + H)
        w, w64 = rand((K, 3, 3, C), "bf16", 51 + H, -0.05, 0.05)
        y_ref, y_na = empty((1, H, H, K), "bf16"), empty((1, H, H, K), "bf16")

        def desc_of(y):
            d = L.OpDesc()
            d.kind, d.dtype, d.act = L.OP_CONV2D, L.BF16, L.ACT_CODE["relu"]
            d.n, d.h, d.w, d.c, d.k, d.kh, d.kw, d.stride, d.pad = 1, H, H, C, K, 3, 3, 1, 1
            d.tile, d.ksplit = 2, 3
            d.x, d.wt, d.y = x.data_ptr(), w.data_ptr(), y.data_ptr()
            return d
        _pair(L, desc_of, y_ref, y_na)
        assert bits(y_na) == bits(y_ref)
        ref = orc.conv2d(x64, w64, stride=1, pad=1, act="relu")
        assert rel_err(to_f64(y_na), ref) <= RTOL["bf16"]


def test_noalloc_rejects_what_does_not_fit():
    from paper_2307_04339_amd import _lib as L
    K = 1 << 18
    x = torch.zeros((16, K), dtype=torch.float16, device="cuda")
    w = torch.zeros((4096, K), dtype=torch.float16, device="cuda")
    y = torch.zeros((16, 4096), dtype=torch.float16, device="cuda")
    d = L.OpDesc()
    d.kind, d.dtype = L.OP_GEMM, L.F16
    d.m, d.nn, d.kk = 16, 4096, K
    d.tile, d.ksplit = 5, 512  # 512 slices of every output tile: 128 MiB of partials, beyond the scratch
    d.x, d.wt, d.y = x.data_ptr(), w.data_ptr(), y.data_ptr()
    rc, h = _create(L, d, True)
    assert rc == L.ERANGE, rc
    assert b"scratch" in L.load().miriam_last_error()
    d.flags = L.INDEX_MEMORY
    d.tile, d.ksplit = 2, 1
    d.kind, d.m, d.nn, d.kk = L.OP_GEMM, 64, 64, 64
    rc, h = _create(L, d, True)
    assert rc == L.EINVAL, rc
