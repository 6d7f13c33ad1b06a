"""Host-side checks of libmiriam.so (no GPU needed): the library loads and exports
every entry point declared in include/miriam.h, the planner matches the oracle,
and operator descriptors are validated before anything could be launched."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2307_04339_amd import _lib as L
    return L.load()


def _declared_functions():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if not fn.endswith(".h"):
            continue
        src = open(os.path.join(ROOT, "include", fn)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_ ]*[\s\*]+(miriam_[a-z0-9_]+)\s*\(",
                             src, flags=re.M):
            names.add(m.group(1))
    return sorted(names)


def test_header_declares_the_boundary():
    names = _declared_functions()
    for must in ["miriam_elastic_launch", "miriam_submit", "miriam_poll", "miriam_op_create",
                 "miriam_init", "miriam_shutdown", "miriam_plan_dichotomy"]:
        assert must in names


def test_library_exports_every_declared_symbol(lib):
    from paper_2307_04339_amd import _lib as L
    missing = [n for n in _declared_functions() if not hasattr(lib, n)]
    assert missing == []
    # and the binding covers them all
    assert sorted(set(_declared_functions()) - set(L.SIGNATURES)) == []


# ------------------------------------------------------------ planner vs oracle
def test_dichotomy_matches_oracle(lib, orc):
    out = (ctypes.c_int64 * 64)()
    for M in list(range(1, 300)) + [1568, 3136, 6272, 401408]:
        n = lib.miriam_plan_dichotomy(M, out, 64)
        assert list(out[:n]) == orc.dichotomy(M)
    assert lib.miriam_plan_dichotomy(0, out, 64) < 0


def test_split_matches_oracle(lib, orc):
    for T in list(range(1, 60)) + [196, 3136, 10**12 + 7]:
        for n in sorted({1, 2, 3, 4, 7, 8, 16, min(T, 64)}):
            if n > T:
                continue
            b = (ctypes.c_int64 * n)()
            l = (ctypes.c_int64 * n)()
            assert lib.miriam_plan_split(T, n, b, l) == 0
            if T < 10**6:
                assert list(zip(b, l)) == orc.balanced_split(T, n)
            else:  # large T: the partition property (the oracle's product j*T would overflow)
                assert b[0] == 0 and b[n - 1] + l[n - 1] == T
                assert all(b[j] + l[j] == b[j + 1] for j in range(n - 1))


def test_wg_rank_matches_oracle(lib, orc):
    for G in list(range(1, 50)) + [255, 256, 257, 1000]:
        for g in range(G):
            assert lib.miriam_plan_wg_rank(g, G, 8) == orc.wg_rank(g, G, 8)


def test_eq2_wiscore_oscore_match_oracle(lib, orc):
    for n_sm in [8, 30, 256]:
        for n_rt in [0, 1, 49, 255, 256, 300]:
            assert lib.miriam_plan_eq2_grid_limit(n_sm, n_rt) == orc.eq2_grid_limit(n_sm, n_rt)
            for s_rt in [64, 256]:
                assert lib.miriam_plan_eq2_block_limit(2048, s_rt) == orc.eq2_block_limit(2048, s_rt)
                for n_be in [1, 7, 64]:
                    for s_be in [64, 128, 256]:
                        assert lib.miriam_plan_wiscore(n_sm, 2048, n_rt, s_rt, n_be, s_be) == \
                            orc.wiscore(n_sm, 2048, n_rt, s_rt, n_be, s_be)
    for lo_b, lo_p, mb, mp in [([1, 2], [0.5, 0.5], 4.0, 2.0), ([1, 3], [0.5, 0.5], 4.0, 2.0),
                               ([1, 2], [1.0, 1.5], 4.0, 2.0)]:
        a = np.array(lo_b, dtype=np.float64)
        b = np.array(lo_p, dtype=np.float64)
        got = lib.miriam_plan_oscore(len(a), a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                     b.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), mb, mp)
        assert got == orc.oscore(lo_b, lo_p, mb, mp)


def test_top_fraction_matches_oracle(lib, orc):
    rng = np.random.default_rng(3)
    for n in [1, 3, 5, 10, 11, 40]:
        sc = rng.choice([0.0, 0.5, 1.0], n).astype(np.float64)
        gr = rng.choice([8, 64, 256], n).astype(np.int64)
        bl = rng.choice([64, 128, 256], n).astype(np.int64)
        keep = (ctypes.c_int * n)()
        k = lib.miriam_plan_top_fraction(n, sc.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                         gr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                         bl.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 0.2, keep)
        assert list(keep[:k]) == orc.top_fraction(sc, gr, bl, 0.2)


def test_tree_head_matches_oracle(lib, orc):
    d = ctypes.c_int()
    for T in [1, 2, 3, 7, 12, 49, 64, 100, 196]:
        for L_ in [1, 2, 3, 5, 16, T]:
            cur = 0
            while cur < T:
                ln = lib.miriam_plan_tree_head(T, cur, L_, ctypes.byref(d))
                assert (ln, d.value) == orc.tree_head(T, cur, L_)
                cur += ln


# --------------------------------------------------------- descriptor checks
def _desc(**kw):
    from paper_2307_04339_amd import _lib as L
    d = L.OpDesc()
    for k, v in kw.items():
        setattr(d, k, v)
    return d


FAKE = 0x100000  # never dereferenced: creation does not touch device memory


def _create(lib, d):
    h = ctypes.c_void_p()
    rc = lib.miriam_op_create(ctypes.byref(d), ctypes.byref(h))
    return rc, h


def test_op_create_rejects_bad_descriptors(lib):
    from paper_2307_04339_amd import _lib as L
    ok = dict(kind=L.OP_CONV2D, dtype=L.F16, n=1, h=8, w=8, c=16, k=16, kh=3, kw=3, stride=1, pad=1,
              x=FAKE, wt=FAKE, y=FAKE)
    rc, h = _create(lib, _desc(**ok))
    assert rc == 0
    info = L.OpInfo()
    assert lib.miriam_op_query(h, ctypes.byref(info)) == 0
    assert info.num_tiles >= 1 and info.logical_block == 256
    # launch validation happens before any device call
    assert lib.miriam_elastic_launch(h, 0, info.num_tiles + 1, 1, 256, None) == L.ERANGE
    assert lib.miriam_elastic_launch(h, -1, 1, 1, 256, None) == L.ERANGE
    assert lib.miriam_elastic_launch(h, 0, 0, 1, 256, None) == L.ERANGE
    assert lib.miriam_elastic_launch(h, 0, 1, 0, 256, None) == L.ERANGE
    assert lib.miriam_elastic_launch(h, 0, 1, 1, 96, None) == L.ERANGE
    assert lib.miriam_op_destroy(h) == 0
    bad = [dict(ok, kind=99), dict(ok, dtype=7), dict(ok, x=None), dict(ok, stride=0),
           dict(ok, kh=20, pad=0), dict(ok, groups=4), dict(ok, act=9), dict(ok, flags=1),
           dict(ok, flags=64), dict(ok, c=0), dict(ok, tile=7),
           # memory-based index function: pipelined contraction kernel only
           dict(ok, c=64, k=64, h=32, w=32, flags=L.INDEX_MEMORY, tile=8),
           dict(ok, c=3, flags=L.INDEX_MEMORY),  # rows not a 16-byte multiple: staged kernel
           dict(ok, kind=L.OP_DWCONV, k=16, groups=16, kh=3, kw=3, wt=FAKE, flags=L.INDEX_MEMORY)]
    for d in bad:
        rc, _ = _create(lib, _desc(**d))
        assert rc == L.EINVAL, d
    assert lib.miriam_last_error()


@pytest.mark.parametrize("M,N,K,tile,T", [(3136, 64, 576, 1, 98 * 2), (3136, 64, 576, 2, 49),
                                          (3136, 64, 576, 3, 25), (49, 512, 4608, 1, 2 * 16)])
def test_gemm_tile_space(lib, M, N, K, tile, T):
    from paper_2307_04339_amd import _lib as L
    rc, h = _create(lib, _desc(kind=L.OP_GEMM, dtype=L.BF16, m=M, nn=N, kk=K, tile=tile,
                               x=FAKE, wt=FAKE, y=FAKE))
    assert rc == 0
    info = L.OpInfo()
    lib.miriam_op_query(h, ctypes.byref(info))
    assert info.num_tiles == T
    assert info.flops == 2.0 * M * N * K
    lib.miriam_op_destroy(h)


@pytest.mark.parametrize("kind,dtype,geo,addr,path", [
    ("conv", "F16", dict(c=64), FAKE, "PATH_DMA_UNIFORM"),       # chunk = 64 channels = one tap
    ("conv", "F16", dict(c=32), FAKE, "PATH_DMA"),               # chunks straddle taps
    ("conv", "F32", dict(c=32), FAKE, "PATH_DMA_UNIFORM"),       # fp32 chunk is 32 elements
    ("conv", "F16", dict(c=64), FAKE + 2, "PATH_STAGED"),        # operand not 16-byte aligned
    ("conv", "F16", dict(c=3), FAKE, "PATH_STAGED"),             # rows not a 16-byte multiple
    ("gemm", "BF16", dict(m=4, kk=512), FAKE, "PATH_SKINNY"),    # small-batch FC
    ("gemm", "BF16", dict(m=64, kk=512), FAKE, "PATH_DMA_UNIFORM"),
    ("gemm", "BF16", dict(m=64, kk=200), FAKE, "PATH_DMA"),      # K tail inside the last chunk
    ("gemm", "F32", dict(m=4, kk=512), FAKE, "PATH_DMA_UNIFORM"),  # no fp32 skinny kernel
    ("conv", "F16", dict(c=64, tile=7), FAKE, "PATH_HALO"),      # direct 3x3 on request
    ("conv", "F32", dict(c=32, tile=7), FAKE, "PATH_HALO"),      # fp32 chunk is 32 channels
    ("conv", "BF16", dict(n=8, h=112, w=112, c=64, k=64), FAKE, "PATH_RESIDENT"),  # chosen: 784 tiles, N = 64
    ("conv", "F16", dict(n=8, h=112, w=112, c=8, k=64), FAKE, "PATH_RESIDENT"),    # 8-channel image stem
    ("conv", "F32", dict(n=8, h=112, w=112, c=64, k=64), FAKE, "PATH_HALO"),       # no fp32 resident kernel
    ("conv", "F16", dict(n=8, h=112, w=112, c=128, k=64), FAKE, "PATH_HALO"),      # C too wide for registers
    ("conv", "BF16", dict(n=8, h=112, w=112, c=64, k=128), FAKE, "PATH_DMA_UNIFORM"),  # wider: implicit GEMM
    ("conv", "F16", dict(c=64, tile=8), FAKE, "PATH_RESIDENT"),  # resident weights on request
    ("conv", "BF16", dict(c=8, k=20, tile=8), FAKE, "PATH_RESIDENT"),
    ("conv", "BF16", dict(n=16, h=224, w=224, c=8, k=32, stride=2), FAKE, "PATH_RESIDENT"),  # stem 3x3/2
    ("conv", "BF16", dict(n=16, h=112, w=112, c=16, k=96, kh=1, kw=1, pad=0), FAKE, "PATH_RESIDENT"),  # 1x1
    ("conv", "F16", dict(n=16, h=56, w=56, c=24, k=144, kh=1, kw=1, pad=0), FAKE, "PATH_RESIDENT"),
    ("conv", "BF16", dict(n=16, h=56, w=56, c=96, k=24, kh=1, kw=1, pad=0), FAKE, "PATH_DMA"),  # C too wide
    ("conv", "F16", dict(c=24, k=200, kh=1, kw=1, pad=0, tile=8), FAKE, "PATH_RESIDENT"),
])
def test_kernel_path_selection(lib, kind, dtype, geo, addr, path):
    from paper_2307_04339_amd import _lib as L
    if kind == "conv":
        d = dict(kind=L.OP_CONV2D, dtype=getattr(L, dtype), n=1, h=9, w=9, c=16, k=32, kh=3, kw=3,
                 stride=1, pad=1, x=addr, wt=FAKE, y=FAKE)
    else:
        d = dict(kind=L.OP_GEMM, dtype=getattr(L, dtype), m=64, nn=96, kk=64, x=addr, wt=FAKE, y=FAKE)
    d.update(geo)
    rc, h = _create(lib, _desc(**d))
    assert rc == 0, lib.miriam_last_error()
    info = L.OpInfo()
    assert lib.miriam_op_query(h, ctypes.byref(info)) == 0
    assert info.path == getattr(L, path)
    assert info.ksplit >= 1
    lib.miriam_op_destroy(h)


@pytest.mark.parametrize("geo", [dict(c=32), dict(c=64, stride=2), dict(c=64, kh=5, kw=5, pad=2),
                                 dict(c=64, ksplit=2)])
def test_direct3x3_rejects_ineligible_convs(lib, geo):
    from paper_2307_04339_amd import _lib as L
    d = dict(kind=L.OP_CONV2D, dtype=L.F16, n=1, h=9, w=9, c=16, k=32, kh=3, kw=3, stride=1, pad=1,
             x=FAKE, wt=FAKE, y=FAKE, tile=7)
    d.update(geo)
    rc, _ = _create(lib, _desc(**d))
    assert rc == L.EINVAL


@pytest.mark.parametrize("geo", [dict(c=24), dict(c=128), dict(c=64, k=96), dict(c=64, stride=2),
                                 dict(c=64, kh=5, kw=5, pad=2), dict(c=64, ksplit=2), dict(c=64, dtype=0),
                                 dict(c=16, stride=2), dict(c=8, k=96, stride=2), dict(c=8, kh=1, kw=1, pad=0),
                                 dict(c=16, kh=1, kw=1, pad=1), dict(c=16, kh=1, kw=1, pad=0, stride=2)])
def test_resident3x3_rejects_ineligible_convs(lib, geo):
    from paper_2307_04339_amd import _lib as L
    d = dict(kind=L.OP_CONV2D, dtype=L.F16, n=1, h=9, w=9, c=16, k=32, kh=3, kw=3, stride=1, pad=1,
             x=FAKE, wt=FAKE, y=FAKE, tile=8)
    d.update(geo)
    rc, _ = _create(lib, _desc(**d))
    assert rc == L.EINVAL


def test_resident3x3_tile_space_and_full_grid(lib):
    from paper_2307_04339_amd import _lib as L
    # 2 x 15 x 37 output: 4 tile rows x 2 tile columns per image; without a device the
    # whole-tile-space grid stays one workgroup per tile
    rc, h = _create(lib, _desc(kind=L.OP_CONV2D, dtype=L.F16, n=2, h=15, w=37, c=64, k=64, kh=3, kw=3,
                               stride=1, pad=1, x=FAKE, wt=FAKE, y=FAKE, tile=8))
    assert rc == 0, lib.miriam_last_error()
    info = L.OpInfo()
    assert lib.miriam_op_query(h, ctypes.byref(info)) == 0
    assert info.num_tiles == 2 * 4 * 2
    assert (info.tile_m, info.tile_n) == (128, 64)
    assert info.full_grid == info.num_tiles
    lib.miriam_op_destroy(h)
