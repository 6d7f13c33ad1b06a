"""Kernels elasticised by the source-to-source transformer, on the GPU: each plain kernel's
elastic form, run as any shard plan (1-8 shards, in random order) under grids of 1, 3, 64 or
shard-length blocks and every allowed physical block, writes bitwise the output of the plain
launch, which matches the CPU oracle (epilogue, max pooling, matrix products and a
two-tap convolution, in float64, rounded once to float32).

Inputs: seeded U[-1, 1] float32 tensors (bias + ReLU over 1000 x 37, max pooling of a
2 x 18 x 22 x 24 image, a 100 x 70 by 70 x 90 product; on 2-D grids and blocks a shifted
sum over a 45 x 70 image and the transpose of a 50 x 37 matrix)."""
import numpy as np
import pytest
import torch

from gpu_util import bits, gpu_available

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


@pytest.fixture(scope="module")
def T():
    from paper_2307_04339_amd.transform import lib
    return lib.load()


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def _p(t):
    return t.data_ptr()


def _f32(a64):
    return np.asarray(a64, dtype=np.float64).astype(np.float32)


def _rel(g, o):
    from gpu_util import rel_err
    return rel_err(np.asarray(g, dtype=np.float64), o)


def _check_elastic(launch_plain, launch_elastic, y, G, blocks, seed):
    from oracle import oracle as orc
    y.fill_(float("nan"))
    assert launch_plain(G) == 0
    torch.cuda.synchronize()
    ref = bits(y)
    rng = np.random.default_rng(seed)
    for n in [1, 2, 3, 5, 8]:
        if n > G:
            continue
        y.fill_(float("nan"))
        plan = orc.balanced_split(G, n)
        for j in rng.permutation(n):
            b, l = plan[j]
            grid = int(rng.choice([1, 3, 64, l]))
            block = int(rng.choice(blocks))
            assert launch_elastic(G, b, l, grid, block) == 0
        torch.cuda.synchronize()
        assert bits(y) == ref, n
    return ref


def test_bias_relu(T):
    rng = np.random.default_rng(0)
    n_rows, c = 1000, 37
    x64 = rng.uniform(-1, 1, (n_rows, c)).astype(np.float32)
    b64 = rng.uniform(-1, 1, c).astype(np.float32)
    x, b = _dev(x64), _dev(b64)
    y = torch.empty((n_rows, c), dtype=torch.float32, device="cuda")
    n = n_rows * c
    G = (n + 255) // 256
    _check_elastic(lambda G: T.plain_bias_relu_plain_launch(_p(x), _p(b), _p(y), n, c, G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_bias_relu_elastic_launch(_p(x), _p(b), _p(y), n, c, G, 1, b0, l, g, bl,
                                                                             None),
                   y, G, [64, 128, 256], seed=1)
    from oracle import oracle as orc
    # one fp32 add and a ReLU: the correctly rounded sum, so the oracle rounded once matches bitwise
    ref = orc.epilogue(x64.astype(np.float64), bias=b64.astype(np.float64), act="relu")
    assert np.array_equal(y.cpu().numpy(), _f32(ref))


def test_maxpool2(T):
    rng = np.random.default_rng(2)
    N, H, W, C = 2, 18, 22, 24
    x64 = rng.uniform(-1, 1, (N, H, W, C)).astype(np.float32)
    x = _dev(x64)
    y = torch.empty((N, H // 2, W // 2, C), dtype=torch.float32, device="cuda")
    G = 7  # a grid-stride kernel: 7 logical blocks of 128 threads cover all 4752 outputs
    _check_elastic(lambda G: T.plain_maxpool2_plain_launch(_p(x), _p(y), N, H, W, C, G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_maxpool2_elastic_launch(_p(x), _p(y), N, H, W, C, G, 1, b0, l, g, bl,
                                                                           None),
                   y, G, [64, 128], seed=3)
    from oracle import oracle as orc
    ref = orc.maxpool(x64.astype(np.float64), 2, 2, 0)
    assert np.array_equal(y.cpu().numpy(), _f32(ref))


def test_tiled_gemm_keeps_its_block(T):
    rng = np.random.default_rng(4)
    M, N, K = 100, 90, 70
    a64 = rng.uniform(-1, 1, (M, K)).astype(np.float32)
    b64 = rng.uniform(-1, 1, (K, N)).astype(np.float32)
    A, B = _dev(a64), _dev(b64)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    G = ((M + 15) // 16) * ((N + 15) // 16)
    _check_elastic(lambda G: T.plain_tiled_gemm_plain_launch(_p(A), _p(B), _p(C), M, N, K, G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_tiled_gemm_elastic_launch(_p(A), _p(B), _p(C), M, N, K, G, 1, b0, l,
                                                                             g, bl, None),
                   C, G, [256], seed=5)
    from oracle import oracle as orc
    ref = orc.gemm_nn(a64.astype(np.float64), b64.astype(np.float64))
    assert _rel(C.cpu().numpy(), ref) <= 1e-4


def test_shift_add2d_on_a_2d_grid(T):
    rng = np.random.default_rng(6)
    R, Cc, a = 45, 70, 0.75
    x64 = rng.uniform(-1, 1, (R, Cc)).astype(np.float32)
    x = _dev(x64)
    y = torch.empty((R, Cc), dtype=torch.float32, device="cuda")
    gx, gy = (Cc + 31) // 32, (R + 7) // 8  # 32 x 8 blocks
    _check_elastic(lambda G: T.plain_shift_add2d_plain_launch(_p(x), _p(y), R, Cc, a, gx, gy, None),
                   lambda G, b0, l, g, bl: T.plain_shift_add2d_elastic_launch(_p(x), _p(y), R, Cc, a, gx, gy, b0, l,
                                                                              g, bl, None),
                   y, gx * gy, [64, 128, 256], seed=7)
    from oracle import oracle as orc
    # y[i, j] = a x[i, j] + x[i, j + 1] (0 past the last column): a 1 x 2 convolution with taps
    # (a, 1) over the image with one zero column appended
    xz = np.zeros((1, R, Cc + 1, 1))
    xz[0, :, :Cc, 0] = x64
    w = np.array([a, 1.0]).reshape(1, 1, 2, 1)
    ref = orc.conv2d(xz, w, stride=1, pad=0)[0, :, :, 0]
    assert ref.shape == (R, Cc)
    assert _rel(y.cpu().numpy(), ref) <= 1e-4


def test_transpose16_keeps_its_2d_block(T):
    rng = np.random.default_rng(8)
    R, Cc = 50, 37
    x64 = rng.uniform(-1, 1, (R, Cc)).astype(np.float32)
    x = _dev(x64)
    y = torch.empty((Cc, R), dtype=torch.float32, device="cuda")
    gx, gy = (Cc + 15) // 16, (R + 15) // 16
    _check_elastic(lambda G: T.plain_transpose16_plain_launch(_p(x), _p(y), R, Cc, gx, gy, None),
                   lambda G, b0, l, g, bl: T.plain_transpose16_elastic_launch(_p(x), _p(y), R, Cc, gx, gy, b0, l, g,
                                                                              bl, None),
                   y, gx * gy, [256], seed=9)
    from oracle import oracle as orc
    # the transpose as the exact product I x^T
    ref = orc.gemm_nt(np.eye(Cc), x64.astype(np.float64))
    assert np.array_equal(y.cpu().numpy(), _f32(ref))
