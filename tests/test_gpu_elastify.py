"""Kernels elasticised by the source-to-source transformer, on the GPU: each plain kernel's
elastic form, run as any shard plan (1-8 shards, in random order) under grids of 1, 3, 64 or
shard-length blocks and every allowed physical block, writes bitwise the output of the plain
launch, which matches the CPU oracle (epilogue, max pooling, matrix products and a
two-tap convolution, in float64, rounded once to float32).

Inputs: seeded U[-1, 1] float32 tensors (bias + ReLU over 1000 x 37, max pooling of a
2 x 18 x 22 x 24 image, a 100 x 70 by 70 x 90 product; on 2-D grids and blocks a shifted
sum over a 45 x 70 image and the transpose of a 50 x 37 matrix).  Network kernels written
plainly: a direct 3x3 convolution with bias and ReLU (2 x 9 x 11 x 13 -> 10 channels, strides 1
and 2) and a depthwise 3x3 convolution with bias and ReLU6 (2 x 10 x 13 x 24, inputs in [-4, 4]
so the clamp at 6 is reached), against the oracle's convolution and epilogue; row softmax
(37 x 300, N(0, 3)) and LayerNorm (29 x 200) with shared-memory reductions, which keep their
block, against the oracle's row operators."""
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


# Network kernels written plainly (one output element per thread, or one block per row with
# shared-memory reductions), elasticised by the same transformer.

@pytest.mark.parametrize("stride", [1, 2])
def test_conv3x3_relu(T, stride):
    rng = np.random.default_rng(10 + stride)
    N, H, W, C, K = 2, 9, 11, 13, 10
    x64 = rng.uniform(-1, 1, (N, H, W, C)).astype(np.float32)
    w64 = rng.uniform(-1, 1, (K, 3, 3, C)).astype(np.float32)
    b64 = rng.uniform(-1, 1, K).astype(np.float32)
    x, w, b = _dev(x64), _dev(w64), _dev(b64)
    Ho, Wo = (H - 1) // stride + 1, (W - 1) // stride + 1
    y = torch.empty((N, Ho, Wo, K), dtype=torch.float32, device="cuda")
    G = (N * Ho * Wo * K + 255) // 256
    _check_elastic(lambda G: T.plain_conv3x3_relu_plain_launch(_p(x), _p(w), _p(b), _p(y), N, H, W, C, K, stride,
                                                               G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_conv3x3_relu_elastic_launch(_p(x), _p(w), _p(b), _p(y), N, H, W, C,
                                                                               K, stride, G, 1, b0, l, g, bl, None),
                   y, G, [64, 128, 256], seed=11)
    from oracle import oracle as orc
    ref = orc.conv2d(x64.astype(np.float64), w64.astype(np.float64), stride=stride, pad=1,
                     bias=b64.astype(np.float64), act="relu")
    # 117 fp32 fused multiply-adds per output against the fp64 sum
    assert _rel(y.cpu().numpy(), ref) <= 1e-5


@pytest.mark.parametrize("stride", [1, 2])
def test_dwconv3x3_relu6(T, stride):
    rng = np.random.default_rng(20 + stride)
    N, H, W, C = 2, 10, 13, 24
    # scaled so that some outputs pass 6 and the clamp is exercised
    x64 = rng.uniform(-4, 4, (N, H, W, C)).astype(np.float32)
    w64 = rng.uniform(-1, 1, (C, 3, 3)).astype(np.float32)
    b64 = rng.uniform(-1, 1, C).astype(np.float32)
    x, w, b = _dev(x64), _dev(w64), _dev(b64)
    Ho, Wo = (H - 1) // stride + 1, (W - 1) // stride + 1
    y = torch.empty((N, Ho, Wo, C), dtype=torch.float32, device="cuda")
    G = (N * Ho * Wo * C + 255) // 256
    _check_elastic(lambda G: T.plain_dwconv3x3_relu6_plain_launch(_p(x), _p(w), _p(b), _p(y), N, H, W, C, stride,
                                                                  G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_dwconv3x3_relu6_elastic_launch(_p(x), _p(w), _p(b), _p(y), N, H, W,
                                                                                  C, stride, G, 1, b0, l, g, bl, None),
                   y, G, [64, 128, 256], seed=21)
    from oracle import oracle as orc
    ref = orc.conv2d(x64.astype(np.float64), w64.astype(np.float64).reshape(C, 3, 3, 1), stride=stride, pad=1,
                     groups=C, bias=b64.astype(np.float64), act="relu6")
    got = y.cpu().numpy()
    assert (ref >= 6.0).any() and (ref <= 0.0).any()
    assert _rel(got, ref) <= 1e-5


def test_softmax_rows_keeps_its_block(T):
    rng = np.random.default_rng(30)
    rows, n = 37, 300  # the row is longer than the block: each thread reduces two strided values
    x64 = rng.normal(0, 3, (rows, n)).astype(np.float32)
    x = _dev(x64)
    y = torch.empty((rows, n), dtype=torch.float32, device="cuda")
    _check_elastic(lambda G: T.plain_softmax_rows_plain_launch(_p(x), _p(y), rows, n, G, 1, None),
                   lambda G, b0, l, g, bl: T.plain_softmax_rows_elastic_launch(_p(x), _p(y), rows, n, G, 1, b0, l, g,
                                                                               bl, None),
                   y, rows, [256], seed=31)
    from oracle import oracle as orc
    ref = orc.softmax_rows(x64.astype(np.float64), 1.0)
    assert _rel(y.cpu().numpy(), ref) <= 1e-5


def test_layernorm_rows_keeps_its_block(T):
    rng = np.random.default_rng(40)
    rows, n, eps = 29, 200, 1e-5
    x64 = rng.normal(0.5, 2, (rows, n)).astype(np.float32)
    g64 = rng.uniform(0.5, 1.5, n).astype(np.float32)
    b64 = rng.uniform(-1, 1, n).astype(np.float32)
    x, g, b = _dev(x64), _dev(g64), _dev(b64)
    y = torch.empty((rows, n), dtype=torch.float32, device="cuda")
    _check_elastic(lambda G: T.plain_layernorm_rows_plain_launch(_p(x), _p(g), _p(b), _p(y), rows, n, eps, G, 1, None),
                   lambda G, b0, l, gr, bl: T.plain_layernorm_rows_elastic_launch(_p(x), _p(g), _p(b), _p(y), rows, n,
                                                                                  eps, G, 1, b0, l, gr, bl, None),
                   y, rows, [128], seed=41)
    from oracle import oracle as orc
    ref = orc.layernorm_rows(x64.astype(np.float64), g64.astype(np.float64), b64.astype(np.float64), eps)
    assert _rel(y.cpu().numpy(), ref) <= 1e-5
