"""GPU parity of the elastic implicit-GEMM convolution against the CPU oracle,
bitwise invariance across elastic configurations, and the device tile map.

The single-conv workload: x 1x64x56x56 and w 64x64x3x3 ~ U[-1,1] (seed 0),
bias ~ U[-1,1], stride 1, pad 1, ReLU, fp32; run unsharded and as 1/2/4/8
shards with blocks of 64/128/256 threads, in forward and reverse shard order.
"""
import numpy as np
import pytest
import torch

from gpu_util import RTOL, bits, empty, f32_dev, gpu_available, ints, rand, rel_err, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


@pytest.fixture(scope="module")
def ops():
    from paper_2307_04339_amd import ops as o
    return o


def _cfg1(ops, tile=0, dtype="f32"):
    x, x64 = rand((1, 56, 56, 64), dtype, seed=0)
    w, w64 = rand((64, 3, 3, 64), dtype, seed=1)
    b64 = np.random.default_rng(2).uniform(-1, 1, 64)
    bias = f32_dev(b64)
    y = empty((1, 56, 56, 64), dtype)
    op = ops.conv2d(x, w, y, stride=1, pad=1, bias=bias, act="relu", tile=tile)
    return op, y, (x64, w64, b64.astype(np.float32).astype(np.float64))


def _persistent_grid(op, block, n_cu=256):
    cap = max(1, op.info.max_wg_per_cu[{64: 0, 128: 1, 256: 2}[block]])
    return n_cu * cap


def test_conv_cfg1_matches_oracle(ops, orc):
    op, y, (x64, w64, b64) = _cfg1(ops)
    op.run()
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, stride=1, pad=1, bias=b64, act="relu")
    err = rel_err(to_f64(y), ref)
    print(f"cfg1 conv fp32: T={op.T} tile={op.info.tile_m} rel={err:.3e}")
    assert err <= RTOL["f32"]


@pytest.mark.parametrize("tile", [1, 2, 3, 4, 7])
def test_conv_cfg1_bitwise_across_elastic_configs(ops, orc, tile):
    op, y, _ = _cfg1(ops, tile=tile)
    op.run()
    torch.cuda.synchronize()
    ref_bits = bits(y)
    T = op.T
    for n in [1, 2, 4, 8]:
        if n > T:
            continue
        plan = orc.balanced_split(T, n)
        for block in [64, 128, 256]:
            for order in ["fwd", "rev"]:
                for gmode in ["persistent", "one-per-tile", "tiny"]:
                    y.fill_(float("nan"))
                    seq = list(range(n)) if order == "fwd" else list(reversed(range(n)))
                    for j in seq:
                        b, l = plan[j]
                        g = {"persistent": min(l, _persistent_grid(op, block)),
                             "one-per-tile": l, "tiny": 3}[gmode]
                        op.launch(b, l, g, block)
                    torch.cuda.synchronize()
                    assert bits(y) == ref_bits, (tile, n, block, order, gmode)


@pytest.mark.parametrize("tile", [1, 7])
def test_conv_tile_map_matches_oracle(ops, orc, tile):
    op, y, _ = _cfg1(ops, tile=tile)
    T = op.T
    for n, grids, block in [(1, [T], 256), (4, [5, 64, 1, 33], 128), (3, [7, 7, 7], 64),
                            (8, [256] * 8, 256)]:
        plan = orc.balanced_split(T, n)
        ow = torch.full((T,), -1, dtype=torch.int32, device="cuda")
        oi = torch.full((T,), -1, dtype=torch.int32, device="cuda")
        cnt = torch.zeros((T,), dtype=torch.int32, device="cuda")
        for (b, l), g in zip(plan, grids):
            op.launch_traced(b, l, g, block, ow, oi, cnt)
        torch.cuda.synchronize()
        _, wg_ref, it_ref, cnt_ref = orc.owner_map(T, plan, grids)
        assert np.array_equal(cnt.cpu().numpy(), cnt_ref)
        assert np.array_equal(ow.cpu().numpy(), wg_ref)
        assert np.array_equal(oi.cpu().numpy(), it_ref)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_conv_integer_inputs_exact(ops, orc, dtype):
    # integer operands in {-2..2}: every partial sum is an integer below 2^11, so
    # fp32 accumulation is exact and GPU == oracle bit for bit (fp16 output exact up to 2048)
    x, x64 = ints((1, 12, 12, 32), dtype, seed=3, lo=-2, hi=2)
    w, w64 = ints((16, 3, 3, 32), dtype, seed=4, lo=-2, hi=2)
    y = empty((1, 12, 12, 16), dtype)
    op = ops.conv2d(x, w, y, stride=1, pad=1)
    op.run()
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, stride=1, pad=1)
    assert np.abs(ref).max() < 2048
    assert np.array_equal(to_f64(y), ref)


CASES = [
    # N, H, W, C, K, KH, stride, pad, act, epilogue
    (1, 56, 56, 64, 64, 3, 1, 1, "relu", "bn"),
    (1, 224, 224, 3, 64, 7, 2, 3, "relu", "bn"),      # ResNet stem: element loads (C=3)
    (2, 17, 13, 32, 48, 3, 2, 1, "none", "bias"),     # ragged tiles
    (1, 14, 14, 256, 512, 1, 2, 0, "none", "bn"),     # 1x1 downsample
    (2, 7, 7, 96, 40, 1, 1, 0, "relu6", "bn_res"),    # residual, K not a tile multiple
    (1, 9, 9, 24, 144, 1, 1, 0, "relu6", "bn"),       # C = 24 (not a chunk multiple)
    (2, 15, 15, 128, 64, 3, 2, 1, "relu", "bn"),      # two chunks per tap, stride 2, padding
    (1, 12, 12, 64, 40, 5, 1, 2, "none", "bias"),     # 5x5 taps, one chunk per tap (16-bit)
]


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("case", CASES)
def test_conv_shapes_match_oracle(ops, orc, dtype, case):
    N, H, W, C, K, KH, s, p, act, epi = case
    seed = abs(hash(case)) % 1000
    x, x64 = rand((N, H, W, C), dtype, seed=seed)
    w, w64 = rand((K, KH, KH, C), dtype, seed=seed + 1, lo=-0.2, hi=0.2)
    Ho, Wo = (H + 2 * p - KH) // s + 1, (W + 2 * p - KH) // s + 1
    rng = np.random.default_rng(seed + 2)
    bias = bn = res = None
    b64 = bn64 = r64 = None
    if "bias" in epi:
        b64 = rng.uniform(-1, 1, K).astype(np.float32).astype(np.float64)
        bias = f32_dev(b64)
    if "bn" in epi:
        g_, be_ = rng.uniform(0.8, 1.2, K), rng.uniform(-0.1, 0.1, K)
        mu, var = rng.uniform(-0.1, 0.1, K), rng.uniform(0.8, 1.2, K)
        bn64 = np.stack([g_, be_, mu, var]).astype(np.float32).astype(np.float64)
        bn = f32_dev(bn64)
    if "res" in epi:
        res, r64 = rand((N, Ho, Wo, K), dtype, seed=seed + 3)
    y = empty((N, Ho, Wo, K), dtype)
    for tile in [1, 2, 3, 4]:
        y.fill_(float("nan"))
        op = ops.conv2d(x, w, y, stride=s, pad=p, bias=bias, bn=bn, residual=res, act=act, tile=tile)
        op.run()
        torch.cuda.synchronize()
        ref = orc.conv2d(x64, w64, stride=s, pad=p, bias=b64,
                         bn=None if bn64 is None else tuple(bn64), residual=r64, act=act)
        err = rel_err(to_f64(y), ref)
        assert err <= RTOL[dtype], (tile, err)


# ---------------------------------------------------------------- split K
SPLIT_CASES = [
    # N, H, W, C, K, KH, stride, pad, ksplit   (deep K over few output tiles)
    (1, 7, 7, 512, 512, 3, 1, 1, 8),
    (1, 14, 14, 256, 256, 3, 1, 1, 3),
    (2, 7, 7, 64, 96, 3, 1, 1, 2),
    (1, 7, 7, 512, 512, 3, 1, 1, 0),   # library choice
]


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("case", SPLIT_CASES)
def test_conv_split_k_matches_oracle_and_is_elastic(ops, orc, dtype, case):
    N, H, W, C, K, KH, s, p, ks = case
    seed = abs(hash(case)) % 1000
    x, x64 = rand((N, H, W, C), dtype, seed=seed)
    w, w64 = rand((K, KH, KH, C), dtype, seed=seed + 1, lo=-0.05, hi=0.05)
    rng = np.random.default_rng(seed + 2)
    bn64 = np.stack([rng.uniform(0.8, 1.2, K), rng.uniform(-0.1, 0.1, K),
                     rng.uniform(-0.1, 0.1, K), rng.uniform(0.8, 1.2, K)]).astype(np.float32).astype(np.float64)
    Ho, Wo = (H + 2 * p - KH) // s + 1, (W + 2 * p - KH) // s + 1
    res, r64 = rand((N, Ho, Wo, K), dtype, seed=seed + 3)
    y = empty((N, Ho, Wo, K), dtype)
    op = ops.conv2d(x, w, y, stride=s, pad=p, bn=f32_dev(bn64), residual=res, act="relu", ksplit=ks)
    if ks == 0:
        # library choice: 1 x 7 x 7 x 512 output at 32x32 tiles is 32 output tiles (under a
        # quarter of a tile per CU) over 72 (fp16) or 144 (fp32) K chunks: 4 slices
        assert op.info.ksplit == 4 and op.T == 32 * 4
    else:
        assert op.info.ksplit == ks
        assert op.T % ks == 0
    op.run()
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, stride=s, pad=p, bn=tuple(bn64), residual=r64, act="relu")
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    ref_bits = bits(y)
    # any shard plan, order, grid and block: the last slice to arrive reduces in fixed order
    rng = np.random.default_rng(seed + 4)
    for n in [1, 2, 3, 5, 8]:
        if n > op.T:
            continue
        plan = orc.balanced_split(op.T, n)
        order = rng.permutation(n)
        for j in order:
            b, l = plan[j]
            op.launch(b, l, int(rng.choice([1, 3, 64, l])), int(rng.choice([64, 128, 256])))
        torch.cuda.synchronize()
        assert bits(y) == ref_bits, (n, order)
    # repeated passes leave the arrival counters clean
    for _ in range(3):
        op.run()
    torch.cuda.synchronize()
    assert bits(y) == ref_bits


# ------------------------------------------------ direct 3x3 kernel (tile 7)
HALO_CASES = [
    # N, H, W, C, K, pad, act, epilogue
    (2, 15, 37, 128, 64, 1, "relu", "bn"),       # ragged tile rows and columns, two 16-bit chunks
    (1, 9, 70, 64, 96, 1, "none", "bias"),       # ragged n tile (96 = 64 + 32), three tile columns
    (1, 30, 33, 64, 64, 0, "relu6", "bn_res"),   # no padding (28 x 31 output), residual
    (3, 8, 32, 192, 40, 1, "none", "bn"),        # odd number of chunks, K < 64, batch 3
]


def _halo_inputs(case, dtype):
    N, H, W, C, K, p, act, epi = case
    seed = abs(hash(case)) % 1000
    x, x64 = rand((N, H, W, C), dtype, seed=seed)
    w, w64 = rand((K, 3, 3, C), dtype, seed=seed + 1, lo=-0.2, hi=0.2)
    Ho, Wo = H + 2 * p - 2, W + 2 * p - 2
    rng = np.random.default_rng(seed + 2)
    bias = bn = res = None
    b64 = bn64 = r64 = None
    if "bias" in epi:
        b64 = rng.uniform(-1, 1, K).astype(np.float32).astype(np.float64)
        bias = f32_dev(b64)
    if "bn" in epi:
        bn64 = np.stack([rng.uniform(0.8, 1.2, K), rng.uniform(-0.1, 0.1, K), rng.uniform(-0.1, 0.1, K),
                         rng.uniform(0.8, 1.2, K)]).astype(np.float32).astype(np.float64)
        bn = f32_dev(bn64)
    if "res" in epi:
        res, r64 = rand((N, Ho, Wo, K), dtype, seed=seed + 3)
    y = empty((N, Ho, Wo, K), dtype)
    ref_args = dict(stride=1, pad=p, bias=b64, bn=None if bn64 is None else tuple(bn64), residual=r64, act=act)
    return (x, w, y, dict(stride=1, pad=p, bias=bias, bn=bn, residual=res, act=act)), (x64, w64, ref_args)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("case", HALO_CASES)
def test_conv_direct3x3_matches_oracle_and_is_elastic(ops, orc, dtype, case):
    from paper_2307_04339_amd import _lib as L
    (x, w, y, kw), (x64, w64, rargs) = _halo_inputs(case, dtype)
    op = ops.conv2d(x, w, y, tile=7, **kw)
    assert op.info.path == L.PATH_HALO
    op.run()
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, **rargs)
    err = rel_err(to_f64(y), ref)
    assert err <= RTOL[dtype], err
    ref_bits = bits(y)
    rng = np.random.default_rng(7)
    for n in [2, 3, 5]:
        if n > op.T:
            continue
        plan = orc.balanced_split(op.T, n)
        for j in rng.permutation(n):
            b, l = plan[j]
            op.launch(b, l, int(rng.choice([1, 2, 7, l])), int(rng.choice([64, 128, 256])))
        torch.cuda.synchronize()
        assert bits(y) == ref_bits, n


def test_conv_direct3x3_chosen_for_wide_layers(ops):
    from paper_2307_04339_amd import _lib as L
    # a 112 x 112 x 64 -> 64 layer at batch 8: 896 tiles, one n tile; fp16 keeps the weights
    # in registers, fp32 streams them through the LDS-patch kernel
    x, _ = rand((8, 112, 112, 64), "f16", seed=0)
    w, _ = rand((64, 3, 3, 64), "f16", seed=1, lo=-0.05, hi=0.05)
    y = empty((8, 112, 112, 64), "f16")
    op = ops.conv2d(x, w, y, stride=1, pad=1)
    assert op.info.path == L.PATH_RESIDENT
    assert 1 <= op.info.full_grid <= op.T
    xf, _ = rand((8, 112, 112, 64), "f32", seed=0)
    wf, _ = rand((64, 3, 3, 64), "f32", seed=1, lo=-0.05, hi=0.05)
    yf = empty((8, 112, 112, 64), "f32")
    assert ops.conv2d(xf, wf, yf, stride=1, pad=1).info.path == L.PATH_HALO
    # stride 2 keeps the implicit GEMM
    y2 = empty((8, 56, 56, 64), "f16")
    assert ops.conv2d(x, w, y2, stride=2, pad=1).info.path not in (L.PATH_HALO, L.PATH_RESIDENT)


# ------------------------------------ direct 3x3 kernel, weights in registers (tile 8)
RW_CASES = [
    # N, H, W, C, K, pad, act, epilogue
    (2, 15, 37, 64, 64, 1, "relu", "bn"),        # ragged tile rows and columns
    (1, 9, 70, 8, 64, 1, "relu", "bias"),        # 8-channel input: two taps per MFMA step, K = 72
    (1, 30, 33, 64, 64, 0, "relu6", "bn_res"),   # no padding (28 x 31 output), residual
    (3, 8, 32, 16, 40, 1, "none", "bn"),         # C = 16, K < 64 (upper channel half partly idle)
    (2, 11, 20, 32, 24, 1, "gelu", "bias"),      # C = 32, only the lower channel half
    (1, 6, 40, 8, 20, 1, "relu", "bias_res"),    # K not a multiple of 8: element stores
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", RW_CASES)
def test_conv_resident3x3_matches_oracle_and_is_elastic(ops, orc, dtype, case):
    from paper_2307_04339_amd import _lib as L
    (x, w, y, kw), (x64, w64, rargs) = _halo_inputs(case, dtype)
    op = ops.conv2d(x, w, y, tile=8, **kw)
    assert op.info.path == L.PATH_RESIDENT
    op.launch(0, op.T, op.T, 256)  # one workgroup per tile
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, **rargs)
    err = rel_err(to_f64(y), ref)
    print(f"resident 3x3 {dtype} {case}: T={op.T} rel={err:.3e}")
    assert err <= RTOL[dtype], err
    ref_bits = bits(y)
    y.fill_(float("nan"))
    op.run()  # full grid
    torch.cuda.synchronize()
    assert bits(y) == ref_bits
    rng = np.random.default_rng(7)
    for n in [1, 2, 3, 5]:
        if n > op.T:
            continue
        for block in [64, 128, 256]:
            y.fill_(float("nan"))
            plan = orc.balanced_split(op.T, n)
            for j in rng.permutation(n):
                b, l = plan[j]
                op.launch(b, l, int(rng.choice([1, 2, 7, l])), block)
            torch.cuda.synchronize()
            assert bits(y) == ref_bits, (n, block)


# 1x1 and 3x3 stride-2 shapes of the resident-weight kernel (N, H, W, C, K, ks, stride, pad, act, epi)
RW_SHAPES = [
    (2, 23, 70, 8, 32, 3, 2, 1, "relu6", "bn"),      # image stem: 3x3 / 2 on 8 channels, ragged
    (1, 16, 33, 8, 64, 3, 2, 1, "relu", "bias"),     # even input size, full 64 channels
    (2, 9, 40, 16, 96, 1, 1, 0, "relu6", "bn"),      # 1x1 expand, two n tiles (96 = 64 + 32)
    (1, 12, 37, 24, 144, 1, 1, 0, "relu6", "bn"),    # 1x1, C = 24 (half-masked last step), 3 n tiles
    (3, 7, 33, 32, 16, 1, 1, 0, "none", "bn_res"),   # 1x1 project with residual, one n tile
    (1, 10, 20, 64, 200, 1, 1, 0, "gelu", "bias"),   # 1x1, 4 n tiles, ragged last one
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("case", RW_SHAPES)
def test_conv_resident_shapes_match_oracle_and_are_elastic(ops, orc, dtype, case):
    from paper_2307_04339_amd import _lib as L
    N, H, W, C, K, ks, st, p, act, epi = case
    seed = abs(hash(case)) % 1000
    x, x64 = rand((N, H, W, C), dtype, seed=seed)
    w, w64 = rand((K, ks, ks, C), dtype, seed=seed + 1, lo=-0.2, hi=0.2)
    Ho, Wo = (H + 2 * p - ks) // st + 1, (W + 2 * p - ks) // st + 1
    rng = np.random.default_rng(seed + 2)
    bias = bn = res = None
    b64 = bn64 = r64 = None
    if "bias" in epi:
        b64 = rng.uniform(-1, 1, K).astype(np.float32).astype(np.float64)
        bias = f32_dev(b64)
    if "bn" in epi:
        bn64 = np.stack([rng.uniform(0.8, 1.2, K), rng.uniform(-0.1, 0.1, K), rng.uniform(-0.1, 0.1, K),
                         rng.uniform(0.8, 1.2, K)]).astype(np.float32).astype(np.float64)
        bn = f32_dev(bn64)
    if "res" in epi:
        res, r64 = rand((N, Ho, Wo, K), dtype, seed=seed + 3)
    y = empty((N, Ho, Wo, K), dtype)
    op = ops.conv2d(x, w, y, stride=st, pad=p, bias=bias, bn=bn, residual=res, act=act, tile=8)
    assert op.info.path == L.PATH_RESIDENT
    assert op.T == N * ((Ho + 3) // 4) * ((Wo + 31) // 32) * ((K + 63) // 64)
    op.launch(0, op.T, op.T, 256)
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, stride=st, pad=p, bias=b64, bn=None if bn64 is None else tuple(bn64),
                     residual=r64, act=act)
    err = rel_err(to_f64(y), ref)
    print(f"resident {ks}x{ks}/{st} {dtype} {case}: T={op.T} rel={err:.3e}")
    assert err <= RTOL[dtype], err
    ref_bits = bits(y)
    y.fill_(float("nan"))
    op.run()
    torch.cuda.synchronize()
    assert bits(y) == ref_bits
    rng = np.random.default_rng(9)
    for n in [1, 2, 5]:
        if n > op.T:
            continue
        for block in [64, 128, 256]:
            y.fill_(float("nan"))
            plan = orc.balanced_split(op.T, n)
            for j in rng.permutation(n):
                b, l = plan[j]
                op.launch(b, l, int(rng.choice([1, 3, 7, l])), block)
            torch.cuda.synchronize()
            assert bits(y) == ref_bits, (n, block)


@pytest.mark.parametrize("C", [8, 64])
def test_conv_resident3x3_integer_inputs_exact(ops, orc, C):
    # integer operands in {-1, 0, 1}: |partial sums| <= 9 C <= 576, exact in fp32 and fp16
    x, x64 = ints((2, 10, 45, C), "f16", seed=5, lo=-1, hi=1)
    w, w64 = ints((64, 3, 3, C), "f16", seed=6, lo=-1, hi=1)
    y = empty((2, 10, 45, 64), "f16")
    op = ops.conv2d(x, w, y, stride=1, pad=1, tile=8)
    op.run()
    torch.cuda.synchronize()
    ref = orc.conv2d(x64, w64, stride=1, pad=1)
    assert np.array_equal(to_f64(y), ref)


def test_conv_resident3x3_tile_map_matches_oracle(ops, orc):
    x, _ = rand((2, 21, 70, 64), "f16", seed=8)
    w, _ = rand((64, 3, 3, 64), "f16", seed=9, lo=-0.1, hi=0.1)
    y = empty((2, 21, 70, 64), "f16")
    op = ops.conv2d(x, w, y, stride=1, pad=1, tile=8)
    T = op.T
    assert T == 2 * 6 * 3
    for n, grids, block in [(1, [T], 256), (4, [5, 64, 1, 3], 128), (3, [7, 7, 7], 64), (2, [4, 2], 256)]:
        plan = orc.balanced_split(T, n)
        ow = torch.full((T,), -1, dtype=torch.int32, device="cuda")
        oi = torch.full((T,), -1, dtype=torch.int32, device="cuda")
        cnt = torch.zeros((T,), dtype=torch.int32, device="cuda")
        for (b, l), g in zip(plan, grids):
            op.launch_traced(b, l, g, block, ow, oi, cnt)
        torch.cuda.synchronize()
        _, wg_ref, it_ref, cnt_ref = orc.owner_map(T, plan, grids)
        assert np.array_equal(cnt.cpu().numpy(), cnt_ref)
        assert np.array_equal(ow.cpu().numpy(), wg_ref)
        assert np.array_equal(oi.cpu().numpy(), it_ref)
