"""GPU parity of the remaining elastic operators against the CPU oracle: GEMM / FC,
strided batched GEMM (attention scores and context), depthwise convolution,
pooling, the standalone epilogue, softmax and layer normalisation; plus bitwise
invariance of each across shard plans and physical blocks."""
import numpy as np
import pytest
import torch

from gpu_util import RTOL, bits, empty, f32_dev, gpu_available, rand, rel_err, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

DTYPES = ["f32", "f16", "bf16"]


@pytest.fixture(scope="module")
def ops():
    from paper_2307_04339_amd import ops as o
    return o


def _elastic_bitwise(op, y, orc, plans=(1, 2, 3, 8), blocks=(64, 128, 256)):
    op.run()
    torch.cuda.synchronize()
    ref = bits(y)
    for n in plans:
        if n > op.T:
            continue
        plan = orc.balanced_split(op.T, n)
        for block in blocks:
            y.fill_(float("nan"))
            for j in reversed(range(n)):
                b, l = plan[j]
                op.launch(b, l, min(l, 37), block)
            torch.cuda.synchronize()
            assert bits(y) == ref, (n, block)


# -------------------------------------------------------------------- GEMM
GEMM_CASES = [
    # M, N, K, epilogue, act
    (1, 1000, 512, "bias", "none"),          # ResNet FC at batch 1
    (8, 4096, 1024, "bias", "relu"),         # VGG-style FC (reduced K)
    (128, 2304, 768, "bias", "none"),        # encoder QKV projection
    (128, 3072, 768, "bias", "gelu"),        # FFN up-projection
    (128, 768, 3072, "bias_res", "none"),    # FFN down-projection + residual
    (77, 45, 33, "bias", "relu"),            # ragged everything, K not a vector multiple
    (16, 1000, 1280, "bias", "none"),        # MobileNetV2 classifier at batch 16
    (3, 77, 200, "bias_res", "relu"),        # skinny with ragged N and a K tail
]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("case", GEMM_CASES)
def test_gemm_matches_oracle(ops, orc, dtype, case):
    M, N, K, epi, act = case
    seed = abs(hash(case)) % 997
    x, x64 = rand((M, K), dtype, seed)
    w, w64 = rand((N, K), dtype, seed + 1, -0.1, 0.1)
    b64 = np.random.default_rng(seed + 2).uniform(-1, 1, N).astype(np.float32).astype(np.float64)
    bias = f32_dev(b64)
    res = r64 = None
    if "res" in epi:
        res, r64 = rand((M, N), dtype, seed + 3)
    y = empty((M, N), dtype)
    ref = orc.linear(x64, w64, bias=b64, residual=r64, act=act)
    tiles = [0, 1, 2, 3, 4]
    if M <= 16 and dtype != "f32" and K % 8 == 0:
        tiles.append(5)  # split-K skinny kernel
    for tile in tiles:
        y.fill_(float("nan"))
        op = ops.gemm(x, w, y, bias=bias, residual=res, act=act, tile=tile)
        op.run()
        torch.cuda.synchronize()
        err = rel_err(to_f64(y), ref)
        assert err <= RTOL[dtype], (tile, err)
    _elastic_bitwise(op, y, orc)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("M,N,K,ksplit", [(4, 300, 4096, 4), (8, 1000, 8192, 0), (2, 64, 3328, 3),
                                          (16, 200, 2048, 2), (4, 2048, 16384, 0), (5, 2040, 16392, 0)])
def test_skinny_split_k_matches_oracle_and_is_elastic(ops, orc, dtype, M, N, K, ksplit):
    # K slices reduced in fixed order by the last-arriving slice; library choice (0): the
    # fewest slices that give every CU a tile.  The two large cases take 32-column tiles (two
    # column groups sharing each activation load; the second with ragged N and a K tail).
    seed = (M * 7 + N * 3 + K) % 991
    x, x64 = rand((M, K), dtype, seed)
    w, w64 = rand((N, K), dtype, seed + 1, -0.05, 0.05)
    b64 = np.random.default_rng(seed + 2).uniform(-1, 1, N).astype(np.float32).astype(np.float64)
    y = empty((M, N), dtype)
    op = ops.gemm(x, w, y, bias=f32_dev(b64), act="relu", tile=5, ksplit=ksplit)
    assert op.info.ksplit > 1
    assert op.info.tile_n == (32 if K >= 16384 else 16)
    assert op.T == op.info.ksplit * ((N + op.info.tile_n - 1) // op.info.tile_n)
    op.run()
    torch.cuda.synchronize()
    ref = orc.linear(x64, w64, bias=b64, act="relu")
    err = rel_err(to_f64(y), ref)
    print(f"skinny split K {dtype} {M}x{N}x{K}: ksplit={op.info.ksplit} T={op.T} rel={err:.3e}")
    assert err <= RTOL[dtype], err
    _elastic_bitwise(op, y, orc, plans=(1, 2, 3, 8))
    # two passes in a row: the arrival counters return to zero after each
    op.run()
    op.run()
    torch.cuda.synchronize()
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("B,S", [(1, 128), (2, 96)])
def test_attention_bgemm_matches_oracle(ops, orc, dtype, B, S):
    # packed QKV [B*S, 3*768]; scores[b,h] = Q_bh K_bh^T; ctx[b*S+i, h*64+j] = P_bh V_bh
    H, D = 12, 64
    hid = H * D
    qkv, qkv64 = rand((B * S, 3 * hid), dtype, seed=S + B)
    scores = empty((B * H, S, S), dtype)
    op_s = ops.bgemm(qkv, qkv[:, hid:], scores, m=S, n=S, k=D, batch=B * H, batch_div=H,
                     ldx=3 * hid, ldw=3 * hid, ldy=S, sx=(S * 3 * hid, D), sw=(S * 3 * hid, D),
                     sy=(H * S * S, S * S))
    op_s.run()
    probs, p64 = rand((B * H, S, S), dtype, seed=S + B + 1, lo=0.0, hi=0.05)
    ctx = empty((B * S, hid), dtype)
    op_c = ops.bgemm(probs, qkv[:, 2 * hid:], ctx, m=S, n=D, k=S, batch=B * H, batch_div=H,
                     ldx=S, ldw=3 * hid, ldy=hid, sx=(H * S * S, S * S), sw=(S * 3 * hid, D),
                     sy=(S * hid, D), b_nmajor=True)
    op_c.run()
    torch.cuda.synchronize()
    q64 = qkv64.reshape(B, S, 3, H, D)
    got_s = to_f64(scores).reshape(B, H, S, S)
    got_c = to_f64(ctx).reshape(B, S, H, D)
    pp = p64.reshape(B, H, S, S)
    for b in range(B):
        for h in range(H):
            ref_s = orc.gemm_nt(q64[b, :, 0, h, :], q64[b, :, 1, h, :])
            assert rel_err(got_s[b, h], ref_s) <= RTOL[dtype]
            ref_c = orc.gemm_nn(pp[b, h], q64[b, :, 2, h, :])
            assert rel_err(got_c[b, :, h, :], ref_c) <= RTOL[dtype]
    _elastic_bitwise(op_c, ctx, orc)


# ------------------------------------------------------------ depthwise conv
DW_CASES = [
    # N, H, W, C, stride, epilogue
    (2, 56, 56, 144, 1, "bn"),
    (2, 28, 28, 192, 2, "bn"),
    (1, 7, 7, 960, 1, "bn"),
    (1, 13, 11, 20, 2, "bias"),   # C not a vector multiple -> element path
    (1, 9, 10, 16, 2, "bias"),    # stride 2, 5-pixel output rows, odd height
    (3, 5, 6, 8, 1, "bn"),        # one channel vector, 6-pixel rows, batch 3
    (16, 56, 54, 144, 1, "bn"),   # strip kernel: 54-pixel rows end in a half strip
    (16, 28, 26, 192, 1, "bn"),   # strip kernel at about one tile per CU: 26-pixel rows, 7 strips
]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("case", DW_CASES)
def test_dwconv_matches_oracle(ops, orc, dtype, case):
    N, H, W, C, s, epi = case
    seed = abs(hash(case)) % 991
    x, x64 = rand((N, H, W, C), dtype, seed)
    w, w64 = rand((3, 3, C), dtype, seed + 1)
    rng = np.random.default_rng(seed + 2)
    bias = bn = None
    b64 = bn64 = None
    if epi == "bias":
        b64 = rng.uniform(-1, 1, C).astype(np.float32).astype(np.float64)
        bias = f32_dev(b64)
    else:
        bn64 = np.stack([rng.uniform(0.8, 1.2, C), rng.uniform(-0.1, 0.1, C),
                         rng.uniform(-0.1, 0.1, C), rng.uniform(0.8, 1.2, C)]).astype(np.float32).astype(np.float64)
        bn = f32_dev(bn64)
    Ho, Wo = (H + 2 - 3) // s + 1, (W + 2 - 3) // s + 1
    y = empty((N, Ho, Wo, C), dtype)
    op = ops.dwconv(x, w, y, stride=s, pad=1, bias=bias, bn=bn, act="relu6")
    if N == 16 and dtype != "f32":
        # 3x3 stride-1 strips of 4 output pixels per 16-byte channel vector
        assert op.T == (N * Ho * ((Wo + 3) // 4) * (C // 8) + 255) // 256
    op.run()
    torch.cuda.synchronize()
    # oracle weights [C][3][3][1] (groups = C)
    w_or = np.ascontiguousarray(w64.transpose(2, 0, 1))[..., None]
    ref = orc.conv2d(x64, w_or, stride=s, pad=1, groups=C, bias=b64,
                     bn=None if bn64 is None else tuple(bn64), act="relu6")
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    _elastic_bitwise(op, y, orc)


# ------------------------------------------------------------------ pooling
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("mode,N,H,C,k,s,p", [
    ("max", 1, 112, 64, 3, 2, 1),   # ResNet stem pool
    ("max", 2, 224, 64, 2, 2, 0),   # VGG pool
    ("avg", 1, 7, 512, 7, 1, 0),    # global average
    ("avg", 2, 9, 24, 3, 2, 1),
    ("max", 1, 10, 5, 3, 2, 1),     # element path
])
def test_pool_matches_oracle(ops, orc, dtype, mode, N, H, C, k, s, p):
    x, x64 = rand((N, H, H, C), dtype, seed=H + C)
    Ho = (H + 2 * p - k) // s + 1
    y = empty((N, Ho, Ho, C), dtype)
    op = ops.pool(x, y, k, s, p, mode)
    op.run()
    torch.cuda.synchronize()
    if mode == "max":
        ref = orc.maxpool(x64, k, s, p)
        assert np.array_equal(to_f64(y), ref)  # max is exact
    else:
        ref = orc.avgpool(x64, k, s, p)
        assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    _elastic_bitwise(op, y, orc)


# ------------------------------------------------------------ bn + act
@pytest.mark.parametrize("dtype", DTYPES)
def test_bn_act_matches_oracle(ops, orc, dtype):
    rows, C = 3 * 56 * 56, 64
    x, x64 = rand((rows, C), dtype, seed=5)
    r, r64 = rand((rows, C), dtype, seed=6)
    rng = np.random.default_rng(7)
    b64 = rng.uniform(-1, 1, C).astype(np.float32).astype(np.float64)
    bn64 = np.stack([rng.uniform(0.8, 1.2, C), rng.uniform(-0.1, 0.1, C),
                     rng.uniform(-0.1, 0.1, C), rng.uniform(0.8, 1.2, C)]).astype(np.float32).astype(np.float64)
    y = empty((rows, C), dtype)
    op = ops.bn_act(x, y, rows, C, bias=f32_dev(b64), bn=f32_dev(bn64), residual=r, act="relu")
    op.run()
    torch.cuda.synchronize()
    ref = orc.epilogue(x64, bias=b64, bn=tuple(bn64), residual=r64, act="relu")
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    _elastic_bitwise(op, y, orc)


# ------------------------------------------------------- softmax / layernorm
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("rows,n", [(12 * 128, 128), (4 * 12 * 256, 256), (5, 100)])
def test_softmax_matches_oracle(ops, orc, dtype, rows, n):
    x, x64 = rand((rows, n), dtype, seed=n, lo=-8, hi=8)
    y = empty((rows, n), dtype)
    op = ops.softmax(x, y, rows, n, scale=0.125)
    op.run()
    torch.cuda.synchronize()
    ref = orc.softmax_rows(x64, scale=0.125)
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    _elastic_bitwise(op, y, orc)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("rows,n,res", [(128, 768, True), (1024, 768, False), (7, 100, True)])
def test_layernorm_matches_oracle(ops, orc, dtype, rows, n, res):
    x, x64 = rand((rows, n), dtype, seed=rows, lo=-2, hi=2)
    r = r64 = None
    if res:
        r, r64 = rand((rows, n), dtype, seed=rows + 1)
    rng = np.random.default_rng(n)
    g64 = rng.uniform(0.5, 1.5, n).astype(np.float32).astype(np.float64)
    be64 = rng.uniform(-1, 1, n).astype(np.float32).astype(np.float64)
    y = empty((rows, n), dtype)
    op = ops.layernorm(x, f32_dev(g64), f32_dev(be64), y, rows, n, residual=r)
    op.run()
    torch.cuda.synchronize()
    ref = orc.layernorm_rows(x64, g64, be64, eps=1e-5, residual=r64)
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    _elastic_bitwise(op, y, orc)


# ------------------------------------------------------------- edge cases
def test_single_tile_and_max_grid(ops, orc):
    x, x64 = rand((1, 4), "f32", 1)
    w, w64 = rand((1, 4), "f32", 2)
    y = empty((1, 1), "f32")
    op = ops.gemm(x, w, y)
    assert op.T == 1
    op.launch(0, 1, 1024, 64)  # surplus workgroups exit at once
    torch.cuda.synchronize()
    assert rel_err(to_f64(y), orc.gemm_nt(x64, w64)) <= 1e-6


def test_launch_errors_do_not_launch(ops):
    from paper_2307_04339_amd import _lib as L
    x, _ = rand((8, 8), "f16", 1)
    y = empty((8, 8), "f16")
    op = ops.softmax(x, y, 8, 8)
    with pytest.raises(L.MiriamError):
        op.launch(0, op.T + 1, 1, 256)
    with pytest.raises(L.MiriamError):
        op.launch(0, 1, 1, 192)
    torch.cuda.synchronize()
    assert torch.isnan(y.float()).all()  # nothing ran


@pytest.mark.parametrize("case", ["vgg_conv5", "resnet_l3_res", "encoder_ffn2"])
def test_library_split_k_matches_oracle_and_is_elastic(ops, orc, case):
    # the library's own split-K choice on the pipelined kernel (slices reduced in fixed order by
    # the last to arrive, partials in fragment layout with 16-byte device-coherent accesses):
    # VGG-16 b8 conv5_x (200 tiles, 2 slices), a ResNet-18 b1 layer-3 convolution with a
    # residual, the encoder b1 FFN2 product; checked against the oracle in full and bitwise
    # across shard plans
    dtype = "f16"
    if case == "encoder_ffn2":
        M, N, K = 128, 768, 3072
        x, x64 = rand((M, K), "bf16", 61)
        w, w64 = rand((N, K), "bf16", 62, -0.03, 0.03)
        b64 = np.random.default_rng(63).uniform(-1, 1, N).astype(np.float32).astype(np.float64)
        y = empty((M, N), "bf16")
        op = ops.gemm(x, w, y, bias=f32_dev(b64), act="gelu")
        ref = orc.linear(x64, w64, bias=b64, act="gelu")
        dtype = "bf16"
    else:
        n, h, c, k, res = (8, 14, 512, 512, False) if case == "vgg_conv5" else (1, 14, 256, 256, True)
        x, x64 = rand((n, h, h, c), dtype, 64)
        w, w64 = rand((k, 3, 3, c), dtype, 65, -0.02, 0.02)
        b64 = np.random.default_rng(66).uniform(-1, 1, k).astype(np.float32).astype(np.float64)
        r, r64 = rand((n, h, h, k), dtype, 67) if res else (None, None)
        y = empty((n, h, h, k), dtype)
        op = ops.conv2d(x, w, y, stride=1, pad=1, bias=f32_dev(b64), residual=r, act="relu")
        ref = orc.conv2d(x64, w64, stride=1, pad=1, bias=b64, residual=r64, act="relu")
    assert op.info.ksplit > 1, case
    op.run()
    torch.cuda.synchronize()
    err = rel_err(to_f64(y), ref)
    print(f"library split K {case}: ksplit={op.info.ksplit} T={op.T} tile={op.info.tile_m}x{op.info.tile_n} rel={err:.3e}")
    assert err <= RTOL[dtype], err
    _elastic_bitwise(op, y, orc, plans=(1, 2, 3, 8))


@pytest.mark.parametrize("tile,shape", [(5, (8, 300, 4096)), (2, None)])
def test_split_k_counters_reset_after_abandoned_pass(ops, orc, tile, shape):
    # a pass that covers only part of a split-K op's tile space leaves arrival counts behind;
    # miriam_op_reset_counters clears them in stream order, and the next whole pass reduces the
    # right slices again (checked against the oracle and bitwise against an untouched pass)
    dtype = "f16"
    if tile == 5:
        M, N, K = shape
        x, x64 = rand((M, K), dtype, 31)
        w, w64 = rand((N, K), dtype, 32, -0.05, 0.05)
        y = empty((M, N), dtype)
        op = ops.gemm(x, w, y, act="relu", tile=5, ksplit=4)
        ref = orc.linear(x64, w64, act="relu")
    else:
        x, x64 = rand((1, 7, 7, 256), dtype, 33)
        w, w64 = rand((64, 3, 3, 256), dtype, 34, -0.05, 0.05)
        y = empty((1, 7, 7, 64), dtype)
        op = ops.conv2d(x, w, y, stride=1, pad=1, act="relu", tile=2, ksplit=3)
        ref = orc.conv2d(x64, w64, stride=1, pad=1, act="relu")
    ks = op.info.ksplit
    assert ks > 1
    op.run()
    torch.cuda.synchronize()
    good = bits(y)
    assert rel_err(to_f64(y), ref) <= RTOL[dtype]
    # abandon a pass after its first slices: every output tile's count is left part-way
    op.launch(0, op.T // 2 + 1, 7, 256)
    op.reset_counters()
    y.fill_(float("nan"))
    op.run()
    torch.cuda.synchronize()
    assert bits(y) == good
    op.run()
    torch.cuda.synchronize()
    assert bits(y) == good
