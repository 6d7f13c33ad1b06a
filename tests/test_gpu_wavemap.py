"""Device trace of the N:1 logical-to-physical wave map (§6.1) against the oracle, for every
kernel family, and the residency figures the library reports for its kernels.

A traced launch records, from the physical wave that ran it, where each logical wave of each
tile ran: the physical wave's index in the workgroup and the logical wave's place among those
that wave runs.  The oracle's or_wave_map gives the expected pair for a logical block of 4
waves and a physical block of P = block / 64 waves; every entry of every tile of the shard must
match bit for bit, whatever the shard plan and the grid, and entries of tiles outside the shard
stay untouched.
"""
import numpy as np
import pytest
import torch

from gpu_util import empty, f32_dev, gpu_available, rand

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

LDS_PER_CU = 160 * 1024


@pytest.fixture(scope="module")
def ops():
    from paper_2307_04339_amd import ops as o
    return o


@pytest.fixture(scope="module")
def L():
    from paper_2307_04339_amd import _lib
    return _lib


def _conv(ops, dtype, n, h, w, c, k, ks=3, stride=1, pad=1, tile=0, ksplit=0, seed=0):
    x, _ = rand((n, h, w, c), dtype, seed)
    wt, _ = rand((k, ks, ks, c), dtype, seed + 1, -0.1, 0.1)
    ho = (h + 2 * pad - ks) // stride + 1
    wo = (w + 2 * pad - ks) // stride + 1
    y = empty((n, ho, wo, k), dtype)
    bias = f32_dev(np.linspace(-1, 1, k))
    return ops.conv2d(x, wt, y, stride=stride, pad=pad, bias=bias, act="relu", tile=tile, ksplit=ksplit)


def _family_ops(ops, L):
    """One op per kernel family and decode variant: (name, op, expected kernel path or None)."""
    out = []
    out.append(("dma-uniform 128x128", _conv(ops, "f16", 1, 24, 24, 64, 128, tile=3), L.PATH_DMA_UNIFORM))
    out.append(("dma-uniform 128x64", _conv(ops, "bf16", 1, 24, 24, 64, 64, tile=4), L.PATH_DMA_UNIFORM))
    out.append(("dma-uniform 64x64", _conv(ops, "f16", 1, 20, 20, 64, 64, tile=2), L.PATH_DMA_UNIFORM))
    out.append(("dma-lane 32x32 fp32", _conv(ops, "f32", 1, 17, 19, 24, 40, tile=1), L.PATH_DMA))
    out.append(("dma split-K", _conv(ops, "f16", 1, 7, 7, 256, 64, tile=2, ksplit=3), L.PATH_DMA_UNIFORM))
    out.append(("halo 3x3", _conv(ops, "f16", 1, 12, 40, 64, 64, tile=7), L.PATH_HALO))
    out.append(("resident 3x3", _conv(ops, "bf16", 1, 12, 40, 32, 64, tile=8), L.PATH_RESIDENT))
    out.append(("resident 1x1", _conv(ops, "f16", 1, 9, 35, 32, 128, ks=1, pad=0, tile=8), L.PATH_RESIDENT))
    # register-staged kernel: N-major right operand (attention context)
    p, _ = rand((2, 40, 40), "f16", 5, 0.0, 0.05)
    v, _ = rand((40, 2 * 64), "f16", 6)
    ctx = empty((40, 2 * 64), "f16")
    out.append(("staged N-major", ops.bgemm(p, v, ctx, m=40, n=64, k=40, batch=2, batch_div=2, ldx=40,
                                            ldw=128, ldy=128, sx=(0, 1600), sw=(0, 64), sy=(0, 64),
                                            b_nmajor=True), L.PATH_STAGED))
    xs, _ = rand((5, 512), "f16", 7)
    ws, _ = rand((300, 512), "f16", 8, -0.1, 0.1)
    ys = empty((5, 300), "f16")
    out.append(("skinny FC", ops.gemm(xs, ws, ys, tile=5, ksplit=2), L.PATH_SKINNY))
    xd, _ = rand((2, 13, 13, 48), "bf16", 9)
    wd, _ = rand((3, 3, 48), "bf16", 10)
    yd = empty((2, 13, 13, 48), "bf16")
    out.append(("depthwise", ops.dwconv(xd, wd, yd, stride=1, pad=1, act="relu6"), L.PATH_OTHER))
    yp = empty((2, 7, 7, 48), "bf16")
    out.append(("max pool", ops.pool(xd, yp, 3, 2, 1, "max"), L.PATH_OTHER))
    xr, _ = rand((37, 96), "f32", 11)
    yr = empty((37, 96), "f32")
    out.append(("softmax", ops.softmax(xr, yr, 37, 96), L.PATH_OTHER))
    g = f32_dev(np.ones(96))
    b = f32_dev(np.zeros(96))
    yl = empty((37, 96), "f32")
    out.append(("layernorm", ops.layernorm(xr, g, b, yl, 37, 96), L.PATH_OTHER))
    return out


def test_wave_map_matches_oracle_for_every_kernel_family(ops, orc, L):
    fam = _family_ops(ops, L)
    for name, op, path in fam:
        if path is not None:
            assert op.info.path == path, (name, op.info.path)
        T = op.T
        for block in (64, 128, 256):
            P = block // 64
            for n, grid_of in ((1, lambda l: l), (3, lambda l: max(1, l // 2)), (2, lambda l: 1)):
                if n > T:
                    continue
                plan = orc.balanced_split(T, n)
                ow = torch.full((T,), -1, dtype=torch.int32, device="cuda")
                oi = torch.full((T,), -1, dtype=torch.int32, device="cuda")
                cnt = torch.zeros((T,), dtype=torch.int32, device="cuda")
                wp = torch.full((4 * T,), -1, dtype=torch.int32, device="cuda")
                ws = torch.full((4 * T,), -1, dtype=torch.int32, device="cuda")
                # only the shards with an odd index are traced: the others leave their entries at -1
                for j, (b, l) in enumerate(plan):
                    if j % 2 == 1 or n == 1:
                        op.launch_traced(b, l, grid_of(l), block, ow, oi, cnt, wave_phys=wp, wave_slot=ws)
                torch.cuda.synchronize()
                got_p = wp.cpu().numpy().reshape(T, 4)
                got_s = ws.cpu().numpy().reshape(T, 4)
                exp = np.array([orc.wave_map(4, P, lam) for lam in range(4)], dtype=np.int32)
                for j, (b, l) in enumerate(plan):
                    traced = j % 2 == 1 or n == 1
                    for t in range(b, b + l):
                        if traced:
                            assert np.array_equal(got_p[t], exp[:, 0]), (name, block, n, t, got_p[t])
                            assert np.array_equal(got_s[t], exp[:, 1]), (name, block, n, t, got_s[t])
                        else:
                            assert (got_p[t] == -1).all() and (got_s[t] == -1).all(), (name, block, n, t)
        print(f"wave map: {name}: T={T} ok")


def test_launch_traced_rejects_half_wave_trace(ops, L):
    op = _conv(ops, "f16", 1, 8, 8, 64, 64, tile=2)
    T = op.T
    a = torch.zeros((T,), dtype=torch.int32, device="cuda")
    w = torch.zeros((4 * T,), dtype=torch.int32, device="cuda")
    with pytest.raises(RuntimeError):
        op.launch_traced(0, T, T, 256, a, a, a, wave_phys=w, wave_slot=None)


def test_residency_figures_match_lds_budget(ops, L):
    """max_wg_per_cu (from the HIP occupancy query) against each kernel's LDS and its launch
    bounds: the pipelined contraction tiles 128x128, 128x64 and 64x64 and the LDS-patch 3x3
    kernel are built for two 4-wave workgroups per CU (their LDS fits twice, not three times,
    and their launch bounds budget registers for two waves per SIMD); every kernel's figure
    respects the LDS of a CU and its 2048 threads."""
    cases = [("128x128", _conv(ops, "f16", 1, 24, 24, 64, 128, tile=3), 2),
             ("128x64", _conv(ops, "f16", 1, 24, 24, 64, 64, tile=4), 2),
             ("64x64", _conv(ops, "bf16", 1, 24, 24, 64, 64, tile=2), 2),
             ("halo", _conv(ops, "f16", 1, 12, 40, 64, 64, tile=7), 2)]
    for name, op, want in cases:
        lds = op.info.lds_bytes
        assert want * lds <= LDS_PER_CU < (want + 1) * lds, (name, lds)
        assert op.info.max_wg_per_cu[2] == want, (name, list(op.info.max_wg_per_cu))
    for name, op, _ in _family_ops(ops, L):
        for i, block in enumerate((64, 128, 256)):
            m = op.info.max_wg_per_cu[i]
            assert m >= 1, (name, block)
            assert m * block <= 2048, (name, block, m)
            if op.info.lds_bytes > 0:
                assert m * op.info.lds_bytes <= LDS_PER_CU, (name, block, m, op.info.lds_bytes)


def test_full_grid_of_pipelined_contraction(ops, L):
    """The unsharded grid of the pipelined contraction: one workgroup per tile up to one round of
    resident workgroups, half as many workgroups (two tiles each) for one to two rounds, one per
    tile beyond; the two-tiles-per-workgroup launch gives the bits of the one-per-tile launch."""
    from gpu_util import bits
    n_cu = ops.device_info().n_cu
    for n, hw, c, k, tile in [(8, 112, 128, 128, 0), (8, 56, 256, 256, 0), (8, 56, 64, 64, 1)]:
        op = _conv(ops, "f16", n, hw, hw, c, k, tile=tile)
        info = op.info
        assert info.path in (L.PATH_DMA, L.PATH_DMA_UNIFORM), (n, hw, c, k, info.path)
        T, slots = op.T, n_cu * info.max_wg_per_cu[2]
        want = (T + 1) // 2 if slots < T <= 2 * slots else T
        assert info.full_grid == want, (T, slots, info.full_grid)
        y = op._keep[2]
        op.run()
        torch.cuda.synchronize()
        ref = bits(y)
        y.fill_(float("nan"))
        op.launch(0, T, T, 256)
        torch.cuda.synchronize()
        assert bits(y) == ref, (T, info.full_grid)
        print(f"full grid: {n}x{hw}x{hw}x{c}->{k}: T={T} slots={slots} grid={info.full_grid}")
