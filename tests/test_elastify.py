"""The source-to-source elastic transformer on the host: parsing of plain kernels, the id
rewrites, rejected inputs, and the generated library's launchers (argument checks only; no
kernel runs without a GPU)."""
import ctypes
import os

import pytest

from paper_2307_04339_amd.transform import elastify


def _plain():
    with open(os.path.join(elastify.PLAIN_DIR, "kernels.hip")) as f:
        return f.read()


def test_parse_plain_kernels():
    ks = {k.name: k for k in elastify.parse(_plain())}
    assert set(ks) == {"plain_bias_relu", "plain_maxpool2", "plain_tiled_gemm", "plain_shift_add2d",
                       "plain_transpose16", "plain_conv3x3_relu", "plain_dwconv3x3_relu6", "plain_softmax_rows",
                       "plain_layernorm_rows"}
    for name in ("plain_conv3x3_relu", "plain_dwconv3x3_relu6"):
        assert (ks[name].block, ks[name].block_elastic) == (256, True)
    for name, blk in (("plain_softmax_rows", 256), ("plain_layernorm_rows", 128)):
        assert (ks[name].block, ks[name].block_elastic, len(ks[name].shared_decls)) == (blk, False, 1)
    assert (ks["plain_shift_add2d"].bx, ks["plain_shift_add2d"].by, ks["plain_shift_add2d"].block_elastic) == (32, 8, True)
    assert (ks["plain_transpose16"].bx, ks["plain_transpose16"].by, ks["plain_transpose16"].block_elastic) == (16, 16, False)
    assert (ks["plain_bias_relu"].block, ks["plain_bias_relu"].block_elastic) == (256, True)
    assert (ks["plain_maxpool2"].block, ks["plain_maxpool2"].block_elastic) == (128, True)
    g = ks["plain_tiled_gemm"]
    assert (g.block, g.block_elastic) == (256, False)
    assert len(g.shared_decls) == 2 and "__shared__" not in g.body
    assert ks["plain_bias_relu"].param_names == ["x", "b", "y", "n", "c"]


def test_ids_become_logical():
    out = elastify.transform(_plain())
    for k in elastify.parse(_plain()):
        start = out.index(f"__global__ void {k.name}_elastic(")
        end = out.index('extern "C"', start)
        kern = out[start:end]
        # physical ids appear only in the shard loop and the logical-thread rounds
        body = kern[kern.index("[&]() {"):]
        for ident in ("blockIdx.x", "gridDim.x", "threadIdx.x", "blockDim.x", "blockIdx.y", "gridDim.y",
                      "threadIdx.y", "blockDim.y"):
            assert ident not in body, (k.name, ident)
        assert "__mi_sh.begin + blockIdx.x" in kern and "__mi_b += gridDim.x" in kern
        if k.block_elastic:
            assert f"{k.block}u / blockDim.x" in kern
        else:
            assert "const unsigned __mi_t = threadIdx.x;" in kern
    assert "__mi_bx * __mi_bdx + __mi_tx" in out
    assert "i += __mi_gx * __mi_bdx" in out  # a grid-stride loop keeps the logical grid
    assert "__mi_by * __mi_bdy + __mi_ty" in out  # 2-D ids from the flattened block and thread
    assert "__mi_by = __mi_gy == 1u ? 0u : __mi_bu / __mi_gx;" in out
    assert "__mi_bx = __mi_bu - __mi_by * __mi_gx;" in out
    assert "__mi_tx = __mi_t % 32u, __mi_ty = __mi_t / 32u" in out


@pytest.mark.parametrize("src,msg", [
    ("// elastic: block 256\n__global__ void k(float *y) { y[blockIdx.z] = 0.0f; }", "not supported"),
    ("// elastic: block 16x12\n__global__ void k(float *y) { y[threadIdx.y] = 0.0f; }", "64, 128 or 256"),
    ("__global__ void k(float *y) { y[blockIdx.x] = 0.0f; }", "no '// elastic: block N'"),
    ("// elastic: block 96\n__global__ void k(float *y) { y[blockIdx.x] = 0.0f; }", "64, 128 or 256"),
    ("// elastic: block 64\n__global__ void k(float *y) { y[0] = 0.0f; ", "unbalanced"),
])
def test_rejects_unsupported_kernels(src, msg):
    with pytest.raises(elastify.TransformError, match=msg):
        elastify.parse(src)


def test_return_ends_one_logical_thread():
    # an early return stays inside the per-thread lambda, so the shard loop goes on
    src = "// elastic: block 64\n__global__ void k(float *y, int n) {\n  if (threadIdx.x >= n) return;\n  y[threadIdx.x] = 1.0f;\n}\n"
    out = elastify.transform(src)
    kern = out[out.index("__global__ void k_elastic("):out.index('extern "C"')]
    assert kern.index("for (long long __mi_b") < kern.index("[&]() {") < kern.index("return;")


def test_launchers_check_arguments():
    from paper_2307_04339_amd.transform import lib as T
    lib = T.load()
    nul = None
    # shard out of range, zero grid, block not dividing the logical block, fixed block changed,
    # empty logical grid
    assert lib.plain_bias_relu_elastic_launch(nul, nul, nul, 10, 2, 4, 1, 2, 3, 1, 256, nul) == -3
    assert lib.plain_bias_relu_elastic_launch(nul, nul, nul, 10, 2, 4, 1, 0, 1, 0, 256, nul) == -3
    assert lib.plain_bias_relu_elastic_launch(nul, nul, nul, 10, 2, 4, 1, 0, 1, 1, 96, nul) == -3
    assert lib.plain_maxpool2_elastic_launch(nul, nul, 1, 4, 4, 8, 2, 1, 0, 2, 1, 256, nul) == -3
    assert lib.plain_tiled_gemm_elastic_launch(nul, nul, nul, 16, 16, 16, 1, 1, 0, 1, 1, 128, nul) == -3
    assert lib.plain_transpose16_elastic_launch(nul, nul, 16, 16, 1, 1, 0, 1, 1, 64, nul) == -3
    assert lib.plain_shift_add2d_elastic_launch(nul, nul, 8, 32, 1.0, 2, 3, 0, 7, 1, 256, nul) == -3
    assert lib.plain_shift_add2d_plain_launch(nul, nul, 8, 32, 1.0, 0, 1, nul) == -3
    assert lib.plain_tiled_gemm_plain_launch(nul, nul, nul, 16, 16, 16, 1, 0, nul) == -3


def test_synchronising_kernels_end_each_logical_block_at_a_barrier():
    # the shared arrays of a fixed-block kernel live at kernel scope across the logical blocks
    # of a shard: each logical block's lambda is followed by a barrier before the next block
    # reuses them; kernels without barriers or shared memory get none
    out = elastify.transform(_plain())
    for k in elastify.parse(_plain()):
        start = out.index(f"__global__ void {k.name}_elastic(")
        kern = out[start:out.index('extern "C"', start)]
        call = kern.index("}();", kern.index("[&]() {"))
        tail = kern[call + len("}();"):]
        if k.syncs:
            assert tail.lstrip().startswith("__syncthreads();"), k.name
            # the barrier sits inside the shard loop, after the logical block
            assert tail.index("__syncthreads();") < tail.index("}")
        else:
            assert "__syncthreads();" not in tail, k.name
    ks = {k.name: k for k in elastify.parse(_plain())}
    assert ks["plain_transpose16"].syncs and ks["plain_tiled_gemm"].syncs
    assert not ks["plain_bias_relu"].syncs
