#!/usr/bin/env python3
"""Miriam co-run benchmark on one MI355X.

Main line (the workload of `value`): the two-task co-run in fp16 whose critical task is a
ResNet-18-shaped CNN at batch 1 released every 20 ms, next to a VGG-16-shaped CNN at batch 8
run closed-loop on 224x224 inputs as best-effort work.  Inputs and weights are seeded synthetic
tensors resident in HBM before timing starts.

One step is a batch of critical release periods (--periods-per-step, 25): W warm-up steps, then
exactly K timed steps, per co-run phase.  Phases: per-kernel timing of the main workload's
networks (roofline of its dominant kernel, elastic-shard overhead and its launch / persistent
decomposition), the single fp32 elastic convolution, the ResNet-18 b1 per-kernel roofline with
seeded shard plans, then the co-run phases (critical task alone, Sequential, Multi-stream, the
inter-stream-barrier baseline, Miriam under the paper's fill rule and under the hold-back rule),
the other two co-run workloads as sub-lines, and the CPU oracle baseline.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

# Hardware queues of this process: one stream per coordinator task (the critical stream and up
# to three normal streams) plus the profiling stream and the framework's own.  With HIP's
# default of 4, kernel traces showed two normal streams sharing one queue (their kernels then
# run in order); 8 gives every stream its own.  Read by the HIP runtime when it starts, so it is
# raised to at least 8 before torch is imported (a larger setting in the environment is kept).
try:
    _hwq = int(os.environ.get("GPU_MAX_HW_QUEUES", "4"))
except ValueError:
    _hwq = 4
os.environ["GPU_MAX_HW_QUEUES"] = str(min(32, max(8, _hwq)))

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "critical p99 latency overhead vs solo; best-effort inf/s; kernel % roofline"
PEAK_TFLOPS = {"f16": 2500.0, "bf16": 2500.0, "f32": 157.3}
PEAK_HBM_GBS = 8000.0

CONFIGS = {
    "corun-resnet18-vgg16-fp16": dict(
        dtype="f16", crit=("resnet18", dict(batch=1)), period_ms=20.0, arrival="periodic",
        be=[("vgg16", dict(batch=8))], be_instances=3),
    "corun-encoder-mobilenetv2-bf16": dict(
        dtype="bf16", crit=("encoder", dict(batch=1, seq=128)), period_ms=10.0, arrival="periodic",
        be=[("mobilenetv2", dict(batch=16))], be_instances=3),
    "mix4-bf16": dict(
        dtype="bf16", crit=("resnet18", dict(batch=1)), period_ms=15.0, arrival="poisson",
        be=[("vgg16", dict(batch=8)), ("encoder", dict(batch=4, seq=256)), ("mobilenetv2", dict(batch=32))],
        be_instances=1),
}
DEFAULT_CONFIG = "corun-resnet18-vgg16-fp16"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pct(xs, q):
    return float(np.percentile(np.asarray(xs, dtype=np.float64), q)) if len(xs) else float("nan")


# ----------------------------------------------------------- kernel timing
class CacheFlush:
    """Evicts the L2 caches and the Infinity Cache before a timed launch by reading a 512 MiB
    buffer (twice the Infinity Cache).  A read pass leaves clean lines behind; a write pass
    would leave dirty lines that the timed kernel then pays to write back."""

    def __init__(self):
        import torch
        self.buf = torch.ones(512 * 1024 * 1024 // 4, dtype=torch.float32, device="cuda")
        self.sink = None

    def __call__(self):
        self.sink = self.buf.sum()


def time_layers(net, reps, flush):
    """Average unsharded duration of every layer, HIP events on torch's current stream."""
    import torch
    out = []
    for layer in net.layers:
        layer.op.run()
        torch.cuda.synchronize()
        total = 0.0
        for _ in range(reps):
            flush()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            layer.op.run()
            e1.record()
            e1.synchronize()
            total += e0.elapsed_time(e1)
        us = 1000.0 * total / reps
        flops = layer.op.info.flops
        if layer.kind == "conv" and layer.params.get("logical_c"):
            # an image stored with zero channels appended: count the logical convolution only
            flops *= layer.params["logical_c"] / layer.t["x"].shape[-1]
        out.append(dict(name=layer.name, us=us, flops=flops, bytes=layer.op.info.bytes,
                        tiles=layer.op.T))
    return out


# HBM traffic of the dominant kernel, from rocprofv3 FETCH_SIZE / WRITE_SIZE runs committed under
# profiles/ (each counter scaled by what it reads for a device copy of known size).  Used only
# while the contraction-kernel sources still hash to the value the counters were taken with.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# device code of the contraction kernels; the host-side choice of kernel is checked through
# the kernel path and tile recorded with the counters
KERNEL_SOURCES = ["conv_halo.h", "conv_rw.h", "igemm_dma.h", "igemm.h", "elastic_common.h", "kargs.h",
                  "kern_igemm_f16.hip", "kern_igemm_bf16.hip", "kern_igemm_f32.hip", "kern_rw.hip", "kern_skinny.hip"]


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2307_04339_amd", "csrc", name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(workload, kernel, tile, path, grid):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None when
    there is none for this workload / kernel path / tile / unsharded grid (where recorded) or
    the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            entries = json.load(f)["entries"]
    except (OSError, ValueError, KeyError):
        return None
    e = entries.get(f"{workload}:{kernel}")
    if (not e or list(e.get("tile", [])) != list(tile) or e.get("path") != path
            or e.get("grid", grid) != grid or e.get("source_sha256") != kernel_source_hash()):
        return None
    fetch = e["fetch_kib"] * 1024.0 * e["copy_bytes"] / (e["copy_fetch_kib"] * 1024.0)
    write = e["write_kib"] * 1024.0 * e["copy_bytes"] / (e["copy_write_kib"] * 1024.0)
    return round(fetch + write)


def roofline_of(k, dtype):
    ai = k["flops"] / max(1.0, k["bytes"])
    ridge = PEAK_TFLOPS[dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    if ai >= ridge:
        ach = k["flops"] / (k["us"] * 1e-6) / 1e12
        return dict(bound="mfma", achieved=round(ach, 2), peak=PEAK_TFLOPS[dtype], unit="TFLOP/s",
                    frac=round(ach / PEAK_TFLOPS[dtype], 4), traffic=None)
    ach = k["bytes"] / (k["us"] * 1e-6) / 1e9
    return dict(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                frac=round(ach / PEAK_HBM_GBS, 4), traffic=None)


def index_function_cost(net, reps, flush, lib_mod):
    """Unsharded time of every layer on the pipelined contraction kernel with the
    computation-based index function (the default) and with the memory-based one (row
    indices from a host-computed table staged in LDS), median over `reps` cold launches."""
    import torch

    def med(op):
        op.run()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            flush()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            op.run()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return 1000.0 * float(np.median(ts))

    rows = []
    for layer in net.layers:
        op = layer.op
        if op.info.path not in (lib_mod.PATH_DMA, lib_mod.PATH_DMA_UNIFORM) or op.info.ksplit > 1:
            continue
        twin = op.variant(flags=op.desc.flags | lib_mod.INDEX_MEMORY)
        try:
            if (twin.info.tile_m, twin.info.tile_n) != (op.info.tile_m, op.info.tile_n):
                continue
            c_us, m_us = med(op), med(twin)
        finally:
            twin.destroy()
        rows.append(dict(name=layer.name, compute_us=round(c_us, 2), memory_us=round(m_us, 2),
                         memory_over_compute=round(m_us / c_us, 4)))
    return rows


def transformed_overhead(reps, flush):
    """Kernels elasticised by the source-to-source transformer: median time of the plain launch
    and of the elastic form unsharded (grid = the plain grid) and as 4 shards, cold caches.
    Workloads: bias + ReLU over 8 x 112 x 112 x 64 fp32, 2x2 max pooling of the same tensor,
    a 1024^3 fp32 product with 16 x 16 shared-memory tiles, a direct 3x3 convolution with bias
    and ReLU (1 x 56 x 56 x 64 -> 64, the single fp32 convolution's shape), a depthwise 3x3
    convolution with bias and ReLU6 (16 x 56 x 56 x 144, a MobileNetV2 b16 layer), and row
    softmax and LayerNorm over the encoder's shapes (4 heads x 128 x 128 scores; 128 x 768)."""
    import torch
    from paper_2307_04339_amd.transform import lib as TL
    T = TL.load()
    g = torch.Generator(device="cuda").manual_seed(0)
    x = torch.rand((8, 112, 112, 64), device="cuda", generator=g) * 2 - 1
    bvec = torch.rand(64, device="cuda", generator=g) * 2 - 1
    y = torch.empty_like(x)
    yp = torch.empty((8, 56, 56, 64), device="cuda")
    A = torch.rand((1024, 1024), device="cuda", generator=g)
    B = torch.rand((1024, 1024), device="cuda", generator=g)
    C = torch.empty((1024, 1024), device="cuda")
    n = x.numel()
    xc = torch.rand((1, 56, 56, 64), device="cuda", generator=g) * 2 - 1
    wc = torch.rand((64, 3, 3, 64), device="cuda", generator=g) * 2 - 1
    yc = torch.empty((1, 56, 56, 64), device="cuda")
    xd = torch.rand((16, 56, 56, 144), device="cuda", generator=g) * 2 - 1
    wd = torch.rand((144, 3, 3), device="cuda", generator=g) * 2 - 1
    bd = torch.rand(144, device="cuda", generator=g) * 2 - 1
    yd = torch.empty_like(xd)
    xs = torch.randn((4 * 128, 128), device="cuda", generator=g)
    ys = torch.empty_like(xs)
    xl = torch.randn((128, 768), device="cuda", generator=g)
    gl = torch.rand(768, device="cuda", generator=g) + 0.5
    bl_ = torch.rand(768, device="cuda", generator=g) - 0.5
    yl = torch.empty_like(xl)
    cases = {
        "bias_relu": ((n + 255) // 256, 256,
                      lambda G, bl: T.plain_bias_relu_plain_launch(x.data_ptr(), bvec.data_ptr(), y.data_ptr(), n, 64,
                                                                   G, 1, None),
                      lambda G, b0, l, gr, bl: T.plain_bias_relu_elastic_launch(
                          x.data_ptr(), bvec.data_ptr(), y.data_ptr(), n, 64, G, 1, b0, l, gr, bl, None)),
        "maxpool2": ((yp.numel() + 127) // 128, 128,
                     lambda G, bl: T.plain_maxpool2_plain_launch(x.data_ptr(), yp.data_ptr(), 8, 112, 112, 64, G, 1,
                                                                 None),
                     lambda G, b0, l, gr, bl: T.plain_maxpool2_elastic_launch(
                         x.data_ptr(), yp.data_ptr(), 8, 112, 112, 64, G, 1, b0, l, gr, bl, None)),
        "tiled_gemm": (64 * 64, 256,
                       lambda G, bl: T.plain_tiled_gemm_plain_launch(A.data_ptr(), B.data_ptr(), C.data_ptr(),
                                                                     1024, 1024, 1024, G, 1, None),
                       lambda G, b0, l, gr, bl: T.plain_tiled_gemm_elastic_launch(
                           A.data_ptr(), B.data_ptr(), C.data_ptr(), 1024, 1024, 1024, G, 1, b0, l, gr, bl, None)),
        "conv3x3_relu": ((yc.numel() + 255) // 256, 256,
                         lambda G, bl: T.plain_conv3x3_relu_plain_launch(
                             xc.data_ptr(), wc.data_ptr(), bvec.data_ptr(), yc.data_ptr(), 1, 56, 56, 64, 64, 1, G, 1,
                             None),
                         lambda G, b0, l, gr, bl: T.plain_conv3x3_relu_elastic_launch(
                             xc.data_ptr(), wc.data_ptr(), bvec.data_ptr(), yc.data_ptr(), 1, 56, 56, 64, 64, 1, G, 1,
                             b0, l, gr, bl, None)),
        "dwconv3x3_relu6": ((yd.numel() + 255) // 256, 256,
                            lambda G, bl: T.plain_dwconv3x3_relu6_plain_launch(
                                xd.data_ptr(), wd.data_ptr(), bd.data_ptr(), yd.data_ptr(), 16, 56, 56, 144, 1, G, 1,
                                None),
                            lambda G, b0, l, gr, bl: T.plain_dwconv3x3_relu6_elastic_launch(
                                xd.data_ptr(), wd.data_ptr(), bd.data_ptr(), yd.data_ptr(), 16, 56, 56, 144, 1, G, 1,
                                b0, l, gr, bl, None)),
        "softmax_rows": (4 * 128, 256,
                         lambda G, bl: T.plain_softmax_rows_plain_launch(xs.data_ptr(), ys.data_ptr(), 4 * 128, 128,
                                                                         G, 1, None),
                         lambda G, b0, l, gr, bl: T.plain_softmax_rows_elastic_launch(
                             xs.data_ptr(), ys.data_ptr(), 4 * 128, 128, G, 1, b0, l, gr, bl, None)),
        "layernorm_rows": (128, 128,
                           lambda G, bl: T.plain_layernorm_rows_plain_launch(
                               xl.data_ptr(), gl.data_ptr(), bl_.data_ptr(), yl.data_ptr(), 128, 768, 1e-5, G, 1, None),
                           lambda G, b0, l, gr, bl: T.plain_layernorm_rows_elastic_launch(
                               xl.data_ptr(), gl.data_ptr(), bl_.data_ptr(), yl.data_ptr(), 128, 768, 1e-5, G, 1, b0, l,
                               gr, bl, None)),
    }

    def med(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            flush()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return 1000.0 * float(np.median(ts))

    out = {}
    for name, (G, blk, plain, elastic) in cases.items():
        q = [(i * G // 4, (i + 1) * G // 4 - i * G // 4) for i in range(4)]
        t_plain = med(lambda: plain(G, blk))
        t_el = med(lambda: elastic(G, 0, G, G, blk))
        t_4 = med(lambda: [elastic(G, b0, l, l, blk) for b0, l in q])
        out[name] = dict(logical_blocks=G, block=blk, plain_us=round(t_plain, 2), elastic_us=round(t_el, 2),
                         shards4_us=round(t_4, 2), elastic_over_plain=round(t_el / t_plain, 4))
    return out


def launch_gap_us(reps=5, n=32):
    """Extra time of one more back-to-back launch on one stream: n launches of a one-tile
    elementwise op over 8 values against one, per launch (the t_launch of the Eq. (5) launch
    term); minimum over reps."""
    import torch
    from paper_2307_04339_amd import ops
    x = torch.zeros((1, 8), dtype=torch.float16, device="cuda")
    y = torch.empty_like(x)
    op = ops.bn_act(x, y, 1, 8, act="relu")
    best = None
    for _ in range(reps):
        ts = []
        for k in (1, n):
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(k):
                op.launch(0, 1, 1, 256)
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        g = 1000.0 * (ts[1] - ts[0]) / (n - 1)
        best = g if best is None else min(best, g)
    return best


def _median_us(run, reps, flush=None):
    """Median over reps of the time between events around run() on torch's current stream (the
    stream every launch here goes to); flush() before each when given."""
    import torch
    ts = []
    for _ in range(reps):
        if flush is not None:
            flush()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        run()
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    return 1000.0 * float(np.median(ts)), 1000.0 * float(np.mean(ts))


def _plan(lib, T, n):
    import ctypes
    b = (ctypes.c_int64 * n)()
    ln = (ctypes.c_int64 * n)()
    lib.miriam_plan_split(T, n, b, ln)
    return [(int(b[j]), int(ln[j])) for j in range(n)]


def shard_overhead(layer, reps, flush, n_cu, lib, gap_us):
    """Unsharded time of the op and of its balanced 1/2/4/8-shard plans run back to back on one
    stream (each shard a persistent grid of its length, up to the resident capacity, block 256),
    medians over cold-cache repetitions.  The overhead t_plan / t_unsharded - 1 is split as in
    Eq. (5): the launch term LO_blk = (n - 1) t_launch (t_launch: the back-to-back launch gap of
    a one-tile kernel) and the rest, LO_pt, the persistent shards' own cost (rounds a shard leaves
    under-filled, its prologue and its tail)."""
    op = layer.op
    T = op.T
    cap = max(1, op.info.max_wg_per_cu[2])
    base, _ = _median_us(lambda: op.launch(0, T, int(op.info.full_grid), 256), reps, flush)
    res = {"unsharded_us": round(base, 2), "launch_gap_us": round(gap_us, 2), "tiles": T}
    for n in (1, 2, 4, 8):
        if n > T:
            continue
        plan = [(b, l, int(min(l, n_cu * cap)), 256) for (b, l) in _plan(lib, T, n)]
        t, _ = _median_us(lambda: [op.launch(b, l, g, bl) for (b, l, g, bl) in plan], reps, flush)
        lo_blk = (n - 1) * gap_us
        res[f"shards{n}_us"] = round(t, 2)
        res[f"shards{n}_overhead"] = round(t / base - 1.0, 4)
        res[f"shards{n}_lo_blk_us"] = round(lo_blk, 2)
        res[f"shards{n}_lo_pt_us"] = round(t - base - lo_blk, 2)
    return res


def config1_phase(reps, n_cu, lib, gap_us):
    """The single elastic fp32 convolution: x 1x56x56x64 and w 64x64x3x3 ~ U[-1, 1] (seeds 0 and
    1), bias ~ U[-1, 1] (seed 2), stride 1, pad 1, ReLU.  Its 1.75 MB working set stays in the
    caches, so launches are timed warm after 50 warm-up launches: the mean of 1000 launches
    back to back between two events, and the median of 1000 single launches between events.  Then every plan n in {1, 2, 4, 8}
    x block {64, 128, 256} x forward / reverse shard order (persistent grids), each checked
    bitwise against the unsharded output."""
    import torch
    from paper_2307_04339_amd import ops, synth
    xs, _ = synth.storage_tensor((1, 56, 56, 64), "f32", seed=0)
    ws, _ = synth.storage_tensor((64, 3, 3, 64), "f32", seed=1)
    bs = np.random.default_rng(2).uniform(-1, 1, 64).astype(np.float32)
    x, w, bias = (torch.from_numpy(a).cuda() for a in (xs, ws, bs))
    y = torch.empty((1, 56, 56, 64), dtype=torch.float32, device="cuda")
    op = ops.conv2d(x, w, y, stride=1, pad=1, bias=bias, act="relu")
    T = op.T
    full = int(op.info.full_grid)
    for _ in range(50):
        op.launch(0, T, full, 256)
    torch.cuda.synchronize()
    ref = y.clone()
    nb = 1000
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(nb):
        op.launch(0, T, full, 256)
    e1.record()
    e1.synchronize()
    mean_b2b = 1000.0 * e0.elapsed_time(e1) / nb
    med_single, _ = _median_us(lambda: op.launch(0, T, full, 256), max(reps, nb))
    flops = op.info.flops
    out = {"workload": "conv 1x56x56x64 * 64x64x3x3 fp32, bias + ReLU", "tiles": T,
           "tile": [op.info.tile_m, op.info.tile_n], "flops": flops,
           "unsharded_us_back_to_back": round(mean_b2b, 3), "unsharded_us_single_median": round(med_single, 3),
           "tflops": round(flops / (mean_b2b * 1e-6) / 1e12, 2)}
    out["frac_fp32_peak"] = round(out["tflops"] / PEAK_TFLOPS["f32"], 4)
    plans = {}
    bitwise = True
    for n in (1, 2, 4, 8):
        shards = _plan(lib, T, n)
        for block in (64, 128, 256):
            cap = max(1, op.info.max_wg_per_cu[{64: 0, 128: 1, 256: 2}[block]])
            for order in ("fwd", "rev"):
                seq = shards if order == "fwd" else shards[::-1]
                plan = [(b, l, int(min(l, n_cu * cap)), block) for (b, l) in seq]
                run = lambda: [op.launch(b, l, g, bl) for (b, l, g, bl) in plan]
                y.fill_(float("nan"))
                run()
                torch.cuda.synchronize()
                bitwise = bitwise and torch.equal(y.view(torch.int32), ref.view(torch.int32))
                e0.record()
                for _ in range(nb):
                    run()
                e1.record()
                e1.synchronize()
                t = 1000.0 * e0.elapsed_time(e1) / nb
                lo_blk = (n - 1) * gap_us
                plans[f"n{n}_b{block}_{order}"] = {"us": round(t, 3), "overhead": round(t / mean_b2b - 1.0, 4),
                                                   "lo_blk_us": round(lo_blk, 3),
                                                   "lo_pt_us": round(t - mean_b2b - lo_blk, 3)}
    out["launch_gap_us"] = round(gap_us, 3)
    out["plans"] = plans
    out["bitwise_identical_all_plans"] = bool(bitwise)
    ovs = [v["overhead"] for v in plans.values()]
    out["overhead_max"] = round(max(ovs), 4)
    out["overhead_by_shards_b256_fwd"] = {n: plans[f"n{n}_b256_fwd"]["overhead"] for n in (1, 2, 4, 8)}
    return out


def config2_phase(reps, flush, dtype="f16", seed=5):
    """ResNet-18 b1 (fp16): every kernel unsharded with cold caches (roofline per kernel), then
    with a seeded shard plan per layer (n in {1, 2, 3, 4, 8}, block in {64, 128, 256}, forward or
    reverse order, persistent grids) and the network's outputs compared bitwise with the
    unsharded forward pass."""
    import torch
    from paper_2307_04339_amd import models
    from paper_2307_04339_amd import _lib as L
    lib = L.load()
    net = models.resnet18(batch=1, dtype=dtype)
    net.forward()
    torch.cuda.synchronize()
    ref = [l.t["y"].clone() for l in net.layers]
    rng = np.random.default_rng(seed)
    rows = []
    plans = {}
    for i, layer in enumerate(net.layers):
        op = layer.op
        T = op.T
        n = int(min(T, rng.choice([1, 2, 3, 4, 8])))
        block = int(rng.choice([64, 128, 256]))
        shards = _plan(lib, T, n)
        if rng.random() < 0.5:
            shards = shards[::-1]
        cap = max(1, op.info.max_wg_per_cu[{64: 0, 128: 1, 256: 2}[block]])
        plans[i] = [(b, l, int(min(l, 256 * cap)), block) for (b, l) in shards]
        t_un, _ = _median_us(lambda: op.run(), reps, flush)
        t_pl, _ = _median_us(lambda: [op.launch(b, l, g, bl) for (b, l, g, bl) in plans[i]], reps, flush)
        flops = op.info.flops
        if layer.kind == "conv" and layer.params.get("logical_c"):
            flops *= layer.params["logical_c"] / layer.t["x"].shape[-1]
        k = dict(name=layer.name, us=t_un, flops=flops, bytes=op.info.bytes, tiles=T)
        rf = roofline_of(k, dtype)
        rows.append(dict(name=layer.name, tiles=T, path=int(op.info.path), unsharded_us=round(t_un, 2),
                         bound=rf["bound"], achieved=rf["achieved"], unit=rf["unit"], frac=rf["frac"],
                         plan=f"{n}x{block}", sharded_us=round(t_pl, 2), shard_overhead=round(t_pl / t_un - 1.0, 4)))
    for l in net.layers:
        l.t["y"].fill_(float("nan"))
    net.forward(plans=plans)
    torch.cuda.synchronize()
    same = all(torch.equal(l.t["y"].view(torch.int16), r.view(torch.int16)) for l, r in zip(net.layers, ref))
    tot = sum(r["unsharded_us"] for r in rows)
    return {"workload": "resnet18 b1 fp16", "kernels": rows, "kernel_sum_us": round(tot, 2),
            "sharded_sum_us": round(sum(r["sharded_us"] for r in rows), 2),
            "flops": net.flops(), "bitwise_identical_sharded_vs_unsharded": bool(same)}


# ----------------------------------------------------------------- co-run
def run_phase(policy, crit_net, be_nets, n_warm, n_steps, period_ms, arrival, seed, ccfg, with_be=True,
              be_inflight=2):
    import torch
    from paper_2307_04339_amd import synth
    from paper_2307_04339_amd.runtime import Coordinator
    torch.cuda.synchronize()
    co = Coordinator(policy=policy, n_be_streams=max(1, len(be_nets)), **ccfg)
    try:
        ct = co.task(crit_net.ops())
        bts = [co.task(n.ops()) for n in be_nets] if with_be else []
        period_ns = int(period_ms * 1e6)
        n_rel = n_warm + n_steps
        if arrival == "poisson":
            rel = synth.poisson_releases(n_rel, period_ns, seed)
        else:
            rel = synth.periodic_releases(n_rel, period_ns)
        t0 = co.now_ns() + 20_000_000
        crit_tickets = {}
        for i, r in enumerate(rel):
            tk = co.submit(ct, True, release_ns=int(t0 + r), deadline_ns=int(t0 + r + period_ns))
            crit_tickets[tk] = i
        t_win0 = int(t0 + rel[n_warm])
        t_end_rel = int(t0 + rel[-1] + period_ns)
        be_out = {}
        be_done = []   # (task index, t_end)
        be_ticket_task = {}
        for j, bt in enumerate(bts):
            for _ in range(be_inflight):
                tk = co.submit(bt, False)
                be_ticket_task[tk] = j
            be_out[j] = 2
        crit_lat = {}
        while len(crit_lat) < n_rel:
            recs = co.poll()
            for r in recs:
                if r.criticality == 1:
                    crit_lat[crit_tickets[r.ticket]] = (r.t_end_ns - r.t_release_ns, r.t_end_ns)
                else:
                    j = be_ticket_task.pop(r.ticket)
                    be_done.append((j, r.t_end_ns))
                    be_out[j] -= 1
                    if co.now_ns() < t_end_rel:
                        tk = co.submit(bts[j], False)
                        be_ticket_task[tk] = j
                        be_out[j] += 1
            if not recs:
                time.sleep(0.0002)
        t_win1 = max(v[1] for v in crit_lat.values())
        co.drain(120000)
        for r in co.poll():
            if r.criticality == 0:
                be_done.append((be_ticket_task.pop(r.ticket), r.t_end_ns))
        st = co.stats()
        torch.cuda.synchronize()
    finally:
        co.shutdown()
    lat_ms = [crit_lat[i][0] / 1e6 for i in range(n_warm, n_rel)]
    win_s = (t_win1 - t_win0) / 1e9
    per_task = []
    for j, n in enumerate(be_nets if with_be else []):
        cnt = sum(1 for (jj, te) in be_done if jj == j and t_win0 <= te <= t_win1)
        per_task.append(dict(net=n.name, batch=n.batch, req_s=cnt / win_s, img_s=cnt * n.batch / win_s))
    return dict(policy=policy, releases=len(lat_ms), p50_ms=pct(lat_ms, 50), p99_ms=pct(lat_ms, 99),
                mean_ms=float(np.mean(lat_ms)), max_ms=float(np.max(lat_ms)), window_s=win_s, be=per_task,
                be_img_s=sum(p["img_s"] for p in per_task), be_req_s=sum(p["req_s"] for p in per_task),
                crit_req_s=n_steps / win_s, launches=st.launches,
                decision_us=st.decision_ns_total / max(1, st.decisions) / 1000.0,
                eq2_violations=st.eq2_violations)


# ------------------------------------------------------------ cpu baseline
def _host_info():
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model,
            "affinity_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}


def _oracle_layers(net_name, kw):
    """Layer shapes of one inference (batch 1) of a workload network, as oracle calls."""
    from paper_2307_04339_amd import models  # shapes only
    net = models.BUILDERS[net_name](**dict(kw, batch=1))
    out = []
    for l in net.layers:
        p = dict(l.params)
        shp = {k: (tuple(v.shape) if hasattr(v, "shape") else None) for k, v in l.t.items()}
        if l.kind == "conv" and p.get("logical_c"):
            lc = p["logical_c"]  # the oracle convolves the logical channels only
            shp["x"] = shp["x"][:-1] + (lc,)
            shp["w"] = shp["w"][:-1] + (lc,)
        out.append((l.kind, shp, p))
    del net
    return out


def _oracle_inference(layers, rng):
    """Run every layer of one inference through the oracle on random inputs of its shape;
    returns the oracle time in seconds (input generation excluded)."""
    from oracle import oracle as orc
    tot = 0.0
    for kind, shp, p in layers:
        if kind == "conv":
            x = rng.uniform(-1, 1, shp["x"])
            w = rng.uniform(-1, 1, shp["w"])
            K = shp["w"][0]
            t0 = time.perf_counter()
            y = orc.conv2d_raw(x, w, stride=p["stride"], pad=p["pad"])
            orc.epilogue(y, bias=np.zeros(K), bn=(np.ones(K), np.zeros(K), np.zeros(K), np.ones(K)),
                         residual=y if shp.get("residual") else None, act=p["act"])
        elif kind == "dwconv":
            x = rng.uniform(-1, 1, shp["x"])
            C = shp["x"][-1]
            w = rng.uniform(-1, 1, (C, 3, 3, 1))
            t0 = time.perf_counter()
            y = orc.conv2d_raw(x, w, stride=p["stride"], pad=p["pad"], groups=C)
            orc.epilogue(y, bn=(np.ones(C), np.zeros(C), np.zeros(C), np.ones(C)), act=p["act"])
        elif kind in ("maxpool", "avgpool"):
            x = rng.uniform(-1, 1, shp["x"])
            fn = orc.maxpool if kind == "maxpool" else orc.avgpool
            t0 = time.perf_counter()
            fn(x, p["k"], p["stride"], p["pad"])
        elif kind == "gemm":
            x = rng.uniform(-1, 1, shp["x"])
            w = rng.uniform(-1, 1, shp["w"])
            t0 = time.perf_counter()
            orc.linear(x, w, bias=np.zeros(shp["w"][0]), residual=np.zeros((shp["x"][0], shp["w"][0]))
                       if shp.get("residual") else None, act=p["act"])
        elif kind == "bgemm":
            B, H, S, D = p["B"], p["H"], p["S"], p["D"]
            q = rng.uniform(-1, 1, (S, D))
            pm = rng.uniform(0, 1, (S, S))
            t0 = time.perf_counter()
            for _ in range(B * H):
                if p["which"] == "qk":
                    orc.gemm_nt(q, q)
                else:
                    orc.gemm_nn(pm, q)
        elif kind == "softmax":
            n = shp["x"][-1]
            x = rng.uniform(-1, 1, (int(np.prod(shp["x"])) // n, n))
            t0 = time.perf_counter()
            orc.softmax_rows(x, scale=p["scale"])
        elif kind == "layernorm":
            x = rng.uniform(-1, 1, shp["x"])
            n = shp["x"][-1]
            t0 = time.perf_counter()
            orc.layernorm_rows(x, np.ones(n), np.zeros(n), eps=p["eps"])
        else:
            raise ValueError(kind)
        tot += time.perf_counter() - t0
    return tot


def cpu_baseline(dtype, seed=0):
    """The CPU oracle (plain C loops in double precision) timed on this host: one inference of
    each workload network (batch 1, every layer in full, random inputs of the layer shapes) and
    the single fp32 convolution (median of 5), single-threaded and on every host core the
    process may use (OpenMP over output elements in the convolution and the products; pooling,
    epilogues, softmax and LayerNorm stay on one thread).  `value` is VGG-16 images per second
    on all cores."""
    from oracle import oracle as orc
    rng = np.random.default_rng(seed)
    host = _host_info()
    all_cores = host["affinity_cpus"] or host["nproc"] or 1
    omp = int(os.environ.get("OMP_NUM_THREADS", "0") or 0)
    if omp > 0:
        all_cores = min(all_cores, omp)
    nets = [("vgg16", {}), ("resnet18", {}), ("mobilenetv2", {}), ("encoder", {"seq": 128})]
    shapes = {n: _oracle_layers(n, dict(kw, dtype=dtype)) for n, kw in nets}
    prev = orc.set_threads()
    res = {}
    t_start = time.time()
    try:
        x = rng.uniform(-1, 1, (1, 56, 56, 64))
        w = rng.uniform(-1, 1, (64, 3, 3, 64))
        for label, th in (("1_thread", 1), (f"{all_cores}_threads", all_cores)):
            used = orc.set_threads(th)
            ts = []
            for _ in range(5):
                t0 = time.perf_counter()
                orc.conv2d(x, w, stride=1, pad=1, bias=np.zeros(64), act="relu")
                ts.append(time.perf_counter() - t0)
            c1 = float(np.median(ts))
            per = {n: _oracle_inference(shapes[n], rng) for n, _ in nets}
            res[label] = {"threads": used, "config1_conv_ms": round(1000 * c1, 2),
                          "config1_conv_gflops": round(231211008 / c1 / 1e9, 2),
                          "ms_per_inference": {n: round(1000 * t, 1) for n, t in per.items()}}
    finally:
        orc.set_threads(prev)
    wall = time.time() - t_start
    top = res[f"{all_cores}_threads"]
    vgg_ms = top["ms_per_inference"]["vgg16"]
    return dict(value=round(1000.0 / vgg_ms, 4), unit="img/s", cores=top["threads"], kind="oracle",
                sample=(f"one VGG-16 image (batch 1, every layer in full, fp64) on {top['threads']} host threads; "
                        f"also ResNet-18, MobileNetV2 and the encoder (seq 128) per image and the single fp32 "
                        f"convolution, on 1 and {top['threads']} threads; {wall:.1f} s of CPU work"),
                host=host, runs=res)


def profile_op(args, cfg):
    """Each listed layer's unsharded launch --reps times back to back (layers in the order
    given), then a plain device copy of 256 MiB --reps times, whose FETCH_SIZE / WRITE_SIZE
    calibrate the traffic counters.  Prints one JSON line per layer and one for the copy."""
    import torch
    from paper_2307_04339_amd import models
    nets = {}
    targets = []
    for item in args.profile_op.split(","):
        net_name, layer_name = item.split(".", 1)
        kw = next((dict(k) for (n, k) in [cfg["crit"]] + cfg["be"] if n == net_name), None)
        if kw is None:
            raise SystemExit(f"{net_name} is not part of workload {args.config}")
        if net_name not in nets:
            nets[net_name] = models.BUILDERS[net_name](dtype=cfg["dtype"], **kw)
            nets[net_name].forward()
        targets.append((item, next(l for l in nets[net_name].layers if l.name == layer_name)))
    src = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for item, layer in targets:
        e0.record()
        for _ in range(args.reps):
            layer.op.run()
        e1.record()
        e1.synchronize()
        us = 1000.0 * e0.elapsed_time(e1) / args.reps
        info = layer.op.info
        print(json.dumps({"op": item, "reps": args.reps, "avg_us": round(us, 3), "tiles": layer.op.T,
                          "tile": [info.tile_m, info.tile_n], "path": int(info.path), "grid": int(info.full_grid),
                          "flops": info.flops, "bytes": info.bytes}), flush=True)
    e0.record()
    for _ in range(args.reps):
        dst.copy_(src)
    e1.record()
    e1.synchronize()
    cus = 1000.0 * e0.elapsed_time(e1) / args.reps
    print(json.dumps({"op": "copy", "reps": args.reps, "copy_bytes_each_way": src.numel() * 4,
                      "copy_avg_us": round(cus, 3)}), flush=True)


# ------------------------------------------------------------------- main
PHASE_POLICY = {"solo": "elastic", "elastic_pause": "elastic", "multistream_cu": "multistream", "elastic_cu": "elastic"}
# co-run phases of the main workload and of the sub-line workloads
MAIN_PHASES = ("solo", "sequential", "multistream", "multistream_cu", "ib", "elastic", "elastic_cu", "elastic_pause")
SUB_PHASES = ("solo", "sequential", "elastic", "elastic_pause")


def coordinator_cfg(args, cfg):
    guard = args.release_guard if args.release_guard >= 0 else int(cfg["arrival"] == "periodic")
    warm = args.warm_critical if args.warm_critical >= 0 else guard
    arm = args.arm_lead_us if args.arm_lead_us >= 0 else (500.0 if guard else 0.0)
    whole = args.whole_when_clear if args.whole_when_clear >= 0 else guard
    inflight_us = args.inflight_us if args.inflight_us >= 0 else 100.0
    event_us = args.event_us if args.event_us >= 0 else inflight_us / 3.0
    return dict(quantum_us=args.quantum_us, inflight_depth=args.depth, inflight_us=inflight_us, event_us=event_us,
                busy_policy=args.busy_policy, profile_reps=3, graphs=args.graphs, release_guard=guard,
                warm_critical=warm, arm_lead_us=arm, segments=args.segments, whole_when_clear=whole,
                whole_margin=args.whole_margin)


def build_workload(cfg, n_inst):
    from paper_2307_04339_amd import models
    dtype = cfg["dtype"]
    cname, ckw = cfg["crit"]
    crit_net = models.BUILDERS[cname](dtype=dtype, **ckw)
    be_nets = [models.BUILDERS[n](dtype=dtype, **kw) for (n, kw) in cfg["be"]]
    be_tasks = []  # every instance of every best-effort network
    for first, (n, kw) in zip(be_nets, cfg["be"]):
        be_tasks.append(first)
        for _ in range(n_inst - 1):
            be_tasks.append(models.BUILDERS[n](dtype=dtype, share=first, **kw))
    crit_net.forward()
    for n in be_tasks:
        n.forward()
    return crit_net, be_nets, be_tasks


def corun(args, cfg, phases, crit_net, be_tasks, ccfg, pps):
    """Run the co-run phases of one workload; returns (runs, summary)."""
    runs = {}
    for ph in MAIN_PHASES:
        if ph not in phases:
            continue
        log(f"  phase {ph} ...")
        policy = PHASE_POLICY.get(ph, ph)
        pcfg = dict(ccfg, busy_policy=1) if ph == "elastic_pause" else dict(ccfg)
        if ph in ("multistream_cu", "elastic_cu"):
            # normal streams masked off the top cu_reserve CUs: a spatial share for the critical
            # stream (which keeps every CU, or only those with --crit-cu-exclusive) next to the
            # paper's fill rule or plain multi-stream
            pcfg = dict(ccfg, be_cu_reserve=args.cu_reserve, crit_cu_exclusive=args.crit_cu_exclusive)
        runs[ph] = run_phase(policy, crit_net, be_tasks, args.warmup * pps, args.steps * pps, cfg["period_ms"],
                             cfg["arrival"], seed=11, ccfg=pcfg, with_be=(ph != "solo"))
        r = runs[ph]
        log(f"    p50 {r['p50_ms']:.3f} ms  p99 {r['p99_ms']:.3f} ms  be {r['be_img_s']:.1f} img/s "
            f"launches {r['launches']} releases {r['releases']}")
    main_name = next((n for n in ("elastic_pause", "elastic") if n in runs), None)
    main_run = runs[main_name] if main_name else next(iter(runs.values()), None)
    summary = {}
    foreknowledge = bool(ccfg["release_guard"] or ccfg["arm_lead_us"] > 0 or ccfg["whole_when_clear"])
    if "solo" in runs and main_run:
        solo = runs["solo"]
        crit = {"policy": main_name, "busy_policy": 1 if main_name == "elastic_pause" else 0,
                "release_foreknowledge": foreknowledge,
                "releases": main_run["releases"],
                "solo_p50_ms": round(solo["p50_ms"], 4), "solo_p99_ms": round(solo["p99_ms"], 4),
                "corun_p50_ms": round(main_run["p50_ms"], 4), "corun_p99_ms": round(main_run["p99_ms"], 4),
                "p99_overhead": round(main_run["p99_ms"] / solo["p99_ms"] - 1.0, 4)}
        for other in ("elastic", "elastic_cu", "multistream", "multistream_cu", "ib", "sequential"):
            if other in runs and other != main_name:
                crit[f"{other}_p99_overhead"] = round(runs[other]["p99_ms"] / solo["p99_ms"] - 1.0, 4)
        summary["critical"] = crit
    if "sequential" in runs and main_run:
        seq = runs["sequential"]
        be = {"policy": main_name,
              "elastic_img_s": round(main_run["be_img_s"], 2), "sequential_img_s": round(seq["be_img_s"], 2),
              "speedup_vs_sequential": round(main_run["be_img_s"] / max(1e-9, seq["be_img_s"]), 3),
              "sequential_p99_ms": round(seq["p99_ms"], 4)}
        summary["best_effort"] = be
    if "elastic" in runs and "solo" in runs:
        el = runs["elastic"]
        pr = {"busy_policy": 0, "release_foreknowledge": foreknowledge,
              "p50_ms": round(el["p50_ms"], 4), "p99_ms": round(el["p99_ms"], 4),
              "p99_overhead": round(el["p99_ms"] / runs["solo"]["p99_ms"] - 1.0, 4),
              "be_img_s": round(el["be_img_s"], 2)}
        if "sequential" in runs:
            pr["speedup_vs_sequential"] = round(el["be_img_s"] / max(1e-9, runs["sequential"]["be_img_s"]), 3)
        summary["paper_rule"] = pr
    if "elastic_cu" in runs and "solo" in runs:
        el = runs["elastic_cu"]
        pr = {"busy_policy": 0, "cu_reserve": args.cu_reserve, "crit_cu_exclusive": args.crit_cu_exclusive,
              "p50_ms": round(el["p50_ms"], 4), "p99_ms": round(el["p99_ms"], 4),
              "p99_overhead": round(el["p99_ms"] / runs["solo"]["p99_ms"] - 1.0, 4),
              "be_img_s": round(el["be_img_s"], 2)}
        if "sequential" in runs:
            pr["speedup_vs_sequential"] = round(el["be_img_s"] / max(1e-9, runs["sequential"]["be_img_s"]), 3)
        summary["paper_rule_cu_masked"] = pr
    phases_out = {ph: {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()} for ph, r in runs.items()}
    return runs, main_name, main_run, summary, phases_out


def vendor_context(layer, reps, flush, ours_us):
    """A convolution's shape through the vendor libraries, for context: torch's
    conv2d on channels-last tensors and on NCHW copies (MIOpen; convolution only, without the
    fused BN and activation) and the equivalent dense product (M = N*Ho*Wo, N = K, K = KH*KW*C; hipBLASLt via
    torch.matmul).  Same eviction read before each launch and HIP events as the per-layer times."""
    import torch
    import torch.nn.functional as F
    t = layer.t
    x, w = t["x"], t["w"]
    stride, pad = layer.params["stride"], layer.params["pad"]
    N, H, W, C = x.shape
    K, KH, KW, _ = w.shape
    xc = x.permute(0, 3, 1, 2)  # NCHW view of the NHWC tensor: channels-last memory
    wc = w.permute(0, 3, 1, 2).contiguous(memory_format=torch.channels_last)
    y = F.conv2d(xc, wc, stride=stride, padding=pad)
    torch.cuda.synchronize()
    conv_us, _ = _median_us(lambda: F.conv2d(xc, wc, stride=stride, padding=pad), reps, flush)
    xn, wn = xc.contiguous(), w.permute(0, 3, 1, 2).contiguous()  # NCHW copies
    F.conv2d(xn, wn, stride=stride, padding=pad)
    torch.cuda.synchronize()
    conv_nchw_us, _ = _median_us(lambda: F.conv2d(xn, wn, stride=stride, padding=pad), reps, flush)
    del xn, wn
    Ho, Wo = y.shape[2], y.shape[3]
    M, Kd = N * Ho * Wo, KH * KW * C
    A = (torch.rand(M, Kd, device="cuda") * 2 - 1).to(x.dtype)
    B = (torch.rand(K, Kd, device="cuda") * 0.1).to(x.dtype)
    gemm_us, _ = _median_us(lambda: A @ B.t(), reps, flush)
    del A, B, y
    return {"ours_us": round(ours_us, 2), "miopen_conv2d_us": round(conv_us, 2),
            "miopen_conv2d_nchw_us": round(conv_nchw_us, 2),
            "hipblaslt_gemm_us": round(gemm_us, 2), "gemm_shape": [M, K, Kd],
            "note": "torch conv2d (MIOpen; channels-last, and NCHW copies) without the fused BN and activation, and the "
                    "equivalent dense GEMM through torch.matmul (hipBLASLt); cold caches, HIP events"}


# kernels whose shard overhead is reported beside the dominant kernel's, per workload
OVERHEAD_KERNELS = {"corun-resnet18-vgg16-fp16": ["vgg16.conv2_2"]}


def kernel_phase(args, cfg, be_nets, crit_net, dev, L, result):
    """Per-kernel timing of the workload's networks; the dominant kernel's roofline, shard
    overhead (with its Eq. (5) decomposition), index functions and transformed kernels."""
    dtype = cfg["dtype"]
    flush = CacheFlush()
    table = []
    for n in be_nets + [crit_net]:
        for k in time_layers(n, args.reps, flush):
            k["net"] = n.name
            table.append(k)
    dom_net = be_nets[0]
    dom = max((k for k in table if k["net"] == dom_net.name), key=lambda k: k["us"])
    kern = roofline_of(dom, dtype)
    kern["kernel"] = f"{dom_net.name}.{dom['name']}"
    kern["launch_us"] = round(dom["us"], 2)
    kern["flops_per_launch"] = dom["flops"]
    kern["bytes_per_launch"] = dom["bytes"]
    layer = next(l for l in dom_net.layers if l.name == dom["name"])
    kern["tile"] = [layer.op.info.tile_m, layer.op.info.tile_n]
    kern["traffic"] = measured_traffic(args.config, kern["kernel"], kern["tile"], layer.op.info.path,
                                       int(layer.op.info.full_grid))
    # the vendor libraries on the longest convolution of the dominant network (the dominant
    # kernel itself when it is one)
    convs = [k for k in table if k["net"] == dom_net.name
             and next(x for x in dom_net.layers if x.name == k["name"]).kind == "conv"]
    vdom = max(convs, key=lambda k: k["us"]) if convs else None
    if vdom is not None:
        vlayer = next(x for x in dom_net.layers if x.name == vdom["name"])
        log("  vendor context ...")
        result["vendor_context"] = {"kernel": f"{dom_net.name}.{vdom['name']}",
                                    **vendor_context(vlayer, args.reps, flush, vdom["us"])}
        # every convolution of the dominant network, same comparison
        per = []
        for k in table:
            if k["net"] != dom_net.name:
                continue
            l = next(x for x in dom_net.layers if x.name == k["name"])
            if l.kind != "conv":
                continue
            v = vendor_context(l, args.reps, flush, k["us"])
            per.append(dict(name=l.name, ours_us=v["ours_us"], miopen_us=min(v["miopen_conv2d_us"],
                                                                               v["miopen_conv2d_nchw_us"]),
                            hipblaslt_gemm_us=v["hipblaslt_gemm_us"]))
        result["vendor_context"]["layers"] = per
    gap = launch_gap_us()
    result["launch_gap_us"] = round(gap, 3)
    log("  shard overhead ...")
    ovh = {"kernel": kern["kernel"], **shard_overhead(layer, args.reps, flush, dev.n_cu, L.load(), gap)}
    result["elastic_overhead"] = ovh
    # the same split for the workload's largest pipelined contraction when another kernel is
    # the longest (the three longest VGG-16 b8 layers are within a few microseconds)
    more = []
    for name in OVERHEAD_KERNELS.get(args.config, []):
        net_name, lname = name.split(".", 1)
        if name == kern["kernel"] or net_name != dom_net.name:
            continue
        l2 = next(l for l in dom_net.layers if l.name == lname)
        more.append({"kernel": name, **shard_overhead(l2, args.reps, flush, dev.n_cu, L.load(), gap)})
    if more:
        result["elastic_overhead_more"] = more
    log("  index functions ...")
    result["index_function"] = {"net": dom_net.name, "layers": index_function_cost(dom_net, args.reps, flush, L)}
    log("  transformed kernels ...")
    result["transformed_kernels"] = transformed_overhead(args.reps, flush)
    result["kernels"] = [dict(net=k["net"], name=k["name"], us=round(k["us"], 2), tiles=k["tiles"],
                              **{kk: vv for kk, vv in roofline_of(k, dtype).items()
                                 if kk in ("bound", "achieved", "unit", "frac")})
                         for k in sorted(table, key=lambda k: -k["us"])[:16]]
    result["be_solo_ms_per_request"] = {n.name: round(sum(k["us"] for k in table if k["net"] == n.name) / 1000, 3)
                                        for n in be_nets}
    result["crit_kernel_sum_ms"] = round(sum(k["us"] for k in table if k["net"] == crit_net.name) / 1000, 3)
    del flush
    return kern


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--periods-per-step", type=int, default=25,
                    help="critical release periods per step: K steps time K x this many releases per phase")
    ap.add_argument("--config", default=DEFAULT_CONFIG, choices=sorted(CONFIGS))
    ap.add_argument("--sub-configs", default="auto",
                    help="comma-separated other co-run workloads reported as sub-lines ('auto': every other "
                         "workload; 'none')")
    ap.add_argument("--reps", type=int, default=20, help="repetitions per kernel timing")
    ap.add_argument("--quantum-us", type=float, default=40.0)
    ap.add_argument("--depth", type=int, default=32)
    ap.add_argument("--inflight-us", type=float, default=-1.0,
                    help="normal work kept queued on the GPU (it bounds the wait of an unannounced critical "
                         "release); -1: 100")
    ap.add_argument("--event-us", type=float, default=-1.0,
                    help="estimated normal work between completion events; -1: a third of the in-flight budget")
    ap.add_argument("--busy-policy", type=int, default=0,
                    help="normal shards next to a running critical kernel in the 'elastic' phase: 0 paper rule, "
                         "1 none, 2 smallest ('elastic_pause' always holds back)")
    ap.add_argument("--graphs", type=int, default=1, choices=(0, 1),
                    help="1: whole-request launches replay each task's captured HIP graph")
    ap.add_argument("--release-guard", type=int, default=-1, choices=(-1, 0, 1),
                    help="1: hold normal shards that would still run at the next timed critical "
                         "release; -1: on for periodic arrivals (release times known ahead), off for Poisson")
    ap.add_argument("--warm-critical", type=int, default=-1, choices=(-1, 0, 1),
                    help="1: warm the critical task's parameters in the caches ahead of each release "
                         "(needs the release guard); -1: follow the release guard")
    ap.add_argument("--arm-lead-us", type=float, default=-1.0,
                    help="queue each timed critical request behind a gate this long before its release "
                         "(0 = launch at the release); -1: 500 with the release guard, else 0")
    ap.add_argument("--segments", type=int, default=0, choices=(0, 1),
                    help="1: runs of short normal ops within one quantum go out as one captured unit")
    ap.add_argument("--be-instances", type=int, default=0,
                    help="instances of each best-effort network (shared weights, separate activation "
                         "buffers), each its own closed-loop task and stream; Sequential still runs one "
                         "request at a time.  0: the workload's default (3 for the two-task co-runs, 1 for "
                         "the four-task mix, whose three networks already give three streams)")
    ap.add_argument("--phases", default="kernels,config1,config2," + ",".join(MAIN_PHASES) + ",sub,cpu",
                    help="kernels, config1 (single fp32 conv), config2 (ResNet-18 b1 per kernel), the co-run "
                         "phases " + ", ".join(MAIN_PHASES) + ", sub (other workloads), cpu (oracle baseline)")
    ap.add_argument("--whole-when-clear", type=int, default=-1,
                    help="launch normal requests whole when they end before the next known critical "
                         "release (-1: with the release guard)")
    ap.add_argument("--whole-margin", type=float, default=0.0,
                    help="factor on the estimate of whole-request launches (0: the library's 2.0)")
    ap.add_argument("--cu-reserve", type=int, default=64,
                    help="multistream_cu / elastic_cu phases: compute units left out of the normal streams' CU mask")
    ap.add_argument("--crit-cu-exclusive", type=int, default=1, choices=(0, 1),
                    help="multistream_cu / elastic_cu phases: the critical stream gets only the reserved CUs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-op", default=None, metavar="NET.LAYER[,NET.LAYER...]",
                    help="only launch the listed layers (unsharded) --reps times each, then a 256 MiB device "
                         "copy --reps times as the counter calibration kernel (for rocprofv3 runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(with several GPUs each critical / best-effort task set runs on a device of its own, "
              "so the co-run is measured on one)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2307_04339_amd import _lib as L
    from paper_2307_04339_amd.ops import device_info

    cfg = CONFIGS[args.config]
    dtype = cfg["dtype"]
    if args.profile_op:
        profile_op(args, cfg)
        return
    pps = max(1, args.periods_per_step)
    dev = device_info()
    log(f"device {dev.arch.decode()} cus={dev.n_cu} config={args.config}")
    phases = set(args.phases.split(","))
    n_inst = args.be_instances if args.be_instances > 0 else cfg["be_instances"]
    result = {}
    kern = None
    if phases & ({"kernels"} | set(MAIN_PHASES)):
        crit_net, be_nets, be_tasks = build_workload(cfg, n_inst)
        torch.cuda.synchronize()
        if "kernels" in phases:
            log("timing kernels ...")
            kern = kernel_phase(args, cfg, be_nets, crit_net, dev, L, result)
            torch.cuda.empty_cache()
    if "config1" in phases:
        log("single fp32 elastic convolution ...")
        result["config1"] = config1_phase(200, dev.n_cu, L.load(), launch_gap_us())
    if "config2" in phases:
        log("resnet18 b1 per kernel ...")
        fl = CacheFlush()
        result["config2"] = config2_phase(args.reps, fl)
        del fl
        torch.cuda.empty_cache()

    ccfg = coordinator_cfg(args, cfg)
    main_name, main_run, summary, phases_out = None, None, {}, {}
    if phases & set(MAIN_PHASES):
        log(f"co-run {args.config} ...")
        _, main_name, main_run, summary, phases_out = corun(args, cfg, phases, crit_net, be_tasks, ccfg, pps)
    value = main_run["be_img_s"] if main_run else float("nan")
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "img/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1000.0 * main_run["window_s"] / args.steps, 4) if main_run else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": args.config, "hw_queues": int(os.environ.get("GPU_MAX_HW_QUEUES", "4")),
                   "critical": f"{cfg['crit'][0]} b{cfg['crit'][1]['batch']} {cfg['arrival']} every {cfg['period_ms']} ms",
                   "best_effort": [f"{n} b{kw['batch']} closed-loop" for n, kw in cfg["be"]],
                   "be_instances": n_inst, "periods_per_step": pps,
                   "releases_timed_per_phase": args.steps * pps,
                   "main_line": "Miriam coordinator, hold-back rule (busy policy 1: no new normal shard while a "
                                "critical kernel runs)" + (", with the known periodic release times (release "
                                "guard, cache warming, armed gate, whole requests before the next release)"
                                if ccfg["release_guard"] else ""),
                   "quantum_us": args.quantum_us, "inflight_depth": args.depth,
                   "inflight_us": ccfg["inflight_us"], "event_us": round(ccfg["event_us"], 2),
                   "busy_policy": 1 if main_name == "elastic_pause" else 0,
                   "graphs": args.graphs, "release_guard": ccfg["release_guard"],
                   "warm_critical": ccfg["warm_critical"], "arm_lead_us": ccfg["arm_lead_us"],
                   "segments": args.segments, "whole_when_clear": ccfg["whole_when_clear"],
                   "cu_reserve_multistream_cu": args.cu_reserve},
    }
    out.update(summary)
    if phases_out:
        out["phases"] = phases_out
    if kern:
        out["roofline"] = kern
    out.update(result)
    if phases & set(MAIN_PHASES):
        del crit_net, be_nets, be_tasks
        torch.cuda.empty_cache()

    if "sub" in phases and args.sub_configs != "none":
        subs = [c for c in sorted(CONFIGS) if c != args.config] if args.sub_configs == "auto" \
            else [c for c in args.sub_configs.split(",") if c]
        out["sub_configs"] = {}
        for name in subs:
            scfg = CONFIGS[name]
            log(f"co-run {name} (sub-line) ...")
            s_inst = scfg["be_instances"]
            c_net, b_nets, b_tasks = build_workload(scfg, s_inst)
            torch.cuda.synchronize()
            s_ccfg = coordinator_cfg(args, scfg)
            _, s_main, s_run, s_sum, s_ph = corun(args, scfg, set(SUB_PHASES), c_net, b_tasks, s_ccfg, pps)
            out["sub_configs"][name] = dict(
                value=round(s_run["be_img_s"], 3), unit="img/s", dtype=scfg["dtype"],
                critical_task=f"{scfg['crit'][0]} b{scfg['crit'][1]['batch']} {scfg['arrival']} every "
                              f"{scfg['period_ms']} ms",
                best_effort_tasks=[f"{n} b{kw['batch']} closed-loop" for n, kw in scfg["be"]], be_instances=s_inst,
                release_guard=s_ccfg["release_guard"], **s_sum, phases=s_ph)
            del c_net, b_nets, b_tasks
            torch.cuda.empty_cache()

    if "cpu" in phases and not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(dtype)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
