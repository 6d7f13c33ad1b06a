#!/usr/bin/env python3
"""Miriam co-run benchmark on one MI355X.

Default workload (two-task co-run, fp16): the critical task is a ResNet-18-shaped
CNN at batch 1 released every 20 ms; the best-effort task is a VGG-16-shaped CNN
at batch 8 run closed-loop on 224x224 inputs.  Inputs and weights are seeded
synthetic tensors resident in HBM before timing starts.

Phases: (1) per-kernel timing of the best-effort network with HIP events (the
roofline object for its dominant kernel and the elastic-shard overhead of that
kernel); (2) critical task alone (solo); (3) the Sequential baseline; (4) Miriam
(elastic policy).  A "step" is one critical release period of the co-run; W
warm-up periods are run first, then exactly K timed periods.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

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


def measured_traffic(workload, kernel, tile, path):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None when
    there is none for this workload / kernel path / tile or the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            entries = json.load(f)["entries"]
    except (OSError, ValueError, KeyError):
        return None
    e = entries.get(f"{workload}:{kernel}")
    if (not e or list(e.get("tile", [])) != list(tile) or e.get("path") != path
            or e.get("source_sha256") != kernel_source_hash()):
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
    and a 1024^3 fp32 product with 16 x 16 shared-memory tiles."""
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


def shard_overhead(layer, reps, flush, n_cu, lib):
    import ctypes
    import torch
    op = layer.op
    T = op.T
    cap = max(1, op.info.max_wg_per_cu[2])

    def timed(plan):
        # median over the repetitions: a single host-side stall between two shard launches
        # would otherwise dominate a 20-sample mean
        ts = []
        for _ in range(reps):
            flush()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for (b, l, g, bl) in plan:
                op.launch(b, l, g, bl)
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return 1000.0 * float(np.median(ts))

    base = timed([(0, T, int(op.info.full_grid), 256)])
    res = {"unsharded_us": round(base, 2)}
    for n in (1, 2, 4, 8):
        if n > T:
            continue
        b = (ctypes.c_int64 * n)()
        ln = (ctypes.c_int64 * n)()
        lib.miriam_plan_split(T, n, b, ln)
        plan = [(b[j], ln[j], int(min(ln[j], n_cu * cap)), 256) for j in range(n)]
        t = timed(plan)
        res[f"shards{n}_us"] = round(t, 2)
        res[f"shards{n}_overhead"] = round(t / base - 1.0, 4)
    return res


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
    return dict(policy=policy, p50_ms=pct(lat_ms, 50), p99_ms=pct(lat_ms, 99), mean_ms=float(np.mean(lat_ms)),
                max_ms=float(np.max(lat_ms)), window_s=win_s, be=per_task,
                be_img_s=sum(p["img_s"] for p in per_task), be_req_s=sum(p["req_s"] for p in per_task),
                crit_req_s=n_steps / win_s, launches=st.launches,
                decision_us=st.decision_ns_total / max(1, st.decisions) / 1000.0,
                eq2_violations=st.eq2_violations)


# ------------------------------------------------------------ cpu baseline
def cpu_baseline(net_name, kw, budget_macs=1.5e9, seed=0):
    """Oracle time of one best-effort inference image, from a bounded sample: each
    convolution computes sampled output pixels (all channels), scaled by the pixel
    count; pooling and FC layers run in full for one image."""
    from oracle import oracle as orc
    from paper_2307_04339_amd import models  # shapes only
    rng = np.random.default_rng(seed)
    shapes = []
    # replay the network's layer shapes on the host (batch 1)
    import torch  # noqa: F401
    net = models.BUILDERS[net_name](**dict(kw, batch=1))
    for l in net.layers:
        x = l.t.get("x")
        xs = None if x is None else tuple(x.shape)
        ws = None if l.t.get("w") is None else tuple(l.t["w"].shape)
        if l.kind == "conv" and l.params.get("logical_c"):
            lc = l.params["logical_c"]  # the oracle convolves the logical channels only
            xs = xs[:-1] + (lc,)
            ws = ws[:-1] + (lc,)
        shapes.append((l.kind, xs, l.t["y"].shape, ws, dict(l.params)))
    del net
    total = 0.0
    t_start = time.time()
    for kind, xs, ys, ws, p in shapes:
        if kind == "conv":
            N, H, W, C = xs
            K, KH, KW, _ = ws
            _, Ho, Wo, _ = ys
            npx = Ho * Wo
            per = K * KH * KW * C
            s = int(max(1, min(npx, budget_macs // per)))
            crops = rng.uniform(-1, 1, (s, KH, KW, C))
            w = rng.uniform(-1, 1, ws)
            t0 = time.perf_counter()
            orc.conv2d(crops, w, stride=1, pad=0, act=p["act"])
            total += (time.perf_counter() - t0) * npx / s
        elif kind in ("maxpool", "avgpool"):
            x = rng.uniform(-1, 1, xs)
            fn = orc.maxpool if kind == "maxpool" else orc.avgpool
            t0 = time.perf_counter()
            fn(x, p["k"], p["stride"], p["pad"])
            total += time.perf_counter() - t0
        elif kind == "gemm":
            x = rng.uniform(-1, 1, (1, xs[1]))
            w = rng.uniform(-1, 1, ws)
            t0 = time.perf_counter()
            orc.linear(x, w, act=p["act"])
            total += time.perf_counter() - t0
    wall = time.time() - t_start
    return dict(value=round(1.0 / total, 5), unit="img/s", cores=1, kind="oracle",
                sample=f"one {net_name} image: <= {budget_macs:.0e} MACs of sampled output pixels per "
                       f"convolution (scaled by pixel count), pooling and FC in full; "
                       f"{wall:.1f} s of CPU work, single thread")


def profile_op(args, cfg):
    """One layer's unsharded launch --reps times, then a plain device copy of 256 MiB
    --reps times (its FETCH_SIZE / WRITE_SIZE calibrate the traffic counters)."""
    import torch
    from paper_2307_04339_amd import models
    net_name, layer_name = args.profile_op.split(".", 1)
    kw = next((dict(k) for (n, k) in [cfg["crit"]] + cfg["be"] if n == net_name), None)
    if kw is None:
        raise SystemExit(f"{net_name} is not part of workload {args.config}")
    net = models.BUILDERS[net_name](dtype=cfg["dtype"], **kw)
    layer = next(l for l in net.layers if l.name == layer_name)
    src = torch.empty(64 * 1024 * 1024, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1.0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.reps):
        layer.op.run()
    e1.record()
    e1.synchronize()
    us = 1000.0 * e0.elapsed_time(e1) / args.reps
    e0.record()
    for _ in range(args.reps):
        dst.copy_(src)
    e1.record()
    e1.synchronize()
    cus = 1000.0 * e0.elapsed_time(e1) / args.reps
    info = layer.op.info
    print(json.dumps({"op": args.profile_op, "reps": args.reps, "avg_us": round(us, 3),
                      "tiles": layer.op.T, "tile": [info.tile_m, info.tile_n],
                      "flops": info.flops, "bytes": info.bytes,
                      "copy_bytes_each_way": src.numel() * 4, "copy_avg_us": round(cus, 3)}), flush=True)


# ------------------------------------------------------------------- main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=500)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default=DEFAULT_CONFIG, choices=sorted(CONFIGS))
    ap.add_argument("--reps", type=int, default=20, help="repetitions per kernel timing")
    ap.add_argument("--quantum-us", type=float, default=40.0)
    ap.add_argument("--depth", type=int, default=32)
    ap.add_argument("--inflight-us", type=float, default=-1.0,
                    help="normal work kept queued on the GPU (it bounds the wait of an unannounced critical "
                         "release; 300 measured 2-6%% more best-effort throughput but slower critical kernels "
                         "next to it); -1: 100")
    ap.add_argument("--event-us", type=float, default=-1.0,
                    help="estimated normal work between completion events; -1: a third of the in-flight budget")
    ap.add_argument("--busy-policy", type=int, default=0,
                    help="normal shards next to a running critical kernel: 0 paper rule, 1 none, 2 smallest")
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
    ap.add_argument("--phases", default="kernels,solo,sequential,multistream,multistream_cu,ib,elastic,elastic_pause")
    ap.add_argument("--whole-when-clear", type=int, default=-1,
                    help="launch normal requests whole when they end before the next known critical "
                         "release (-1: with the release guard)")
    ap.add_argument("--whole-margin", type=float, default=0.0,
                    help="factor on the estimate of whole-request launches (0: the library's 2.0)")
    ap.add_argument("--cu-reserve", type=int, default=64,
                    help="multistream_cu phase: compute units left out of the normal streams' CU mask")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-op", default=None, metavar="NET.LAYER",
                    help="only launch one layer (unsharded) --reps times, then a 256 MiB device copy "
                         "--reps times as the counter calibration kernel (for rocprofv3 runs)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported "
              "(with several GPUs each critical / best-effort task set runs on a device of its own, "
              "so the co-run is measured on one)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2307_04339_amd import _lib as L
    from paper_2307_04339_amd import models
    from paper_2307_04339_amd.ops import device_info

    cfg = CONFIGS[args.config]
    dtype = cfg["dtype"]
    if args.profile_op:
        profile_op(args, cfg)
        return
    dev = device_info()
    log(f"device {dev.arch.decode()} cus={dev.n_cu} config={args.config}")
    cname, ckw = cfg["crit"]
    crit_net = models.BUILDERS[cname](dtype=dtype, **ckw)
    be_nets = [models.BUILDERS[n](dtype=dtype, **kw) for (n, kw) in cfg["be"]]
    be_tasks = []  # every instance of every best-effort network
    n_inst = args.be_instances if args.be_instances > 0 else cfg["be_instances"]
    for first, (n, kw) in zip(be_nets, cfg["be"]):
        be_tasks.append(first)
        for _ in range(n_inst - 1):
            be_tasks.append(models.BUILDERS[n](dtype=dtype, share=first, **kw))
    crit_net.forward()
    for n in be_tasks:
        n.forward()
    torch.cuda.synchronize()
    phases = set(args.phases.split(","))
    flush = CacheFlush()
    result = {}

    kern = None
    if "kernels" in phases:
        log("timing kernels ...")
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
        kern["traffic"] = measured_traffic(args.config, kern["kernel"], kern["tile"], layer.op.info.path)
        result["elastic_overhead"] = dict(kernel=kern["kernel"],
                                          **shard_overhead(layer, args.reps, flush, dev.n_cu, L.load()))
        log("index functions ...")
        result["index_function"] = {"net": dom_net.name,
                                    "layers": index_function_cost(dom_net, args.reps, flush, L)}
        log("transformed kernels ...")
        result["transformed_kernels"] = transformed_overhead(args.reps, flush)
        result["kernels"] = [dict(net=k["net"], name=k["name"], us=round(k["us"], 2), tiles=k["tiles"],
                                  **{kk: vv for kk, vv in roofline_of(k, dtype).items()
                                     if kk in ("bound", "achieved", "unit", "frac")})
                             for k in sorted(table, key=lambda k: -k["us"])[:12]]
        result["be_solo_ms_per_request"] = {n.name: round(sum(k["us"] for k in table if k["net"] == n.name) / 1000, 3)
                                            for n in be_nets}
        result["crit_kernel_sum_ms"] = round(sum(k["us"] for k in table if k["net"] == crit_net.name) / 1000, 3)
    del flush
    torch.cuda.empty_cache()

    guard = args.release_guard if args.release_guard >= 0 else int(cfg["arrival"] == "periodic")
    warm = args.warm_critical if args.warm_critical >= 0 else guard
    arm = args.arm_lead_us if args.arm_lead_us >= 0 else (500.0 if guard else 0.0)
    whole = args.whole_when_clear if args.whole_when_clear >= 0 else guard
    inflight_us = args.inflight_us if args.inflight_us >= 0 else 100.0
    event_us = args.event_us if args.event_us >= 0 else inflight_us / 3.0
    ccfg = dict(quantum_us=args.quantum_us, inflight_depth=args.depth, inflight_us=inflight_us, event_us=event_us,
                busy_policy=args.busy_policy, profile_reps=3, graphs=args.graphs, release_guard=guard,
                warm_critical=warm, arm_lead_us=arm, segments=args.segments, whole_when_clear=whole,
                whole_margin=args.whole_margin)
    runs = {}
    for ph in ("solo", "sequential", "multistream", "multistream_cu", "ib", "elastic", "elastic_pause"):
        if ph not in phases:
            continue
        log(f"phase {ph} ...")
        policy = {"solo": "elastic", "elastic_pause": "elastic", "multistream_cu": "multistream"}.get(ph, ph)
        pcfg = dict(ccfg, busy_policy=1) if ph == "elastic_pause" else ccfg
        if ph == "multistream_cu":
            pcfg = dict(ccfg, be_cu_reserve=args.cu_reserve)
        runs[ph] = run_phase(policy, crit_net, be_tasks, args.warmup, args.steps, cfg["period_ms"],
                             cfg["arrival"], seed=11, ccfg=pcfg, with_be=(ph != "solo"))
        r = runs[ph]
        log(f"  p50 {r['p50_ms']:.3f} ms  p99 {r['p99_ms']:.3f} ms  be {r['be_img_s']:.1f} img/s "
            f"launches {r['launches']}")

    # main line: Miriam with normal shards held back while a critical kernel runs (the paper's
    # padding rule is reported beside it as "elastic")
    main_name = next((n for n in ("elastic_pause", "elastic") if n in runs), None)
    main_run = runs[main_name] if main_name else next(iter(runs.values()), None)
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
        "config": {"workload": args.config,
                   "critical": f"{cname} b{ckw['batch']} {cfg['arrival']} every {cfg['period_ms']} ms",
                   "best_effort": [f"{n} b{kw['batch']} closed-loop" for n, kw in cfg["be"]],
                   "be_instances": n_inst,
                   "quantum_us": args.quantum_us, "inflight_depth": args.depth,
                   "inflight_us": inflight_us, "event_us": round(event_us, 2),
                   "busy_policy": 1 if main_name == "elastic_pause" else args.busy_policy,
                   "graphs": args.graphs, "release_guard": guard, "warm_critical": warm,
                   "arm_lead_us": arm, "segments": args.segments, "whole_when_clear": whole,
                   "cu_reserve_multistream_cu": args.cu_reserve},
    }
    if "solo" in runs and main_run:
        solo = runs["solo"]
        out["critical"] = {
            "policy": main_name,
            "solo_p50_ms": round(solo["p50_ms"], 4), "solo_p99_ms": round(solo["p99_ms"], 4),
            "corun_p50_ms": round(main_run["p50_ms"], 4), "corun_p99_ms": round(main_run["p99_ms"], 4),
            "p99_overhead": round(main_run["p99_ms"] / solo["p99_ms"] - 1.0, 4)}
        for other in ("elastic", "multistream", "multistream_cu", "ib", "sequential"):
            if other in runs and other != main_name:
                out["critical"][f"{other}_p99_overhead"] = round(runs[other]["p99_ms"] / solo["p99_ms"] - 1.0, 4)
    for ph, r in runs.items():
        out.setdefault("phases", {})[ph] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()}
    if "sequential" in runs and main_run:
        seq = runs["sequential"]
        out["best_effort"] = {
            "policy": main_name,
            "elastic_img_s": round(main_run["be_img_s"], 2), "sequential_img_s": round(seq["be_img_s"], 2),
            "speedup_vs_sequential": round(main_run["be_img_s"] / max(1e-9, seq["be_img_s"]), 3),
            "sequential_p99_ms": round(seq["p99_ms"], 4)}
    if kern:
        out["roofline"] = kern
    out.update({k: v for k, v in result.items()})
    if not args.no_cpu_baseline:
        bname, bkw = cfg["be"][0]
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(bname, dict(bkw, dtype=dtype))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
