"""Full-tensor oracle parity of the dominant layers at the workloads' real shapes.

The network tests check contractions on sampled outputs; here every output element of the
largest contraction layers is compared with the oracle, run on the layer's own GPU input bits
(the oracle spreads output elements over host threads; each element keeps its loop order).
Covered: VGG-16 b8 (fp16 and bf16) conv1_2 (resident-weight kernel), conv2_2 (the co-run's
dominant kernel, 128x128 pipelined tiles), conv3_2, conv4_2 (128x64), conv5_2 (64x64) and fc6
(split-K skinny kernel); MobileNetV2 b32 expand and depthwise layers; the encoder b4 s256 FFN.
"""
import time

import numpy as np
import pytest
import torch

from gpu_util import RTOL, gpu_available, rel_err, to_f64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]


def _bn(t):
    return None if t is None else tuple(to_f64(t))


def _full_ref(layer, orc):
    t, p = layer.t, layer.params
    if layer.kind == "conv":
        return orc.conv2d(to_f64(t["x"]), to_f64(t["w"]), stride=p["stride"], pad=p["pad"],
                          bias=None if t.get("bias") is None else to_f64(t["bias"]), bn=_bn(t.get("bn")),
                          eps=p.get("eps", 1e-5),
                          residual=None if t.get("residual") is None else to_f64(t["residual"]), act=p["act"])
    if layer.kind == "dwconv":
        w = to_f64(t["w"])
        w_or = np.ascontiguousarray(w.transpose(2, 0, 1))[..., None]
        C = w.shape[-1]
        return orc.conv2d(to_f64(t["x"]), w_or, stride=p["stride"], pad=p["pad"], groups=C,
                          bias=None if t.get("bias") is None else to_f64(t["bias"]), bn=_bn(t.get("bn")),
                          eps=p.get("eps", 1e-5), act=p["act"])
    if layer.kind == "gemm":
        return orc.linear(to_f64(t["x"]), to_f64(t["w"]), bias=to_f64(t["bias"]),
                          residual=None if t.get("residual") is None else to_f64(t["residual"]), act=p["act"])
    raise ValueError(layer.kind)


CASES = [
    ("vgg16", dict(batch=8, dtype="f16"), ["conv1_2", "conv2_2", "conv3_2", "conv4_2", "conv5_2", "fc6"]),
    ("vgg16", dict(batch=8, dtype="bf16"), ["conv2_2", "conv4_2"]),
    ("mobilenetv2", dict(batch=32, dtype="bf16"), None),
    ("encoder", dict(batch=4, seq=256, dtype="bf16"), None),
]


@pytest.mark.parametrize("name,kw,layers", CASES, ids=[f"{c[0]}-{c[1]['dtype']}" for c in CASES])
def test_dominant_layers_match_oracle_in_full(orc, name, kw, layers):
    from paper_2307_04339_amd import models
    net = models.BUILDERS[name](**kw)
    net.forward()
    torch.cuda.synchronize()
    if layers is None:
        # the four slowest contraction / depthwise layers of the network by algorithmic work
        cand = [l for l in net.layers if l.kind in ("conv", "dwconv", "gemm")]
        cand.sort(key=lambda l: -l.op.info.flops)
        chosen = cand[:3] + [l for l in cand if l.kind == "dwconv"][:1]
    else:
        by = {l.name: l for l in net.layers}
        chosen = [by[n] for n in layers]
    for layer in chosen:
        t0 = time.time()
        ref = _full_ref(layer, orc)
        got = to_f64(layer.t["y"])
        assert got.shape == ref.shape, (layer.name, got.shape, ref.shape)
        err = rel_err(got, ref)
        print(f"{name} {kw['dtype']} {layer.name}: {got.size} outputs, path {layer.op.info.path}, "
              f"rel {err:.2e}, oracle {time.time() - t0:.1f} s", flush=True)
        assert err <= RTOL[kw["dtype"]], (layer.name, err)
