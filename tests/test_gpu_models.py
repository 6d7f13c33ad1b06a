"""Network-level GPU checks at the workloads' full sizes: every layer of the
ResNet-18-, VGG-16-, encoder- and MobileNetV2-shaped networks against the
oracle (on that layer's own GPU inputs; sampled outputs for contractions), and
the ResNet-18 forward pass bitwise identical under seeded random per-layer
shard plans (n in {1,2,3,4,8}, block in {64,128,256})."""
import numpy as np
import pytest
import torch

from gpu_util import RTOL, bits, gpu_available
from layer_check import check_layer

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs an MI355X")]

NETS = [
    ("resnet18", dict(batch=1, dtype="f16")),
    ("vgg16", dict(batch=8, dtype="f16")),
    ("encoder", dict(batch=1, seq=128, dtype="bf16")),
    ("mobilenetv2", dict(batch=16, dtype="bf16")),
    ("resnet18", dict(batch=1, dtype="bf16")),
    ("vgg16", dict(batch=8, dtype="bf16")),
    ("encoder", dict(batch=4, seq=256, dtype="bf16")),
    ("mobilenetv2", dict(batch=32, dtype="bf16")),
]


@pytest.mark.parametrize("name,kw", NETS, ids=[f"{n}-{k['dtype']}-b{k['batch']}" for n, k in NETS])
def test_network_layers_match_oracle(orc, name, kw):
    from paper_2307_04339_amd import models
    net = models.BUILDERS[name](**kw)
    net.forward()
    torch.cuda.synchronize()
    worst = 0.0
    for i, layer in enumerate(net.layers):
        err = check_layer(layer, orc, samples=32, seed=i)
        worst = max(worst, err)
        assert err <= RTOL[kw["dtype"]], (layer.name, err)
    out = net.output.float()
    assert torch.isfinite(out).all()
    print(f"{name} {kw}: {len(net.layers)} layers, worst rel err {worst:.2e}")


def _random_plans(net, seed):
    from oracle import oracle as orc  # the plan generator's definition, host only
    rng = np.random.default_rng(seed)
    plans = {}
    for i, layer in enumerate(net.layers):
        T = layer.op.T
        n = int(rng.choice([1, 2, 3, 4, 8]))
        n = min(n, T)
        shards = orc.balanced_split(T, n)
        if rng.random() < 0.5:
            shards = shards[::-1]
        seq = []
        for (b, l) in shards:
            block = int(rng.choice([64, 128, 256]))
            g = int(rng.choice([1, 7, 64, 256, l]))
            seq.append((b, l, max(1, min(g, l)), block))
        plans[i] = seq
    return plans


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_resnet18_bitwise_under_random_shard_plans(dtype):
    from paper_2307_04339_amd import models
    net = models.resnet18(batch=1, dtype=dtype)
    net.forward()
    torch.cuda.synchronize()
    ref = [bits(l.t["y"]) for l in net.layers]
    for seed in range(3):
        for l in net.layers:
            l.t["y"].fill_(float("nan"))
        net.forward(plans=_random_plans(net, seed))
        torch.cuda.synchronize()
        for l, r in zip(net.layers, ref):
            assert bits(l.t["y"]) == r, (seed, l.name)
