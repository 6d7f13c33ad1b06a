"""Graph builders for the synthetic workloads: ResNet-18-, VGG-16-, BERT-encoder-
and MobileNetV2-shaped networks as ordered lists of elastic operators over
preallocated device buffers (NHWC activations, one buffer per layer output so a
forward pass keeps every intermediate for layer-by-layer checks).

Weights are seeded random (no trained weights exist here): He-uniform
U(+-sqrt(6/fan_in)) for conv / FC weights, U(+-1/sqrt(fan_in)) biases, batch-norm
gamma, running var ~ U(0.8, 1.2), beta, running mean ~ U(-0.1, 0.1); encoder
linears U(+-1/sqrt(fan_in)), LayerNorm gamma = 1, beta = 0; inputs U[-1, 1].
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

from . import ops as O
from . import synth

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


@dataclass
class Layer:
    name: str
    kind: str                  # conv | dwconv | gemm | bgemm | maxpool | avgpool | softmax | layernorm
    op: O.ElasticOp
    params: dict = field(default_factory=dict)
    t: dict = field(default_factory=dict)   # device tensors: x, w, bias, bn, residual, y, ...


class Net:
    def __init__(self, name: str, dtype: str, batch: int, seed: int, share=None):
        """share: a network built by the same builder with the same arguments whose read-only
        tensors (weights, biases, BN / LN vectors, the input) this one reuses; activation
        buffers are always its own, so the two can run requests concurrently."""
        self.name = name
        self.dtype = dtype
        self.batch = batch
        self.seed = seed
        self.layers: list[Layer] = []
        self._n = 0
        self.input = None
        self.output = None
        self._share = share
        self._params: list = []

    # ----------------------------------------------------------- tensors
    def _dev(self, x64, dtype=None):
        dtype = dtype or self.dtype
        s = synth.to_storage(x64, dtype)
        if dtype == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(s).view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(s))
        return t.cuda()

    def _param(self, make, dtype=None):
        """Read-only tensor: built from make() (a float64 array), or taken from the shared network."""
        i = len(self._params)
        if self._share is not None:
            t = self._share._params[i]
        else:
            t = make() if callable(make) and not isinstance(make, np.ndarray) else make
            t = self._dev(t, dtype) if isinstance(t, np.ndarray) else t
        self._params.append(t)
        return t

    def _u(self, shape, bound, name, dtype=None):
        sd = synth.tensor_seed(self.seed, self._n, name)
        return self._param(lambda: synth.uniform(shape, -bound, bound, sd), dtype)

    def _bn(self, C):
        sd = synth.tensor_seed(self.seed, self._n, "bn")

        def make():
            rng = np.random.default_rng(sd)
            return np.stack([rng.uniform(0.8, 1.2, C), rng.uniform(-0.1, 0.1, C),
                             rng.uniform(-0.1, 0.1, C), rng.uniform(0.8, 1.2, C)])
        return self._param(make, "f32")

    def act_buf(self, shape):
        return torch.empty(shape, dtype=TORCH[self.dtype], device="cuda")

    def _add(self, layer: Layer):
        self.layers.append(layer)
        self._n += 1
        return layer.t["y"]

    # ------------------------------------------------------------ layers
    def conv(self, x, K, k, stride, pad, bn=True, bias=False, act="relu", residual=None, name=None,
             logical_c=None):
        """logical_c: channels that carry data when x is stored with zero channels appended
        (the padded weights of those channels are zero, so the result is the logical conv)."""
        N, H, W, C = x.shape
        lc = logical_c or C
        fan = lc * k * k
        sd = synth.tensor_seed(self.seed, self._n, "w")

        def make_w():
            w64 = synth.uniform((K, k, k, lc), -math.sqrt(6.0 / fan), math.sqrt(6.0 / fan), sd)
            if lc != C:
                w64 = np.concatenate([w64, np.zeros((K, k, k, C - lc))], axis=3)
            return w64
        w = self._param(make_w)
        b = self._u((K,), 1.0 / math.sqrt(fan), "b", "f32") if bias else None
        bnp = self._bn(K) if bn else None
        Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
        y = self.act_buf((N, Ho, Wo, K))
        op = O.conv2d(x, w, y, stride=stride, pad=pad, bias=b, bn=bnp, residual=residual, act=act)
        return self._add(Layer(name or f"conv{self._n}", "conv", op,
                               dict(stride=stride, pad=pad, act=act, eps=1e-5, logical_c=lc),
                               dict(x=x, w=w, bias=b, bn=bnp, residual=residual, y=y)))

    def dwconv(self, x, stride, act="relu6", name=None):
        N, H, W, C = x.shape
        w = self._u((3, 3, C), math.sqrt(6.0 / 9.0), "w")
        bnp = self._bn(C)
        Ho, Wo = (H + 2 - 3) // stride + 1, (W + 2 - 3) // stride + 1
        y = self.act_buf((N, Ho, Wo, C))
        op = O.dwconv(x, w, y, stride=stride, pad=1, bn=bnp, act=act)
        return self._add(Layer(name or f"dw{self._n}", "dwconv", op,
                               dict(stride=stride, pad=1, act=act, eps=1e-5),
                               dict(x=x, w=w, bias=None, bn=bnp, residual=None, y=y)))

    def pool(self, x, k, stride, pad, mode, name=None):
        N, H, W, C = x.shape
        Ho, Wo = (H + 2 * pad - k) // stride + 1, (W + 2 * pad - k) // stride + 1
        y = self.act_buf((N, Ho, Wo, C))
        op = O.pool(x, y, k, stride, pad, mode)
        return self._add(Layer(name or f"{mode}pool{self._n}", f"{mode}pool", op,
                               dict(k=k, stride=stride, pad=pad), dict(x=x, y=y)))

    def linear(self, x2d, nout, act="none", residual=None, w_bound=None, name=None):
        M, Kin = x2d.shape
        wb = w_bound if w_bound is not None else math.sqrt(6.0 / Kin)
        w = self._u((nout, Kin), wb, "w")
        b = self._u((nout,), 1.0 / math.sqrt(Kin), "b", "f32")
        y = self.act_buf((M, nout))
        op = O.gemm(x2d, w, y, bias=b, residual=residual, act=act)
        return self._add(Layer(name or f"fc{self._n}", "gemm", op, dict(act=act),
                               dict(x=x2d, w=w, bias=b, residual=residual, y=y)))

    # ------------------------------------------------------------- run
    def ops(self):
        return [l.op for l in self.layers]

    def forward(self, plans=None, stream=None):
        """Launch every layer; plans maps layer index -> list of (begin, len, grid, block)."""
        for i, l in enumerate(self.layers):
            if plans and i in plans:
                for (b, ln, g, bl) in plans[i]:
                    l.op.launch(b, ln, g, bl, stream)
            else:
                l.op.run(stream)

    def flops(self):
        return sum(l.op.info.flops for l in self.layers)

    def bytes(self):
        return sum(l.op.info.bytes for l in self.layers)


# ------------------------------------------------------------------ networks
IMAGE_C = 8  # storage channels of a 3-channel input image (16-byte pixels)


def image_input(batch, seed):
    """Batch of 224x224 RGB images ~ U[-1, 1], stored NHWC with the 3 data channels
    padded by zeros to 8 so every pixel is one 16-byte vector."""
    x = synth.uniform((batch, 224, 224, 3), -1, 1, synth.tensor_seed(seed, -1, "input"))
    return np.concatenate([x, np.zeros((batch, 224, 224, IMAGE_C - 3))], axis=3)



def resnet18(batch=1, dtype="f16", seed=0, num_classes=1000, share=None) -> Net:
    """7x7/2 stem, 3x3/2 max pool, 4 stages of two 3x3 basic blocks (64/128/256/512),
    global average pool, FC 512 -> classes.  23 operators."""
    net = Net("resnet18", dtype, batch, seed, share)
    x = net._param(lambda: image_input(batch, seed))
    net.input = x
    h = net.conv(x, 64, 7, 2, 3, name="stem", logical_c=3)
    h = net.pool(h, 3, 2, 1, "max", name="maxpool")
    cin = 64
    for stage, cout in enumerate([64, 128, 256, 512]):
        for blk in range(2):
            stride = 2 if (stage > 0 and blk == 0) else 1
            ident = h
            if stride != 1 or cin != cout:
                ident = net.conv(h, cout, 1, stride, 0, act="none", name=f"l{stage + 1}.{blk}.down")
            t = net.conv(h, cout, 3, stride, 1, act="relu", name=f"l{stage + 1}.{blk}.conv1")
            h = net.conv(t, cout, 3, 1, 1, act="relu", residual=ident, name=f"l{stage + 1}.{blk}.conv2")
            cin = cout
    h = net.pool(h, h.shape[1], 1, 0, "avg", name="avgpool")
    net.output = net.linear(h.view(batch, 512), num_classes, name="fc")
    return net


def vgg16(batch=8, dtype="f16", seed=1, num_classes=1000, share=None) -> Net:
    """13 3x3 convs (64..512, bias + ReLU), 5 2x2 max pools, FC 25088->4096->4096->classes."""
    net = Net("vgg16", dtype, batch, seed, share)
    x = net._param(lambda: image_input(batch, seed))
    net.input = x
    h = x
    for si, (c, n) in enumerate([(64, 2), (128, 2), (256, 3), (512, 3), (512, 3)]):
        for j in range(n):
            h = net.conv(h, c, 3, 1, 1, bn=False, bias=True, act="relu", name=f"conv{si + 1}_{j + 1}",
                         logical_c=3 if (si, j) == (0, 0) else None)
        h = net.pool(h, 2, 2, 0, "max", name=f"pool{si + 1}")
    f = h.reshape(batch, 7 * 7 * 512)
    f = net.linear(f, 4096, act="relu", name="fc6")
    f = net.linear(f, 4096, act="relu", name="fc7")
    net.output = net.linear(f, num_classes, name="fc8")
    return net


def mobilenetv2(batch=16, dtype="bf16", seed=2, num_classes=1000, share=None) -> Net:
    """Stem 3x3/2 conv 3->32, inverted residual blocks (expansion 6, width 1.0),
    1x1 conv 320->1280, global average pool, FC 1280->classes."""
    net = Net("mobilenetv2", dtype, batch, seed, share)
    x = net._param(lambda: image_input(batch, seed))
    net.input = x
    h = net.conv(x, 32, 3, 2, 1, act="relu6", name="stem", logical_c=3)
    cin = 32
    for bi, (t, c, n, s) in enumerate([(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2),
                                       (6, 96, 3, 1), (6, 160, 3, 2), (6, 320, 1, 1)]):
        for j in range(n):
            stride = s if j == 0 else 1
            inp = h
            e = h
            if t != 1:
                e = net.conv(h, cin * t, 1, 1, 0, act="relu6", name=f"b{bi}.{j}.expand")
            d = net.dwconv(e, stride, act="relu6", name=f"b{bi}.{j}.dw")
            res = inp if (stride == 1 and cin == c) else None
            h = net.conv(d, c, 1, 1, 0, act="none", residual=res, name=f"b{bi}.{j}.project")
            cin = c
    h = net.conv(h, 1280, 1, 1, 0, act="relu6", name="head")
    h = net.pool(h, h.shape[1], 1, 0, "avg", name="avgpool")
    net.output = net.linear(h.view(batch, 1280), num_classes, name="fc")
    return net


def encoder(batch=1, seq=128, layers=12, hidden=768, heads=12, ffn=3072, dtype="bf16", seed=3, share=None) -> Net:
    """Post-LN BERT-style encoder: per layer QKV projection, scores = Q K^T (per head),
    softmax(scores / sqrt(64)), context = P V, output projection + residual, LayerNorm,
    FFN (GELU) + residual, LayerNorm.  No attention mask."""
    net = Net("encoder", dtype, batch, seed, share)
    M = batch * seq
    D = hidden // heads
    x = net._param(lambda: synth.uniform((M, hidden), -1, 1, synth.tensor_seed(seed, -1, "input")))
    net.input = x
    ones = net._param(lambda: torch.ones(hidden, dtype=torch.float32, device="cuda"))
    zeros = net._param(lambda: torch.zeros(hidden, dtype=torch.float32, device="cuda"))
    h = x
    for li in range(layers):
        bnd = 1.0 / math.sqrt(hidden)
        qkv = net.linear(h, 3 * hidden, w_bound=bnd, name=f"L{li}.qkv")
        scores = net.act_buf((batch * heads, seq, seq))
        op = O.bgemm(qkv, qkv[:, hidden:], scores, m=seq, n=seq, k=D, batch=batch * heads,
                     batch_div=heads, ldx=3 * hidden, ldw=3 * hidden, ldy=seq,
                     sx=(seq * 3 * hidden, D), sw=(seq * 3 * hidden, D), sy=(heads * seq * seq, seq * seq))
        net._add(Layer(f"L{li}.scores", "bgemm", op,
                       dict(B=batch, H=heads, S=seq, D=D, hidden=hidden, which="qk"),
                       dict(qkv=qkv, y=scores)))
        probs = net.act_buf((batch * heads, seq, seq))
        op = O.softmax(scores, probs, batch * heads * seq, seq, scale=1.0 / math.sqrt(D))
        net._add(Layer(f"L{li}.softmax", "softmax", op, dict(scale=1.0 / math.sqrt(D)),
                       dict(x=scores, y=probs)))
        ctx = net.act_buf((M, hidden))
        op = O.bgemm(probs, qkv[:, 2 * hidden:], ctx, m=seq, n=D, k=seq, batch=batch * heads,
                     batch_div=heads, ldx=seq, ldw=3 * hidden, ldy=hidden,
                     sx=(heads * seq * seq, seq * seq), sw=(seq * 3 * hidden, D), sy=(seq * hidden, D),
                     b_nmajor=True)
        net._add(Layer(f"L{li}.context", "bgemm", op,
                       dict(B=batch, H=heads, S=seq, D=D, hidden=hidden, which="pv"),
                       dict(probs=probs, qkv=qkv, y=ctx)))
        t1 = net.linear(ctx, hidden, residual=h, w_bound=bnd, name=f"L{li}.attn_out")
        x1 = net.act_buf((M, hidden))
        op = O.layernorm(t1, ones, zeros, x1, M, hidden)
        net._add(Layer(f"L{li}.ln1", "layernorm", op, dict(eps=1e-5),
                       dict(x=t1, gamma=ones, beta=zeros, residual=None, y=x1)))
        f1 = net.linear(x1, ffn, act="gelu", w_bound=bnd, name=f"L{li}.ffn1")
        t2 = net.linear(f1, hidden, residual=x1, w_bound=1.0 / math.sqrt(ffn), name=f"L{li}.ffn2")
        x2 = net.act_buf((M, hidden))
        op = O.layernorm(t2, ones, zeros, x2, M, hidden)
        h = net._add(Layer(f"L{li}.ln2", "layernorm", op, dict(eps=1e-5),
                           dict(x=t2, gamma=ones, beta=zeros, residual=None, y=x2)))
    net.output = h
    return net


BUILDERS = {"resnet18": resnet18, "vgg16": vgg16, "mobilenetv2": mobilenetv2, "encoder": encoder}
