"""Layer-by-layer oracle check of a network built by paper_2307_04339_amd.models.

Each layer is checked on the GPU's own input bits for that layer (so the error
does not compound through the network).  Contractions are checked on sampled
outputs that the oracle computes one by one: for a convolution, the input window
of each sampled output pixel is cut out (zero padding made explicit) and the
oracle convolves it; for a GEMM, sampled rows; for attention, sampled heads.
Bandwidth-bound layers are checked in full.
"""
import numpy as np

from gpu_util import rel_err, to_f64


def _window(x64, n, p, q, KH, KW, stride, pad):
    """Input window of output pixel (n, p, q), zero-padded: [KH, KW, C]."""
    N, H, W, C = x64.shape
    out = np.zeros((KH, KW, C))
    for r in range(KH):
        h = p * stride - pad + r
        if h < 0 or h >= H:
            continue
        for s in range(KW):
            w = q * stride - pad + s
            if 0 <= w < W:
                out[r, s] = x64[n, h, w]
    return out


def _sample_pixels(N, Ho, Wo, k, rng):
    pix = {(0, 0, 0), (N - 1, Ho - 1, Wo - 1), (0, 0, Wo - 1), (N - 1, Ho - 1, 0)}
    while len(pix) < min(k, N * Ho * Wo):
        pix.add((int(rng.integers(N)), int(rng.integers(Ho)), int(rng.integers(Wo))))
    return sorted(pix)


def _bn_tuple(t):
    return None if t is None else tuple(to_f64(t))


def check_layer(layer, orc, samples=48, seed=0):
    """Relative error of one layer's GPU output against the oracle."""
    rng = np.random.default_rng(seed)
    t, p = layer.t, layer.params
    y = to_f64(t["y"])
    if layer.kind in ("conv", "dwconv"):
        x64 = to_f64(t["x"])
        w64 = to_f64(t["w"])
        N, H, W, C = x64.shape
        _, Ho, Wo, K = y.shape
        if layer.kind == "conv":
            KH, KW = w64.shape[1], w64.shape[2]
            w_or, groups = w64, 1
        else:
            KH, KW = w64.shape[0], w64.shape[1]
            w_or, groups = np.ascontiguousarray(w64.transpose(2, 0, 1))[..., None], C
        pix = _sample_pixels(N, Ho, Wo, samples, rng)
        crops = np.stack([_window(x64, n, pp, q, KH, KW, p["stride"], p["pad"]) for (n, pp, q) in pix])
        raw = orc.conv2d_raw(crops, w_or, stride=1, pad=0, groups=groups)[:, 0, 0, :]
        res = None
        if t.get("residual") is not None:
            r64 = to_f64(t["residual"])
            res = np.stack([r64[n, pp, q] for (n, pp, q) in pix])
        ref = orc.epilogue(raw, bias=None if t.get("bias") is None else to_f64(t["bias"]),
                           bn=_bn_tuple(t.get("bn")), eps=p.get("eps", 1e-5), residual=res, act=p["act"])
        got = np.stack([y[n, pp, q] for (n, pp, q) in pix])
        return rel_err(got, ref)
    if layer.kind == "gemm":
        x64 = to_f64(t["x"])
        w64 = to_f64(t["w"])
        M = x64.shape[0]
        rows = sorted({0, M - 1} | set(rng.integers(0, M, min(samples, M)).tolist()))
        res = None if t.get("residual") is None else to_f64(t["residual"])[rows]
        ref = orc.linear(x64[rows], w64, bias=to_f64(t["bias"]), residual=res, act=p["act"])
        return rel_err(y[rows], ref)
    if layer.kind == "bgemm":
        B, H, S, D, hid = p["B"], p["H"], p["S"], p["D"], p["hidden"]
        q64 = to_f64(t["qkv"]).reshape(B, S, 3, H, D)
        heads = sorted({(0, 0), (B - 1, H - 1)} | {(int(rng.integers(B)), int(rng.integers(H)))
                                                    for _ in range(3)})
        errs = []
        if p["which"] == "qk":
            yy = y.reshape(B, H, S, S)
            for b, h in heads:
                errs.append(rel_err(yy[b, h], orc.gemm_nt(q64[b, :, 0, h], q64[b, :, 1, h])))
        else:
            pr = to_f64(t["probs"]).reshape(B, H, S, S)
            yy = y.reshape(B, S, H, D)
            for b, h in heads:
                errs.append(rel_err(yy[b, :, h], orc.gemm_nn(pr[b, h], q64[b, :, 2, h])))
        return max(errs)
    if layer.kind in ("maxpool", "avgpool"):
        x64 = to_f64(t["x"])
        fn = orc.maxpool if layer.kind == "maxpool" else orc.avgpool
        return rel_err(y, fn(x64, p["k"], p["stride"], p["pad"]))
    if layer.kind == "softmax":
        x64 = to_f64(t["x"])
        n = x64.shape[-1]
        return rel_err(y.reshape(-1, n), orc.softmax_rows(x64.reshape(-1, n), scale=p["scale"]))
    if layer.kind == "layernorm":
        x64 = to_f64(t["x"])
        return rel_err(y, orc.layernorm_rows(x64, to_f64(t["gamma"]), to_f64(t["beta"]), eps=p["eps"]))
    raise ValueError(layer.kind)
