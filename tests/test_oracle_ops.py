"""Pins of the oracle's operator definitions (CPU only).

Each operator is pinned by closed forms (all-ones / delta kernels, ramps,
constant rows), hand-worked fixtures under tests/golden/, and independent
library routines in float64 (PyTorch CPU convolution / pooling / softmax /
layer norm / batch norm, SciPy correlation, NumPy matmul).  None of these
shares code with the oracle's plain loops.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _torch_conv_nhwc(x, w, stride, pad, groups):
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2)))
    wt = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2)))
    y = F.conv2d(xt, wt, stride=stride, padding=pad, groups=groups)
    return y.numpy().transpose(0, 2, 3, 1)


# ------------------------------------------------------------------ conv2d
def test_conv_all_ones_counts_valid_taps(orc):
    # 1x56x56x64 input and 64x3x3x64 weights of ones, stride 1, pad 1:
    # interior pixels see 9 taps * 64 channels = 576, edges 6*64 = 384, corners 4*64 = 256
    x = np.ones((1, 56, 56, 64))
    w = np.ones((64, 3, 3, 64))
    y = orc.conv2d_raw(x, w, stride=1, pad=1)
    assert y.shape == (1, 56, 56, 64)
    assert (y[0, 1:-1, 1:-1, :] == 576).all()
    assert (y[0, 0, 1:-1, :] == 384).all() and (y[0, -1, 1:-1, :] == 384).all()
    assert (y[0, 1:-1, 0, :] == 384).all() and (y[0, 1:-1, -1, :] == 384).all()
    for (p, q) in [(0, 0), (0, 55), (55, 0), (55, 55)]:
        assert (y[0, p, q, :] == 256).all()


def test_conv_delta_kernel_copies(orc):
    rng = _rng(1)
    x = rng.uniform(-1, 1, (2, 7, 5, 6))
    w = np.zeros((6, 3, 3, 6))
    for c in range(6):
        w[c, 1, 1, c] = 1.0
    y = orc.conv2d_raw(x, w, stride=1, pad=1)
    assert np.array_equal(y, x)
    # an off-centre delta shifts the image (tap (0,2) reads x[p-1][q+1])
    w2 = np.zeros((6, 3, 3, 6))
    for c in range(6):
        w2[c, 0, 2, c] = 1.0
    y2 = orc.conv2d_raw(x, w2, stride=1, pad=1)
    assert np.array_equal(y2[:, 1:, :-1, :], x[:, :-1, 1:, :])
    assert (y2[:, 0, :, :] == 0).all() and (y2[:, :, -1, :] == 0).all()


def test_conv_golden_hand_cases(orc):
    with open(os.path.join(GOLD, "conv_tiny.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        x = np.array(case["x_hw"], dtype=np.float64)[None, :, :, None]
        w = np.array(case["w_hw"], dtype=np.float64)[None, :, :, None]
        y = orc.conv2d_raw(x, w, stride=case["stride"], pad=case["pad"])
        assert np.array_equal(y[0, :, :, 0], np.array(case["y_hw"], dtype=np.float64)), case["what"]


@pytest.mark.parametrize("shape", [
    # N, H, W, C, K, KH, stride, pad, groups
    (1, 5, 5, 2, 3, 3, 1, 1, 1),
    (2, 9, 7, 4, 6, 3, 2, 1, 1),
    (1, 12, 12, 3, 8, 7, 2, 3, 1),
    (1, 6, 6, 8, 4, 1, 1, 0, 1),
    (1, 6, 8, 8, 8, 3, 1, 1, 8),     # depthwise
    (2, 7, 7, 6, 6, 3, 2, 1, 6),     # depthwise, stride 2
    (1, 8, 8, 8, 4, 3, 1, 1, 2),     # grouped
])
def test_conv_matches_torch_float64(orc, shape):
    N, H, W, C, K, KH, s, p, g = shape
    rng = _rng(hash(shape) & 0xFFFF)
    x = rng.uniform(-1, 1, (N, H, W, C))
    w = rng.uniform(-1, 1, (K, KH, KH, C // g))
    y = orc.conv2d_raw(x, w, stride=s, pad=p, groups=g)
    ref = _torch_conv_nhwc(x, w, s, p, g)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_depthwise_matches_scipy_correlate(orc):
    from scipy.signal import correlate2d
    rng = _rng(7)
    x = rng.uniform(-1, 1, (1, 9, 11, 5))
    w = rng.uniform(-1, 1, (5, 3, 3, 1))
    y = orc.conv2d_raw(x, w, stride=1, pad=1, groups=5)
    for c in range(5):
        ref = correlate2d(x[0, :, :, c], w[c, :, :, 0], mode="same", boundary="fill")
        np.testing.assert_allclose(y[0, :, :, c], ref, rtol=1e-12, atol=1e-12)


def test_conv_1x1_equals_matmul(orc):
    rng = _rng(3)
    x = rng.uniform(-1, 1, (2, 4, 5, 16))
    w = rng.uniform(-1, 1, (12, 1, 1, 16))
    y = orc.conv2d_raw(x, w)
    ref = x.reshape(-1, 16) @ w.reshape(12, 16).T
    np.testing.assert_allclose(y.reshape(-1, 12), ref, rtol=1e-12, atol=1e-12)


def test_conv_rejects_bad_groups(orc):
    with pytest.raises(ValueError):
        orc.conv2d_raw(np.zeros((1, 4, 4, 6)), np.zeros((4, 3, 3, 2)), groups=4)


# -------------------------------------------------------------------- GEMM
def test_gemm_identity_and_numpy(orc):
    rng = _rng(11)
    X = rng.uniform(-1, 1, (37, 19))
    assert np.array_equal(orc.gemm_nt(X, np.eye(19)), X)
    W = rng.uniform(-1, 1, (23, 19))
    np.testing.assert_allclose(orc.gemm_nt(X, W), X @ W.T, rtol=1e-12, atol=1e-12)
    B = rng.uniform(-1, 1, (19, 29))
    np.testing.assert_allclose(orc.gemm_nn(X, B), X @ B, rtol=1e-12, atol=1e-12)
    # integer operands give exact products
    Xi = rng.integers(-3, 4, (8, 40)).astype(float)
    Wi = rng.integers(-3, 4, (5, 40)).astype(float)
    assert np.array_equal(orc.gemm_nt(Xi, Wi), Xi @ Wi.T)


# ---------------------------------------------------------------- epilogue
def test_bn_identity_case(orc):
    rng = _rng(2)
    y = rng.uniform(-3, 3, (10, 7))
    eps = 1e-5
    C = 7
    bn = (np.ones(C), np.zeros(C), np.zeros(C), np.full(C, 1 - eps))
    out = orc.epilogue(y, bn=bn, eps=eps)
    np.testing.assert_allclose(out, y, rtol=1e-15, atol=1e-15)


def test_epilogue_matches_torch(orc):
    rng = _rng(4)
    C = 6
    y = rng.uniform(-3, 3, (4, 5, C))
    bias = rng.uniform(-1, 1, C)
    gamma, beta = rng.uniform(0.8, 1.2, C), rng.uniform(-0.1, 0.1, C)
    mean, var = rng.uniform(-0.1, 0.1, C), rng.uniform(0.8, 1.2, C)
    res = rng.uniform(-1, 1, y.shape)
    for act, fn in [("none", lambda t: t), ("relu", F.relu), ("relu6", F.relu6),
                    ("gelu", lambda t: F.gelu(t, approximate="none"))]:
        out = orc.epilogue(y, bias=bias, bn=(gamma, beta, mean, var), eps=1e-5,
                           residual=res, act=act)
        t = torch.from_numpy(y + bias).reshape(-1, C)
        t = F.batch_norm(t, torch.from_numpy(mean), torch.from_numpy(var),
                         torch.from_numpy(gamma), torch.from_numpy(beta), training=False, eps=1e-5)
        t = fn(t + torch.from_numpy(res).reshape(-1, C))
        np.testing.assert_allclose(out.reshape(-1, C), t.numpy(), rtol=1e-12, atol=1e-12)


def test_activation_closed_forms(orc):
    v = np.array([[-7.0, -1.0, 0.0, 0.5, 6.0, 9.0]])
    assert orc.epilogue(v, act="relu").tolist() == [[0, 0, 0, 0.5, 6, 9]]
    assert orc.epilogue(v, act="relu6").tolist() == [[0, 0, 0, 0.5, 6, 6]]
    g = orc.epilogue(v, act="gelu")
    gn = orc.epilogue(-v, act="gelu")
    assert g[0, 2] == 0.0
    np.testing.assert_allclose(g - gn, v, rtol=1e-14, atol=1e-14)  # gelu(x) - gelu(-x) = x


# ----------------------------------------------------------------- pooling
def test_maxpool_ramp_closed_form(orc):
    # strictly increasing ramp along h and w: the max of a window is its
    # bottom-right in-bounds tap
    N, H, W, C = 1, 9, 8, 3
    x = np.zeros((N, H, W, C))
    for h in range(H):
        for w in range(W):
            x[0, h, w, :] = 100 * h + w + np.arange(C) * 0.25
    y = orc.maxpool(x, 3, 2, 1)
    Ho, Wo = (H + 2 - 3) // 2 + 1, (W + 2 - 3) // 2 + 1
    assert y.shape == (1, Ho, Wo, C)
    for p in range(Ho):
        for q in range(Wo):
            h = min(2 * p - 1 + 2, H - 1)
            w = min(2 * q - 1 + 2, W - 1)
            assert (y[0, p, q] == x[0, h, w]).all()


def test_pools_match_torch(orc):
    rng = _rng(9)
    x = rng.uniform(-1, 1, (2, 11, 10, 5))
    xt = torch.from_numpy(np.ascontiguousarray(x.transpose(0, 3, 1, 2)))
    for (k, s, p) in [(3, 2, 1), (2, 2, 0), (3, 1, 1)]:
        ref = F.max_pool2d(xt, k, s, p).numpy().transpose(0, 2, 3, 1)
        assert np.array_equal(orc.maxpool(x, k, s, p), ref)
        ref = F.avg_pool2d(xt, k, s, p, count_include_pad=True).numpy().transpose(0, 2, 3, 1)
        np.testing.assert_allclose(orc.avgpool(x, k, s, p), ref, rtol=1e-13, atol=1e-14)


def test_global_avgpool_constant_and_mean(orc):
    x = np.full((2, 7, 7, 4), 0.375)
    assert (orc.global_avgpool(x) == 0.375).all()
    rng = _rng(5)
    x = rng.uniform(-1, 1, (3, 7, 7, 6))
    np.testing.assert_allclose(orc.global_avgpool(x)[:, 0, 0, :], x.mean(axis=(1, 2)),
                               rtol=1e-13, atol=1e-14)


# ----------------------------------------------------------------- softmax
def test_softmax_constant_row_and_sums(orc):
    y = orc.softmax_rows(np.full((3, 128), 2.5))
    assert np.allclose(y, 1 / 128, rtol=0, atol=1e-17)
    rng = _rng(6)
    x = rng.uniform(-8, 8, (5, 256))
    y = orc.softmax_rows(x)
    np.testing.assert_allclose(y.sum(axis=1), 1.0, rtol=0, atol=1e-13)
    np.testing.assert_allclose(orc.softmax_rows(x + 3.0), y, rtol=1e-12, atol=1e-15)
    ref = torch.softmax(torch.from_numpy(x * 0.125), dim=-1).numpy()
    np.testing.assert_allclose(orc.softmax_rows(x, scale=0.125), ref, rtol=1e-12, atol=1e-15)


# --------------------------------------------------------------- layernorm
def test_layernorm_constant_row_gives_beta(orc):
    n = 768
    rng = _rng(8)
    gamma, beta = rng.uniform(0.5, 1.5, n), rng.uniform(-1, 1, n)
    y = orc.layernorm_rows(np.full((2, n), 3.25), gamma, beta)
    np.testing.assert_allclose(y, np.broadcast_to(beta, (2, n)), rtol=0, atol=1e-15)


def test_layernorm_moments_and_torch(orc):
    n = 768
    rng = _rng(10)
    x = rng.uniform(-2, 2, (6, n))
    r = rng.uniform(-1, 1, (6, n))
    y = orc.layernorm_rows(x, np.ones(n), np.zeros(n), eps=0.0, residual=r)
    np.testing.assert_allclose(y.mean(axis=1), 0.0, atol=1e-13)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1.0, atol=1e-12)
    gamma, beta = rng.uniform(0.5, 1.5, n), rng.uniform(-1, 1, n)
    y = orc.layernorm_rows(x, gamma, beta, eps=1e-5, residual=r)
    ref = F.layer_norm(torch.from_numpy(x + r), (n,), torch.from_numpy(gamma),
                       torch.from_numpy(beta), eps=1e-5).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_thread_count_does_not_change_results(orc):
    # the convolution and the products spread whole output elements over host threads; each
    # element keeps its loop order, so the results are bitwise the same for any count
    rng = np.random.default_rng(5)
    x = rng.uniform(-1, 1, (2, 9, 11, 24))
    w = rng.uniform(-1, 1, (10, 3, 3, 24))
    A = rng.uniform(-1, 1, (37, 53))
    B = rng.uniform(-1, 1, (41, 53))
    prev = orc.set_threads()
    try:
        outs = []
        for n in (1, 3):
            assert orc.set_threads(n) == n
            outs.append((orc.conv2d_raw(x, w, 2, 1), orc.gemm_nt(A, B), orc.gemm_nn(A, B.T.copy())))
        for a, b in zip(outs[0], outs[1]):
            assert np.array_equal(a, b)
    finally:
        orc.set_threads(prev)
