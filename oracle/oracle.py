"""Miriam CPU oracle, Python side — TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper over ``miriam_oracle.c`` (plain C loops in double
precision).  Only the test suite, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this module; the product path
(``paper_2307_04339_amd``) never does and shares no code with it.

Every function widens its numpy inputs to float64 (exact for fp32/fp16/bf16
values), calls the C routine and returns float64 results.  Composite helpers
(``conv2d`` with its epilogue, ``attention``) only chain the C routines in the
order the operator's definition gives.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "miriam_oracle.c")
_LIB = os.path.join(_HERE, "libmiriam_oracle.so")

ACT = {"none": 0, "relu": 1, "relu6": 2, "gelu": 3}

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no GPU code, no shared headers)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fno-fast-math", "-fopenmp",
             "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = ctypes.CDLL(_LIB)
        _declare(_lib)
    return _lib


_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.POINTER(ctypes.c_int64)
_I32 = ctypes.POINTER(ctypes.c_int32)
_INT = ctypes.POINTER(ctypes.c_int)
i64 = ctypes.c_int64


def set_threads(n: int = 0) -> int:
    """Host threads of the convolution and matrix products (0: report only)."""
    return int(lib().or_set_threads(int(n)))


def _declare(L):
    L.or_set_threads.argtypes = [ctypes.c_int]
    L.or_set_threads.restype = ctypes.c_int
    L.or_dichotomy.argtypes = [i64, _I64, ctypes.c_int]
    L.or_balanced_split.argtypes = [i64, i64, _I64, _I64]
    L.or_wg_rank.argtypes = [i64, i64, i64]
    L.or_wg_rank.restype = i64
    L.or_owner_map.argtypes = [i64, i64, _I64, _I64, _I64, i64, _I32, _I32, _I32, _I32]
    L.or_wave_map.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _INT, _INT]
    L.or_tile_coords.argtypes = [i64, i64, i64, i64, i64, _I64, _I64, _I64]
    L.or_eq2_grid_limit.argtypes = [i64, i64]
    L.or_eq2_grid_limit.restype = i64
    L.or_eq2_block_limit.argtypes = [i64, i64]
    L.or_eq2_block_limit.restype = i64
    L.or_eq2_feasible.argtypes = [i64] * 6
    L.or_wiscore.argtypes = [i64] * 6
    L.or_wiscore.restype = ctypes.c_double
    L.or_oscore.argtypes = [i64, _D, _D, ctypes.c_double, ctypes.c_double]
    L.or_top_fraction.argtypes = [ctypes.c_int, _D, _I64, _I64, ctypes.c_double, _INT]
    L.or_tree_head.argtypes = [i64, i64, i64, _INT]
    L.or_tree_head.restype = i64
    L.or_conv2d.argtypes = [_D, i64, i64, i64, i64, _D, i64, i64, i64, i64, i64, i64, _D]
    L.or_gemm_nt.argtypes = [_D, _D, i64, i64, i64, _D]
    L.or_gemm_nn.argtypes = [_D, _D, i64, i64, i64, _D]
    L.or_epilogue.argtypes = [_D, i64, i64, _D, _D, ctypes.c_double, _D, ctypes.c_int]
    L.or_maxpool.argtypes = [_D, i64, i64, i64, i64, i64, i64, i64, i64, _D]
    L.or_avgpool.argtypes = [_D, i64, i64, i64, i64, i64, i64, i64, i64, _D]
    L.or_softmax_rows.argtypes = [_D, i64, i64, ctypes.c_double, _D]
    L.or_layernorm_rows.argtypes = [_D, _D, i64, i64, _D, _D, ctypes.c_double, _D]


def _d(a):
    """Contiguous float64 copy/view and its pointer."""
    a = np.ascontiguousarray(np.asarray(a, dtype=np.float64))
    return a, a.ctypes.data_as(_D)


def _dn(a):
    if a is None:
        return None, None
    return _d(a)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what}: bad arguments (rc={rc})")


# ----------------------------------------------------------------- tile maps
def dichotomy(M: int):
    """Eq. (1) slice widths, smallest first."""
    out = np.zeros(64, dtype=np.int64)
    n = lib().or_dichotomy(M, out.ctypes.data_as(_I64), 64)
    if n < 0:
        raise ValueError("dichotomy: M must be >= 1")
    return [int(v) for v in out[:n]]


def balanced_split(T: int, n: int):
    b = np.zeros(n, dtype=np.int64)
    l = np.zeros(n, dtype=np.int64)
    _check(lib().or_balanced_split(T, n, b.ctypes.data_as(_I64), l.ctypes.data_as(_I64)),
           "balanced_split")
    return list(zip(b.tolist(), l.tolist()))


def wg_rank(g: int, G: int, X: int) -> int:
    return int(lib().or_wg_rank(g, G, X))


def owner_map(T: int, shards, grids, X: int = 8):
    """shards: list of (begin, len); grids: list of G per shard.
    Returns (owner_shard, owner_wg, owner_iter, count) int32 arrays of length T."""
    n = len(shards)
    b = np.array([s[0] for s in shards], dtype=np.int64)
    l = np.array([s[1] for s in shards], dtype=np.int64)
    G = np.array(grids, dtype=np.int64)
    outs = [np.zeros(max(T, 1), dtype=np.int32) for _ in range(4)]
    rc = lib().or_owner_map(T, n, b.ctypes.data_as(_I64), l.ctypes.data_as(_I64),
                            G.ctypes.data_as(_I64), X, *[o.ctypes.data_as(_I32) for o in outs])
    _check(rc, "owner_map")
    return tuple(o[:T] for o in outs)


def wave_map(L: int, P: int, lam: int):
    pw, rd = ctypes.c_int(), ctypes.c_int()
    _check(lib().or_wave_map(L, P, lam, ctypes.byref(pw), ctypes.byref(rd)), "wave_map")
    return pw.value, rd.value


def tile_coords(t, M, N, TM, TN):
    bi, mt, nt = i64(), i64(), i64()
    _check(lib().or_tile_coords(t, M, N, TM, TN, ctypes.byref(bi), ctypes.byref(mt),
                                ctypes.byref(nt)), "tile_coords")
    return bi.value, mt.value, nt.value


# ------------------------------------------------------- design-space shrinking
def eq2_grid_limit(n_sm, n_blk_rt):
    return int(lib().or_eq2_grid_limit(n_sm, n_blk_rt))


def eq2_block_limit(l_threads, s_blk_rt):
    return int(lib().or_eq2_block_limit(l_threads, s_blk_rt))


def eq2_feasible(n_sm, l_threads, n_blk_rt, s_blk_rt, n_blk_be, s_blk_be):
    return bool(lib().or_eq2_feasible(n_sm, l_threads, n_blk_rt, s_blk_rt, n_blk_be, s_blk_be))


def wiscore(n_sm, l_threads, n_blk_rt, s_blk_rt, n_blk_be, s_blk_be):
    return float(lib().or_wiscore(n_sm, l_threads, n_blk_rt, s_blk_rt, n_blk_be, s_blk_be))


def oscore(lo_blk, lo_pt, max_blk, max_pt):
    a, pa = _d(lo_blk)
    b, pb = _d(lo_pt)
    return int(lib().or_oscore(len(a), pa, pb, max_blk, max_pt))


def top_fraction(scores, grids, blocks, frac=0.2):
    s, ps = _d(scores)
    g = np.ascontiguousarray(grids, dtype=np.int64)
    bl = np.ascontiguousarray(blocks, dtype=np.int64)
    keep = np.zeros(max(len(s), 1), dtype=np.intc)
    k = lib().or_top_fraction(len(s), ps, g.ctypes.data_as(_I64), bl.ctypes.data_as(_I64),
                              frac, keep.ctypes.data_as(_INT))
    return keep[:k].tolist()


def tree_head(T, cursor, max_len):
    depth = ctypes.c_int(-1)
    ln = lib().or_tree_head(T, cursor, max_len, ctypes.byref(depth))
    if ln < 0:
        raise ValueError("tree_head: bad arguments")
    return int(ln), depth.value


# ------------------------------------------------------------------ operators
def conv2d_raw(x, w, stride=1, pad=0, groups=1):
    """x: [N,H,W,C] (NHWC), w: [K,KH,KW,C/groups]; returns [N,Ho,Wo,K] float64."""
    x, px = _d(x)
    w, pw = _d(w)
    N, H, W, C = x.shape
    K, KH, KW, _ = w.shape
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (W + 2 * pad - KW) // stride + 1
    y = np.zeros((N, Ho, Wo, K), dtype=np.float64)
    _check(lib().or_conv2d(px, N, H, W, C, pw, K, KH, KW, stride, pad, groups,
                           y.ctypes.data_as(_D)), "conv2d")
    return y


def epilogue(y, bias=None, bn=None, eps=1e-5, residual=None, act="none"):
    """In-order per-channel epilogue on a float64 array whose last dim is C.
    bn: (gamma, beta, mean, var) tuple or None."""
    y = np.array(y, dtype=np.float64, order="C", copy=True)
    C = y.shape[-1]
    rows = y.size // C if C else 0
    biasarr, pb = _dn(bias)
    bnarr = None
    pbn = None
    if bn is not None:
        bnarr, pbn = _d(np.concatenate([np.asarray(v, dtype=np.float64).reshape(C) for v in bn]))
    res, pr = _dn(None if residual is None else np.asarray(residual).reshape(y.shape))
    _check(lib().or_epilogue(y.ctypes.data_as(_D), rows, C, pb, pbn, eps, pr, ACT[act]),
           "epilogue")
    return y


def conv2d(x, w, stride=1, pad=0, groups=1, bias=None, bn=None, eps=1e-5,
           residual=None, act="none"):
    return epilogue(conv2d_raw(x, w, stride, pad, groups), bias, bn, eps, residual, act)


def gemm_nt(X, W):
    X, px = _d(X)
    W, pw = _d(W)
    M, K = X.shape
    N = W.shape[0]
    Y = np.zeros((M, N), dtype=np.float64)
    _check(lib().or_gemm_nt(px, pw, M, N, K, Y.ctypes.data_as(_D)), "gemm_nt")
    return Y


def gemm_nn(X, B):
    X, px = _d(X)
    B, pb = _d(B)
    M, K = X.shape
    N = B.shape[1]
    Y = np.zeros((M, N), dtype=np.float64)
    _check(lib().or_gemm_nn(px, pb, M, N, K, Y.ctypes.data_as(_D)), "gemm_nn")
    return Y


def linear(X, W, bias=None, residual=None, act="none"):
    """Fully connected layer Y = X W^T + b (+ residual), then act."""
    return epilogue(gemm_nt(X, W), bias=bias, residual=residual, act=act)


def maxpool(x, k, stride, pad):
    x, px = _d(x)
    N, H, W, C = x.shape
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    y = np.zeros((N, Ho, Wo, C))
    _check(lib().or_maxpool(px, N, H, W, C, k, k, stride, pad, y.ctypes.data_as(_D)), "maxpool")
    return y


def avgpool(x, k, stride, pad):
    x, px = _d(x)
    N, H, W, C = x.shape
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    y = np.zeros((N, Ho, Wo, C))
    _check(lib().or_avgpool(px, N, H, W, C, k, k, stride, pad, y.ctypes.data_as(_D)), "avgpool")
    return y


def global_avgpool(x):
    x = np.asarray(x)
    N, H, W, C = x.shape
    assert H == W
    return avgpool(x, H, 1, 0)


def softmax_rows(x, scale=1.0):
    x, px = _d(x)
    n = x.shape[-1]
    rows = x.size // n
    y = np.zeros_like(x)
    _check(lib().or_softmax_rows(px, rows, n, scale, y.ctypes.data_as(_D)), "softmax")
    return y


def layernorm_rows(x, gamma, beta, eps=1e-5, residual=None):
    x, px = _d(x)
    n = x.shape[-1]
    rows = x.size // n
    resarr, pr = _dn(None if residual is None else np.asarray(residual).reshape(x.shape))
    g, pg = _d(gamma)
    b, pb = _d(beta)
    y = np.zeros_like(x)
    _check(lib().or_layernorm_rows(px, pr, rows, n, pg, pb, eps, y.ctypes.data_as(_D)),
           "layernorm")
    return y
