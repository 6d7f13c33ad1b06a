"""Python view of the elastic operators: builds miriam_op_desc from torch tensors
(device memory only) and forwards to the C ABI.  No arithmetic happens here."""
from __future__ import annotations

import ctypes

import torch

from . import _lib as L

TORCH_DTYPE = {torch.float32: L.F32, torch.float16: L.F16, torch.bfloat16: L.BF16}


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("operator tensors must live in device memory")
    return t.data_ptr()


def _stream_handle(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class ElasticOp:
    """One elastic operator over caller-owned device tensors."""

    def __init__(self, kind: int, dtype: torch.dtype, *, keep=(), **fields):
        lib = L.load()
        d = L.OpDesc()
        d.kind = kind
        d.dtype = TORCH_DTYPE[dtype]
        for k, v in fields.items():
            if isinstance(v, torch.Tensor):
                v = _ptr(v)
            setattr(d, k, v)
        self.desc = d
        self._keep = tuple(keep)  # tensors borrowed by the op
        h = ctypes.c_void_p()
        L.check(lib.miriam_op_create(ctypes.byref(d), ctypes.byref(h)), "miriam_op_create")
        self.handle = h
        info = L.OpInfo()
        L.check(lib.miriam_op_query(h, ctypes.byref(info)), "miriam_op_query")
        self.info = info
        self.T = int(info.num_tiles)

    # --------------------------------------------------------------- launches
    def launch(self, begin: int, length: int, grid: int, block: int = 256, stream=None) -> None:
        L.check(L.load().miriam_elastic_launch(self.handle, begin, length, grid, block,
                                               _stream_handle(stream)), "miriam_elastic_launch")

    def launch_traced(self, begin, length, grid, block, owner_wg, owner_iter, count, stream=None,
                      wave_phys=None, wave_slot=None):
        def ptr(t):
            return None if t is None else ctypes.c_void_p(t.data_ptr())
        L.check(L.load().miriam_elastic_launch_traced(
            self.handle, begin, length, grid, block, _stream_handle(stream),
            ptr(owner_wg), ptr(owner_iter), ptr(count), ptr(wave_phys), ptr(wave_slot)),
            "miriam_elastic_launch_traced")

    def reset_counters(self, stream=None) -> None:
        """Clear the split-K arrival counters (stream-ordered) after a pass that did not cover
        the whole tile space."""
        L.check(L.load().miriam_op_reset_counters(self.handle, _stream_handle(stream)),
                "miriam_op_reset_counters")

    def variant(self, **changes) -> "ElasticOp":
        """A second op over the same tensors, from this op's descriptor with `changes` applied
        (for example flags=op.desc.flags | INDEX_MEMORY)."""
        lib = L.load()
        new = ElasticOp.__new__(ElasticOp)
        d = L.OpDesc.from_buffer_copy(self.desc)
        for k, v in changes.items():
            setattr(d, k, v)
        new.desc = d
        new._keep = self._keep
        h = ctypes.c_void_p()
        L.check(lib.miriam_op_create(ctypes.byref(d), ctypes.byref(h)), "miriam_op_create")
        new.handle = h
        info = L.OpInfo()
        L.check(lib.miriam_op_query(h, ctypes.byref(info)), "miriam_op_query")
        new.info = info
        new.T = int(info.num_tiles)
        return new

    def run(self, stream=None) -> None:
        """Unsharded launch: the whole tile space at the op's full grid (one workgroup per
        tile, or the resident capacity for kernels that keep operands across tiles), block 256."""
        self.launch(0, self.T, int(self.info.full_grid), 256, stream)

    def run_plan(self, shards, grids, blocks, stream=None) -> None:
        for (b, l), g, bl in zip(shards, grids, blocks):
            self.launch(b, l, g, bl, stream)

    def destroy(self) -> None:
        if self.handle:
            L.check(L.load().miriam_op_destroy(self.handle), "miriam_op_destroy")
            self.handle = None

    def __del__(self):
        try:
            if self.handle:
                L.load().miriam_op_destroy(self.handle)
        except Exception:
            pass


# ------------------------------------------------------------ constructors
def _epi(bias, bn, residual):
    flags = 0
    if bias is not None:
        flags |= L.EPI_BIAS
    if bn is not None:
        flags |= L.EPI_BN
    if residual is not None:
        flags |= L.EPI_RESIDUAL
    return flags


def conv2d(x, w, y, stride=1, pad=0, bias=None, bn=None, residual=None, act="none", eps=1e-5, tile=0,
           ksplit=0, memory_index=False):
    """x [N,H,W,C], w [K,KH,KW,C], y [N,Ho,Wo,K]; bias [K] f32; bn [4,K] f32.
    memory_index: output-row indices from a host-computed table instead of in-kernel division."""
    N, H, W, C = x.shape
    K, KH, KW, C2 = w.shape
    assert C2 == C
    return ElasticOp(L.OP_CONV2D, x.dtype, keep=(x, w, y, bias, bn, residual),
                     n=N, h=H, w=W, c=C, k=K, kh=KH, kw=KW, stride=stride, pad=pad, groups=1,
                     x=x, wt=w, y=y, bias=bias, bn=bn, residual=residual,
                     flags=_epi(bias, bn, residual) | (L.INDEX_MEMORY if memory_index else 0),
                     act=L.ACT_CODE[act], eps=eps, tile=tile, ksplit=ksplit)


def gemm(x, w, y, bias=None, residual=None, act="none", tile=0, ldx=0, ldw=0, ldy=0, m=None, n=None, k=None,
         ksplit=0, memory_index=False):
    """y[m][n] = act(x[m][:] . w[n][:] + bias + residual)."""
    M = m if m is not None else x.shape[0]
    Kk = k if k is not None else x.shape[-1]
    Nn = n if n is not None else w.shape[0]
    return ElasticOp(L.OP_GEMM, x.dtype, keep=(x, w, y, bias, residual),
                     m=M, nn=Nn, kk=Kk, ldx=ldx, ldw=ldw, ldy=ldy, x=x, wt=w, y=y, bias=bias,
                     residual=residual, flags=_epi(bias, None, residual) | (L.INDEX_MEMORY if memory_index else 0),
                     act=L.ACT_CODE[act], tile=tile, ksplit=ksplit)


def bgemm(x, w, y, m, n, k, batch, batch_div, ldx, ldw, ldy, sx=(0, 0), sw=(0, 0), sy=(0, 0),
          b_nmajor=False, tile=0):
    return ElasticOp(L.OP_BGEMM, x.dtype, keep=(x, w, y),
                     m=m, nn=n, kk=k, batch=batch, batch_div=batch_div, ldx=ldx, ldw=ldw, ldy=ldy,
                     sx0=sx[0], sx1=sx[1], sw0=sw[0], sw1=sw[1], sy0=sy[0], sy1=sy[1],
                     b_nmajor=1 if b_nmajor else 0, x=x, wt=w, y=y, tile=tile)


def dwconv(x, w, y, stride=1, pad=1, bias=None, bn=None, residual=None, act="none", eps=1e-5):
    """x [N,H,W,C], w [KH,KW,C], y [N,Ho,Wo,C]."""
    N, H, W, C = x.shape
    KH, KW, C2 = w.shape
    assert C2 == C
    return ElasticOp(L.OP_DWCONV, x.dtype, keep=(x, w, y, bias, bn, residual),
                     n=N, h=H, w=W, c=C, k=C, kh=KH, kw=KW, stride=stride, pad=pad, groups=C,
                     x=x, wt=w, y=y, bias=bias, bn=bn, residual=residual,
                     flags=_epi(bias, bn, residual), act=L.ACT_CODE[act], eps=eps)


def pool(x, y, k, stride, pad, mode="max"):
    N, H, W, C = x.shape
    kind = L.OP_POOL_MAX if mode == "max" else L.OP_POOL_AVG
    return ElasticOp(kind, x.dtype, keep=(x, y), n=N, h=H, w=W, c=C, k=C, kh=k, kw=k,
                     stride=stride, pad=pad, x=x, y=y)


def softmax(x, y, rows, n, scale=1.0, ldx=0, ldy=0):
    return ElasticOp(L.OP_SOFTMAX, x.dtype, keep=(x, y), m=rows, nn=n, ldx=ldx, ldy=ldy,
                     scale=scale, x=x, y=y)


def layernorm(x, gamma, beta, y, rows, n, residual=None, eps=1e-5):
    return ElasticOp(L.OP_LAYERNORM, x.dtype, keep=(x, gamma, beta, y, residual), m=rows, nn=n,
                     x=x, wt=gamma, bias=beta, y=y, residual=residual,
                     flags=L.EPI_RESIDUAL if residual is not None else 0, eps=eps)


def bn_act(x, y, rows, channels, bias=None, bn=None, residual=None, act="none", eps=1e-5):
    return ElasticOp(L.OP_BN_ACT, x.dtype, keep=(x, y, bias, bn, residual), m=rows, nn=channels,
                     x=x, y=y, bias=bias, bn=bn, residual=residual,
                     flags=_epi(bias, bn, residual), act=L.ACT_CODE[act], eps=eps)


def device_info():
    dd = L.DeviceDesc()
    L.check(L.load().miriam_device_query(ctypes.byref(dd)), "miriam_device_query")
    return dd
