"""Python binding of the router library: torch tensors in, torch tensors out.

Every function here only checks tensor metadata, allocates outputs and workspace with
torch on the tensors' device, and passes raw device pointers and the current HIP stream to
libmore.so.  All arithmetic runs in the library's HIP kernels.

Layouts (see include/more.h): x [T][h] bf16; R1t = R1^T [r][h] bf16 (the paper's
down-projection); R2t = R2^T [M][r] bf16 (the paper's expert vectors, one row per expert);
Wt [M][h] bf16 (the full-rank router matrix, one row per expert).
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import Optional

import torch

from . import _lib


@dataclasses.dataclass
class Routing:
    idx: torch.Tensor  # int32 [T][k], experts in selection order
    gate: torch.Tensor  # float32 [T][k], softmax over the selected logits
    topval: Optional[torch.Tensor] = None  # float32 [T][k], the selected logits
    counts: Optional[torch.Tensor] = None  # int32 [M], selections per expert


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check_bf16(name: str, t: torch.Tensor, ndim: int):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != torch.bfloat16:
        raise TypeError("%s must be bfloat16, got %s" % (name, t.dtype))
    if t.dim() != ndim or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %d-D tensor" % (name, ndim))
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU device" % name)


def lowrank_workspace_size(T: int, h: int, r: int, M: int, k: int, m_chunks: int = 0) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().more_route_lowrank_workspace_size_ex(T, h, r, M, k, m_chunks,
                                                                ctypes.byref(n)),
               "more_route_lowrank_workspace_size_ex")
    return n.value


def lowrank_plan(T: int, h: int, r: int, M: int, k: int) -> int:
    """Number of expert-axis chunks the library picks for this shape (0: the fused or the
    single-pass route, which no m_chunks >= 1 selects)."""
    c = ctypes.c_int32(0)
    _lib.check(_lib.load().more_route_lowrank_plan(T, h, r, M, k, ctypes.byref(c)),
               "more_route_lowrank_plan")
    return c.value


ROUTE_NAMES = {0: "expert-resident", 1: "fused", 2: "fused-local", 3: "single-pass", 4: "wide"}


def lowrank_route(T: int, h: int, r: int, M: int, k: int) -> str:
    """Name of the route more_route_lowrank takes for this shape."""
    c = ctypes.c_int32(0)
    _lib.check(_lib.load().more_route_lowrank_route(T, h, r, M, k, ctypes.byref(c)),
               "more_route_lowrank_route")
    return ROUTE_NAMES[c.value]


def fullrank_workspace_size(T: int, h: int, M: int, k: int, logit_bits: int = 32) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().more_route_fullrank_workspace_size(T, h, M, k, logit_bits,
                                                              ctypes.byref(n)),
               "more_route_fullrank_workspace_size")
    return n.value


class LowrankRouter:
    """Pre-allocated outputs and workspace for repeated calls with one shape.

    `__call__` only launches; results land in the tensors held by `out`.
    """

    def __init__(self, T: int, h: int, r: int, M: int, k: int, *, device=None,
                 topval: bool = False, histogram: bool = False, m_chunks: int = 0):
        self.shape = (T, h, r, M, k)
        self.m_chunks = m_chunks
        self.device = torch.device(device or "cuda")
        dev = self.device
        self.out = Routing(
            idx=torch.empty((T, k), dtype=torch.int32, device=dev),
            gate=torch.empty((T, k), dtype=torch.float32, device=dev),
            topval=torch.empty((T, k), dtype=torch.float32, device=dev) if topval else None,
            counts=torch.empty((M,), dtype=torch.int32, device=dev) if histogram else None,
        )
        nbytes = lowrank_workspace_size(T, h, r, M, k, m_chunks)
        self.workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
        self.workspace_bytes = nbytes

    def __call__(self, x: torch.Tensor, R1t: torch.Tensor, R2t: torch.Tensor) -> Routing:
        T, h, r, M, k = self.shape
        _check_bf16("x", x, 2)
        _check_bf16("R1t", R1t, 2)
        _check_bf16("R2t", R2t, 2)
        if tuple(x.shape) != (T, h) or tuple(R1t.shape) != (r, h) or tuple(R2t.shape) != (M, r):
            raise ValueError("shapes %s %s %s do not match the router's (T=%d, h=%d, r=%d, M=%d)"
                             % (tuple(x.shape), tuple(R1t.shape), tuple(R2t.shape), T, h, r, M))
        o = self.out
        ws = _ptr(self.workspace) if self.workspace_bytes else None
        lib = _lib.load()
        if self.m_chunks == 0:  # the library's own plan: the plain entry point
            st = lib.more_route_lowrank(_ptr(x), _ptr(R1t), _ptr(R2t), T, h, r, M, k,
                                        _ptr(o.idx), _ptr(o.gate), _ptr(o.topval),
                                        _ptr(o.counts), ws, self.workspace_bytes,
                                        _stream(x.device))
            _lib.check(st, "more_route_lowrank")
        else:
            st = lib.more_route_lowrank_ex(_ptr(x), _ptr(R1t), _ptr(R2t), T, h, r, M, k,
                                           self.m_chunks, _ptr(o.idx), _ptr(o.gate),
                                           _ptr(o.topval), _ptr(o.counts), ws,
                                           self.workspace_bytes, _stream(x.device))
            _lib.check(st, "more_route_lowrank_ex")
        return o


def route_lowrank(x: torch.Tensor, R1t: torch.Tensor, R2t: torch.Tensor, k: int, *,
                  topval: bool = False, histogram: bool = False, m_chunks: int = 0) -> Routing:
    """softmax(TopK(x R1 R2)) for every row of x; R1t = R1^T [r][h], R2t = R2^T [M][r]."""
    _check_bf16("x", x, 2)
    _check_bf16("R1t", R1t, 2)
    _check_bf16("R2t", R2t, 2)
    T, h = x.shape
    r, h2 = R1t.shape
    M, r2 = R2t.shape
    if h2 != h or r2 != r:
        raise ValueError("inconsistent shapes x %s R1t %s R2t %s"
                         % (tuple(x.shape), tuple(R1t.shape), tuple(R2t.shape)))
    router = LowrankRouter(T, h, r, M, k, device=x.device, topval=topval, histogram=histogram,
                           m_chunks=m_chunks)
    return router(x, R1t, R2t)


@dataclasses.dataclass
class TrainRouting(Routing):
    """Routing plus the softmax statistics of the training forward pass."""
    m: Optional[torch.Tensor] = None  # float32 [T], the top-1 logit
    Z: Optional[torch.Tensor] = None  # float32 [T], sum_e exp(l_te - m_t)
    psum: Optional[torch.Tensor] = None  # float32 [M], sum_t exp(l_te - m_t) / Z_t


def lowrank_train_workspace_size(T: int, h: int, r: int, M: int, k: int) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().more_route_lowrank_train_workspace_size(T, h, r, M, k,
                                                                   ctypes.byref(n)),
               "more_route_lowrank_train_workspace_size")
    return n.value


class LowrankTrainRouter:
    """Pre-allocated outputs and workspace for repeated training-forward calls with one shape
    (more_route_lowrank_train): the routing plus m, Z and psum."""

    def __init__(self, T: int, h: int, r: int, M: int, k: int, *, device=None,
                 topval: bool = False, histogram: bool = True):
        self.shape = (T, h, r, M, k)
        self.device = torch.device(device or "cuda")
        dev = self.device
        f32 = torch.float32
        self.out = TrainRouting(
            idx=torch.empty((T, k), dtype=torch.int32, device=dev),
            gate=torch.empty((T, k), dtype=f32, device=dev),
            topval=torch.empty((T, k), dtype=f32, device=dev) if topval else None,
            counts=torch.empty((M,), dtype=torch.int32, device=dev) if histogram else None,
            m=torch.empty((T,), dtype=f32, device=dev),
            Z=torch.empty((T,), dtype=f32, device=dev),
            psum=torch.empty((M,), dtype=f32, device=dev),
        )
        nbytes = lowrank_train_workspace_size(T, h, r, M, k)
        self.workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
        self.workspace_bytes = nbytes

    def __call__(self, x: torch.Tensor, R1t: torch.Tensor, R2t: torch.Tensor) -> TrainRouting:
        T, h, r, M, k = self.shape
        _check_bf16("x", x, 2)
        _check_bf16("R1t", R1t, 2)
        _check_bf16("R2t", R2t, 2)
        if tuple(x.shape) != (T, h) or tuple(R1t.shape) != (r, h) or tuple(R2t.shape) != (M, r):
            raise ValueError("shapes %s %s %s do not match the router's (T=%d, h=%d, r=%d, M=%d)"
                             % (tuple(x.shape), tuple(R1t.shape), tuple(R2t.shape), T, h, r, M))
        o = self.out
        ws = _ptr(self.workspace) if self.workspace_bytes else None
        st = _lib.load().more_route_lowrank_train(
            _ptr(x), _ptr(R1t), _ptr(R2t), T, h, r, M, k, _ptr(o.idx), _ptr(o.gate),
            _ptr(o.topval), _ptr(o.counts), _ptr(o.m), _ptr(o.Z), _ptr(o.psum), ws,
            self.workspace_bytes, _stream(x.device))
        _lib.check(st, "more_route_lowrank_train")
        return o


def route_lowrank_train(x: torch.Tensor, R1t: torch.Tensor, R2t: torch.Tensor, k: int, *,
                        topval: bool = False, histogram: bool = True) -> TrainRouting:
    """Training forward pass of the low-rank router: route_lowrank plus the row maximum m,
    the softmax normaliser Z over all experts and the column sums psum of the row softmax."""
    _check_bf16("x", x, 2)
    _check_bf16("R1t", R1t, 2)
    _check_bf16("R2t", R2t, 2)
    T, h = x.shape
    r, h2 = R1t.shape
    M, r2 = R2t.shape
    if h2 != h or r2 != r:
        raise ValueError("inconsistent shapes x %s R1t %s R2t %s"
                         % (tuple(x.shape), tuple(R1t.shape), tuple(R2t.shape)))
    router = LowrankTrainRouter(T, h, r, M, k, device=x.device, topval=topval,
                                histogram=histogram)
    return router(x, R1t, R2t)


@dataclasses.dataclass
class Gradients:
    """Gradients of the training backward pass (float32)."""
    dx: torch.Tensor    # [T][h]
    dR1t: torch.Tensor  # [r][h]
    dR2t: torch.Tensor  # [M][r]


def lowrank_backward_workspace_size(T: int, h: int, r: int, M: int, k: int,
                                    balance: bool = True) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().more_route_lowrank_backward_workspace_size(T, h, r, M, k, int(balance),
                                                                      ctypes.byref(n)),
               "more_route_lowrank_backward_workspace_size")
    return n.value


def _check_dev(name: str, t: torch.Tensor, dtype, shape):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError("%s must be a contiguous tensor of shape %s, got %s"
                         % (name, tuple(shape), tuple(t.shape)))
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU device" % name)


class LowrankBackward:
    """Pre-allocated gradients and workspace for repeated backward calls with one shape
    (more_route_lowrank_backward); balance=False leaves out the psum term (pbar)."""

    def __init__(self, T: int, h: int, r: int, M: int, k: int, *, balance: bool = True,
                 device=None):
        self.shape = (T, h, r, M, k)
        self.balance = balance
        dev = torch.device(device or "cuda")
        f32 = torch.float32
        self.out = Gradients(dx=torch.empty((T, h), dtype=f32, device=dev),
                             dR1t=torch.empty((r, h), dtype=f32, device=dev),
                             dR2t=torch.empty((M, r), dtype=f32, device=dev))
        nbytes = lowrank_backward_workspace_size(T, h, r, M, k, balance)
        self.workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
        self.workspace_bytes = nbytes

    def __call__(self, x, R1t, R2t, idx, dtop, pbar=None, m=None, Z=None) -> Gradients:
        T, h, r, M, k = self.shape
        _check_bf16("x", x, 2)
        _check_bf16("R1t", R1t, 2)
        _check_bf16("R2t", R2t, 2)
        if tuple(x.shape) != (T, h) or tuple(R1t.shape) != (r, h) or tuple(R2t.shape) != (M, r):
            raise ValueError("shapes %s %s %s do not match (T=%d, h=%d, r=%d, M=%d)"
                             % (tuple(x.shape), tuple(R1t.shape), tuple(R2t.shape), T, h, r, M))
        _check_dev("idx", idx, torch.int32, (T, k))
        _check_dev("dtop", dtop, torch.float32, (T, k))
        if (pbar is not None) != self.balance:
            raise ValueError("pbar must be given exactly when the backward was set up with "
                             "balance=True")
        if pbar is not None:
            _check_dev("pbar", pbar, torch.float32, (M,))
            _check_dev("m", m, torch.float32, (T,))
            _check_dev("Z", Z, torch.float32, (T,))
        o = self.out
        ws = _ptr(self.workspace) if self.workspace_bytes else None
        st = _lib.load().more_route_lowrank_backward(
            _ptr(x), _ptr(R1t), _ptr(R2t), T, h, r, M, k, _ptr(idx), _ptr(dtop), _ptr(pbar),
            _ptr(m), _ptr(Z), _ptr(o.dx), _ptr(o.dR1t), _ptr(o.dR2t), ws, self.workspace_bytes,
            _stream(x.device))
        _lib.check(st, "more_route_lowrank_backward")
        return o


def route_lowrank_backward(x, R1t, R2t, idx, dtop, pbar=None, m=None, Z=None) -> Gradients:
    """Training backward pass of the low-rank router: the gradients of x, R1t and R2t given the
    gradient dtop [T][k] with respect to the selected logits and, optionally, pbar [M] with
    respect to psum (then m and Z [T] are the statistics of the training forward pass)."""
    _check_bf16("x", x, 2)
    _check_bf16("R1t", R1t, 2)
    _check_bf16("R2t", R2t, 2)
    T, h = x.shape
    r = R1t.shape[0]
    M = R2t.shape[0]
    k = idx.shape[1] if idx.dim() == 2 else 0
    return LowrankBackward(T, h, r, M, k, balance=pbar is not None, device=x.device)(
        x, R1t, R2t, idx, dtop, pbar, m, Z)


class FullrankRouter:
    """Pre-allocated outputs and workspace (logits + GEMM scratch) for the full-rank router."""

    def __init__(self, T: int, h: int, M: int, k: int, *, device=None, topval: bool = False,
                 logit_bits: int = 32):
        self.shape = (T, h, M, k)
        self.logit_bits = logit_bits
        dev = torch.device(device or "cuda")
        self.out = Routing(
            idx=torch.empty((T, k), dtype=torch.int32, device=dev),
            gate=torch.empty((T, k), dtype=torch.float32, device=dev),
            topval=torch.empty((T, k), dtype=torch.float32, device=dev) if topval else None)
        self.workspace_bytes = fullrank_workspace_size(T, h, M, k, logit_bits)
        self.workspace = torch.empty((max(self.workspace_bytes, 1),), dtype=torch.uint8,
                                     device=dev)

    def __call__(self, x: torch.Tensor, Wt: torch.Tensor) -> Routing:
        T, h, M, k = self.shape
        _check_bf16("x", x, 2)
        _check_bf16("Wt", Wt, 2)
        if tuple(x.shape) != (T, h) or tuple(Wt.shape) != (M, h):
            raise ValueError("shapes %s %s do not match (T=%d, h=%d, M=%d)"
                             % (tuple(x.shape), tuple(Wt.shape), T, h, M))
        o = self.out
        st = _lib.load().more_route_fullrank(_ptr(x), _ptr(Wt), T, h, M, k, self.logit_bits,
                                             _ptr(o.idx), _ptr(o.gate), _ptr(o.topval),
                                             _ptr(self.workspace), self.workspace_bytes,
                                             _stream(x.device))
        _lib.check(st, "more_route_fullrank")
        return o


def route_fullrank(x: torch.Tensor, Wt: torch.Tensor, k: int, *, topval: bool = False,
                   logit_bits: int = 32) -> Routing:
    """softmax(TopK(x W)) with Wt = W^T [M][h] (the standard router; logits materialised)."""
    _check_bf16("x", x, 2)
    _check_bf16("Wt", Wt, 2)
    T, h = x.shape
    M, h2 = Wt.shape
    if h2 != h:
        raise ValueError("inconsistent shapes x %s Wt %s" % (tuple(x.shape), tuple(Wt.shape)))
    return FullrankRouter(T, h, M, k, device=x.device, topval=topval, logit_bits=logit_bits)(x, Wt)


def fullrank_fused_workspace_size(T: int, h: int, M: int, k: int) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.load().more_route_fullrank_fused_workspace_size(T, h, M, k, ctypes.byref(n)),
               "more_route_fullrank_fused_workspace_size")
    return n.value


class FusedFullrankRouter:
    """Pre-allocated outputs and workspace for the fused full-rank router (no logits written)."""

    def __init__(self, T: int, h: int, M: int, k: int, *, device=None, topval: bool = False):
        self.shape = (T, h, M, k)
        dev = torch.device(device or "cuda")
        self.out = Routing(
            idx=torch.empty((T, k), dtype=torch.int32, device=dev),
            gate=torch.empty((T, k), dtype=torch.float32, device=dev),
            topval=torch.empty((T, k), dtype=torch.float32, device=dev) if topval else None)
        self.workspace_bytes = fullrank_fused_workspace_size(T, h, M, k)
        self.workspace = torch.empty((max(self.workspace_bytes, 1),), dtype=torch.uint8,
                                     device=dev)

    def __call__(self, x: torch.Tensor, Wt: torch.Tensor) -> Routing:
        T, h, M, k = self.shape
        _check_bf16("x", x, 2)
        _check_bf16("Wt", Wt, 2)
        if tuple(x.shape) != (T, h) or tuple(Wt.shape) != (M, h):
            raise ValueError("shapes %s %s do not match (T=%d, h=%d, M=%d)"
                             % (tuple(x.shape), tuple(Wt.shape), T, h, M))
        o = self.out
        ws = _ptr(self.workspace) if self.workspace_bytes else None
        st = _lib.load().more_route_fullrank_fused(_ptr(x), _ptr(Wt), T, h, M, k, _ptr(o.idx),
                                                   _ptr(o.gate), _ptr(o.topval), ws,
                                                   self.workspace_bytes, _stream(x.device))
        _lib.check(st, "more_route_fullrank_fused")
        return o


def route_fullrank_fused(x: torch.Tensor, Wt: torch.Tensor, k: int, *,
                         topval: bool = False) -> Routing:
    """softmax(TopK(x W)) with Wt = W^T [M][h], fused: no logits written (h <= 2112)."""
    _check_bf16("x", x, 2)
    _check_bf16("Wt", Wt, 2)
    T, h = x.shape
    M, h2 = Wt.shape
    if h2 != h:
        raise ValueError("inconsistent shapes x %s Wt %s" % (tuple(x.shape), tuple(Wt.shape)))
    return FusedFullrankRouter(T, h, M, k, device=x.device, topval=topval)(x, Wt)


def expert_histogram(idx: torch.Tensor, M: int) -> torch.Tensor:
    """counts[e] = number of entries of idx (int32 [T][k]) equal to e."""
    if idx.dtype != torch.int32 or idx.dim() != 2 or not idx.is_contiguous():
        raise ValueError("idx must be a contiguous int32 [T][k] tensor")
    if idx.device.type != "cuda":
        raise ValueError("idx must be on a GPU device")
    T, k = idx.shape
    counts = torch.empty((M,), dtype=torch.int32, device=idx.device)
    st = _lib.load().more_expert_histogram(_ptr(idx), T, k, M, _ptr(counts), _stream(idx.device))
    _lib.check(st, "more_expert_histogram")
    return counts


def dispatch_sort(idx: torch.Tensor, M: int) -> tuple[torch.Tensor, torch.Tensor]:
    """(offsets int32 [M + 1], sorted int32 [T k]): the positions p = t k + j of idx
    (int32 [T][k]) grouped by expert id, increasing p within an expert, ids outside [0, M)
    after all experts; offsets[e] = number of entries with a smaller id (more_dispatch_sort)."""
    if idx.dtype != torch.int32 or idx.dim() != 2 or not idx.is_contiguous():
        raise ValueError("idx must be a contiguous int32 [T][k] tensor")
    if idx.device.type != "cuda":
        raise ValueError("idx must be on a GPU device")
    T, k = idx.shape
    lib = _lib.load()
    n = ctypes.c_size_t(0)
    _lib.check(lib.more_dispatch_sort_workspace_size(T, k, M, ctypes.byref(n)),
               "more_dispatch_sort_workspace_size")
    ws = torch.empty((max(n.value, 1),), dtype=torch.uint8, device=idx.device)
    offsets = torch.empty((M + 1,), dtype=torch.int32, device=idx.device)
    srt = torch.empty((T * k,), dtype=torch.int32, device=idx.device)
    st = lib.more_dispatch_sort(_ptr(idx), T, k, M, _ptr(offsets), _ptr(srt), _ptr(ws), n.value,
                                _stream(idx.device))
    _lib.check(st, "more_dispatch_sort")
    return offsets, srt


class DispatchSorter:
    """Pre-allocated outputs and workspace for repeated more_dispatch_sort calls on one shape
    (no allocation per call, so a call can be captured in a HIP graph)."""

    def __init__(self, T: int, k: int, M: int, device="cuda"):
        self.T, self.k, self.M = T, k, M
        dev = torch.device(device)
        n = ctypes.c_size_t(0)
        _lib.check(_lib.load().more_dispatch_sort_workspace_size(T, k, M, ctypes.byref(n)),
                   "more_dispatch_sort_workspace_size")
        self.workspace_bytes = n.value
        self.workspace = torch.empty((max(n.value, 1),), dtype=torch.uint8, device=dev)
        self.offsets = torch.empty((M + 1,), dtype=torch.int32, device=dev)
        self.sorted = torch.empty((T * k,), dtype=torch.int32, device=dev)

    def __call__(self, idx: torch.Tensor):
        if idx.dtype != torch.int32 or tuple(idx.shape) != (self.T, self.k) or not idx.is_contiguous():
            raise ValueError("idx must be a contiguous int32 [%d][%d] tensor" % (self.T, self.k))
        st = _lib.load().more_dispatch_sort(_ptr(idx), self.T, self.k, self.M, _ptr(self.offsets),
                                            _ptr(self.sorted), _ptr(self.workspace),
                                            self.workspace_bytes, _stream(idx.device))
        _lib.check(st, "more_dispatch_sort")
        return self.offsets, self.sorted
