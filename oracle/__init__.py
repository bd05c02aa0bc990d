"""fp64 CPU oracle for the MoRE router (test infrastructure).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's CPU-baseline
leg are the only callers.  The library under `paper_2609_36301_amd` never imports this
package, and this package never imports the library.

The arithmetic lives in `oracle.c` (plain C, double precision); this module compiles it
with gcc and wraps it with ctypes.  Every function here is argument marshalling only.

Functions and the passage they follow:
  route_lowrank   softmax(TopK(x R1 R2)), the MoRE router ("Preliminaries", MoRE layer)
  route_fullrank  softmax(TopK(x W)), the standard router ("Preliminaries")
  histogram       per-expert selection counts (Appendix "Training", statistic f)
  route_stats     training-forward softmax statistics m, Z and psum (Appendix "Pseudocode",
                  training forward, eqs. app_softmax, app_psum, app_online)
  route_backward  training backward: gradients of x, R1 and R2 from those of the selected
                  logits and of psum (Appendix "Pseudocode", backward pass, eqs. app_chain,
                  app_jac, app_kernelgrad)
  dispatch_sort   "Sort + Count": positions grouped by expert plus offsets (MoE layer
                  forward pass, efficiency appendix)
  logits_at       the logits x R1 R2 at given (token, expert) pairs ("Preliminaries"), to
                  check a selection made elsewhere expert by expert
  fullrank_logits_at  the same for the full-rank logits x W (W as bf16 bits)
  parity          the comparison rules of a routing result against this oracle
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load_library(path: str):
    """Open a compiled oracle library at `path` and declare its entry points."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    lib.oracle_route_lowrank.argtypes = [P, P, P, i64, i32, i32, i32, i32, P, i64, P, P, P, P, i32]
    lib.oracle_route_lowrank.restype = ctypes.c_int
    for name in ("oracle_route_fullrank_f64", "oracle_route_fullrank_bf16"):
        fn = getattr(lib, name)
        fn.argtypes = [P, P, i64, i32, i32, i32, P, i64, P, P, P, P, i32]
        fn.restype = ctypes.c_int
    lib.oracle_histogram.argtypes = [P, i64, i32, i32, P]
    lib.oracle_dispatch_sort.argtypes = [P, i64, i32, i32, P, P]
    lib.oracle_route_stats.argtypes = [P, P, P, i64, i32, i32, i32, P, P, P, i32]
    lib.oracle_route_backward.argtypes = [P, P, P, i64, i32, i32, i32, i32, P, P, P, P, P, P, P,
                                          P, P, P, i32]
    lib.oracle_route_backward.restype = ctypes.c_int
    lib.oracle_histogram.restype = ctypes.c_int
    lib.oracle_logits_at.argtypes = [P, P, P, i64, i32, i32, i32, P, i64, P, i32, P, i32]
    lib.oracle_logits_at.restype = ctypes.c_int
    lib.oracle_fullrank_logits_at.argtypes = [P, P, i64, i32, i32, P, i64, P, i32, P]
    lib.oracle_fullrank_logits_at.restype = ctypes.c_int
    return lib


def _load(lib=None):
    global _lib
    if lib is not None:
        return lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build(force=True)
    _lib = load_library(_LIB_PATH)
    return _lib


_ERRORS = {1: "invalid argument", 2: "non-finite input", 3: "out of memory"}


def _check(status: int):
    if status != 0:
        raise ValueError("oracle: " + _ERRORS.get(status, "error %d" % status))


@dataclasses.dataclass
class OracleResult:
    idx: np.ndarray  # int32 [n][k], experts in (logit desc, index asc) order
    gate: np.ndarray  # float64 [n][k]
    topval: np.ndarray  # float64 [n][k], the selected logits
    next: np.ndarray  # float64 [n], the best unselected logit (-inf when k == M)

    @property
    def kth(self) -> np.ndarray:
        return self.topval[:, -1]


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _rows_arg(rows, T):
    if rows is None:
        return None, 0, T
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    return rows, rows.size, rows.size


def _threads(threads):
    if threads is None:
        try:
            return len(os.sched_getaffinity(0))
        except AttributeError:  # pragma: no cover
            return os.cpu_count() or 1
    return int(threads)


def _u16(a, shape_len=2):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16 or a.ndim != shape_len:
        raise TypeError("expected a %d-D uint16 array of bfloat16 bits" % shape_len)
    return a


def route_lowrank(x, R1, R2, k: int, rows=None, threads=None, lib=None) -> OracleResult:
    """x: bf16 bits [T][h]; R1: [h][r]; R2: [r][M] (row-major, mathematical orientation)."""
    x, R1, R2 = _u16(x), _u16(R1), _u16(R2)
    T, h = x.shape
    h2, r = R1.shape
    r2, M = R2.shape
    if h2 != h or r2 != r:
        raise ValueError("shape mismatch")
    rows_a, nrows, n = _rows_arg(rows, T)
    out = OracleResult(np.zeros((n, k), np.int32), np.zeros((n, k)), np.zeros((n, k)), np.zeros(n))
    lib = _load(lib)
    _check(lib.oracle_route_lowrank(_ptr(x), _ptr(R1), _ptr(R2), T, h, r, M, k,
                                    None if rows_a is None else _ptr(rows_a), nrows,
                                    _ptr(out.idx), _ptr(out.gate), _ptr(out.topval),
                                    _ptr(out.next), _threads(threads)))
    return out


def route_fullrank(x, W, k: int, rows=None, threads=None, lib=None) -> OracleResult:
    """x: bf16 bits [T][h]; W: [h][M] as float64 values or as bf16 bits (uint16)."""
    x = _u16(x)
    W = np.ascontiguousarray(W)
    T, h = x.shape
    h2, M = W.shape
    if h2 != h:
        raise ValueError("shape mismatch")
    rows_a, nrows, n = _rows_arg(rows, T)
    out = OracleResult(np.zeros((n, k), np.int32), np.zeros((n, k)), np.zeros((n, k)), np.zeros(n))
    lib = _load(lib)
    if W.dtype == np.uint16:
        fn = lib.oracle_route_fullrank_bf16
    elif W.dtype == np.float64:
        fn = lib.oracle_route_fullrank_f64
    else:
        raise TypeError("W must be float64 values or uint16 bfloat16 bits")
    _check(fn(_ptr(x), _ptr(W), T, h, M, k, None if rows_a is None else _ptr(rows_a), nrows,
              _ptr(out.idx), _ptr(out.gate), _ptr(out.topval), _ptr(out.next), _threads(threads)))
    return out


def logits_at(x, R1, R2, rows, experts, threads=None, lib=None) -> np.ndarray:
    """fp64 logits l[rows[i], experts[i][j]] ([n][m] float64); the same sums as route_lowrank."""
    x, R1, R2 = _u16(x), _u16(R1), _u16(R2)
    T, h = x.shape
    h2, r = R1.shape
    r2, M = R2.shape
    if h2 != h or r2 != r:
        raise ValueError("shape mismatch")
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    experts = np.ascontiguousarray(experts, dtype=np.int32)
    if rows.ndim != 1 or experts.ndim != 2 or experts.shape[0] != rows.size:
        raise ValueError("rows must be [n] and experts [n][m]")
    out = np.zeros(experts.shape, np.float64)
    _check(_load(lib).oracle_logits_at(_ptr(x), _ptr(R1), _ptr(R2), T, h, r, M, _ptr(rows),
                                       rows.size, _ptr(experts), experts.shape[1], _ptr(out),
                                       _threads(threads)))
    return out


def fullrank_logits_at(x, W, rows, experts, lib=None) -> np.ndarray:
    """fp64 logits (x W)[rows[i], experts[i][j]] with W bf16 bits [h][M]; [n][m] float64."""
    x, W = _u16(x), _u16(W)
    T, h = x.shape
    h2, M = W.shape
    if h2 != h:
        raise ValueError("shape mismatch")
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    experts = np.ascontiguousarray(experts, dtype=np.int32)
    if rows.ndim != 1 or experts.ndim != 2 or experts.shape[0] != rows.size:
        raise ValueError("rows must be [n] and experts [n][m]")
    out = np.zeros(experts.shape, np.float64)
    _check(_load(lib).oracle_fullrank_logits_at(_ptr(x), _ptr(W), T, h, M, _ptr(rows), rows.size,
                                                _ptr(experts), experts.shape[1], _ptr(out)))
    return out


def histogram(idx, M: int, lib=None) -> np.ndarray:
    """counts[e] = number of entries of idx ([n][k] int32) equal to e."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    if idx.ndim != 2:
        raise ValueError("idx must be [n][k]")
    counts = np.zeros(M, np.int64)
    _check(_load(lib).oracle_histogram(_ptr(idx), idx.shape[0], idx.shape[1], M, _ptr(counts)))
    return counts


def dispatch_sort(idx, M: int, lib=None):
    """(offsets [M + 1], sorted [n k]) of the entries of idx ([n][k] int32): positions
    p = t k + j grouped by expert id (ids outside [0, M) last), increasing within a group;
    offsets[e] = number of entries with a smaller key.  int64 arrays."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    if idx.ndim != 2:
        raise ValueError("idx must be [n][k]")
    offsets = np.zeros(M + 1, np.int64)
    srt = np.zeros(idx.size, np.int64)
    _check(_load(lib).oracle_dispatch_sort(_ptr(idx), idx.shape[0], idx.shape[1], M,
                                           _ptr(offsets), _ptr(srt)))
    return offsets, srt


def route_stats(x, R1, R2, threads=None, lib=None):
    """(m [T], Z [T], psum [M]) in fp64: the row maximum of the logits x R1 R2, the softmax
    normaliser sum_e exp(l - m), and the column sums of the row softmax over all experts."""
    x, R1, R2 = _u16(x), _u16(R1), _u16(R2)
    T, h = x.shape
    r, M = R2.shape
    if R1.shape != (h, r):
        raise ValueError("R1 must be [h][r]")
    m = np.zeros(T, np.float64)
    Z = np.zeros(T, np.float64)
    psum = np.zeros(M, np.float64)
    _check(_load(lib).oracle_route_stats(_ptr(x), _ptr(R1), _ptr(R2), T, h, r, M, _ptr(m),
                                         _ptr(Z), _ptr(psum), _threads(threads)))
    return m, Z, psum


@dataclasses.dataclass
class BackwardResult:
    dx: np.ndarray   # float64 [T][h]
    dR1: np.ndarray  # float64 [h][r]
    dR2: np.ndarray  # float64 [r][M]
    g: np.ndarray    # float64 [T], sum_e pbar_e P_te (0 without pbar)
    dz: np.ndarray   # float64 [T][r]


def route_backward(x, R1, R2, idx, dtop, pbar=None, m=None, Z=None, threads=None, lib=None):
    """Gradients of a loss with respect to x [T][h], R1 [h][r] and R2 [r][M] (bf16 bits), given
    its gradient dtop [T][k] with respect to the selected logits l_t[idx[t][j]] and pbar [M]
    with respect to psum (None: no balancing term; then m and Z are not read), with the saved
    statistics m [T], Z [T] defining P = exp(l - m) / Z.  fp64 throughout."""
    x, R1, R2 = _u16(x), _u16(R1), _u16(R2)
    T, h = x.shape
    r, M = R2.shape
    if R1.shape != (h, r):
        raise ValueError("R1 must be [h][r]")
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    dtop = np.ascontiguousarray(dtop, dtype=np.float64)
    if idx.ndim != 2 or idx.shape[0] != T or dtop.shape != idx.shape:
        raise ValueError("idx and dtop must be [T][k]")
    k = idx.shape[1]
    if pbar is not None:
        pbar = np.ascontiguousarray(pbar, dtype=np.float64)
        m = np.ascontiguousarray(m, dtype=np.float64)
        Z = np.ascontiguousarray(Z, dtype=np.float64)
        if pbar.shape != (M,) or m.shape != (T,) or Z.shape != (T,):
            raise ValueError("pbar must be [M], m and Z [T]")
    res = BackwardResult(dx=np.zeros((T, h)), dR1=np.zeros((h, r)), dR2=np.zeros((r, M)),
                         g=np.zeros(T), dz=np.zeros((T, r)))
    opt = (lambda a: None if a is None else _ptr(a))
    _check(_load(lib).oracle_route_backward(
        _ptr(x), _ptr(R1), _ptr(R2), T, h, r, M, k, _ptr(idx), _ptr(dtop), opt(pbar), opt(m),
        opt(Z), _ptr(res.dx), _ptr(res.dR1), _ptr(res.dR2), _ptr(res.g), _ptr(res.dz),
        _threads(threads)))
    return res
