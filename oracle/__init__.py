"""CPU oracle for the sparse DNN forward pass.

TEST INFRASTRUCTURE ONLY: the reference that the GPU library is checked
against.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
may import this package; the library never does and shares no code with it.

It wraps ``oracle.c`` (plain C, fp64 accumulation, one rounding to fp32 per
layer; see that file's header for the equations it follows: Sec. III of
Kepner et al., arXiv:1708.02937, batched inference with ReLU, in the
orientation Y_{k+1} = h(Y_k W_k + 1 b_k^T)).
"""

from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle.so")

_lib = None


class _Layer(ctypes.Structure):
    _fields_ = [
        ("row_ptr", ctypes.c_void_p),
        ("col", ctypes.c_void_p),
        ("val", ctypes.c_void_p),
        ("bias", ctypes.c_void_p),
    ]


def build(out_path: str = LIB_PATH, src: str = _SRC) -> str:
    """Compile the oracle with gcc (contraction off, so the source's operation order is the one run)."""
    tmp = out_path + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                           "-pthread", "-o", tmp, src, "-lm"])
    os.replace(tmp, out_path)
    return out_path


def load(path: str | None = None):
    """Load (building first if absent) the oracle library; `path` selects another build of it."""
    global _lib
    if path is not None:
        return _declare(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


def _declare(lib):
    lib.oracle_forward.restype = ctypes.c_int
    lib.oracle_forward.argtypes = [
        ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_Layer), ctypes.c_double, ctypes.c_int,
        ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    lib.oracle_mxm.restype = ctypes.c_int
    lib.oracle_mxm.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.POINTER(_Layer), ctypes.c_int64,
                               ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_preact.restype = ctypes.c_int
    lib.oracle_preact.argtypes = [
        ctypes.c_int64, ctypes.POINTER(_Layer), ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int]
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data if a.size else None


def _layer_structs(layers, keep):
    arr = (_Layer * max(1, len(layers)))()
    for k, l in enumerate(layers):
        rp = np.ascontiguousarray(l.row_ptr, dtype=np.int64)
        c = np.ascontiguousarray(l.col, dtype=np.int32)
        v = np.ascontiguousarray(l.val, dtype=np.float32)
        b = np.ascontiguousarray(l.bias, dtype=np.float32)
        keep.extend([rp, c, v, b])
        arr[k] = _Layer(rp.ctypes.data, _ptr(c), _ptr(v), b.ctypes.data)
    return arr


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count() or 1)


def forward(n: int, layers, ymax: float, y_csr, k0: int = 0, k1: int | None = None,
            threads: int | None = None, trace: bool = False, lib=None, bias_mode: int = 0):
    """Y_{k1} for the CSR rows `y_csr` = (row_ptr, col, val) taken as Y_{k0}.

    bias_mode 0 adds the bias at every position (the dense equation); 1 only where Y_k W_k has a
    structural entry (the pattern semantics of the Fig. 4 listing).

    Returns the output CSR (row_ptr int64, col int32, val float32); with
    ``trace=True`` also the per-layer nnz of Y_{k0+1} .. Y_{k1} summed over rows.
    """
    lib = lib or load()
    k1 = len(layers) if k1 is None else k1
    row_ptr = np.ascontiguousarray(y_csr[0], dtype=np.int64)
    col = np.ascontiguousarray(y_csr[1], dtype=np.int32)
    val = np.ascontiguousarray(y_csr[2], dtype=np.float32)
    nrows = len(row_ptr) - 1
    keep = []
    ls = _layer_structs(layers, keep)
    cnt = np.zeros(max(1, nrows), dtype=np.int64)
    oc = np.empty(max(1, nrows * n), dtype=np.int32)
    ov = np.empty(max(1, nrows * n), dtype=np.float32)
    lnnz = np.zeros(max(1, k1 - k0), dtype=np.int64)
    rc = lib.oracle_forward(n, k0, k1, ls, float(ymax), int(bias_mode), nrows, row_ptr.ctypes.data, _ptr(col), _ptr(val),
                            cnt.ctypes.data, oc.ctypes.data, ov.ctypes.data, lnnz.ctypes.data,
                            threads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_forward failed with status {rc}")
    cnt = cnt[:nrows]
    out_ptr = np.zeros(nrows + 1, dtype=np.int64)
    np.cumsum(cnt, out=out_ptr[1:])
    idx = np.repeat(np.arange(nrows, dtype=np.int64) * n - out_ptr[:-1], cnt) + np.arange(out_ptr[-1])
    out = (out_ptr, oc[idx], ov[idx])
    if trace:
        return out, lnnz[: k1 - k0]
    return out


def preact(n: int, layer, y_csr, threads: int | None = None, lib=None):
    """Dense fp64 (z, s) of one layer for the CSR rows `y_csr`: z = Y W + b, s = |Y||W| + |b|."""
    lib = lib or load()
    row_ptr = np.ascontiguousarray(y_csr[0], dtype=np.int64)
    col = np.ascontiguousarray(y_csr[1], dtype=np.int32)
    val = np.ascontiguousarray(y_csr[2], dtype=np.float32)
    nrows = len(row_ptr) - 1
    keep = []
    ls = _layer_structs([layer], keep)
    z = np.empty((max(1, nrows), n), dtype=np.float64)
    s = np.empty((max(1, nrows), n), dtype=np.float64)
    rc = lib.oracle_preact(n, ls, nrows, row_ptr.ctypes.data, _ptr(col), _ptr(val), z.ctypes.data,
                           s.ctypes.data, threads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_preact failed with status {rc}")
    return z[:nrows], s[:nrows]


def csr_to_dense(csr, n: int) -> np.ndarray:
    row_ptr, col, val = csr
    nrows = len(row_ptr) - 1
    out = np.zeros((nrows, n), dtype=np.float32)
    rows = np.repeat(np.arange(nrows), np.diff(row_ptr))
    out[rows, col] = val
    return out


INF = math.inf


SEMIRINGS = {"plus_times": 0, "max_plus": 1, "max_min": 2, "min_max": 3, "xor_and": 4}


def mxm(semiring, n: int, layer, y_dense, lib=None):
    """Z = Y (+).(x) W over one of SEMIRINGS (name or id) for dense rows y_dense (rows x n float32)."""
    lib = lib or load()
    sr = SEMIRINGS[semiring] if isinstance(semiring, str) else int(semiring)
    y = np.ascontiguousarray(y_dense, dtype=np.float32).reshape(-1, n)
    keep = []
    ls = _layer_structs([layer], keep)
    z = np.empty((max(1, y.shape[0]), n), dtype=np.float32)
    rc = lib.oracle_mxm(sr, n, ls, y.shape[0], _ptr(y), z.ctypes.data)
    if rc != 0:
        raise ValueError(f"oracle_mxm failed with status {rc}")
    return z[: y.shape[0]]
