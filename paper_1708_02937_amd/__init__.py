"""Python binding of libsdnn.so, the MI355X sparse DNN forward pass (C ABI in include/sdnn.h).

The functions below carry the C names and only marshal arguments: every step of the
forward pass runs in the library's HIP kernels.  PyTorch supplies device memory and
the stream.  Importing this package fails if libsdnn.so has not been built
(``python paper_1708_02937_amd/build.py``); there is no fallback.

The paper computes Y_{k+1} = h(W_k Y_k + B_k) with ReLU h (Kepner et al.,
arXiv:1708.02937, Sec. III) via the GraphBLAS loop of Fig. 4 (Sec. IV); here the
same step is Y_{k+1} = h(Y_k W_k + 1 b_k^T) with Y batch x n.
"""

from __future__ import annotations

import ctypes
import math
import os
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsdnn.so")

SDNN_OK = 0
SDNN_ARM_SPARSE = 0
SDNN_ARM_DENSE = 1
SDNN_ARM_DENSE_F32 = 2
SDNN_ARENA_DENSE_F64 = 1
SDNN_ARENA_DENSE_F32 = 2
SDNN_BIAS_EVERYWHERE = 0
SDNN_BIAS_PATTERN = 1
SDNN_SEMIRING_PLUS_TIMES = 0
SDNN_SEMIRING_MAX_PLUS = 1
SDNN_SEMIRING_MAX_MIN = 2
SDNN_SEMIRING_MIN_MAX = 3
SDNN_SEMIRING_XOR_AND = 4

# kernel ids of the profiling log (SDNN_KERNEL_*) and the kernels they stand for
KERNEL_NAMES = {
    0: "transpose_kernel", 1: "spmm_fanin_kernel", 2: "spmm_narrow_kernel", 3: "spmm_slots_kernel",
    4: "spmm_tiled_kernel", 5: "gemm_dense_layer_kernel", 6: "spgemm_layer", 7: "densify", 8: "pack_dense_to_csr",
    9: "compact_rows", 10: "spmm_blocked_kernel", 11: "gemm32_dense_layer_kernel",
}

STATUS_NAMES = {
    0: "SDNN_OK", 1: "SDNN_ERR_NULL_POINTER", 2: "SDNN_ERR_INVALID_VALUE", 3: "SDNN_ERR_INVALID_INDEX",
    4: "SDNN_ERR_DIMENSION_MISMATCH", 5: "SDNN_ERR_INVALID_OBJECT", 6: "SDNN_ERR_WORKSPACE_TOO_SMALL",
    7: "SDNN_ERR_OUT_OF_MEMORY", 8: "SDNN_ERR_DEVICE", 9: "SDNN_ERR_UNSUPPORTED",
}


class SdnnError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        self.name = STATUS_NAMES.get(status, f"status {status}")
        super().__init__(f"{self.name}: {message}")


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python {os.path.join(_HERE, 'build.py')}` first")

_c = ctypes
lib = ctypes.CDLL(LIB_PATH)
_P = _c.c_void_p
_I64 = _c.c_int64
_I32 = _c.c_int32
_sig = {
    "sdnn_net_create": [_c.POINTER(_P), _I64, _I32, _c.c_float, _c.POINTER(_I64), _I32, _P, _I64, _P],
    "sdnn_net_arena_size": [_I64, _I32, _c.POINTER(_I64), _I32, _c.POINTER(_I64)],
    "sdnn_net_set_stream": [_P, _P],
    "sdnn_net_set_bias_mode": [_P, _I32],
    "sdnn_net_set_layer": [_P, _I32, _I64, _P, _P, _P, _P],
    "sdnn_net_build_dense": [_P],
    "sdnn_workspace_size": [_P, _I64, _I32, _c.POINTER(_I64)],
    "sdnn_forward_dense": [_P, _I32, _I32, _I64, _P, _P, _P, _I64, _I32],
    "sdnn_forward_dense_noalloc": [_P, _I32, _I32, _I64, _P, _P, _I32],
    "sdnn_forward_csr": [_P, _I32, _I32, _I64, _P, _P, _P, _P, _I64, _P, _c.POINTER(_P), _c.POINTER(_P),
                         _c.POINTER(_I64)],
    "sdnn_mxm_dense": [_P, _I32, _I32, _I64, _P, _P, _P, _I64],
    "sdnn_mxm_csr": [_P, _I32, _I32, _I64, _P, _P, _P, _P, _P, _I64],
    "sdnn_net_free": [_P],
    "sdnn_net_set_profiling": [_P, _I32],
}


class KernelTime(ctypes.Structure):
    _fields_ = [("layer", ctypes.c_int32), ("kernel", ctypes.c_int32), ("ms", ctypes.c_float)]


lib_read_profile_args = [_P, _c.POINTER(KernelTime), _I32, _c.POINTER(_I32)]
for _name, _args in _sig.items():
    getattr(lib, _name).argtypes = _args
    getattr(lib, _name).restype = _c.c_int
lib.sdnn_net_read_profile.argtypes = lib_read_profile_args
lib.sdnn_net_read_profile.restype = _c.c_int
lib.sdnn_noalloc_scratch_bytes.argtypes = []
lib.sdnn_noalloc_scratch_bytes.restype = _I64
lib.sdnn_status_string.argtypes = [_c.c_int]
lib.sdnn_status_string.restype = _c.c_char_p
lib.sdnn_last_error.argtypes = []
lib.sdnn_last_error.restype = _c.c_char_p


def _check(status: int):
    if status != SDNN_OK:
        raise SdnnError(status, lib.sdnn_last_error().decode())


def _ptr(x):
    """Device address of a torch tensor, or an int / None passed through."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def sdnn_status_string(status: int) -> str:
    return lib.sdnn_status_string(status).decode()


def sdnn_last_error() -> str:
    return lib.sdnn_last_error().decode()


def _caps(nnz_per_layer):
    arr = (_I64 * max(1, len(nnz_per_layer)))(*[int(x) for x in nnz_per_layer])
    return arr


def sdnn_net_arena_size(n: int, L: int, nnz_per_layer, dense_flags: int = 0) -> int:
    out = _I64()
    _check(lib.sdnn_net_arena_size(n, L, _caps(nnz_per_layer), dense_flags, _c.byref(out)))
    return out.value


def sdnn_net_create(n: int, L: int, ymax: float, nnz_per_layer, dense_flags: int, arena, arena_bytes: int,
                    stream=None):
    """Returns the opaque net handle (an int); arena: device memory of at least sdnn_net_arena_size bytes."""
    h = _P()
    _check(lib.sdnn_net_create(_c.byref(h), n, L, ymax, _caps(nnz_per_layer), dense_flags, _ptr(arena), arena_bytes,
                               _ptr(stream)))
    return h.value


def sdnn_net_set_stream(net, stream):
    _check(lib.sdnn_net_set_stream(net, _ptr(stream)))


def sdnn_net_set_bias_mode(net, mode: int):
    _check(lib.sdnn_net_set_bias_mode(net, mode))


def sdnn_net_set_layer(net, k: int, nnz: int, row_ptr, col_idx, val, bias):
    _check(lib.sdnn_net_set_layer(net, k, nnz, _ptr(row_ptr), _ptr(col_idx), _ptr(val), _ptr(bias)))


def sdnn_net_build_dense(net):
    _check(lib.sdnn_net_build_dense(net))


def sdnn_workspace_size(net, batch: int, y_is_csr: int) -> int:
    out = _I64()
    _check(lib.sdnn_workspace_size(net, batch, y_is_csr, _c.byref(out)))
    return out.value


def sdnn_forward_dense(net, k0: int, k1: int, batch: int, y_in, y_out, ws, ws_bytes: int, arm: int = SDNN_ARM_SPARSE):
    _check(lib.sdnn_forward_dense(net, k0, k1, batch, _ptr(y_in), _ptr(y_out), _ptr(ws), ws_bytes, arm))


def sdnn_forward_dense_noalloc(net, k0: int, k1: int, batch: int, y_in, y_out, arm: int = SDNN_ARM_SPARSE):
    _check(lib.sdnn_forward_dense_noalloc(net, k0, k1, batch, _ptr(y_in), _ptr(y_out), arm))


def sdnn_noalloc_scratch_bytes() -> int:
    return int(lib.sdnn_noalloc_scratch_bytes())


def sdnn_forward_csr(net, k0: int, k1: int, batch: int, y_row_ptr, y_col, y_val, ws, ws_bytes: int, out_row_ptr):
    """Returns (device address of out_col, device address of out_val, nnz)."""
    oc, ov, nnz = _P(), _P(), _I64()
    _check(lib.sdnn_forward_csr(net, k0, k1, batch, _ptr(y_row_ptr), _ptr(y_col), _ptr(y_val), _ptr(ws), ws_bytes,
                                _ptr(out_row_ptr), _c.byref(oc), _c.byref(ov), _c.byref(nnz)))
    return oc.value or 0, ov.value or 0, nnz.value


def sdnn_mxm_dense(net, k: int, semiring: int, batch: int, y, z, ws, ws_bytes: int):
    _check(lib.sdnn_mxm_dense(net, k, semiring, batch, _ptr(y), _ptr(z), _ptr(ws), ws_bytes))


def sdnn_mxm_csr(net, k: int, semiring: int, batch: int, y_row_ptr, y_col, y_val, z, ws, ws_bytes: int):
    _check(lib.sdnn_mxm_csr(net, k, semiring, batch, _ptr(y_row_ptr), _ptr(y_col), _ptr(y_val), _ptr(z),
                            _ptr(ws), ws_bytes))


def sdnn_net_free(net):
    _check(lib.sdnn_net_free(net))


def sdnn_net_set_profiling(net, enable: bool):
    _check(lib.sdnn_net_set_profiling(net, 1 if enable else 0))


def sdnn_net_read_profile(net, max_records: int = 1 << 16):
    """Up to max_records entries of the profiling log as (layer, kernel id, ms), oldest first; clears it."""
    buf = (KernelTime * max(1, max_records))()
    count = _I32()
    _check(lib.sdnn_net_read_profile(net, buf, max_records, _c.byref(count)))
    return [(r.layer, r.kernel, r.ms) for r in buf[:min(count.value, max_records)]]


class Net:
    """Owns a net handle, its arena (a torch uint8 tensor) and the device tensors its layers reference (they
    must outlive it).  nnz_per_layer: the most entries each layer will hold (an int applies to every layer);
    dense: SDNN_ARENA_DENSE_* flags (True means the fp64 copy) for the dense arms."""

    def __init__(self, n: int, L: int, ymax: float = math.inf, device: str = "cuda:0", nnz_per_layer=None,
                 dense=0):
        import torch

        self.torch = torch
        self.device = torch.device(device)
        self.n, self.L, self.ymax = n, L, ymax
        if nnz_per_layer is None:
            raise ValueError("nnz_per_layer (the entry capacity of each layer) is required")
        caps = [int(nnz_per_layer)] * L if isinstance(nnz_per_layer, int) else [int(x) for x in nnz_per_layer]
        flags = SDNN_ARENA_DENSE_F64 if dense is True else int(dense or 0)
        self.arena_bytes = sdnn_net_arena_size(n, L, caps, flags)
        self.arena = torch.empty(max(self.arena_bytes, 1), dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            self.handle = sdnn_net_create(n, L, ymax, caps, flags, self.arena, self.arena_bytes,
                                          torch.cuda.current_stream(self.device).cuda_stream)
        self._keep = [None] * L
        self._ws = {}

    def _dev(self, a, dtype):
        t = self.torch
        if isinstance(a, t.Tensor):
            return a.to(self.device, dtype).contiguous()
        return t.from_numpy(a).to(self.device, dtype).contiguous()

    def set_layer(self, k: int, row_ptr, col, val, bias):
        t = self.torch
        rp = self._dev(row_ptr, t.int64)
        c = self._dev(col, t.int32)
        v = self._dev(val, t.float32)
        b = self._dev(bias, t.float32)
        nnz = int(v.numel())
        sdnn_net_set_layer(self.handle, k, nnz, rp, c if nnz else None, v if nnz else None, b)
        self._keep[k] = (rp, c, v, b)

    def build_dense(self):
        sdnn_net_build_dense(self.handle)

    def set_bias_mode(self, mode: int):
        sdnn_net_set_bias_mode(self.handle, mode)

    def workspace(self, batch: int, y_is_csr: int):
        key = (batch, y_is_csr)
        need = sdnn_workspace_size(self.handle, batch, y_is_csr)
        ws = self._ws.get(key)
        if ws is None or ws.numel() < need:
            self._ws.clear()
            ws = self.torch.empty(max(need, 1), dtype=self.torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    def forward_dense(self, y, k0: int = 0, k1: int | None = None, arm: int = SDNN_ARM_SPARSE, out=None):
        t = self.torch
        k1 = self.L if k1 is None else k1
        y = self._dev(y, t.float32)
        batch = y.shape[0]
        out = t.empty_like(y) if out is None else out
        ws = self.workspace(batch, 0)
        sdnn_forward_dense(self.handle, k0, k1, batch, y, out, ws, ws.numel(), arm)
        return out

    def capture_forward_dense(self, y, out, k0: int = 0, k1: int | None = None, arm: int = SDNN_ARM_SPARSE):
        """Record forward_dense(y -> out) as a HIP graph (a torch.cuda.CUDAGraph); g.replay() launches the same
        kernels from the graph instead of one call at a time, on the current stream.  y and out (device,
        float32, contiguous, batch x n) and the workspace stay bound to the graph: write new inputs into y
        before a replay and read out after it."""
        t = self.torch
        k1 = self.L if k1 is None else k1
        if not (isinstance(y, t.Tensor) and isinstance(out, t.Tensor) and y.is_contiguous() and out.is_contiguous()
                and y.dtype == t.float32 and out.dtype == t.float32 and y.device == self.device
                and out.shape == y.shape and y.dim() == 2 and y.shape[1] == self.n):
            raise ValueError("y and out must be contiguous float32 batch x n tensors on the net's device")
        batch = y.shape[0]
        ws = self.workspace(batch, 0)
        self.forward_dense(y, k0, k1, arm, out)  # any one-time device set-up happens outside the capture
        t.cuda.synchronize(self.device)
        prev = t.cuda.current_stream(self.device).cuda_stream
        g = t.cuda.CUDAGraph()
        try:
            with t.cuda.graph(g, stream=t.cuda.Stream(device=self.device)):
                sdnn_net_set_stream(self.handle, t.cuda.current_stream(self.device).cuda_stream)
                sdnn_forward_dense(self.handle, k0, k1, batch, y, out, ws, ws.numel(), arm)
        finally:
            sdnn_net_set_stream(self.handle, prev)
        g.sdnn_buffers = (y, out, ws)  # the graph reads and writes these addresses
        return g

    def mxm(self, k: int, semiring: int, y, out=None):
        """Z = Y (+).(x) W_k over a semiring (dense batch x n in and out)."""
        t = self.torch
        y = self._dev(y, t.float32)
        batch = y.shape[0]
        out = t.empty_like(y) if out is None else out
        ws = self.workspace(batch, 0)
        sdnn_mxm_dense(self.handle, k, semiring, batch, y, out, ws, ws.numel())
        return out

    def mxm_csr(self, k: int, semiring: int, row_ptr, col, val):
        """Z = Y (+).(x) W_k for a CSR batch (unstored entries are the 0-element); Z dense batch x n."""
        t = self.torch
        rp = self._dev(row_ptr, t.int64)
        c = self._dev(col, t.int32)
        v = self._dev(val, t.float32)
        batch = rp.numel() - 1
        out = t.empty((batch, self.n), dtype=t.float32, device=self.device)
        sdnn_mxm_csr(self.handle, k, semiring, batch, rp, c if c.numel() else None, v if v.numel() else None,
                     out, None, 0)
        return out

    def forward_csr(self, row_ptr, col, val, k0: int = 0, k1: int | None = None):
        """Returns (row_ptr, col, val) device tensors; col/val are views into the net's workspace."""
        t = self.torch
        k1 = self.L if k1 is None else k1
        rp = self._dev(row_ptr, t.int64)
        c = self._dev(col, t.int32)
        v = self._dev(val, t.float32)
        batch = rp.numel() - 1
        ws = self.workspace(batch, 1)
        out_rp = t.empty(batch + 1, dtype=t.int64, device=self.device)
        oc, ov, nnz = sdnn_forward_csr(self.handle, k0, k1, batch, rp, c if c.numel() else None,
                                       v if v.numel() else None, ws, ws.numel(), out_rp)
        base = ws.data_ptr()
        col_t = ws[oc - base: oc - base + 4 * nnz].view(t.int32)
        val_t = ws[ov - base: ov - base + 4 * nnz].view(t.float32)
        return out_rp, col_t, val_t

    def set_profiling(self, enable: bool = True):
        sdnn_net_set_profiling(self.handle, enable)

    def read_profile(self, max_records: int = 1 << 16):
        """The profiling log as a list of (layer, kernel name, ms); clears it."""
        return [(layer, KERNEL_NAMES.get(k, str(k)), ms)
                for layer, k, ms in sdnn_net_read_profile(self.handle, max_records)]

    def free(self):
        if getattr(self, "handle", None):
            sdnn_net_free(self.handle)
            self.handle = None
            self._keep = []
            self._ws.clear()
            self.arena = None

    def __del__(self, _finalizing=sys.is_finalizing):
        # At interpreter shutdown the HIP runtime (and any tool layered on it) may already be torn down, so
        # no HIP call is made from here then; the process exit releases the device memory.  (The check is
        # bound at definition: module globals such as sys may already be cleared when this runs.)
        if _finalizing():
            return
        try:
            self.free()
        except Exception:
            pass


def net_from_problem(problem, device: str = "cuda:0", dense=0, bias_mode: int = SDNN_BIAS_EVERYWHERE) -> Net:
    """Upload every layer of a workloads.Problem (dense: SDNN_ARENA_DENSE_* flags, True for the fp64 copy;
    the dense copies are built)."""
    net = Net(problem.n, problem.L, problem.ymax, device, nnz_per_layer=[l.nnz for l in problem.layers],
              dense=dense)
    if bias_mode != SDNN_BIAS_EVERYWHERE:
        net.set_bias_mode(bias_mode)
    for k, l in enumerate(problem.layers):
        net.set_layer(k, l.row_ptr, l.col, l.val, l.bias)
    if dense:
        net.build_dense()
    return net
