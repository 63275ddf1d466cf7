"""Python binding of the MI355X DARB library (libdarb.so, C ABI in include/darb.h).

Argument marshalling only: every step of DARB runs in the library's HIP
kernels.  torch supplies device memory and the current HIP stream; numpy
arrays are accepted for host-side inputs (row densities).

    plan = Plan(M, N, row_density, matrix_density, mode=ROUND_FLOOR, b_min=4, b_max=64)
    # or, from the device-side irregular pruning of W (k largest magnitudes):
    #   plan = Plan.from_counts(N, prune_counts(W, k), k, ROUND_FLOOR, 4, 64)
    plan.upload()                           # device metadata into a torch workspace
    values, offsets = plan.encode(W)        # W: cuda tensor [M, N] fp32/fp16
    y = plan.spmv(values, offsets, x)       # fp32 [M]
    Y = plan.spmm(values, offsets, X)       # X: [N, B], fp32 [M, B]
    packed = plan.pack_offsets(offsets)     # log2 b bits per weight (section 4.2)
    y = plan.spmv_packed(values, packed, x) # same result, bit for bit

The library must have been built (``python paper_1911_08020_amd/build.py`` or
``__graft_entry__.build()``); importing this package fails loudly otherwise.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdarb.so")

OK = 0
E_INVALID = -1
E_DTYPE = -2
E_NOT_UPLOADED = -3
E_HIP = -4
E_NOMEM = -5
E_WORKSPACE = -6

F32 = 0
F16 = 1
ROUND_FLOOR = 0
ROUND_PAPER = 1


class DarbError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {_strerror(code)} ({code}): {detail}")
        self.code = code


class _Bin(ctypes.Structure):
    _fields_ = [("log2b", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("first_row", ctypes.c_int64), ("rows", ctypes.c_int64),
                ("first_elem", ctypes.c_int64), ("nblk", ctypes.c_int64),
                ("first_word", ctypes.c_int64)]


class _Info(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("workspace_bytes", ctypes.c_int64), ("packed_words", ctypes.c_int64),
                ("nbins", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("bins", _Bin * 8)]


def _load_library():
    # torch carries its own HIP runtime (same soname as /opt/rocm's).  Loading it
    # first makes libdarb.so bind to that one, so the process has a single HIP
    # runtime and the library sees the devices and streams torch uses.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"DARB HIP library not built: {LIB_PATH} is missing. "
            "Run `python paper_1911_08020_amd/build.py` (hipcc, gfx950) first.")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    sig = {
        "darb_version": ([], I),
        "darb_strerror": ([I], ctypes.c_char_p),
        "darb_last_error": ([], ctypes.c_char_p),
        "darb_plan_create": ([I64, I64, P, ctypes.c_double, I, I, I, ctypes.POINTER(P)], I),
        "darb_plan_info": ([P, ctypes.POINTER(_Info)], I),
        "darb_plan_export": ([P, P, P, P], I),
        "darb_plan_upload": ([P, P, I64, P], I),
        "darb_plan_destroy": ([P], None),
        "darb_encode": ([P, I, P, I64, P, P, P], I),
        "darb_decode": ([P, I, P, P, P, I64, P], I),
        "darb_spmv": ([P, I, P, P, I, P, P, P], I),
        "darb_spmm": ([P, I, P, P, I, I64, P, I64, P, I64, P], I),
        "darb_plan_create_counts": ([I64, I64, P, I64, I, I, I, ctypes.POINTER(P)], I),
        "darb_plan_device_workspace": ([I64, ctypes.POINTER(I64)], I),
        "darb_plan_create_device": ([I64, I64, P, I64, I, I, I, P, I64, P, ctypes.POINTER(P)], I),
        "darb_prune_workspace": ([I64, I64, I, ctypes.POINTER(I64)], I),
        "darb_prune_counts": ([I64, I64, I, P, I64, I64, P, P, I64, P], I),
        "darb_prune_counts_noalloc": ([I64, I64, I, P, I64, I64, P, P], I),
        "darb_pack_offsets": ([P, P, P, P], I),
        "darb_unpack_offsets": ([P, P, P, P], I),
        "darb_spmv_packed": ([P, I, P, P, I, P, P, P], I),
        "darb_spmm_packed": ([P, I, P, P, I, I64, P, I64, P, I64, P], I),
        "darb_quantize_i8": ([P, I, P, P, P, P], I),
        "darb_spmv_i8": ([P, P, P, P, P, I, P, P, P], I),
        "darb_spmm_i8": ([P, P, P, P, P, I, I64, P, I64, P, I64, P], I),
        "darb_lstm_layer": ([P, P, P, P, P, P, I, I64, I64, I64, P, P, P, P, P, I64, P], I),
        "darb_lstm_workspace": ([I64, I64, I64, ctypes.POINTER(I64)], I),
        "darb_stream_read": ([P, I64, P, P], I),
        "darb_stream_read_shape": ([P, I64, I, I, P, P], I),
        "darb_stream_copy": ([P, P, I64, P], I),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load_library()

#: every symbol include/darb.h declares
EXPORTED = ("darb_plan_create", "darb_plan_create_counts", "darb_plan_device_workspace",
            "darb_plan_create_device", "darb_prune_workspace",
            "darb_prune_counts", "darb_prune_counts_noalloc", "darb_plan_info", "darb_plan_export", "darb_plan_upload",
            "darb_plan_destroy", "darb_encode", "darb_decode", "darb_spmv", "darb_spmm",
            "darb_pack_offsets", "darb_unpack_offsets", "darb_spmv_packed", "darb_spmm_packed",
            "darb_quantize_i8", "darb_spmv_i8", "darb_spmm_i8", "darb_lstm_layer",
            "darb_lstm_workspace", "darb_stream_read", "darb_stream_read_shape", "darb_stream_copy", "darb_strerror",
            "darb_last_error", "darb_version")


def lib():
    return _lib


def _strerror(code: int) -> str:
    return _lib.darb_strerror(code).decode()


def _check(rc: int, where: str):
    if rc != OK:
        raise DarbError(rc, where, _lib.darb_last_error().decode())


def _torch():
    import torch
    return torch


def _stream_ptr(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.float16:
        return F16
    raise TypeError(f"unsupported dtype {t.dtype} (fp32 or fp16)")


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(t.data_ptr())


def _require_cuda(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("device tensors required (torch cuda tensors)")


def _check_format(t, n: int, name: str, dtypes=None):
    """A flat device buffer of at least n elements (of one of `dtypes`)."""
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} must be one of {dtypes}, got {t.dtype}")
    if not t.is_contiguous() or t.numel() < n:
        raise ValueError(f"{name} must be contiguous with >= {n} elements, got {t.numel()}")


def _row_major_ld(t, rows: int, cols: int, name: str) -> int:
    if t.dim() != 2 or t.shape[0] != rows or t.shape[1] != cols:
        raise ValueError(f"{name} must be [{rows}, {cols}], got {tuple(t.shape)}")
    if t.stride(1) != 1:
        raise ValueError(f"{name} must have unit column stride")
    return t.stride(0) if rows > 1 else max(cols, t.stride(0))


class Plan:
    """A DARB plan: block sizes and grouped layout from row densities (section 3.2)."""

    def __init__(self, M: int, N: int, row_density, matrix_density: float,
                 mode: int = ROUND_FLOOR, b_min: int = 1, b_max: int = 128, *, _counts=None):
        h = ctypes.c_void_p()
        if _counts is None:
            d = np.ascontiguousarray(row_density, dtype=np.float64)
            if d.shape != (M,):
                raise ValueError(f"row_density must have shape ({M},)")
            _check(_lib.darb_plan_create(int(M), int(N), d.ctypes.data_as(ctypes.c_void_p),
                                         float(matrix_density), int(mode), int(b_min),
                                         int(b_max), ctypes.byref(h)), "darb_plan_create")
        else:
            c, kept = _counts
            _check(_lib.darb_plan_create_counts(int(M), int(N), c.ctypes.data_as(ctypes.c_void_p),
                                                int(kept), int(mode), int(b_min), int(b_max),
                                                ctypes.byref(h)), "darb_plan_create_counts")
        self._take(h)
        self.workspace = None

    def _take(self, h):
        self._h = h
        info = _Info()
        _check(_lib.darb_plan_info(h, ctypes.byref(info)), "darb_plan_info")
        self.M, self.N, self.nnz = info.M, info.N, info.nnz
        self.workspace_bytes = info.workspace_bytes
        self.packed_words = info.packed_words
        self.bins = [dict(log2b=b.log2b, first_row=b.first_row, rows=b.rows,
                          first_elem=b.first_elem, nblk=b.nblk, first_word=b.first_word)
                     for b in info.bins[:info.nbins]]

    @classmethod
    def from_device_counts(cls, N: int, row_count, kept: int, mode: int = ROUND_FLOOR,
                           b_min: int = 1, b_max: int = 128, stream=None):
        """Plan built on the device from kept counts in device memory (``prune_counts``'s
        output, never copied to the host); comes back uploaded, its workspace being the
        one the tables were built in."""
        torch = _torch()
        _require_cuda(row_count)
        if row_count.dim() != 1:
            raise ValueError("row_count must be 1-D")
        M = row_count.shape[0]
        _check_format(row_count, M, "row_count", (torch.int64,))
        need = ctypes.c_int64()
        _check(_lib.darb_plan_device_workspace(M, ctypes.byref(need)), "darb_plan_device_workspace")
        ws = torch.empty(need.value, dtype=torch.uint8, device=row_count.device)
        h = ctypes.c_void_p()
        with torch.cuda.device(row_count.device):
            _check(_lib.darb_plan_create_device(int(M), int(N), _ptr(row_count), int(kept),
                                                int(mode), int(b_min), int(b_max), _ptr(ws),
                                                ws.numel(), _stream_ptr(stream), ctypes.byref(h)),
                   "darb_plan_create_device")
        self = cls.__new__(cls)
        self._take(h)
        self.workspace = ws
        return self

    @classmethod
    def from_counts(cls, N: int, row_count, kept: int, mode: int = ROUND_FLOOR, b_min: int = 1,
                    b_max: int = 128):
        """Plan from per-row kept counts (e.g. ``prune_counts``): d_r = count_r / N."""
        if hasattr(row_count, "is_cuda"):
            row_count = row_count.cpu().numpy()
        c = np.ascontiguousarray(row_count, dtype=np.int64)
        if c.ndim != 1:
            raise ValueError("row_count must be 1-D")
        return cls(c.shape[0], N, None, 0.0, mode, b_min, b_max, _counts=(c, kept))

    # bound at class creation: module globals may already be cleared when a plan is
    # collected at interpreter exit
    def __del__(self, _destroy=_lib.darb_plan_destroy):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def export(self) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        log2b = np.zeros(self.M, dtype=np.uint8)
        row_start = np.zeros(self.M, dtype=np.int64)
        perm = np.zeros(self.M, dtype=np.int32)
        _check(_lib.darb_plan_export(self._h, log2b.ctypes.data_as(ctypes.c_void_p),
                                     row_start.ctypes.data_as(ctypes.c_void_p),
                                     perm.ctypes.data_as(ctypes.c_void_p)), "darb_plan_export")
        return log2b, row_start, perm

    def upload(self, device=None, stream=None):
        torch = _torch()
        dev = torch.device("cuda") if device is None else torch.device(device)
        with torch.cuda.device(dev):
            ws = torch.empty(self.workspace_bytes, dtype=torch.uint8, device=dev)
            _check(_lib.darb_plan_upload(self._h, _ptr(ws), self.workspace_bytes,
                                         _stream_ptr(stream)), "darb_plan_upload")
        self.workspace = ws
        return self

    # -- device calls -----------------------------------------------------------------
    def empty_format(self, dtype, device=None):
        torch = _torch()
        dev = self.workspace.device if device is None else device
        return (torch.empty(self.nnz, dtype=dtype, device=dev),
                torch.empty(self.nnz, dtype=torch.uint8, device=dev))

    def encode(self, W, values=None, offsets=None, stream=None):
        """BMWM encode of W [M, N] (cuda, fp32/fp16, unit column stride)."""
        _require_cuda(W)
        ldw = _row_major_ld(W, self.M, self.N, "W")
        if values is None or offsets is None:
            values, offsets = self.empty_format(W.dtype, W.device)
        _require_cuda(values, offsets)
        self._check_values_offsets(values, offsets)
        if values.dtype != W.dtype:
            raise TypeError("values must have W's dtype")
        _check(_lib.darb_encode(self._h, _dtype_code(W), _ptr(W), ldw, _ptr(values),
                                _ptr(offsets), _stream_ptr(stream)), "darb_encode")
        return values, offsets

    def decode(self, values, offsets, out=None, stream=None):
        torch = _torch()
        _require_cuda(values, offsets)
        self._check_values_offsets(values, offsets)
        if out is None:
            out = torch.empty((self.M, self.N), dtype=values.dtype, device=values.device)
        if out.dtype != values.dtype:
            raise TypeError("out must have the values' dtype")
        ldw = _row_major_ld(out, self.M, self.N, "out")
        _check(_lib.darb_decode(self._h, _dtype_code(values), _ptr(values), _ptr(offsets),
                                _ptr(out), ldw, _stream_ptr(stream)), "darb_decode")
        return out

    def spmv(self, values, offsets, x, y=None, stream=None):
        torch = _torch()
        _require_cuda(values, offsets, x)
        self._check_values_offsets(values, offsets)
        y = self._vector_out(x, y)
        _check(_lib.darb_spmv(self._h, _dtype_code(values), _ptr(values), _ptr(offsets),
                              _dtype_code(x), _ptr(x), _ptr(y), _stream_ptr(stream)),
               "darb_spmv")
        return y

    def spmm(self, values, offsets, X, Y=None, stream=None):
        torch = _torch()
        _require_cuda(values, offsets, X)
        self._check_values_offsets(values, offsets)
        B, ldx, Y, ldy = self._matrix_out(X, Y)
        _check(_lib.darb_spmm(self._h, _dtype_code(values), _ptr(values), _ptr(offsets),
                              _dtype_code(X), B, _ptr(X), ldx, _ptr(Y), ldy,
                              _stream_ptr(stream)), "darb_spmm")
        return Y

    # -- bit-packed offsets (section 4.2) ---------------------------------------------
    def empty_packed(self, device=None):
        torch = _torch()
        dev = self.workspace.device if device is None else device
        return torch.empty(max(self.packed_words, 1), dtype=torch.int32, device=dev)

    def pack_offsets(self, offsets, packed=None, stream=None):
        """Byte offsets [nnz] -> packed words (int32 tensor holding the uint32 words)."""
        torch = _torch()
        _require_cuda(offsets)
        _check_format(offsets, self.nnz, "offsets", (torch.uint8,))
        if packed is None:
            packed = self.empty_packed(offsets.device)
        self._check_packed(packed)
        _check(_lib.darb_pack_offsets(self._h, _ptr(offsets), _ptr(packed), _stream_ptr(stream)),
               "darb_pack_offsets")
        return packed

    def unpack_offsets(self, packed, offsets=None, stream=None):
        torch = _torch()
        _require_cuda(packed)
        self._check_packed(packed)
        if offsets is None:
            offsets = torch.empty(self.nnz, dtype=torch.uint8, device=packed.device)
        _check_format(offsets, self.nnz, "offsets", (torch.uint8,))
        _check(_lib.darb_unpack_offsets(self._h, _ptr(packed), _ptr(offsets),
                                        _stream_ptr(stream)), "darb_unpack_offsets")
        return offsets

    def spmv_packed(self, values, packed, x, y=None, stream=None):
        _require_cuda(values, packed, x)
        self._check_values(values)
        self._check_packed(packed)
        y = self._vector_out(x, y)
        _check(_lib.darb_spmv_packed(self._h, _dtype_code(values), _ptr(values), _ptr(packed),
                                     _dtype_code(x), _ptr(x), _ptr(y), _stream_ptr(stream)),
               "darb_spmv_packed")
        return y

    def spmm_packed(self, values, packed, X, Y=None, stream=None):
        _require_cuda(values, packed, X)
        self._check_values(values)
        self._check_packed(packed)
        B, ldx, Y, ldy = self._matrix_out(X, Y)
        _check(_lib.darb_spmm_packed(self._h, _dtype_code(values), _ptr(values), _ptr(packed),
                                     _dtype_code(X), B, _ptr(X), ldx, _ptr(Y), ldy,
                                     _stream_ptr(stream)), "darb_spmm_packed")
        return Y

    # -- INT8 values ------------------------------------------------------------------
    def quantize_i8(self, values, codes=None, scales=None, stream=None):
        """Retained values -> (codes int8 [nnz], scales fp32 [M] by original row).

        Per-row symmetric INT8 (section 4.2 assumes INT8 weights): s_r = max|v| / 127,
        q = rint(v * 127 / max|v|); see darb_quantize_i8 in include/darb.h.
        """
        torch = _torch()
        _require_cuda(values)
        self._check_values(values)
        if codes is None:
            codes = torch.empty(self.nnz, dtype=torch.int8, device=values.device)
        if scales is None:
            scales = torch.empty(self.M, dtype=torch.float32, device=values.device)
        self._check_i8(codes, scales)
        _check(_lib.darb_quantize_i8(self._h, _dtype_code(values), _ptr(values), _ptr(codes),
                                     _ptr(scales), _stream_ptr(stream)), "darb_quantize_i8")
        return codes, scales

    def _i8_offsets(self, offsets, packed):
        if (offsets is None) == (packed is None):
            raise ValueError("pass exactly one of offsets (bytes) and packed (words)")
        if offsets is not None:
            _require_cuda(offsets)
            _check_format(offsets, self.nnz, "offsets", (_torch().uint8,))
            return _ptr(offsets), None
        _require_cuda(packed)
        self._check_packed(packed)
        return None, _ptr(packed)

    def spmv_i8(self, codes, scales, x, offsets=None, packed=None, y=None, stream=None):
        """y = diag(scales) (W_i8 x), offsets as bytes or packed words."""
        _require_cuda(codes, scales, x)
        self._check_i8(codes, scales)
        po, pp = self._i8_offsets(offsets, packed)
        y = self._vector_out(x, y)
        _check(_lib.darb_spmv_i8(self._h, _ptr(codes), _ptr(scales), po, pp, _dtype_code(x),
                                 _ptr(x), _ptr(y), _stream_ptr(stream)), "darb_spmv_i8")
        return y

    def spmm_i8(self, codes, scales, X, offsets=None, packed=None, Y=None, stream=None):
        """Y = diag(scales) (W_i8 X), offsets as bytes or packed words."""
        _require_cuda(codes, scales, X)
        self._check_i8(codes, scales)
        po, pp = self._i8_offsets(offsets, packed)
        B, ldx, Y, ldy = self._matrix_out(X, Y)
        _check(_lib.darb_spmm_i8(self._h, _ptr(codes), _ptr(scales), po, pp, _dtype_code(X), B,
                                 _ptr(X), ldx, _ptr(Y), ldy, _stream_ptr(stream)),
               "darb_spmm_i8")
        return Y

    # -- argument checks --------------------------------------------------------------
    def _check_i8(self, codes, scales):
        torch = _torch()
        _check_format(codes, self.nnz, "codes", (torch.int8,))
        _check_format(scales, self.M, "scales", (torch.float32,))

    def _check_values(self, values):
        torch = _torch()
        _check_format(values, self.nnz, "values", (torch.float32, torch.float16))

    def _check_values_offsets(self, values, offsets):
        torch = _torch()
        self._check_values(values)
        _check_format(offsets, self.nnz, "offsets", (torch.uint8,))

    def _check_packed(self, packed):
        torch = _torch()
        _check_format(packed, self.packed_words, "packed", (torch.int32,))

    def _vector_out(self, x, y):
        torch = _torch()
        if x.dim() != 1 or x.shape[0] != self.N or not x.is_contiguous():
            raise ValueError(f"x must be a contiguous [{self.N}] tensor")
        if y is None:
            y = torch.empty(self.M, dtype=torch.float32, device=x.device)
        _check_format(y, self.M, "y", (torch.float32,))
        return y

    def _matrix_out(self, X, Y):
        torch = _torch()
        if X.dim() != 2 or X.shape[0] != self.N:
            raise ValueError(f"X must be [{self.N}, B]")
        B = X.shape[1]
        ldx = _row_major_ld(X, self.N, B, "X")
        if Y is None:
            Y = torch.empty((self.M, B), dtype=torch.float32, device=X.device)
        if Y.dtype != torch.float32:
            raise TypeError("Y must be fp32")
        ldy = _row_major_ld(Y, self.M, B, "Y")
        return B, ldx, Y, ldy


def prune_counts(W, k: int, counts=None, workspace=None, stream=None):
    """Per-row counts of the k largest-magnitude elements of W (cuda, fp32/fp16).

    The irregular-pruning step DARB starts from (section 3.2), on the device.
    Returns an int64 cuda tensor [M].
    """
    torch = _torch()
    _require_cuda(W)
    if W.dim() != 2:
        raise ValueError("W must be 2-D")
    M, N = W.shape
    ldw = _row_major_ld(W, M, N, "W")
    code = _dtype_code(W)
    need = ctypes.c_int64()
    _check(_lib.darb_prune_workspace(M, N, code, ctypes.byref(need)), "darb_prune_workspace")
    if workspace is None:
        workspace = torch.empty(need.value, dtype=torch.uint8, device=W.device)
    if counts is None:
        counts = torch.empty(M, dtype=torch.int64, device=W.device)
    _check_format(counts, M, "counts", (torch.int64,))
    _check_format(workspace, need.value, "workspace", (torch.uint8,))
    _check(_lib.darb_prune_counts(M, N, code, _ptr(W), ldw, int(k), _ptr(counts), _ptr(workspace),
                                  workspace.numel(), _stream_ptr(stream)), "darb_prune_counts")
    return counts


def lstm_workspace_floats(hidden: int, seq_len: int, batch: int) -> int:
    n = ctypes.c_int64()
    _check(_lib.darb_lstm_workspace(hidden, seq_len, batch, ctypes.byref(n)),
           "darb_lstm_workspace")
    return n.value


def lstm_layer(wih: Tuple[Plan, object, object], whh: Tuple[Plan, object, object], x_seq,
               hidden: int, seq_len: int, batch: int, h=None, c=None, h_seq=None,
               workspace=None, stream=None):
    """One LSTM layer over a sequence with DARB weights (gate order i, f, g, o, no bias).

    ``wih``/``whh`` are (plan, values, offsets); ``x_seq`` is fp32 [I, T*batch].
    Returns (h_seq [H, T*batch], h [H, batch], c [H, batch]).
    """
    torch = _torch()
    H, T, Bt = hidden, seq_len, batch
    dev = x_seq.device
    if h is None:
        h = torch.zeros((H, Bt), dtype=torch.float32, device=dev)
    if c is None:
        c = torch.zeros((H, Bt), dtype=torch.float32, device=dev)
    if h_seq is None:
        h_seq = torch.empty((H, T * Bt), dtype=torch.float32, device=dev)
    need = lstm_workspace_floats(H, T, Bt)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.float32, device=dev)
    for t in (x_seq, h, c, h_seq, workspace):
        if t.dtype != torch.float32 or not t.is_contiguous():
            raise ValueError("LSTM state and sequences must be contiguous fp32")
    if x_seq.shape != (wih[0].N, T * Bt):
        raise ValueError("x_seq must be [I, T*batch]")
    for t, shape in ((h, (H, Bt)), (c, (H, Bt)), (h_seq, (H, T * Bt))):
        if tuple(t.shape) != shape:
            raise ValueError(f"LSTM buffer must be {shape}, got {tuple(t.shape)}")
    for (p, v, o), name in ((wih, "wih"), (whh, "whh")):
        _require_cuda(v, o)
        p._check_values_offsets(v, o)
    _check(_lib.darb_lstm_layer(wih[0].handle, _ptr(wih[1]), _ptr(wih[2]), whh[0].handle,
                                _ptr(whh[1]), _ptr(whh[2]), _dtype_code(wih[1]), H, T, Bt,
                                _ptr(x_seq), _ptr(h_seq), _ptr(h), _ptr(c), _ptr(workspace),
                                workspace.numel(), _stream_ptr(stream)), "darb_lstm_layer")
    return h_seq, h, c


def stream_read(buf, sink, stream=None):
    _check(_lib.darb_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                 _stream_ptr(stream)), "darb_stream_read")


def stream_copy(dst, src, stream=None):
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than src")
    _check(_lib.darb_stream_copy(_ptr(dst), _ptr(src), nbytes, _stream_ptr(stream)),
           "darb_stream_copy")
