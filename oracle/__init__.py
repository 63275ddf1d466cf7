"""DARB CPU oracle -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it; the only module both sides use is ``workloads`` (the
seeded input generator).

The arithmetic lives in ``darb_oracle.c`` (plain C, fp64 products); this file
only marshals numpy arrays.  The recurrent workload's gate math is plain numpy
in fp64 (``lstm_forward``).  Functions and the paper passages they follow:

* ``block_log2``   -- section 3.2, block size from row density (both rounding modes)
* ``layout``       -- section 3.2 (power-of-two density groups make storage regular),
                      section 4.2 / Table 7 (ceil(N/b) blocks per row)
* ``encode``       -- section 3.1, block-max weight masking, per row with its own b
* ``decode``       -- the masked dense matrix the format stands for
* ``spmm``         -- section 2 / 3.2, product over retained weights, offsets select activations
* ``pack_offsets``  -- section 4.2, log2(b)-bit indices (and ``unpack_offsets``)
* ``quantize_i8``  -- section 4.2's storage accounting (INT8 weights): per-row
                      symmetric codes and scales (``spmm_i8`` is their product)
* ``prune_counts`` -- section 3.2's first step (irregular top-K magnitude pruning,
                      section 2), per-row kept counts that give the row densities
* ``dense_masked_product`` -- the plain definition of the product: a dense fp64 matmul
* ``lstm_forward`` -- the LSTM recurrence of the recurrent workload on the decoded
                      masked matrices (dense fp64 products)
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "darb_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

ROUND_FLOOR = 0
ROUND_PAPER = 1
_DT = {np.dtype(np.float32): 0, np.dtype(np.float16): 1}
_BITS = {np.dtype(np.float32): np.uint32, np.dtype(np.float16): np.uint16}

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with the host C compiler (gcc, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH) or \
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared",
                               "-fno-fast-math", "-ffp-contract=off",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build(force=False)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I = ctypes.c_int
    lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_double.restype = ctypes.c_double
    lib.oracle_block_log2.argtypes = [I64, P, ctypes.c_double, I, I, I, P]
    lib.oracle_block_log2.restype = I
    lib.oracle_layout.argtypes = [I64, I64, P, P, P]
    lib.oracle_layout.restype = I64
    lib.oracle_encode_f32.argtypes = [I64, I64, P, I64, P, P, P, P]
    lib.oracle_encode_f32.restype = None
    lib.oracle_encode_f16.argtypes = [I64, I64, P, I64, P, P, P, P]
    lib.oracle_encode_f16.restype = None
    lib.oracle_decode.argtypes = [I64, I64, I, P, P, P, P, P, I64]
    lib.oracle_decode.restype = I
    lib.oracle_spmm_f64.argtypes = [I64, I64, I, P, P, P, P, I, P, I64, I64, P, I64]
    lib.oracle_spmm_f64.restype = I
    lib.oracle_spmm_absdot_f64.argtypes = [I64, I64, I, P, P, P, P, I, P, I64, I64, P, I64]
    lib.oracle_spmm_absdot_f64.restype = I
    lib.oracle_packed_layout.argtypes = [I64, I64, P, P]
    lib.oracle_packed_layout.restype = I64
    lib.oracle_pack_offsets.argtypes = [I64, I64, P, P, P, P]
    lib.oracle_pack_offsets.restype = None
    lib.oracle_unpack_offsets.argtypes = [I64, I64, P, P, P, P]
    lib.oracle_unpack_offsets.restype = None
    lib.oracle_prune_counts.argtypes = [I64, I64, I, P, I64, I64, P]
    lib.oracle_prune_counts.restype = I
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def half_to_double(bits: int) -> float:
    return _load().oracle_half_to_double(int(bits))


def block_log2(row_density, matrix_density: float, mode: int, b_min: int, b_max: int) -> np.ndarray:
    """log2 of each row's block size (section 3.2).  Raises ValueError on bad input."""
    d = np.ascontiguousarray(row_density, dtype=np.float64)
    out = np.zeros(d.shape[0], dtype=np.uint8)
    rc = _load().oracle_block_log2(d.shape[0], _ptr(d), float(matrix_density), int(mode),
                                   int(b_min), int(b_max), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_block_log2 rejected its arguments")
    return out


@dataclasses.dataclass
class Layout:
    M: int
    N: int
    log2b: np.ndarray      # uint8 [M]
    perm: np.ndarray       # int32 [M]: original row stored i-th
    row_start: np.ndarray  # int64 [M]: first slot of each original row
    nnz: int

    @property
    def nblk(self) -> np.ndarray:
        b = np.left_shift(1, self.log2b.astype(np.int64))
        return (self.N + b - 1) // b


def layout(N: int, log2b: np.ndarray) -> Layout:
    lb = np.ascontiguousarray(log2b, dtype=np.uint8)
    M = lb.shape[0]
    perm = np.zeros(M, dtype=np.int32)
    row_start = np.zeros(M, dtype=np.int64)
    nnz = _load().oracle_layout(M, int(N), _ptr(lb), _ptr(perm), _ptr(row_start))
    if nnz < 0:
        raise ValueError("oracle_layout rejected its arguments")
    return Layout(M, int(N), lb, perm, row_start, int(nnz))


def plan(N: int, row_density, matrix_density: float, mode: int, b_min: int, b_max: int) -> Layout:
    return layout(N, block_log2(row_density, matrix_density, mode, b_min, b_max))


def encode(W: np.ndarray, lay: Layout):
    """BMWM with per-row block sizes (section 3.1 / 3.2) -> (values, offsets)."""
    W = np.asarray(W)
    if W.dtype not in _BITS:
        raise TypeError(f"unsupported dtype {W.dtype}")
    if W.ndim != 2 or W.shape[0] != lay.M or W.shape[1] < lay.N:
        raise ValueError("W shape does not match the layout")
    if W.strides[1] != W.itemsize:
        W = np.ascontiguousarray(W)
    ldw = W.strides[0] // W.itemsize
    bits = W.view(_BITS[W.dtype])
    values = np.zeros(lay.nnz, dtype=W.dtype)
    offsets = np.zeros(lay.nnz, dtype=np.uint8)
    fn = _load().oracle_encode_f32 if W.dtype == np.float32 else _load().oracle_encode_f16
    fn(lay.M, lay.N, _ptr(bits), ldw, _ptr(lay.log2b), _ptr(lay.row_start), _ptr(values),
       _ptr(offsets))
    return values, offsets


def _at(a: np.ndarray, first: int):
    """Pointer to element `first` along a's first axis (C-contiguous arrays)."""
    return ctypes.c_void_p(a.ctypes.data + int(first) * a.strides[0])


def encode_rows(W: np.ndarray, lay: Layout, r0: int, r1: int, values: np.ndarray,
                offsets: np.ndarray) -> None:
    """encode() restricted to the original rows [r0, r1), writing their slots of the
    caller's values / offsets (the same arithmetic; only the row range is narrowed,
    so several calls on disjoint ranges can run on separate threads)."""
    W = np.ascontiguousarray(W)
    bits = W.view(_BITS[W.dtype])
    fn = _load().oracle_encode_f32 if W.dtype == np.float32 else _load().oracle_encode_f16
    fn(r1 - r0, lay.N, _at(bits, r0), bits.shape[1], _at(lay.log2b, r0), _at(lay.row_start, r0),
       _ptr(values), _ptr(offsets))


def spmm_rows(values: np.ndarray, offsets: np.ndarray, lay: Layout, X: np.ndarray, r0: int,
              r1: int, Y: np.ndarray) -> None:
    """spmm() restricted to the original rows [r0, r1), written to those rows of the
    caller's fp64 Y [M, B] (same arithmetic; for running row ranges on threads)."""
    X2 = _as_2d(X)
    B = X2.shape[1]
    rc = _load().oracle_spmm_f64(r1 - r0, lay.N, _DT[values.dtype], _ptr(values), _ptr(offsets),
                                 _at(lay.log2b, r0), _at(lay.row_start, r0), _DT[X2.dtype],
                                 _ptr(X2), B, B, _at(Y, r0), B)
    if rc != 0:
        raise ValueError("malformed DARB format (offset outside its block or row)")


def decode(values: np.ndarray, offsets: np.ndarray, lay: Layout) -> np.ndarray:
    values = np.ascontiguousarray(values)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint8)
    out = np.empty((lay.M, lay.N), dtype=values.dtype)
    rc = _load().oracle_decode(lay.M, lay.N, values.itemsize, _ptr(values), _ptr(offsets),
                               _ptr(lay.log2b), _ptr(lay.row_start), _ptr(out), lay.N)
    if rc != 0:
        raise ValueError("malformed DARB format (offset outside its block or row)")
    return out


def _as_2d(X: np.ndarray) -> np.ndarray:
    X = np.ascontiguousarray(X)
    return X.reshape(X.shape[0], 1) if X.ndim == 1 else X


def spmm(values: np.ndarray, offsets: np.ndarray, lay: Layout, X: np.ndarray) -> np.ndarray:
    """fp64 Y = W_darb X in the format's own order (retained weights only)."""
    values = np.ascontiguousarray(values)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint8)
    vec = np.asarray(X).ndim == 1
    X2 = _as_2d(X)
    if X2.dtype not in _DT or values.dtype not in _DT:
        raise TypeError("values and X must be fp32 or fp16")
    if X2.shape[0] != lay.N:
        raise ValueError("X must have N rows")
    B = X2.shape[1]
    Y = np.zeros((lay.M, B), dtype=np.float64)
    rc = _load().oracle_spmm_f64(lay.M, lay.N, _DT[values.dtype], _ptr(values), _ptr(offsets),
                                 _ptr(lay.log2b), _ptr(lay.row_start), _DT[X2.dtype], _ptr(X2),
                                 B, B, _ptr(Y), B)
    if rc != 0:
        raise ValueError("malformed DARB format (offset outside its block or row)")
    return Y[:, 0] if vec else Y


def spmm_absdot(values: np.ndarray, offsets: np.ndarray, lay: Layout, X: np.ndarray) -> np.ndarray:
    """fp64 sum_k |v * x| per output: the scale of a dot product's rounding error."""
    values = np.ascontiguousarray(values)
    offsets = np.ascontiguousarray(offsets, dtype=np.uint8)
    vec = np.asarray(X).ndim == 1
    X2 = _as_2d(X)
    B = X2.shape[1]
    A = np.zeros((lay.M, B), dtype=np.float64)
    rc = _load().oracle_spmm_absdot_f64(lay.M, lay.N, _DT[values.dtype], _ptr(values),
                                        _ptr(offsets), _ptr(lay.log2b), _ptr(lay.row_start),
                                        _DT[X2.dtype], _ptr(X2), B, B, _ptr(A), B)
    if rc != 0:
        raise ValueError("malformed DARB format")
    return A[:, 0] if vec else A


def packed_layout(lay: Layout):
    """(total 32-bit words, first word of each block-size group l = 0..7)."""
    first = np.zeros(8, dtype=np.int64)
    words = _load().oracle_packed_layout(lay.M, lay.N, _ptr(lay.log2b), _ptr(first))
    return int(words), first


def pack_offsets(offsets: np.ndarray, lay: Layout) -> np.ndarray:
    """Offsets as log2(b)-bit fields in 32-slot runs of l words per group (section 4.2)."""
    offsets = np.ascontiguousarray(offsets, dtype=np.uint8)
    words, _ = packed_layout(lay)
    out = np.zeros(max(words, 1), dtype=np.uint32)
    _load().oracle_pack_offsets(lay.M, lay.N, _ptr(lay.log2b), _ptr(lay.row_start),
                                _ptr(offsets), _ptr(out))
    return out[:words]


def unpack_offsets(packed: np.ndarray, lay: Layout) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint32)
    if packed.size == 0:
        packed = np.zeros(1, dtype=np.uint32)
    out = np.zeros(lay.nnz, dtype=np.uint8)
    _load().oracle_unpack_offsets(lay.M, lay.N, _ptr(lay.log2b), _ptr(lay.row_start),
                                  _ptr(packed), _ptr(out))
    return out


def prune_counts(W: np.ndarray, k: int) -> np.ndarray:
    """Per-row counts of the k largest-magnitude elements of W (sections 2 and 3.2).

    Magnitude is the stored bits with the sign cleared; equal magnitudes go to the
    lower flat index.  Returns int64 [M].
    """
    W = np.asarray(W)
    if W.ndim != 2 or W.dtype not in _DT:
        raise TypeError("W must be a 2-D fp32 or fp16 array")
    M, N = W.shape
    Wc = np.ascontiguousarray(W)
    counts = np.zeros(M, dtype=np.int64)
    rc = _load().oracle_prune_counts(M, N, _DT[W.dtype], _ptr(Wc), N, int(k), _ptr(counts))
    if rc != 0:
        raise ValueError("invalid pruning arguments")
    return counts


# Rows whose largest retained magnitude is below this quantise to zero: 127 / absmax
# must stay finite in fp32.
I8_MIN_ABSMAX = np.float32(2.0 ** -120)


def quantize_i8(values: np.ndarray, lay: Layout):
    """INT8 retained weights (section 4.2's storage accounting assumes INT8 weights).

    Reading of the paper, which does not fix the scheme: symmetric, one scale per
    row over the row's retained weights.  With a = max |v| over the row (fp32),
    inv = 127 / a and every code is q = rint(v * inv) (round half to even), clamped to
    [-127, 127]; the row's scale is s = a / 127 so that v ~ s * q.  Every operation
    is a single correctly rounded fp32 operation, in this order.  Rows with
    a < 2^-120 (all zero, or so small that 127 / a would overflow) get s = 0 and
    q = 0.  Values must be finite.

    Returns (codes int8 [nnz] in the format's slot order, scales float32 [M] by
    original row).
    """
    v32 = np.ascontiguousarray(values).astype(np.float32)   # fp16 -> fp32 is exact
    if not np.all(np.isfinite(v32)):
        raise ValueError("INT8 quantisation needs finite values")
    codes = np.zeros(lay.nnz, dtype=np.int8)
    scales = np.zeros(lay.M, dtype=np.float32)
    nblk = lay.nblk
    c127 = np.float32(127.0)
    for r in range(lay.M):
        s0, n = int(lay.row_start[r]), int(nblk[r])
        row = v32[s0:s0 + n]
        a = np.max(np.abs(row)) if n else np.float32(0.0)
        if not a >= I8_MIN_ABSMAX:
            continue
        inv = np.float32(c127 / a)
        q = np.rint(row * inv)                                # fp32 product, half to even
        codes[s0:s0 + n] = np.clip(q, -127, 127).astype(np.int8)
        scales[r] = np.float32(a / c127)
    return codes, scales


def spmm_i8(codes: np.ndarray, scales: np.ndarray, offsets: np.ndarray, lay: Layout,
            X: np.ndarray) -> np.ndarray:
    """fp64 product of the INT8 format: y[r] = s_r * sum_k q[r,k] * x[k*b_r + off]."""
    q = np.ascontiguousarray(codes, dtype=np.int8).astype(np.float32)   # exact
    Y = spmm(q, offsets, lay, X)
    s = np.asarray(scales, dtype=np.float64)
    return Y * (s if Y.ndim == 1 else s[:, None])


def spmm_i8_absdot(codes: np.ndarray, scales: np.ndarray, offsets: np.ndarray, lay: Layout,
                   X: np.ndarray) -> np.ndarray:
    """fp64 |s_r| * sum_k |q * x|: the rounding-error scale of the INT8 product."""
    q = np.ascontiguousarray(codes, dtype=np.int8).astype(np.float32)
    A = spmm_absdot(q, offsets, lay, X)
    s = np.abs(np.asarray(scales, dtype=np.float64))
    return A * (s if A.ndim == 1 else s[:, None])


def dense_masked_product(Wm: np.ndarray, X: np.ndarray) -> np.ndarray:
    """The plain definition of the product: dense fp64 matmul of the masked matrix."""
    return np.asarray(Wm, dtype=np.float64) @ np.asarray(X, dtype=np.float64)


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def lstm_forward(masked_layers, xs: np.ndarray, hidden: int, seq_len: int, batch: int):
    """Multi-layer LSTM without bias, gate order (i, f, g, o), all in fp64.

    ``masked_layers`` is a list of (Wm_ih, Wm_hh): the decoded masked dense
    matrices, [4*hidden x in] and [4*hidden x hidden].  ``xs`` is
    [in x (T*batch)] with column t*batch + n.  Returns the last layer's h for
    every step, [hidden x (T*batch)], and the final (h, c) of every layer.
    """
    H, T, Bt = hidden, seq_len, batch
    inp = np.asarray(xs, dtype=np.float64)
    finals = []
    out = None
    for (wih, whh) in masked_layers:
        wih = np.asarray(wih, dtype=np.float64)
        whh = np.asarray(whh, dtype=np.float64)
        U = wih @ inp                                       # input products of all steps
        h = np.zeros((H, Bt), dtype=np.float64)
        c = np.zeros((H, Bt), dtype=np.float64)
        out = np.zeros((H, T * Bt), dtype=np.float64)
        for t in range(T):
            g = U[:, t * Bt:(t + 1) * Bt] + whh @ h
            i = _sigmoid(g[0:H])
            f = _sigmoid(g[H:2 * H])
            gg = np.tanh(g[2 * H:3 * H])
            o = _sigmoid(g[3 * H:4 * H])
            c = f * c + i * gg
            h = o * np.tanh(c)
            out[:, t * Bt:(t + 1) * Bt] = h
        finals.append((h, c))
        inp = out
    return out, finals
