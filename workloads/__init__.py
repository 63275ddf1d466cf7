"""Seeded synthetic inputs for the DARB encode and the DARB products.

This module is the only code shared by the CPU oracle and the HIP path.  It
draws dense weight matrices, activations and the irregular-pruning row
densities that DARB starts from, and it contains none of the method's own
arithmetic (no block-size rule, no block-max selection, no product).

The paper evaluates on trained PTB / TIMIT / ImageNet models that are not
available here; the shapes below stand in for them:

* ``lstm_tiny``  W fp32 [1024 x 256]   (4 gates x hidden 256), keep 10 %, b in [4, 32]
* ``lstm_1024``  W fp32 [4096 x 2048]  (LSTM hidden 1024, input+hidden), keep 6 %, b in [4, 64]
* ``gru_1536``   W fp16 [4608 x 3072]  (GRU hidden 1536, 3 gates), keep 5 %, b in [4, 64]
* ``fc_9216``    W fp32 [4096 x 9216]  (AlexNet FC6-shaped head, Laplace weights), keep 4 %, b in [8, 128]
* ``lstm2_seq``  2-layer LSTM, hidden 1024, four fp16 [4096 x 1024] matrices, keep 5 %, b in [4, 64],
  sequence 200, batch 32

Recipe (every config, seed 0 unless told otherwise):

1. ``rng = numpy.random.default_rng(seed)``.
2. Row scales ``s ~ LogNormal(0, sigma)`` (M draws).
3. Weights in fp64: Normal ``w = 0.05 * s_r * z`` with ``z ~ N(0, 1)``, or Laplace
   ``w = 0.01 * s_r * l`` with ``l ~ Laplace(0, 1)``; M*N draws, row-major; then cast to the
   stored dtype with round-to-nearest-even.
4. Activations ``~ N(0, 1)`` in fp64, cast to their dtype, drawn after the weights.
5. Irregular magnitude pruning (paper section 2, "Irregular Pruning"; section 3.1 uses it only to
   obtain a mask and row densities): keep exactly ``k = floor(p*M*N + 0.5)`` weights, the largest
   by magnitude of the *stored* value, ties broken by ascending flat index.  Row density
   ``d_r = count_r / N``; matrix density ``D = k / (M*N)``.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

__all__ = [
    "CONFIGS",
    "Config",
    "MatrixInput",
    "make_matrix",
    "irregular_densities",
    "make_activations",
    "make_config",
    "make_lstm_inputs",
]


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    M: int
    N: int
    wdtype: str          # "f32" | "f16"
    dist: str            # "normal" | "laplace"
    sigma: float         # LogNormal(0, sigma) row-scale spread
    keep: float          # fraction retained by the irregular threshold
    b_min: int
    b_max: int
    batch: int           # batch of the product this config is quoted on (1 = SpMV)
    xdtype: str          # activation dtype
    note: str = ""


CONFIGS: Dict[str, Config] = {
    c.name: c
    for c in [
        Config("lstm_tiny", 1024, 256, "f32", "normal", 0.5, 0.10, 4, 32, 1, "f32",
               "tiny LSTM gate matrix (4 gates x hidden 256), SpMV"),
        Config("lstm_1024", 4096, 2048, "f32", "normal", 0.5, 0.06, 4, 64, 1, "f32",
               "LSTM layer hidden 1024 with input concatenated, encode on device + SpMV"),
        Config("gru_1536", 4608, 3072, "f16", "normal", 0.7, 0.05, 4, 64, 16, "f16",
               "GRU layer hidden 1536, SpMM with fp16 X, fp32 accumulate"),
        Config("fc_9216", 4096, 9216, "f32", "laplace", 0.5, 0.04, 8, 128, 64, "f32",
               "FC head shaped like AlexNet FC6, SpMM B=64 plus SpMV B=1"),
        Config("lstm2_seq", 4096, 1024, "f16", "normal", 0.5, 0.05, 4, 64, 32, "f32",
               "2-layer LSTM hidden 1024, T=200, batch 32; four matrices of this shape"),
    ]
}

LSTM_SEQ = dict(layers=2, hidden=1024, seq_len=200, batch=32)

_NP_DTYPE = {"f32": np.float32, "f16": np.float16}
_KEY_MASK = {"f32": (np.uint32, 0x7FFFFFFF), "f16": (np.uint16, 0x7FFF)}


@dataclasses.dataclass
class MatrixInput:
    """One dense weight matrix plus the irregular-pruning statistics DARB consumes."""

    W: np.ndarray            # [M, N] stored dtype, C-contiguous
    row_density: np.ndarray  # fp64 [M], d_r = count_r / N
    matrix_density: float    # D = k / (M*N)
    mask: np.ndarray         # bool [M, N], the irregular mask (generator output only)
    k: int


def _draw_weights(rng: np.random.Generator, M: int, N: int, dist: str, sigma: float,
                  wdtype: str) -> np.ndarray:
    s = rng.lognormal(0.0, sigma, size=M)
    if dist == "normal":
        z = rng.standard_normal((M, N))
        w = (0.05 * s)[:, None] * z
    elif dist == "laplace":
        z = rng.laplace(0.0, 1.0, size=(M, N))
        w = (0.01 * s)[:, None] * z
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return np.ascontiguousarray(w.astype(_NP_DTYPE[wdtype]))


def irregular_densities(W: np.ndarray, keep: float) -> Tuple[np.ndarray, float, np.ndarray, int]:
    """Exact-k global magnitude mask and its row densities.

    Magnitude is compared on the stored bits with the sign cleared, so the order
    is exactly |w| for finite values and ties (frequent in fp16) are broken by
    ascending flat index.  Returns (row_density fp64[M], D, mask, k).
    """
    M, N = W.shape
    if W.dtype == np.float32:
        ut, m = _KEY_MASK["f32"]
    elif W.dtype == np.float16:
        ut, m = _KEY_MASK["f16"]
    else:
        raise TypeError(f"unsupported weight dtype {W.dtype}")
    size = M * N
    k = int(np.floor(keep * size + 0.5))
    k = max(0, min(k, size))
    keys = (W.reshape(-1).view(ut) & ut(m)).astype(np.int64)
    mask = np.zeros(size, dtype=bool)
    if k > 0:
        t = np.partition(keys, size - k)[size - k]   # k-th largest key
        mask = keys > t
        need = k - int(mask.sum())
        eq = np.flatnonzero(keys == t)[:need]
        mask[eq] = True
    mask = mask.reshape(M, N)
    counts = mask.sum(axis=1).astype(np.int64)
    row_density = counts.astype(np.float64) / float(N)
    D = float(k) / float(size)
    return row_density, D, mask, k


def make_matrix(M: int, N: int, *, wdtype: str = "f32", dist: str = "normal",
                sigma: float = 0.5, keep: float = 0.1, seed: int = 0,
                rng: Optional[np.random.Generator] = None) -> MatrixInput:
    """Draw one weight matrix and its irregular densities (recipe steps 1-3 and 5)."""
    if rng is None:
        rng = np.random.default_rng(seed)
    W = _draw_weights(rng, M, N, dist, sigma, wdtype)
    d, D, mask, k = irregular_densities(W, keep)
    return MatrixInput(W=W, row_density=d, matrix_density=D, mask=mask, k=k)


def make_activations(rng: np.random.Generator, shape, xdtype: str) -> np.ndarray:
    """Activations ~ N(0, 1), cast to ``xdtype`` (recipe step 4)."""
    return np.ascontiguousarray(rng.standard_normal(shape).astype(_NP_DTYPE[xdtype]))


def make_config(name: str, seed: int = 0, batch: Optional[int] = None,
                with_vector: bool = True):
    """Inputs of one named matrix config: (Config, MatrixInput, x [N], X [N, B]).

    X is row-major [N x B] (the B values of one input feature are contiguous),
    which is the layout the products gather from.  ``x`` is the batch-1 vector.
    """
    cfg = CONFIGS[name]
    rng = np.random.default_rng(seed)
    mi = make_matrix(cfg.M, cfg.N, wdtype=cfg.wdtype, dist=cfg.dist, sigma=cfg.sigma,
                     keep=cfg.keep, rng=rng)
    B = cfg.batch if batch is None else batch
    X = make_activations(rng, (cfg.N, B), cfg.xdtype)
    x = make_activations(rng, (cfg.N,), cfg.xdtype) if with_vector else None
    return cfg, mi, x, X


def make_lstm_inputs(seed: int = 0, seq_len: Optional[int] = None,
                     batch: Optional[int] = None, hidden: Optional[int] = None,
                     layers: Optional[int] = None):
    """The recurrent workload: per layer (W_ih, W_hh) and the input sequence.

    Each matrix is [4*hidden x hidden] fp16 (input size = hidden), drawn in the
    order layer-0 W_ih, layer-0 W_hh, layer-1 W_ih, ..., each with its own
    irregular threshold.  The input sequence is fp32, laid out [hidden x (T*batch)]
    with column index t*batch + n, i.e. feature-major so it can be the X operand
    of a product directly.
    """
    cfg = CONFIGS["lstm2_seq"]
    H = LSTM_SEQ["hidden"] if hidden is None else hidden
    T = LSTM_SEQ["seq_len"] if seq_len is None else seq_len
    Bt = LSTM_SEQ["batch"] if batch is None else batch
    L = LSTM_SEQ["layers"] if layers is None else layers
    rng = np.random.default_rng(seed)
    mats: List[Tuple[MatrixInput, MatrixInput]] = []
    for _ in range(L):
        wih = make_matrix(4 * H, H, wdtype=cfg.wdtype, dist=cfg.dist, sigma=cfg.sigma,
                          keep=cfg.keep, rng=rng)
        whh = make_matrix(4 * H, H, wdtype=cfg.wdtype, dist=cfg.dist, sigma=cfg.sigma,
                          keep=cfg.keep, rng=rng)
        mats.append((wih, whh))
    xs = make_activations(rng, (H, T * Bt), "f32")
    return cfg, mats, xs, dict(hidden=H, seq_len=T, batch=Bt, layers=L)
