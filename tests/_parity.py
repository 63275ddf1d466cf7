"""The product tolerance check shared by the GPU parity tests.

Per output, |y - y64| / sum_k |v_k * x_k| must stay within the tolerance (1e-5
for fp32 and INT8 weights, 2e-3 for fp16 weights); an output whose terms are all
zero must be exactly zero.  y64 is the oracle's fp64 product and the
denominator, the oracle's error scale, is the scale of a dot product's rounding
error.  The normwise error max |y - y64| / max |y64| is printed beside it.
"""
import sys

import numpy as np


def compare(Y, ref, scale, tol, label=""):
    """Assert the componentwise bound; print both error measures; return the worst
    componentwise error."""
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.asarray(scale, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64).reshape(ref.shape)
    assert scale.shape == ref.shape, label
    err = np.abs(Y - ref)
    zero = scale == 0
    assert np.all(Y[zero] == 0.0), f"{label}: nonzero output where every term is 0"
    rel = err[~zero] / scale[~zero]
    worst = float(rel.max()) if rel.size else 0.0
    peak = float(np.abs(ref).max()) if ref.size else 0.0
    normwise = float(err.max()) / peak if peak > 0 else float(err.max() if err.size else 0.0)
    print(f"  {label}: max rel err {worst:.3e} (tol {tol:.0e}), "
          f"normwise {normwise:.3e}", flush=True, file=sys.stderr)
    assert worst <= tol, label
    return worst
