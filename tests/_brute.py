"""Brute-force restatements of DARB's definitions, for tiny inputs only.

These are written from the definitions, not from the oracle's loops, so that
the oracle can be pinned to something other than itself:

* block sizes are chosen by enumerating power-of-two fractions with exact
  rational arithmetic (``fractions.Fraction``);
* the kept weight of a block is found with a per-element predicate on Python
  float magnitudes ("no element of the block is larger, and no earlier element
  is as large"), not with a running argmax over integer keys.
"""
from fractions import Fraction

import numpy as np


def block_size_brute(count: int, N: int, D: Fraction, mode: str, b_min: int, b_max: int) -> int:
    """Block size of a row holding ``count`` irregular survivors out of N.

    mode "floor": the row density is always rounded up to a power-of-two
    fraction; mode "paper": rounded up when d >= D, down when d < D.
    """
    d = Fraction(count, N)
    cands = [1 << e for e in range(0, 64)]
    if d == 0:
        b = b_max
    else:
        up = max(b for b in cands if Fraction(1, b) >= d)           # smallest fraction >= d
        if mode == "floor" or d >= D:
            b = up
        else:
            b = min(b for b in cands if Fraction(1, b) <= d)        # largest fraction <= d
    return min(max(b, b_min), b_max)


def kept_positions(row: np.ndarray, b: int):
    """Columns kept by block-max masking of one row (floats, no NaN)."""
    N = row.shape[0]
    mags = [abs(float(v)) for v in row]
    kept = []
    for c in range(N):
        k = c // b
        block = range(k * b, min(k * b + b, N))
        larger = any(mags[o] > mags[c] for o in block)
        earlier_equal = any(mags[o] == mags[c] for o in block if o < c)
        if not larger and not earlier_equal:
            kept.append(c)
    return kept


def encode_brute(W: np.ndarray, block_sizes):
    """Per row: list of (column, value bits) kept, in column order."""
    out = []
    for r in range(W.shape[0]):
        cols = kept_positions(W[r], int(block_sizes[r]))
        out.append(cols)
    return out
