"""Brute-force restatements of DARB's definitions, for tiny inputs only.

These are written from the definitions, not from the oracle's loops, so that
the oracle can be pinned to something other than itself:

* block sizes are chosen by enumerating power-of-two fractions with exact
  rational arithmetic (``fractions.Fraction``);
* the kept weight of a block is found with a per-element predicate on Python
  float magnitudes ("no element of the block is larger, and no earlier element
  is as large"), not with a running argmax over integer keys;
* the irregular top-K mask ranks every element with Python's sort on
  (magnitude key descending, flat index ascending) and counts the first K.
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


def prune_brute(W, k):
    """Brute force: rank every element by (magnitude bits desc, flat index asc)."""
    ut = np.uint32 if W.dtype == np.float32 else np.uint16
    mag = 0x7FFFFFFF if W.dtype == np.float32 else 0x7FFF
    keys = [int(b) & mag for b in W.reshape(-1).view(ut)]
    order = sorted(range(len(keys)), key=lambda i: (-keys[i], i))
    counts = [0] * W.shape[0]
    for i in order[:k]:
        counts[i // W.shape[1]] += 1
    return counts
