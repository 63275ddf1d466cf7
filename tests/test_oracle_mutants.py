"""Plant mistakes in copies of the oracle and check that the pins catch each one.

Each mutant is a textual change to a copy of oracle/darb_oracle.c (compiled on
the CPU into a temporary library) or of the oracle's Python wrapper, driven
through a fresh copy of that wrapper.  The real oracle must pass ``pin_suite``; every mutant must fail it.
"""
import importlib.util
import os
import shutil
import sys
from fractions import Fraction

import numpy as np
import pytest

import oracle
from tests._brute import block_size_brute, kept_positions, prune_brute

ORACLE_DIR = os.path.dirname(oracle.__file__)

MUTANTS = {
    "tie_goes_to_last": [("if (key > best_key)", "if (key >= best_key)")],
    "sign_not_cleared": [("& 0x7FFFFFFFu;\n            for", "& 0xFFFFFFFFu;\n            for"),
                         ("uint32_t key = row[k * b + j] & 0x7FFFFFFFu",
                          "uint32_t key = row[k * b + j] & 0xFFFFFFFFu")],
    "tail_block_dropped": [("(N + b - 1) / b", "N / b")],
    "rounding_direction_swapped": [("d >= matrix_density", "d < matrix_density")],
    "round_down_off_by_one": [("(f * d == 1.0) ? f : 2.0 * f", "2.0 * f")],
    "gather_index_wrong": [("int64_t c = k * b + offsets[s];", "int64_t c = k + offsets[s];")],
    "product_sign_flipped": [("y[j] += v *", "y[j] -= v *")],
    "bins_in_wrong_order": [("for (int l = 0; l <= 7; ++l)", "for (int l = 7; l >= 0; --l)")],
    "half_exponent_bias": [("e - 25", "e - 24")],
    "pack_bit_order": [("uint32_t v = (offsets[row_start[r] + k] >> t) & 1u;",
                        "uint32_t v = (offsets[row_start[r] + k] >> (l - 1 - t)) & 1u;")],
    "pack_run_length": [("int64_t bit = (j % 32) * l;\n            uint32_t *run = packed + first_word[l] + (j / 32) * l;",
                         "int64_t bit = (j % 16) * l;\n            uint32_t *run = packed + first_word[l] + (j / 16) * l;")],
    "prune_ties_to_high_index": [("return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);",
                                  "return x->idx > y->idx ? -1 : (x->idx < y->idx ? 1 : 0);")],
    "prune_sign_kept": [("key = ((const uint32_t *)W)[r * ldw + c] & 0x7FFFFFFFu;",
                         "key = ((const uint32_t *)W)[r * ldw + c];")],
    "prune_keeps_one_less": [("for (int64_t i = 0; i < k; ++i) counts",
                              "for (int64_t i = 1; i < k; ++i) counts")],
    # the error scale of the product checks, sum_k |v_k * x_k|
    "absdot_fabs_dropped": [("a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));",
                             "a[j] += v * load_elem(xdtype, X, c * ldx + j);")],
    "absdot_term_doubled": [("a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));",
                             "a[j] += 2.0 * fabs(v * load_elem(xdtype, X, c * ldx + j));")],
    "absdot_offset_dropped": [("a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));",
                               "a[j] += fabs(v * load_elem(xdtype, X, (k * b) * ldx + j));")],
    "absdot_batch_column_fixed": [("a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));",
                                   "a[j] += fabs(v * load_elem(xdtype, X, c * ldx));")],
    "absdot_sums_all_columns": [
        ("for (int64_t j = 0; j < B; ++j) a[j] += fabs(v * load_elem(xdtype, X, c * ldx + j));",
         "for (int64_t j = 0; j < B; ++j) for (int64_t i = 0; i < B; ++i) "
         "a[j] += fabs(v * load_elem(xdtype, X, c * ldx + i));")],
    "i8_absdot_scale_dropped": [("py", "return A * (s if A.ndim == 1 else s[:, None])",
                                 "return A")],
    "i8_absdot_scale_signed": [("py", "s = np.abs(np.asarray(scales, dtype=np.float64))",
                                "s = np.asarray(scales, dtype=np.float64)")],
    # INT8 values (edits of the Python wrapper, where that arithmetic lives)
    "i8_round_half_up": [("py", "q = np.rint(row * inv)",
                          "q = np.floor(row * inv + np.float32(0.5))")],
    "i8_scale_128": [("py", "inv = np.float32(c127 / a)", "inv = np.float32(np.float32(128.0) / a)")],
    "i8_matrix_absmax": [("py", "a = np.max(np.abs(row)) if n else np.float32(0.0)",
                          "a = np.max(np.abs(v32))")],
    "i8_scale_inverted": [("py", "scales[r] = np.float32(a / c127)",
                           "scales[r] = np.float32(c127 / a)")],
}


def _load_variant(tmp_path, name, edits):
    """Edits are (old, new) on darb_oracle.c or ("py", old, new) on __init__.py."""
    src = open(os.path.join(ORACLE_DIR, "darb_oracle.c")).read()
    py = open(os.path.join(ORACLE_DIR, "__init__.py")).read()
    for e in edits:
        if e[0] == "py":
            assert e[1] in py, (name, e[1])
            py = py.replace(e[1], e[2])
        else:
            assert e[0] in src, (name, e[0])
            src = src.replace(e[0], e[1])
    d = tmp_path / name
    d.mkdir()
    (d / "darb_oracle.c").write_text(src)
    (d / "__init__.py").write_text(py)
    spec = importlib.util.spec_from_file_location(f"oracle_mutant_{name}", str(d / "__init__.py"))
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod          # dataclasses look their module up here
    spec.loader.exec_module(mod)
    return mod


def pin_suite(orc):
    """A compact run of the pins; raises AssertionError on the first miss."""
    # section 3.2 worked example (paper mode) and the floor rule's closed form
    for D, d, b in [(0.2188, 0.375, 2), (0.2188, 0.1875, 8), (0.2188, 0.25, 4)]:
        assert (1 << int(orc.block_log2(np.array([d]), D, orc.ROUND_PAPER, 1, 128)[0])) == b
    counts = np.arange(0, 257)
    got = orc.block_log2(counts / 256.0, 0.3, orc.ROUND_PAPER, 1, 128)
    for c in counts:
        want = block_size_brute(int(c), 256, Fraction(0.3), "paper", 1, 128)
        assert (1 << int(got[c])) == want
    # Table 7: sum of ceil(1500/b), b = 2..64, is 1478
    assert orc.layout(1500, np.arange(1, 7, dtype=np.uint8)).nnz == 1478
    # rows grouped by block size, smallest first
    assert list(orc.layout(100, np.array([3, 1, 3, 0], dtype=np.uint8)).perm) == [3, 1, 0, 2]
    # BMWM against the brute-force predicate, with ties and negative values
    rng = np.random.default_rng(0)
    for dtype, ut in [(np.float32, np.uint32), (np.float16, np.uint16)]:
        for _ in range(6):
            M, N = int(rng.integers(2, 6)), int(rng.integers(5, 40))
            W = (rng.integers(-3, 4, size=(M, N)) * 0.5).astype(dtype)
            log2b = rng.integers(0, 5, size=M).astype(np.uint8)
            lay = orc.layout(N, log2b)
            v, o = orc.encode(W, lay)
            kept = np.zeros((M, N), dtype=bool)
            for r in range(M):
                b = 1 << int(log2b[r])
                s = int(lay.row_start[r])
                cols = [k * b + int(o[s + k]) for k in range(-(-N // b))]
                assert cols == kept_positions(W[r], b)
                kept[r, cols] = True
            Wm = orc.decode(v, o, lay)
            assert np.array_equal(Wm.view(ut), np.where(kept, W, dtype(0)).view(ut))
            X = rng.standard_normal((N, 3)).astype(np.float32)
            Y = orc.spmm(v, o, lay, X)
            ref = np.where(kept, W, 0).astype(np.float64) @ X.astype(np.float64)
            assert np.allclose(Y, ref, rtol=0, atol=1e-12)
    # packed offsets: the hand example and a round trip through the unmutated reader
    lay = orc.layout(24, np.array([3], dtype=np.uint8))
    assert orc.pack_offsets(np.array([5, 1, 7], dtype=np.uint8), lay).tolist() == [461, 0, 0]
    lay = orc.layout(97, np.array([3, 5, 7, 2], dtype=np.uint8))
    o = np.random.default_rng(1).integers(0, 4, size=lay.nnz).astype(np.uint8)
    assert np.array_equal(oracle.unpack_offsets(orc.pack_offsets(o, lay), lay), o)
    # irregular pruning counts against brute force, ties and negative values included
    for dtype in (np.float32, np.float16):
        W = (rng.integers(-3, 4, size=(4, 9)) * 0.5).astype(dtype)
        for k in (0, 1, 5, 17, 36):
            assert orc.prune_counts(W, k).tolist() == prune_brute(W, k), (dtype, k)
    # INT8 values: the hand example (ties to even, per-row scale, zero row)
    lay = orc.layout(8, np.array([1, 2, 3], dtype=np.uint8))
    vals = np.zeros(lay.nnz, dtype=np.float32)
    for r, row in enumerate([[127.0, 2.5, -3.5, 0.5], [-2.0, 1.0], [0.0]]):
        vals[int(lay.row_start[r]):int(lay.row_start[r]) + len(row)] = row
    q, s = orc.quantize_i8(vals, lay)
    assert [q[int(lay.row_start[r]):int(lay.row_start[r]) + int(lay.nblk[r])].tolist()
            for r in range(3)] == [[127, 2, -4, 0], [-127, 64], [0]]
    assert s.tolist() == [1.0, float(np.float32(2.0) / np.float32(127.0)), 0.0]
    # the products' error scale against a library matmul of the magnitudes, and its
    # INT8 form with scales of either sign
    lay = orc.layout(37, np.array([0, 2, 5, 3, 7], dtype=np.uint8))
    W = rng.standard_normal((5, 37)).astype(np.float32)
    v, o = orc.encode(W, lay)
    Wa = np.abs(orc.decode(v, o, lay).astype(np.float64))
    for B in (1, 3):
        X = rng.standard_normal((37, B)).astype(np.float32)
        act = X[:, 0].copy() if B == 1 else X
        assert np.allclose(orc.spmm_absdot(v, o, lay, act), Wa @ np.abs(act.astype(np.float64)),
                           rtol=1e-14, atol=0)
        q = rng.integers(-127, 128, size=lay.nnz).astype(np.int8)
        sc = np.array([0.5, -2.0, 0.0, 1.5, -0.25], dtype=np.float32)
        ref = np.abs(orc.decode(q.astype(np.float32), o, lay).astype(np.float64)) @ \
            np.abs(act.astype(np.float64))
        ref = ref * (np.abs(sc) if B == 1 else np.abs(sc)[:, None])
        assert np.allclose(orc.spmm_i8_absdot(q, sc, o, lay, act), ref, rtol=1e-14, atol=0)
    # fp16 decoding of a few bit patterns against numpy
    for bits in [0x3C00, 0x0001, 0x7BFF, 0xC000, 0x0400]:
        assert orc.half_to_double(bits) == float(np.array([bits], np.uint16).view(np.float16)[0])


def test_real_oracle_passes_pin_suite():
    pin_suite(oracle)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(tmp_path, name):
    mod = _load_variant(tmp_path, name, MUTANTS[name])
    with pytest.raises((AssertionError, ValueError)):
        pin_suite(mod)
