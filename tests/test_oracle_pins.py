"""Pins for the CPU oracle: worked examples, closed forms, brute force, invariants.

Nothing here needs a GPU.  Every check compares the oracle with something other
than the oracle itself: numbers the paper states (tests/golden/), exact
rational brute force, numpy library routines, or algebraic invariants.
"""
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from tests._brute import block_size_brute, encode_brute, kept_positions, prune_brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]


# ----------------------------------------------------------------------------------
# block-size rule (section 3.2)
# ----------------------------------------------------------------------------------

def test_block_size_worked_example_paper_mode():
    for D, d, b in _rows("block_size_worked_example.txt"):
        got = oracle.block_log2(np.array([float(d)]), float(D), oracle.ROUND_PAPER, 1, 128)
        assert (1 << int(got[0])) == int(b), (D, d, b)


def test_worked_example_differs_between_modes():
    # floor mode always rounds the density up: 0.1875 -> 0.25 -> block size 4
    got = oracle.block_log2(np.array([0.1875]), 0.2188, oracle.ROUND_FLOOR, 1, 128)
    assert (1 << int(got[0])) == 4


@pytest.mark.parametrize("N", [256, 1500, 3072, 9216, 1000, 7])
def test_floor_rule_exhaustive_counts(N):
    """Floor mode equals 'largest 2^k with 2^k * count <= N' for every count."""
    counts = np.arange(N + 1)
    d = counts / float(N)
    got = oracle.block_log2(d, 0.5, oracle.ROUND_FLOOR, 1, 128)
    for c in range(N + 1):
        if c == 0:
            want = 128
        else:
            want = 1
            while 2 * want * c <= N:
                want *= 2
            want = min(want, 128)
        assert (1 << int(got[c])) == want, (N, c)


@pytest.mark.parametrize("N", [256, 1500, 2048, 9216])
@pytest.mark.parametrize("bounds", [(1, 128), (4, 32), (8, 128), (4, 64)])
def test_paper_rule_vs_rational_brute_force(N, bounds):
    b_min, b_max = bounds
    rng = np.random.default_rng(N + b_min)
    counts = np.unique(np.concatenate([np.arange(0, 40), rng.integers(0, N + 1, 400),
                                       [N, N // 2, N // 4, N // 8, N // 3]]))
    k_total = int(counts.sum())
    D = k_total / float(N * counts.size)
    Dexact = Fraction(D)          # the rule compares against the fp64 value it is given
    d = counts / float(N)
    for mode, name in [(oracle.ROUND_PAPER, "paper"), (oracle.ROUND_FLOOR, "floor")]:
        got = oracle.block_log2(d, D, mode, b_min, b_max)
        for i, c in enumerate(counts):
            want = block_size_brute(int(c), N, Dexact, name, b_min, b_max)
            assert (1 << int(got[i])) == want, (name, N, c, bounds)


def test_row_density_equal_to_matrix_density_rounds_up():
    # reading: a row exactly at the matrix density is treated like a denser row
    got = oracle.block_log2(np.array([0.3]), 0.3, oracle.ROUND_PAPER, 1, 128)
    assert (1 << int(got[0])) == 2   # 0.3 -> up to 0.5
    got = oracle.block_log2(np.array([0.3]), 0.30000001, oracle.ROUND_PAPER, 1, 128)
    assert (1 << int(got[0])) == 4   # 0.3 -> down to 0.25


def test_empty_and_full_rows_and_clamp():
    got = oracle.block_log2(np.array([0.0, 1.0, 0.9, 1e-300]), 0.1, oracle.ROUND_PAPER, 4, 64)
    assert [1 << int(v) for v in got] == [64, 4, 4, 64]


@pytest.mark.parametrize("bad", [
    dict(d=[float("nan")]), dict(d=[-0.1]), dict(d=[1.5]), dict(b_min=3), dict(b_max=256),
    dict(b_min=64, b_max=8), dict(mode=7), dict(D=float("nan")),
])
def test_block_rule_rejects_bad_arguments(bad):
    args = dict(d=[0.1], D=0.1, mode=0, b_min=4, b_max=64)
    args.update(bad)
    with pytest.raises(ValueError):
        oracle.block_log2(np.array(args["d"]), args["D"], args["mode"], args["b_min"], args["b_max"])


# ----------------------------------------------------------------------------------
# layout and block counts (section 3.2, section 4.2 / Table 7)
# ----------------------------------------------------------------------------------

def test_table7_decoding_total_pins_tail_block():
    (n, bs, total), = _rows("decoding_table7.txt")
    bs = [int(b) for b in bs.split(",")]
    log2b = np.array([int(np.log2(b)) for b in bs], dtype=np.uint8)
    lay = oracle.layout(int(n), log2b)
    assert lay.nnz == int(total)


def test_stated_block_counts():
    for n, b, blocks in _rows("bmwm_block_counts.txt"):
        n, b, blocks = int(n), int(b), int(blocks)
        # one kept weight per block: a row of n elements keeps exactly n/b weights
        row = np.random.default_rng(1).standard_normal(n).astype(np.float32)
        assert len(kept_positions(row, b)) == blocks
        if b & (b - 1) == 0:
            lay = oracle.layout(n, np.array([int(np.log2(b))], dtype=np.uint8))
            assert lay.nnz == blocks


def test_layout_groups_rows_by_block_size():
    log2b = np.array([3, 1, 3, 0, 7, 1, 2], dtype=np.uint8)
    N = 100
    lay = oracle.layout(N, log2b)
    assert list(lay.perm) == [3, 1, 5, 6, 0, 2, 4]
    nblk = [(N + (1 << l) - 1) >> l for l in log2b]
    pos = 0
    for r in lay.perm:
        assert lay.row_start[r] == pos
        pos += nblk[r]
    assert lay.nnz == pos == sum(nblk)


# ----------------------------------------------------------------------------------
# BMWM (section 3.1) against brute force and library special cases
# ----------------------------------------------------------------------------------

def _tiny_matrix(rng, M, N, dtype):
    # small integers make equal magnitudes (ties) and signed zeros frequent
    vals = rng.integers(-3, 4, size=(M, N)).astype(np.float64)
    vals *= rng.choice([1.0, 0.5, 0.25], size=(M, N))
    W = vals.astype(dtype)
    negz = rng.random((M, N)) < 0.1
    W[negz] = -0.0
    return W


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_bmwm_vs_brute_force(dtype):
    rng = np.random.default_rng(11)
    for trial in range(40):
        M = int(rng.integers(1, 9))
        N = int(rng.integers(1, 41))
        W = _tiny_matrix(rng, M, N, dtype)
        log2b = rng.integers(0, 6, size=M).astype(np.uint8)
        lay = oracle.layout(N, log2b)
        values, offsets = oracle.encode(W, lay)
        ref = encode_brute(W, [1 << int(l) for l in log2b])
        for r in range(M):
            b = 1 << int(log2b[r])
            s = int(lay.row_start[r])
            cols = [k * b + int(offsets[s + k]) for k in range(int(lay.nblk[r]))]
            assert cols == ref[r], (trial, r)
            got_bits = values[s:s + len(cols)].view(np.uint32 if dtype == np.float32 else np.uint16)
            want_bits = W[r, cols].view(got_bits.dtype)
            assert np.array_equal(got_bits, want_bits)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("b", [1, 2, 4])
def test_bmwm_exhaustive_tie_patterns(dtype, b):
    alphabet = np.array([-2.0, -1.0, -0.0, 0.0, 1.0, 2.0], dtype=dtype)
    grid = np.stack(np.meshgrid(*([np.arange(6)] * b), indexing="ij"), -1).reshape(-1, b)
    W = alphabet[grid]                              # every pattern is one row of one block
    lay = oracle.layout(b, np.full(W.shape[0], int(np.log2(b)), dtype=np.uint8))
    values, offsets = oracle.encode(W, lay)
    for r in range(W.shape[0]):
        assert kept_positions(W[r], b) == [int(offsets[lay.row_start[r]])]


def test_bmwm_special_values_fp32():
    f = np.float32
    den = np.array([1e-45, 3e-45], dtype=f)     # denormals
    row = np.array([0.0, -0.0, den[0], -den[1], np.inf, -np.inf, 1.0, 2.0], dtype=f)
    lay = oracle.layout(8, np.array([1], dtype=np.uint8))   # blocks of 2
    values, offsets = oracle.encode(row[None, :], lay)
    assert list(offsets) == [0, 1, 0, 1]                     # +0 vs -0 tie -> first
    assert values.view(np.uint32)[1] == row[3:4].view(np.uint32)[0]   # sign kept
    assert np.isinf(values[2]) and values[2] > 0


def test_bmwm_nan_outranks_inf_by_bits():
    # reading: the magnitude key is the sign-cleared bit pattern, so NaN beats inf
    row = np.array([np.inf, np.nan, 1.0, 2.0], dtype=np.float32)
    lay = oracle.layout(4, np.array([2], dtype=np.uint8))
    values, offsets = oracle.encode(row[None, :], lay)
    assert int(offsets[0]) == 1 and np.isnan(values[0])


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_block_wider_than_row_is_numpy_argmax(dtype):
    rng = np.random.default_rng(5)
    W = rng.standard_normal((64, 37)).astype(dtype)
    W[::7, 3] = W[::7, 11]                       # some exact ties
    lay = oracle.layout(37, np.full(64, 6, dtype=np.uint8))   # b = 64 > N
    values, offsets = oracle.encode(W, lay)
    assert lay.nnz == 64
    want = np.argmax(np.abs(W.astype(np.float64)), axis=1)    # first occurrence
    assert np.array_equal(offsets.astype(np.int64), want)


def test_block_size_one_is_identity():
    W = np.random.default_rng(3).standard_normal((5, 13)).astype(np.float32)
    lay = oracle.layout(13, np.zeros(5, dtype=np.uint8))
    values, offsets = oracle.encode(W, lay)
    assert not offsets.any()
    assert np.array_equal(values.reshape(5, 13), W)


def test_half_conversion_all_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


# ----------------------------------------------------------------------------------
# format invariants
# ----------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_format_invariants_and_roundtrip(dtype):
    rng = np.random.default_rng(21)
    M, N = 37, 203                                  # N not a multiple of any b > 1
    W = rng.standard_normal((M, N)).astype(dtype)
    W[rng.random((M, N)) < 0.05] = -0.0
    log2b = rng.integers(0, 8, size=M).astype(np.uint8)
    lay = oracle.layout(N, log2b)
    values, offsets = oracle.encode(W, lay)
    kept = np.zeros((M, N), dtype=bool)
    for r in range(M):
        b = 1 << int(log2b[r])
        nb = int(lay.nblk[r])
        assert nb == -(-N // b)
        s = int(lay.row_start[r])
        offs = offsets[s:s + nb].astype(np.int64)
        assert (offs < b).all()
        cols = np.arange(nb) * b + offs
        assert (cols < N).all()
        kept[r, cols] = True
        # exactly one kept weight per block
        assert np.array_equal(np.bincount(cols // b, minlength=nb), np.ones(nb))
    Wm = oracle.decode(values, offsets, lay)
    ut = np.uint32 if dtype == np.float32 else np.uint16
    want = np.where(kept, W, dtype(0.0))
    assert np.array_equal(Wm.view(ut), want.view(ut))        # +0.0 where not kept


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_negation_and_power_of_two_scaling_equivariance(dtype):
    rng = np.random.default_rng(8)
    W = rng.standard_normal((20, 70)).astype(dtype)
    lay = oracle.layout(70, rng.integers(0, 7, size=20).astype(np.uint8))
    v, o = oracle.encode(W, lay)
    vn, on = oracle.encode(-W, lay)
    v2, o2 = oracle.encode(W * dtype(2.0), lay)
    assert np.array_equal(o, on) and np.array_equal(o, o2)
    assert np.array_equal(vn, -v) and np.array_equal(v2, v * dtype(2.0))


# ----------------------------------------------------------------------------------
# products (sections 2 / 3.2): equal to the dense masked product
# ----------------------------------------------------------------------------------

@pytest.mark.parametrize("wdt,xdt", [(np.float32, np.float32), (np.float16, np.float16),
                                     (np.float16, np.float32)])
def test_product_equals_dense_masked_matmul(wdt, xdt):
    rng = np.random.default_rng(4)
    M, N, B = 50, 300, 7
    W = rng.standard_normal((M, N)).astype(wdt)
    lay = oracle.layout(N, rng.integers(0, 8, size=M).astype(np.uint8))
    v, o = oracle.encode(W, lay)
    X = rng.standard_normal((N, B)).astype(xdt)
    Y = oracle.spmm(v, o, lay, X)
    ref = oracle.dense_masked_product(oracle.decode(v, o, lay), X)
    scale = oracle.spmm_absdot(v, o, lay, X)
    assert np.all(np.abs(Y - ref) <= 1e-14 * scale + 1e-300)
    y = oracle.spmm(v, o, lay, X[:, 0].copy())
    assert np.array_equal(y, Y[:, 0])


# The error scale every product parity check divides by, sum_k |v_k * x_k| per
# output, is pinned against a library matmul of the magnitudes: |decode(W)| @ |X|
# has exactly the same terms (the masked matrix is zero off the kept columns).

def _random_format(rng, wdt, M, N):
    """A format over every block size 1..128 (rows cycle through them, N ragged)."""
    W = rng.standard_normal((M, N)).astype(wdt)
    W[rng.random((M, N)) < 0.05] = 0                    # exact zeros, both signs kept
    log2b = (np.arange(M) % 8).astype(np.uint8)
    rng.shuffle(log2b)
    lay = oracle.layout(N, log2b)
    v, o = oracle.encode(W, lay)
    return lay, v, o


@pytest.mark.parametrize("wdt,xdt", [(np.float32, np.float32), (np.float16, np.float16),
                                     (np.float16, np.float32), (np.float32, np.float16)])
@pytest.mark.parametrize("B", [1, 6])
def test_error_scale_equals_abs_matmul(wdt, xdt, B):
    rng = np.random.default_rng(21 + B)
    for M, N in [(16, 300), (11, 1), (24, 129), (9, 1000)]:
        lay, v, o = _random_format(rng, wdt, M, N)
        X = rng.standard_normal((N, B)).astype(xdt)
        X[rng.random((N, B)) < 0.05] = 0
        act = X[:, 0].copy() if B == 1 else X
        A = oracle.spmm_absdot(v, o, lay, act)
        ref = np.abs(oracle.decode(v, o, lay).astype(np.float64)) @ \
            np.abs(act.astype(np.float64))
        assert A.shape == ref.shape == ((M,) if B == 1 else (M, B))
        assert np.array_equal(A == 0, ref == 0)
        assert np.all(np.abs(A - ref) <= 1e-14 * ref), (M, N)


def test_error_scale_is_abs_of_product_when_terms_share_sign():
    """With W >= 0 and X >= 0 no term cancels: the scale equals the product itself,
    and with mixed signs it bounds the product's magnitude."""
    rng = np.random.default_rng(23)
    lay, v, o = _random_format(rng, np.float32, 20, 257)
    X = rng.standard_normal((257, 4)).astype(np.float32)
    A = oracle.spmm_absdot(v, o, lay, X)
    assert np.all(np.abs(oracle.spmm(v, o, lay, X)) <= A * (1 + 1e-14))
    vp, Xp = np.abs(v), np.abs(X)
    assert np.allclose(oracle.spmm_absdot(vp, o, lay, Xp), oracle.spmm(vp, o, lay, Xp),
                       rtol=1e-14, atol=0)


def test_int8_error_scale_equals_abs_matmul():
    """|s_r| * (|Dq| @ |X|), Dq the decoded matrix of the codes; scales of either sign."""
    rng = np.random.default_rng(25)
    for B in (1, 5):
        lay, v, o = _random_format(rng, np.float32, 18, 333)
        q = rng.integers(-127, 128, size=lay.nnz).astype(np.int8)
        s = rng.standard_normal(lay.M).astype(np.float32)
        s[::5] = 0
        X = rng.standard_normal((lay.N, B)).astype(np.float32)
        act = X[:, 0].copy() if B == 1 else X
        A = oracle.spmm_i8_absdot(q, s, o, lay, act)
        Dq = oracle.decode(q.astype(np.float32), o, lay).astype(np.float64)
        ref = np.abs(Dq) @ np.abs(act.astype(np.float64))
        ref = ref * (np.abs(s.astype(np.float64)) if B == 1 else
                     np.abs(s.astype(np.float64))[:, None])
        assert A.shape == ref.shape
        assert np.all(np.abs(A - ref) <= 1e-14 * ref)
        assert np.all(A[s == 0] == 0)


def test_product_with_unit_vector_returns_masked_column():
    rng = np.random.default_rng(6)
    M, N = 30, 90
    W = rng.standard_normal((M, N)).astype(np.float32)
    lay = oracle.layout(N, rng.integers(0, 6, size=M).astype(np.uint8))
    v, o = oracle.encode(W, lay)
    Wm = oracle.decode(v, o, lay)
    for c in [0, 1, 45, 89]:
        e = np.zeros(N, dtype=np.float32)
        e[c] = 1.0
        assert np.array_equal(oracle.spmm(v, o, lay, e), Wm[:, c].astype(np.float64))


def test_block_size_one_product_is_dense_gemv():
    rng = np.random.default_rng(7)
    W = rng.standard_normal((16, 40)).astype(np.float32)
    x = rng.standard_normal(40).astype(np.float32)
    lay = oracle.layout(40, np.zeros(16, dtype=np.uint8))
    v, o = oracle.encode(W, lay)
    y = oracle.spmm(v, o, lay, x)
    assert np.allclose(y, W.astype(np.float64) @ x.astype(np.float64), rtol=0, atol=1e-13)


def test_malformed_offsets_are_rejected():
    lay = oracle.layout(10, np.array([2], dtype=np.uint8))    # b = 4, 3 blocks, tail of 2
    v = np.ones(3, dtype=np.float32)
    o = np.array([0, 1, 3], dtype=np.uint8)                    # 8 + 3 = 11 >= 10
    with pytest.raises(ValueError):
        oracle.decode(v, o, lay)
    with pytest.raises(ValueError):
        oracle.spmm(v, o, lay, np.ones(10, dtype=np.float32))


# ----------------------------------------------------------------------------------
# the recurrent workload's LSTM against torch.nn.LSTM (library routine)
# ----------------------------------------------------------------------------------

def test_lstm_forward_matches_torch_lstm():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(9)
    H, T, Bt, L = 8, 5, 3, 2
    masked = []
    for _ in range(L):
        pair = []
        for _ in range(2):
            W = (0.3 * rng.standard_normal((4 * H, H))).astype(np.float16)
            lay = oracle.layout(H, rng.integers(0, 3, size=4 * H).astype(np.uint8))
            v, o = oracle.encode(W, lay)
            pair.append(oracle.decode(v, o, lay).astype(np.float64))
        masked.append(tuple(pair))
    xs = rng.standard_normal((H, T * Bt)).astype(np.float32)
    out, finals = oracle.lstm_forward(masked, xs, H, T, Bt)
    lstm = torch.nn.LSTM(H, H, num_layers=L, bias=False).double()
    with torch.no_grad():
        for l in range(L):
            getattr(lstm, f"weight_ih_l{l}").copy_(torch.from_numpy(masked[l][0]))
            getattr(lstm, f"weight_hh_l{l}").copy_(torch.from_numpy(masked[l][1]))
        seq = torch.from_numpy(xs.astype(np.float64)).reshape(H, T, Bt).permute(1, 2, 0)
        ref, (hn, cn) = lstm(seq)
    ref = ref.permute(2, 0, 1).reshape(H, T * Bt).numpy()
    assert np.allclose(out, ref, rtol=0, atol=1e-12)
    for l in range(L):
        assert np.allclose(finals[l][1], cn[l].numpy().T, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------------
# bit-packed offsets (section 4.2: log2(b) bits per index)
# ----------------------------------------------------------------------------------

def test_packed_offsets_hand_example():
    # one row of 24 columns, b = 8 (3 bits per index): offsets 5, 1, 7 become the bit
    # string 101 100 111 (LSB first per field) = 5 + (1 << 3) + (7 << 6) in word 0 of
    # the group's first run, which is 3 words long
    lay = oracle.layout(24, np.array([3], dtype=np.uint8))
    packed = oracle.pack_offsets(np.array([5, 1, 7], dtype=np.uint8), lay)
    assert packed.tolist() == [5 + (1 << 3) + (7 << 6), 0, 0]


def test_packed_offsets_word_counts_and_bits_per_index():
    N = 300
    log2b = np.array([0, 1, 2, 3, 4, 5, 6, 7, 3, 3], dtype=np.uint8)
    lay = oracle.layout(N, log2b)
    words, first = oracle.packed_layout(lay)
    want = 0
    for l in range(8):
        slots = int((log2b == l).sum()) * -(-N // (1 << l))
        assert first[l] == want
        want += -(-slots // 32) * l          # runs of 32 slots, l words each
    assert words == want


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_packed_offsets_round_trip(seed):
    rng = np.random.default_rng(seed)
    M, N = int(rng.integers(1, 60)), int(rng.integers(1, 700))
    log2b = rng.integers(0, 8, size=M).astype(np.uint8)
    lay = oracle.layout(N, log2b)
    W = rng.standard_normal((M, N)).astype(np.float32)
    v, o = oracle.encode(W, lay)
    packed = oracle.pack_offsets(o, lay)
    assert np.array_equal(oracle.unpack_offsets(packed, lay), o)
    # each index occupies exactly log2 b bits: count the set bits both ways
    ones = sum(bin(int(w)).count("1") for w in packed)
    assert ones == sum(bin(int(x)).count("1") for x in o)


# ----------------------------------------------------------------------------------
# irregular top-K magnitude pruning: per-row kept counts (sections 2 and 3.2)
# ----------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_prune_counts_brute_force(dtype, seed):
    rng = np.random.default_rng(seed)
    M, N = int(rng.integers(1, 9)), int(rng.integers(1, 13))
    # few distinct magnitudes with both signs: many ties, +0 / -0 among them
    W = (rng.integers(-3, 4, size=(M, N)) * 0.5).astype(dtype)
    W[rng.random((M, N)) < 0.1] = -0.0
    for k in range(0, M * N + 1):
        assert oracle.prune_counts(W, k).tolist() == prune_brute(W, k), k


def test_prune_counts_special_values():
    W = np.array([[np.inf, 1.0, np.nan], [-np.inf, -0.0, 0.0]], dtype=np.float32)
    # key order: NaN (0x7FC00000) > +inf == -inf > 1.0 > +0 == -0
    assert oracle.prune_counts(W, 1).tolist() == [1, 0]          # the NaN
    assert oracle.prune_counts(W, 2).tolist() == [2, 0]          # + inf at column 0
    assert oracle.prune_counts(W, 3).tolist() == [2, 1]          # - inf
    assert oracle.prune_counts(W, 4).tolist() == [3, 1]          # 1.0
    assert oracle.prune_counts(W, 5).tolist() == [3, 2]          # -0 before +0 (lower index)


def test_prune_counts_all_ties_take_flat_order():
    M, N = 5, 7
    W = np.full((M, N), -2.5, dtype=np.float16)
    for k in (0, 1, 6, 7, 8, 20, 35):
        want = [min(N, max(0, k - r * N)) for r in range(M)]
        assert oracle.prune_counts(W, k).tolist() == want


def test_prune_counts_invariants_and_generator_agreement():
    # distinct magnitudes: the kept set is the k largest |w|, whatever the tie rule
    rng = np.random.default_rng(9)
    W = rng.standard_normal((64, 300)).astype(np.float32)
    k = 1920
    c = oracle.prune_counts(W, k)
    assert c.sum() == k and (c >= 0).all() and (c <= 300).all()
    thr = np.sort(np.abs(W).reshape(-1))[-k]
    assert np.array_equal(c, (np.abs(W) >= thr).sum(axis=1))
    # the input generator's own exact-k selection (np.partition) agrees on a workload
    mi = workloads.make_matrix(256, 512, wdtype="f16", dist="normal", sigma=0.7, keep=0.05,
                               seed=3)
    assert np.array_equal(oracle.prune_counts(mi.W, mi.k), mi.mask.sum(axis=1))


# --------------------------------------------------------------------------------
# INT8 values (section 4.2's storage accounting assumes INT8 weights; the scheme is
# the reading documented on oracle.quantize_i8)
# --------------------------------------------------------------------------------

def _rows_to_slots(lay, rows):
    """values in slot order from a list of per-original-row value lists."""
    vals = np.zeros(lay.nnz, dtype=np.float32)
    for r, row in enumerate(rows):
        s = int(lay.row_start[r])
        vals[s:s + len(row)] = row
    return vals


def test_int8_hand_example():
    # row 0 (b = 2, four blocks): absmax 127, so 127 / a = 1 and the codes are rint of
    # the values: 2.5 -> 2 and -3.5 -> -4 (ties to even), 0.5 -> 0; scale 1.
    # row 1 (b = 4, two blocks): absmax 2, 127 / 2 = 63.5 exactly: -2 -> -127,
    # 1 -> 63.5 -> 64 (even); scale 2 / 127.  row 2: all zero -> scale 0, codes 0.
    lay = oracle.layout(8, np.array([1, 2, 3], dtype=np.uint8))
    vals = _rows_to_slots(lay, [[127.0, 2.5, -3.5, 0.5], [-2.0, 1.0], [0.0]])
    q, s = oracle.quantize_i8(vals, lay)
    got = [q[int(lay.row_start[r]):int(lay.row_start[r]) + int(lay.nblk[r])].tolist()
           for r in range(3)]
    assert got == [[127, 2, -4, 0], [-127, 64], [0]]
    assert s.dtype == np.float32
    assert s[0] == np.float32(1.0) and s[1] == np.float32(2.0) / np.float32(127.0) and s[2] == 0


def test_int8_small_absmax_threshold():
    # one row of two blocks (b = 1): absmax exactly 2^-120 still quantises (127 / a
    # is finite), half of it does not
    lay = oracle.layout(2, np.array([0], dtype=np.uint8))
    t = float(oracle.I8_MIN_ABSMAX)
    q, s = oracle.quantize_i8(np.array([t, -t / 2], dtype=np.float32), lay)
    assert q.tolist() == [127, -64] and s[0] > 0        # -63.5 -> -64 (ties to even)
    q, s = oracle.quantize_i8(np.array([t / 2, 0.0], dtype=np.float32), lay)
    assert q.tolist() == [0, 0] and s.tolist() == [0.0]
    with pytest.raises(ValueError):
        oracle.quantize_i8(np.array([np.inf, 1.0], dtype=np.float32), lay)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_int8_invariants_and_error_bound(dtype):
    rng = np.random.default_rng(5)
    M, N = 40, 300
    W = (rng.standard_normal((M, N)) * np.exp(rng.uniform(-6, 3, size=(M, 1)))).astype(dtype)
    lay = oracle.layout(N, rng.integers(0, 7, size=M).astype(np.uint8))
    vals, _ = oracle.encode(W, lay)
    q, s = oracle.quantize_i8(vals, lay)
    v = vals.astype(np.float64)
    for r in range(M):
        sl = slice(int(lay.row_start[r]), int(lay.row_start[r]) + int(lay.nblk[r]))
        qa = np.abs(q[sl].astype(np.int64))
        assert qa.max() == 127                                    # the largest maps to 127
        # round to nearest: |s q - v| <= s / 2, up to the two fp32 roundings of s and v*inv
        err = np.abs(float(s[r]) * q[sl].astype(np.float64) - v[sl])
        assert (err <= float(s[r]) * (0.5 + 1e-5) + 1e-30).all()
    # fp16 values quantise exactly as the same values widened to fp32
    if dtype == np.float16:
        q2, s2 = oracle.quantize_i8(vals.astype(np.float32), lay)
        assert np.array_equal(q, q2) and np.array_equal(s, s2)


def test_int8_product_is_dequantised_masked_column():
    # y = W_i8 e_c picks column c of the dequantised masked matrix s_r * q
    rng = np.random.default_rng(8)
    M, N = 12, 40
    W = rng.standard_normal((M, N)).astype(np.float32)
    lay = oracle.layout(N, rng.integers(0, 4, size=M).astype(np.uint8))
    vals, offs = oracle.encode(W, lay)
    q, s = oracle.quantize_i8(vals, lay)
    Dq = oracle.decode(q.astype(np.float32), offs, lay).astype(np.float64) * \
        s.astype(np.float64)[:, None]
    for c in range(N):
        e = np.zeros(N, dtype=np.float32)
        e[c] = 1.0
        assert np.array_equal(oracle.spmm_i8(q, s, offs, lay, e), Dq[:, c])
    X = rng.standard_normal((N, 3)).astype(np.float32)
    assert np.allclose(oracle.spmm_i8(q, s, offs, lay, X), Dq @ X.astype(np.float64),
                       rtol=0, atol=1e-12)
