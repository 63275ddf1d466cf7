"""The seeded input generator: exact-k irregular threshold, determinism, Table 1."""
import os

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_exact_k_and_densities():
    mi = workloads.make_matrix(300, 170, keep=0.07, seed=3)
    k = int(np.floor(0.07 * 300 * 170 + 0.5))
    assert mi.k == k and mi.mask.sum() == k
    assert np.array_equal(mi.row_density, mi.mask.sum(1) / 170.0)
    assert mi.matrix_density == k / (300 * 170)
    # every kept magnitude is >= every dropped magnitude
    a = np.abs(mi.W.astype(np.float64))
    assert a[mi.mask].min() >= a[~mi.mask].max()


def test_fp16_ties_broken_by_flat_index():
    W = np.array([[1, 2, 2, 3], [2, 2, 1, 0]], dtype=np.float16)
    d, D, mask, k = workloads.irregular_densities(W, 0.5)      # k = 4
    assert k == 4
    # 3 wins, then the first three 2's in flat order
    assert mask.tolist() == [[False, True, True, True], [True, False, False, False]]
    assert list(d) == [0.75, 0.25]


def test_generator_is_deterministic():
    a = workloads.make_matrix(64, 40, wdtype="f16", keep=0.1, seed=9)
    b = workloads.make_matrix(64, 40, wdtype="f16", keep=0.1, seed=9)
    assert np.array_equal(a.W.view(np.uint16), b.W.view(np.uint16))
    assert np.array_equal(a.row_density, b.row_density)


def test_table1_block_occupancy_with_uniform_row_scale():
    """Section 3.1, Table 1: after 90 % irregular pruning, size-10 blocks hold 0 / 1 / >1
    survivors about 34.9 / 38.7 / 26.4 % of the time.  With one row scale (sigma = 0) the
    generator's mask is a uniformly random exact-k subset, which reproduces the table."""
    mi = workloads.make_matrix(650, 6500, dist="normal", sigma=0.0, keep=0.10, seed=0)
    occ = mi.mask.reshape(650, 650, 10).sum(-1).ravel()
    got = 100.0 * np.array([(occ == 0).mean(), (occ == 1).mean(), (occ > 1).mean()])
    with open(os.path.join(GOLDEN, "table1_block_occupancy.txt")) as f:
        rows = [ln.split() for ln in f if ln.strip() and not ln.startswith("#")]
    for name, z, one, more in rows:
        want = np.array([float(z), float(one), float(more)])
        assert np.all(np.abs(got - want) < 0.5), (name, got, want)


def test_config_table():
    c = workloads.CONFIGS
    assert (c["fc_9216"].M, c["fc_9216"].N, c["fc_9216"].b_max) == (4096, 9216, 128)
    assert c["gru_1536"].wdtype == "f16" and c["gru_1536"].batch == 16
    assert c["lstm_tiny"].keep == 0.10
