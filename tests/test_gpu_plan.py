"""The plan built on the device from kept counts (section 3.2: block sizes from the
irregular mask's row densities) against the oracle's layout and the host-built plan:
block sizes, first slots and storage order bit for bit, in both rounding modes, on the
workloads' matrices and on random densities; and the all-device path W -> pruning
counts -> plan -> encode -> products with no host copy of the counts."""
import sys

import numpy as np
import pytest

import oracle
import workloads
from tests._parity import compare

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def darb():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_1911_08020_amd as d
    return d


def check_plan(darb, counts, N, kept, mode, bmin, bmax, label):
    M = counts.shape[0]
    say(f"device plan: {label} M={M} N={N} kept={kept} mode={mode} b {bmin}..{bmax}")
    dp = darb.Plan.from_device_counts(N, torch.from_numpy(counts).cuda(), kept, mode, bmin, bmax)
    hp = darb.Plan.from_counts(N, counts, kept, mode, bmin, bmax)
    lay = oracle.layout(N, oracle.block_log2(counts / N, kept / (M * N), mode, bmin, bmax))
    l2, rs, pm = dp.export()
    assert np.array_equal(l2, lay.log2b), label
    assert np.array_equal(rs, lay.row_start), label
    assert np.array_equal(pm, lay.perm), label
    assert (dp.nnz, dp.packed_words, dp.bins) == (hp.nnz, hp.packed_words, hp.bins), label
    assert dp.nnz == lay.nnz
    return dp, hp, lay


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216", "lstm2_seq"])
@pytest.mark.parametrize("mode", [0, 1])
def test_device_plan_on_workloads(darb, name, mode):
    if name == "lstm2_seq":
        cfg, mats, _, _ = workloads.make_lstm_inputs(seed=0)
        mi = mats[0][1]
    else:
        cfg, mi, _, _ = workloads.make_config(name, seed=0)
    counts = mi.mask.sum(axis=1).astype(np.int64)
    check_plan(darb, counts, mi.W.shape[1], mi.k, mode, cfg.b_min, cfg.b_max, name)


@pytest.mark.parametrize("seed", range(6))
def test_device_plan_on_random_densities(darb, seed):
    rng = np.random.default_rng(100 + seed)
    for mode in (0, 1):
        M = int(rng.integers(1, 5000))
        N = int(rng.integers(1, 3000))
        counts = rng.integers(0, N + 1, size=M).astype(np.int64)
        counts[rng.random(M) < 0.1] = 0
        counts[rng.random(M) < 0.05] = N
        lo = int(rng.integers(0, 8))
        bmin, bmax = 1 << lo, 1 << int(rng.integers(lo, 8))
        kept = int(rng.integers(0, M * N + 1))
        check_plan(darb, counts, N, kept, mode, bmin, bmax, f"random seed {seed}")


def test_device_plan_rows_across_workgroups(darb):
    # more rows than one workgroup of the build takes (1024), every group present
    N = 1000
    M = 3 * 1024 + 17
    counts = (np.arange(M) * 7919 % (N + 1)).astype(np.int64)
    check_plan(darb, counts, N, int(counts.sum()), 1, 1, 128, "multi-workgroup")


def test_all_device_path(darb):
    """W -> device pruning counts -> device plan -> encode -> SpMV / SpMM: the counts never
    leave the device; every result equals the oracle's."""
    cfg, mi, x, X = workloads.make_config("fc_9216", seed=0, batch=64)
    W = torch.from_numpy(mi.W).cuda()
    counts = darb.prune_counts(W, mi.k)
    plan = darb.Plan.from_device_counts(cfg.N, counts, mi.k, darb.ROUND_FLOOR, cfg.b_min,
                                        cfg.b_max)
    v, o = plan.encode(W)
    y = plan.spmv(v, o, torch.from_numpy(x).cuda())
    Y = plan.spmm(v, o, torch.from_numpy(X).cuda())
    torch.cuda.synchronize()
    lay = oracle.plan(cfg.N, mi.row_density, mi.matrix_density, oracle.ROUND_FLOOR, cfg.b_min,
                      cfg.b_max)
    vr, orf = oracle.encode(mi.W, lay)
    assert np.array_equal(o.cpu().numpy(), orf)
    assert np.array_equal(v.cpu().numpy().view(np.uint32), vr.view(np.uint32))
    compare(y.cpu().numpy(), oracle.spmm(vr, orf, lay, x), oracle.spmm_absdot(vr, orf, lay, x),
            1e-5, "all-device spmv")
    compare(Y.cpu().numpy(), oracle.spmm(vr, orf, lay, X), oracle.spmm_absdot(vr, orf, lay, X),
            1e-5, "all-device spmm")
