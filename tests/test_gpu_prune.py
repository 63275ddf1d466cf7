"""GPU parity of the device-side irregular pruning (section 3.2's first step).

The per-row kept counts of the k largest-magnitude elements are integers and
unique (ties go to the lower flat index), so the HIP result must equal the
oracle's exactly.
"""
import ctypes
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


def dev(a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_counts(darb, Wd, k):
    c = darb.prune_counts(Wd, k)
    torch.cuda.synchronize()
    return c.cpu().numpy()


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216", "lstm2_seq"])
def test_config_counts_equal_oracle(darb, name):
    cfg, mi, _, _ = workloads.make_config(name, seed=0)
    say(f"{name}: prune {cfg.M}x{cfg.N} {cfg.wdtype}, k = {mi.k}")
    got = gpu_counts(darb, dev(mi.W), mi.k)
    assert got.sum() == mi.k
    assert np.array_equal(got, oracle.prune_counts(mi.W, mi.k))
    # the plan built on the device counts is the plan of the generator's densities
    a = darb.Plan.from_counts(cfg.N, got, mi.k, darb.ROUND_FLOOR, cfg.b_min, cfg.b_max)
    b = darb.Plan(cfg.M, cfg.N, mi.row_density, mi.matrix_density, darb.ROUND_FLOOR,
                  cfg.b_min, cfg.b_max)
    for x, y in zip(a.export(), b.export()):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("seed", range(4))
def test_random_ties_and_every_k_class(darb, dtype, seed):
    # few distinct magnitudes (heavy ties at the threshold), ragged shapes
    rng = np.random.default_rng(seed)
    M, N = int(rng.integers(1, 90)), int(rng.integers(1, 5000))
    W = (rng.integers(-6, 7, size=(M, N)) * 0.25).astype(dtype)
    W[rng.random((M, N)) < 0.05] = -0.0
    Wd = dev(W)
    size = M * N
    for k in sorted({0, 1, 2, size // 7, size // 2, size - 1, size}):
        if k < 0:
            continue
        say(f"  {dtype.__name__} {M}x{N} k={k}")
        assert np.array_equal(gpu_counts(darb, Wd, k), oracle.prune_counts(W, k)), k


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_continuous_values_many_digits(darb, dtype):
    # distinct magnitudes spread over many exponents: every radix digit matters
    rng = np.random.default_rng(11)
    M, N = 300, 2500
    W = (rng.standard_normal((M, N)) * np.exp(rng.uniform(-8, 4, size=(M, N)))).astype(dtype)
    Wd = dev(W)
    for keep in (0.003, 0.05, 0.5, 0.97):
        k = int(np.floor(keep * M * N + 0.5))
        assert np.array_equal(gpu_counts(darb, Wd, k), oracle.prune_counts(W, k)), keep


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("N", [1, 3, 7, 9, 17])
def test_narrow_rows_many_rows_per_wave(darb, dtype, N):
    # W is split evenly over the waves as padded rows; with narrow rows one wave's
    # range crosses many rows, and rows end inside a 16-byte vector
    rng = np.random.default_rng(100 + N)
    M = 20000 // N + 13
    W = (rng.integers(-40, 41, size=(M, N)) * 0.125).astype(dtype)
    Wd = dev(W)
    size = M * N
    for k in (1, size // 3, size - 5):
        say(f"  {np.dtype(dtype).name} {M}x{N} k={k}")
        assert np.array_equal(gpu_counts(darb, Wd, k), oracle.prune_counts(W, k)), k


def test_special_values(darb):
    W = np.zeros((6, 40), dtype=np.float32)
    W[0, 3], W[1, 0], W[2, 39], W[3, 7] = np.nan, np.inf, -np.inf, 1e-45
    W[4, :] = -0.0
    W[5, 10:20] = 3.0
    for k in range(0, 240, 7):
        assert np.array_equal(gpu_counts(darb, dev(W), k), oracle.prune_counts(W, k)), k


def test_all_equal_takes_flat_order(darb):
    M, N = 37, 1111
    W = np.full((M, N), 0.5, dtype=np.float16)
    for k in (1, N - 1, N, 5 * N + 3, M * N - 2):
        want = np.array([min(N, max(0, k - r * N)) for r in range(M)], dtype=np.int64)
        assert np.array_equal(gpu_counts(darb, dev(W), k), want), k


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_strided_and_misaligned_rows(darb, dtype):
    rng = np.random.default_rng(21)
    M, N = 50, 1500
    W = rng.standard_normal((M, N)).astype(dtype)
    k = 4321
    ref = oracle.prune_counts(W, k)
    # a leading dimension larger than N, and rows starting off a 16-byte boundary
    big = torch.zeros((M, N + 9), dtype=torch.float32 if dtype == np.float32 else torch.float16,
                      device="cuda")
    big[:, 1:N + 1] = dev(W)
    view = big[:, 1:N + 1]
    assert view.stride(0) == N + 9
    assert np.array_equal(gpu_counts(darb, view, k), ref)


def test_repeat_calls_reuse_workspace(darb):
    # a workspace reused across calls holds the previous call's state: results
    # must not depend on it
    rng = np.random.default_rng(3)
    W = rng.standard_normal((64, 777)).astype(np.float32)
    Wd = dev(W)
    nbytes = ctypes.c_int64()
    assert darb.lib().darb_prune_workspace(64, 777, darb.F32, ctypes.byref(nbytes)) == 0
    ws = torch.full((nbytes.value,), 0xAB, dtype=torch.uint8, device="cuda")
    for k in (5000, 17, 5000, 0, 49000):
        c = darb.prune_counts(Wd, k, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(c.cpu().numpy(), oracle.prune_counts(W, k)), k


def test_split_with_a_workspace_that_held_other_data(darb):
    # at the split size the sample's histogram starts as the workspace holds it (the
    # count pass of a call leaves it at zero): a workspace that held other data
    # biases the first call's bracket, which may cost passes over W, never the counts
    rng = np.random.default_rng(21)
    W = rng.standard_normal((4096, 4096)).astype(np.float32)      # 64 MiB of W
    Wd = dev(W)
    nbytes = ctypes.c_int64()
    assert darb.lib().darb_prune_workspace(4096, 4096, darb.F32, ctypes.byref(nbytes)) == 0
    ks = (int(0.1 * W.size), 12345)
    ref = {k: oracle.prune_counts(W, k) for k in ks}
    for fill in (0xAB, 0x00, 0x3F):
        ws = torch.full((nbytes.value,), fill, dtype=torch.uint8, device="cuda")
        for k in ks + ks:                               # each k on a used workspace too
            say(f"split-size workspace filled with {fill:#x}, k = {k}")
            c = darb.prune_counts(Wd, k, workspace=ws)
            torch.cuda.synchronize()
            assert np.array_equal(c.cpu().numpy(), ref[k]), (fill, k)


@pytest.mark.parametrize("name", ["lstm_tiny", "gru_1536"])
def test_whole_pipeline_on_device(darb, name):
    # W -> device pruning counts -> plan -> encode -> bit-packed offsets -> products,
    # against the oracle's own chain (its pruning, plan, encode and packing)
    cfg, mi, x, X = workloads.make_config(name, seed=0)
    say(f"{name}: whole pipeline")
    Wd = dev(mi.W)
    counts = gpu_counts(darb, Wd, mi.k)
    plan = darb.Plan.from_counts(cfg.N, counts, mi.k, darb.ROUND_FLOOR, cfg.b_min,
                                 cfg.b_max).upload()
    values, offsets = plan.encode(Wd)
    packed = plan.pack_offsets(offsets)
    y = plan.spmv_packed(values, packed, dev(x))
    Y = plan.spmm_packed(values, packed, dev(X))
    torch.cuda.synchronize()

    ref_counts = oracle.prune_counts(mi.W, mi.k)
    lay = oracle.plan(cfg.N, ref_counts / cfg.N, mi.k / (cfg.M * cfg.N), oracle.ROUND_FLOOR,
                      cfg.b_min, cfg.b_max)
    vr, orf = oracle.encode(mi.W, lay)
    ut = np.uint32 if mi.W.dtype == np.float32 else np.uint16
    assert np.array_equal(values.cpu().numpy().view(ut), vr.view(ut))
    assert np.array_equal(offsets.cpu().numpy(), orf)
    assert np.array_equal(packed.cpu().numpy()[:plan.packed_words].view(np.uint32),
                          oracle.pack_offsets(orf, lay))
    tol = 1e-5 if mi.W.dtype == np.float32 else 2e-3
    for got, act, what in ((y.cpu().numpy(), x, "spmv"), (Y.cpu().numpy(), X, "spmm")):
        compare(got, oracle.spmm(vr, orf, lay, act), oracle.spmm_absdot(vr, orf, lay, act), tol,
                f"pruned {what}")


@pytest.mark.parametrize("kind", ["normal", "ties"])
def test_fp16_sampled_bracket(darb, kind):
    # 64 MiB of fp16 takes the sample and split path (8-bit first digit): normal
    # values kept at 0.5 % give a one-digit bracket with room for its keys; 61
    # distinct magnitudes kept at 5 % put 1.6 % of W in the threshold's digit, more
    # than half the room, so the split pass takes the exact first digit of W instead
    # and the later passes stream W
    rng = np.random.default_rng(8)
    M, N = 512, 65536
    if kind == "normal":
        W = (rng.standard_normal((M, N)) * 0.7).astype(np.float16)
        k = int(0.005 * M * N)
    else:
        W = (rng.integers(-60, 61, size=(M, N)) * 0.015625).astype(np.float16)
        k = int(0.05 * M * N)
    say(f"fp16 sampled bracket ({kind}): {M}x{N}, k = {k}")
    assert np.array_equal(gpu_counts(darb, dev(W), k), oracle.prune_counts(W, k))


def test_biased_sample_falls_back_to_w(darb):
    # from 64 MiB the first digit's candidates come from a bracket proposed by a
    # sample of W (ranges at a fixed stride); the split pass counts the keys above
    # the bracket, and the threshold must lie between that count and it plus the
    # candidates.  Rows exactly one sample stride long put every
    # sampled range at the same columns (the first 1024, with the library's present
    # sample); values spread over 20 octaves only there make the sample propose a
    # narrow bracket near the top while the true threshold lies in the rest of W,
    # so the check must send the later passes back to W, with the oracle's counts.
    rng = np.random.default_rng(5)
    M, N = 512, 32 * 1024 + 37 * 4
    W = rng.uniform(0.0, 0.5, size=(M, N)).astype(np.float32)
    W[:, :1024] = np.exp2(rng.uniform(0.0, 20.0, size=(M, 1024))).astype(np.float32)
    k = int(0.05 * M * N)
    say(f"biased sample: {M}x{N} fp32, k = {k}")
    assert np.array_equal(gpu_counts(darb, dev(W), k), oracle.prune_counts(W, k))


@pytest.mark.parametrize("case", ["candidates_fit", "candidate_room_overflows",
                                  "workgroup_lds_overflows"])
def test_split_pass_paths(darb, case):
    # after the first digit the pass copies the keys sharing the threshold's first
    # digit (candidates) and later passes read only them; when they do not fit (the
    # workspace's room, M*N/32, or one workgroup's LDS) later passes stream W
    # again.  Both must give the oracle's counts.  (64 MiB of fp32: the smallest W
    # that takes the split pass.)
    rng = np.random.default_rng(31)
    M, N = 256, 65536
    W = rng.uniform(0.0, 0.5, size=(M, N)).astype(np.float32)
    if case == "candidates_fit":
        ties = rng.random((M, N)) < 1.0 / 256           # ~66 k equal keys: fit
    elif case == "candidate_room_overflows":
        ties = rng.random((M, N)) < 1.0 / 16            # ~1 M > the room of 524 k
    else:
        ties = np.zeros((M, N), dtype=bool)
        ties[:2] = True                                 # 131 k ties in two rows: one
    W[ties] = 1.0                                       # workgroup's share > its LDS
    k = int(ties.sum()) // 2 + 7
    say(f"split pass {case}: {int(ties.sum())} keys equal to the threshold, k = {k}")
    assert np.array_equal(gpu_counts(darb, dev(W), k), oracle.prune_counts(W, k))


@pytest.mark.parametrize("keep", [0.10, 0.30])
def test_gaussian_weights_at_split_size(darb, keep):
    # 64 MiB of i.i.d. Gaussian fp32 weights takes the sample and split path.  At
    # 10 % keep the threshold's 11-bit leading digit holds about 3 % of W, more than
    # half the candidate room: the sample's 14-bit bracket is what keeps the
    # candidates few (and at 30 % the density at the threshold is higher still).
    # Which path ran is not visible here; the counts must be the oracle's either way.
    rng = np.random.default_rng(11)
    W = (rng.standard_normal((4096, 4096)) * 0.05).astype(np.float32)
    k = int(keep * W.size)
    say(f"gaussian 4096x4096 fp32, keep {keep}, k = {k}")
    assert np.array_equal(gpu_counts(darb, dev(W), k), oracle.prune_counts(W, k))
