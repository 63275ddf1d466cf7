"""The C-ABI library on the host: symbols, plan vs oracle, argument errors.

No kernel runs here: the plan is host code, and every device entry point is
called only in ways that must fail before touching the GPU (plan not uploaded,
NULL buffers, bad sizes).
"""
import ctypes
import functools
import os
import re

import numpy as np
import pytest

import oracle
import paper_1911_08020_amd as darb
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    src = open(os.path.join(ROOT, "include", "darb.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(darb_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    declared = _declared_symbols()
    assert len(declared) >= 15
    lib = ctypes.CDLL(darb.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(darb.EXPORTED) == declared


def test_binding_and_oracle_are_separate():
    # the product binding never loads the oracle's library or package
    src = open(darb.__file__).read()
    assert "oracle" not in src.replace("DarbError", "")
    for f in os.listdir(os.path.join(ROOT, "paper_1911_08020_amd", "csrc")):
        assert "oracle" not in open(os.path.join(ROOT, "paper_1911_08020_amd", "csrc", f)).read()


def _plan_matches_oracle(M, N, d, D, mode, bmin, bmax):
    p = darb.Plan(M, N, d, D, mode, bmin, bmax)
    lay = oracle.plan(N, d, D, mode, bmin, bmax)
    log2b, row_start, perm = p.export()
    assert p.nnz == lay.nnz
    assert np.array_equal(log2b, lay.log2b)
    assert np.array_equal(row_start, lay.row_start)
    assert np.array_equal(perm, lay.perm)
    # the group table describes the same layout
    for b in p.bins:
        rows = perm[b["first_row"]:b["first_row"] + b["rows"]]
        assert (log2b[rows] == b["log2b"]).all()
        assert row_start[rows[0]] == b["first_elem"]
        assert b["nblk"] == -(-N // (1 << b["log2b"]))
    # the bit-packed offsets take the oracle's word count and group starts
    words, first = oracle.packed_layout(lay)
    assert p.packed_words == words
    for b in p.bins:
        assert b["first_word"] == first[b["log2b"]]
    return p


@functools.lru_cache(maxsize=None)
def _config_densities(name):
    cfg = workloads.CONFIGS[name]
    mi = workloads.make_matrix(cfg.M, cfg.N, wdtype=cfg.wdtype, dist=cfg.dist, sigma=cfg.sigma,
                               keep=cfg.keep, seed=0)
    return mi.row_density, mi.matrix_density


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216", "lstm2_seq"])
@pytest.mark.parametrize("mode", [darb.ROUND_FLOOR, darb.ROUND_PAPER])
def test_plan_equals_oracle_on_configs(name, mode):
    cfg = workloads.CONFIGS[name]
    d, D = _config_densities(name)
    _plan_matches_oracle(cfg.M, cfg.N, d, D, mode, cfg.b_min, cfg.b_max)


def test_plan_random_densities_and_bounds():
    rng = np.random.default_rng(2)
    for trial in range(30):
        M = int(rng.integers(1, 300))
        N = int(rng.integers(1, 5000))
        counts = rng.integers(0, N + 1, size=M)
        counts[rng.random(M) < 0.2] = 0
        d = counts / float(N)
        D = float(rng.random())
        bmin = 1 << int(rng.integers(0, 8))
        bmax = 1 << int(rng.integers(int(np.log2(bmin)), 8))
        for mode in (darb.ROUND_FLOOR, darb.ROUND_PAPER):
            _plan_matches_oracle(M, N, d, D, mode, bmin, bmax)


def test_plan_packed_words_table7():
    # one row per block size 2 ... 64 over 1500 columns (Table 7's decoders): the
    # offsets take sum_b ceil(ceil(1500 / b) / 32) * log2 b words
    p = darb.Plan(6, 1500, np.array([0.5, 0.25, 0.125, 1 / 16, 1 / 32, 1 / 64]), 0.1,
                  darb.ROUND_FLOOR, 1, 128)
    want = sum(-(-(-(-1500 // b)) // 32) * l for l, b in enumerate([2, 4, 8, 16, 32, 64], 1))
    assert p.packed_words == want == 24 + 24 + 18 + 12 + 10 + 6


def test_plan_from_counts_equals_plan_from_densities():
    rng = np.random.default_rng(4)
    M, N = 200, 1000
    counts = rng.integers(0, N + 1, size=M)
    counts[:7] = 0
    kept = int(counts.sum())
    for mode in (darb.ROUND_FLOOR, darb.ROUND_PAPER):
        a = darb.Plan.from_counts(N, counts, kept, mode, 2, 128)
        b = darb.Plan(M, N, counts / N, kept / (M * N), mode, 2, 128)
        for x, y in zip(a.export(), b.export()):
            assert np.array_equal(x, y)
    L = darb.lib()
    h = ctypes.c_void_p()
    c = np.array([1, 2, 3], dtype=np.int64)
    P = c.ctypes.data_as(ctypes.c_void_p)
    assert L.darb_plan_create_counts(3, 2, P, 3, 0, 1, 2, ctypes.byref(h)) == darb.E_INVALID
    assert L.darb_plan_create_counts(3, 4, P, 13, 0, 1, 2, ctypes.byref(h)) == darb.E_INVALID
    assert L.darb_plan_create_counts(3, 4, None, 3, 0, 1, 2, ctypes.byref(h)) == darb.E_INVALID


def test_prune_argument_checks():
    L = darb.lib()
    nbytes = ctypes.c_int64()
    assert L.darb_prune_workspace(64, 300, darb.F32, ctypes.byref(nbytes)) == 0
    assert nbytes.value > 0 and nbytes.value % 256 == 0
    assert L.darb_prune_workspace(64, 300, 7, ctypes.byref(nbytes)) == darb.E_DTYPE
    assert L.darb_prune_workspace(0, 300, darb.F32, ctypes.byref(nbytes)) == darb.E_INVALID
    buf = ctypes.c_void_p(0x1000)
    # every check fails before any HIP work
    assert L.darb_prune_counts(4, 8, darb.F32, buf, 8, 33, buf, buf, 1 << 20, None) \
        == darb.E_INVALID                                     # k > M*N
    assert L.darb_prune_counts(4, 8, darb.F32, buf, 7, 3, buf, buf, 1 << 20, None) \
        == darb.E_INVALID                                     # ldw < N
    assert L.darb_prune_counts(4, 8, darb.F32, None, 8, 3, buf, buf, 1 << 20, None) \
        == darb.E_INVALID
    assert L.darb_prune_counts(4, 8, darb.F32, buf, 8, 3, buf, ctypes.c_void_p(0x1010),
                               1 << 20, None) == darb.E_INVALID  # workspace alignment
    assert L.darb_prune_counts(4, 8, darb.F32, buf, 8, 3, buf, buf, 16, None) \
        == darb.E_WORKSPACE
    assert L.darb_prune_counts(4, 8, 9, buf, 8, 3, buf, buf, 1 << 20, None) == darb.E_DTYPE


def test_plan_table7_and_worked_example():
    p = darb.Plan(6, 1500, np.array([0.5, 0.25, 0.125, 1 / 16, 1 / 32, 1 / 64]), 0.1,
                  darb.ROUND_FLOOR, 1, 128)
    assert p.nnz == 1478
    p = darb.Plan(2, 16, np.array([0.375, 0.1875]), 0.2188, darb.ROUND_PAPER, 1, 128)
    assert [1 << int(v) for v in p.export()[0]] == [2, 8]


@pytest.mark.parametrize("kw,code", [
    (dict(M=0), darb.E_INVALID), (dict(N=0), darb.E_INVALID), (dict(M=-3), darb.E_INVALID),
    (dict(N=(1 << 31) - 255), darb.E_INVALID), (dict(M=1 << 31), darb.E_INVALID),
    (dict(b_min=3), darb.E_INVALID), (dict(b_max=256), darb.E_INVALID),
    (dict(b_min=64, b_max=8), darb.E_INVALID), (dict(mode=5), darb.E_INVALID),
    (dict(D=float("nan")), darb.E_INVALID), (dict(D=1.5), darb.E_INVALID),
    (dict(d=[0.1, float("nan"), 0.2]), darb.E_INVALID), (dict(d=[0.1, -0.01, 0.2]), darb.E_INVALID),
    (dict(d=[0.1, 1.01, 0.2]), darb.E_INVALID),
])
def test_plan_create_rejects(kw, code):
    args = dict(M=3, N=64, d=[0.1, 0.2, 0.3], D=0.2, mode=0, b_min=4, b_max=64)
    args.update(kw)
    d = np.asarray(args["d"], dtype=np.float64)
    h = ctypes.c_void_p(1234)
    rc = darb.lib().darb_plan_create(args["M"], args["N"], d.ctypes.data_as(ctypes.c_void_p),
                                     args["D"], args["mode"], args["b_min"], args["b_max"],
                                     ctypes.byref(h))
    assert rc == code
    assert h.value is None                         # *out cleared on error
    assert darb.lib().darb_last_error().decode() != ""


def test_null_arguments_and_not_uploaded():
    L = darb.lib()
    h = ctypes.c_void_p()
    d = np.array([0.1, 0.2], dtype=np.float64)
    assert L.darb_plan_create(2, 8, None, 0.1, 0, 1, 8, ctypes.byref(h)) == darb.E_INVALID
    assert L.darb_plan_create(2, 8, d.ctypes.data_as(ctypes.c_void_p), 0.1, 0, 1, 8, None) \
        == darb.E_INVALID
    p = darb.Plan(2, 8, d, 0.1, 0, 1, 8)
    buf = ctypes.c_void_p(0x1000)
    # every device call on a plan that was never uploaded fails before any HIP work
    assert L.darb_encode(p.handle, 0, buf, 8, buf, buf, None) == darb.E_NOT_UPLOADED
    assert L.darb_decode(p.handle, 0, buf, buf, buf, 8, None) == darb.E_NOT_UPLOADED
    assert L.darb_spmv(p.handle, 0, buf, buf, 0, buf, buf, None) == darb.E_NOT_UPLOADED
    assert L.darb_spmm(p.handle, 0, buf, buf, 0, 4, buf, 4, buf, 4, None) == darb.E_NOT_UPLOADED
    assert L.darb_pack_offsets(p.handle, buf, buf, None) == darb.E_NOT_UPLOADED
    assert L.darb_unpack_offsets(p.handle, buf, buf, None) == darb.E_NOT_UPLOADED
    assert L.darb_spmv_packed(p.handle, 0, buf, buf, 0, buf, buf, None) == darb.E_NOT_UPLOADED
    assert L.darb_spmm_packed(p.handle, 0, buf, buf, 0, 4, buf, 4, buf, 4, None) \
        == darb.E_NOT_UPLOADED
    assert L.darb_spmv_packed(None, 0, buf, buf, 0, buf, buf, None) == darb.E_INVALID
    assert L.darb_encode(None, 0, buf, 8, buf, buf, None) == darb.E_INVALID
    assert L.darb_plan_info(None, None) == darb.E_INVALID
    assert L.darb_plan_upload(p.handle, None, 1024, None) == darb.E_INVALID
    assert L.darb_plan_upload(p.handle, ctypes.c_void_p(0x1001), 1024, None) == darb.E_INVALID
    assert L.darb_plan_upload(p.handle, ctypes.c_void_p(0x1000), 4, None) == darb.E_WORKSPACE
    assert L.darb_stream_read(None, 16, buf, None) == darb.E_INVALID
    assert L.darb_stream_copy(buf, buf, 15, None) == darb.E_INVALID
    # the pruning call without a workspace names its row limit before touching a device
    assert L.darb_prune_counts_noalloc(1 << 20, 4, darb.F32, buf, 4, 0, buf, None) == \
        darb.E_INVALID
    assert b"fixed pruning scratch" in L.darb_last_error()
    assert L.darb_prune_counts_noalloc(4, 4, 7, buf, 4, 0, buf, None) == darb.E_DTYPE
    # the device-built plan checks its arguments before touching a device
    nb = ctypes.c_int64()
    assert L.darb_plan_device_workspace(1000, ctypes.byref(nb)) == darb.OK and nb.value > 12000
    assert L.darb_plan_device_workspace(0, ctypes.byref(nb)) == darb.E_INVALID
    hp = ctypes.c_void_p()
    ws = ctypes.c_void_p(0x100000)
    assert L.darb_plan_create_device(10, 10, buf, 5, 0, 1, 128, None, 1 << 20, None,
                                     ctypes.byref(hp)) == darb.E_INVALID
    assert L.darb_plan_create_device(10, 10, buf, 5, 0, 1, 128, ctypes.c_void_p(0x100010),
                                     1 << 20, None, ctypes.byref(hp)) == darb.E_INVALID
    assert L.darb_plan_create_device(10, 10, buf, 5, 2, 1, 128, ws, 1 << 20, None,
                                     ctypes.byref(hp)) == darb.E_INVALID
    assert L.darb_plan_create_device(10, 10, buf, 101, 0, 1, 128, ws, 1 << 20, None,
                                     ctypes.byref(hp)) == darb.E_INVALID
    assert L.darb_plan_create_device(10, 10, buf, 5, 0, 4, 2, ws, 1 << 20, None,
                                     ctypes.byref(hp)) == darb.E_INVALID
    assert L.darb_plan_create_device(10, 10, buf, 5, 0, 1, 128, ws, 16, None,
                                     ctypes.byref(hp)) == darb.E_WORKSPACE
    L.darb_plan_destroy(None)                        # ignored


def test_strerror_covers_codes():
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert darb.lib().darb_strerror(code).decode() not in ("", "unknown error code")
    assert darb.lib().darb_strerror(-99).decode() == "unknown error code"


def test_binding_rejects_host_tensors():
    torch = pytest.importorskip("torch")
    p = darb.Plan(4, 16, np.full(4, 0.25), 0.25, 0, 1, 16)
    with pytest.raises(ValueError):
        p.encode(torch.zeros(4, 16))


def test_single_hip_runtime_in_process():
    # libdarb.so must share torch's HIP runtime, not load a second copy
    import torch  # noqa: F401
    maps = open("/proc/self/maps").read()
    paths = {ln.split()[-1] for ln in maps.splitlines() if "libamdhip64" in ln}
    assert len(paths) == 1, paths


def test_bench_refuses_more_than_one_gpu():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
