"""GPU parity: the HIP kernels against the CPU oracle, through the C ABI.

Encode, decode and the plan are compared bit for bit.  Products are compared
per output with err = |y - y64| / sum_k |v_k x_k| (the scale of a dot
product's rounding error; an output whose scale is 0 must be exactly 0),
bounded by 1e-5 for fp32 weights and 2e-3 for fp16 weights.
"""
import functools
import sys

import numpy as np
import pytest

import oracle
import workloads
from tests._parity import compare

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TOL = {np.dtype(np.float32): 1e-5, np.dtype(np.float16): 2e-3}
_TDT = {np.dtype(np.float32): torch.float32, np.dtype(np.float16): torch.float16}
_UT = {np.dtype(np.float32): np.uint32, np.dtype(np.float16): np.uint16}


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.fixture(scope="module")
def darb():
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_1911_08020_amd as d
    return d


def dev(a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy()


def check_product(Y, vals, offs, lay, X, wdtype, label=""):
    compare(Y, oracle.spmm(vals, offs, lay, X), oracle.spmm_absdot(vals, offs, lay, X),
            TOL[np.dtype(wdtype)], label)


def encode_both(darb, W, d, D, mode, bmin, bmax, W_dev=None):
    """Plan + encode on the GPU and in the oracle; assert bit-exact equality."""
    M, N = W.shape
    plan = darb.Plan(M, N, d, D, mode, bmin, bmax).upload()
    lay = oracle.plan(N, d, D, mode, bmin, bmax)
    log2b, row_start, perm = plan.export()
    assert np.array_equal(log2b, lay.log2b) and np.array_equal(perm, lay.perm)
    vals_ref, offs_ref = oracle.encode(W, lay)
    Wd = dev(W) if W_dev is None else W_dev
    v, o = plan.encode(Wd)
    v, o = host(v), host(o)
    ut = _UT[W.dtype]
    assert np.array_equal(o, offs_ref), "offsets differ"
    assert np.array_equal(v.view(ut), vals_ref.view(ut)), "values differ"
    return plan, lay, vals_ref, offs_ref


# --------------------------------------------------------------------------------
# encode
# --------------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", [np.float32, np.float16])
@pytest.mark.parametrize("shape", [(1, 1), (3, 7), (37, 203), (130, 1030), (64, 4100), (9, 2049)])
def test_encode_small_shapes_ties_and_tails(darb, dtype, shape):
    M, N = shape
    say(f"encode small {shape} {np.dtype(dtype).name}")
    rng = np.random.default_rng(M * 1000 + N)
    W = (rng.integers(-4, 5, size=(M, N)) * 0.5).astype(dtype)      # many ties
    W[rng.random((M, N)) < 0.05] = -0.0
    counts = rng.integers(0, N + 1, size=M)
    for mode in (0, 1):
        encode_both(darb, W, counts / float(N), float(counts.mean() / N), mode, 1, 128)


@pytest.mark.parametrize("dtype", [np.float32, np.float16])
def test_encode_special_values(darb, dtype):
    say(f"encode special values {np.dtype(dtype).name}")
    rng = np.random.default_rng(5)
    M, N = 48, 517
    W = rng.standard_normal((M, N)).astype(dtype)
    specials = np.array([np.inf, -np.inf, 0.0, -0.0, np.finfo(dtype).tiny,
                         np.finfo(dtype).max, -np.finfo(dtype).max], dtype=dtype)
    sel = rng.random((M, N)) < 0.1
    W[sel] = rng.choice(specials, size=int(sel.sum()))
    W[::5] *= dtype(1e-30) if dtype == np.float32 else dtype(0)     # denormals / zeros
    W[3, 10] = np.nan
    W[7, 100:140] = np.nan
    d = np.full(M, 0.01)
    d[::3] = 0.3
    encode_both(darb, W, d, 0.1, 0, 1, 128)


def test_encode_strided_and_misaligned_rows(darb):
    say("encode strided W (ldw > N, rows not 16-byte aligned)")
    rng = np.random.default_rng(6)
    M, N = 70, 999
    big = rng.standard_normal((M, N + 3)).astype(np.float32)
    W = big[:, :N]
    d = rng.integers(0, N, size=M) / N
    plan = darb.Plan(M, N, d, 0.05, 0, 2, 64).upload()
    lay = oracle.plan(N, d, 0.05, 0, 2, 64)
    vr, orf = oracle.encode(np.ascontiguousarray(W), lay)
    Wd = dev(big)[:, :N]
    assert Wd.stride(0) == N + 3
    v, o = plan.encode(Wd)
    assert np.array_equal(host(o), orf)
    assert np.array_equal(host(v).view(np.uint32), vr.view(np.uint32))


@functools.lru_cache(maxsize=None)
def _config(name):
    return workloads.make_config(name, seed=0)


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216"])
def test_config_encode_decode_spmv_spmm(darb, name):
    cfg, mi, x, X = _config(name)
    say(f"config {name}: encode {cfg.M}x{cfg.N} {cfg.wdtype}")
    plan, lay, vals, offs = encode_both(darb, mi.W, mi.row_density, mi.matrix_density, 0,
                                        cfg.b_min, cfg.b_max)
    vd, od = dev(vals), dev(offs)
    say(f"config {name}: decode")
    Wm = host(plan.decode(vd, od))
    ut = _UT[mi.W.dtype]
    assert np.array_equal(Wm.view(ut), oracle.decode(vals, offs, lay).view(ut))
    say(f"config {name}: spmv")
    y = host(plan.spmv(vd, od, dev(x)))
    check_product(y, vals, offs, lay, x, mi.W.dtype, f"{name} spmv")
    say(f"config {name}: spmm B={X.shape[1]}")
    Y = host(plan.spmm(vd, od, dev(X)))
    check_product(Y, vals, offs, lay, X, mi.W.dtype, f"{name} spmm B={X.shape[1]}")


def test_fc_spmm_and_spmv_deterministic(darb):
    cfg, mi, x, X = _config("fc_9216")
    say("fc_9216: repeat products, bitwise equal")
    plan = darb.Plan(cfg.M, cfg.N, mi.row_density, mi.matrix_density, 0, cfg.b_min,
                     cfg.b_max).upload()
    v, o = plan.encode(dev(mi.W))
    xd, Xd = dev(x), dev(X)
    y1, y2 = host(plan.spmv(v, o, xd)), host(plan.spmv(v, o, xd))
    Y1, Y2 = host(plan.spmm(v, o, Xd)), host(plan.spmm(v, o, Xd))
    assert np.array_equal(y1.view(np.uint32), y2.view(np.uint32))
    assert np.array_equal(Y1.view(np.uint32), Y2.view(np.uint32))


# --------------------------------------------------------------------------------
# products: batch sizes, strides, dtypes, degenerate layouts
# --------------------------------------------------------------------------------

@pytest.mark.parametrize("B", [1, 2, 3, 16, 33, 64, 65, 130])
@pytest.mark.parametrize("wx", [("f32", "f32"), ("f16", "f16"), ("f16", "f32")])
def test_spmm_batches(darb, B, wx):
    wdt, xdt = {"f32": np.float32, "f16": np.float16}[wx[0]], {"f32": np.float32,
                                                              "f16": np.float16}[wx[1]]
    say(f"spmm B={B} w={wx[0]} x={wx[1]}")
    rng = np.random.default_rng(B)
    M, N = 300, 777
    W = rng.standard_normal((M, N)).astype(wdt)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 1, 128)
    X = rng.standard_normal((N, B)).astype(xdt)
    # X and Y with leading dimensions larger than B
    Xbig = np.zeros((N, B + 5), dtype=xdt)
    Xbig[:, :B] = X
    Xd = dev(Xbig)[:, :B]
    Yd = torch.full((M, B + 3), float("nan"), device="cuda")[:, :B]
    plan.spmm(dev(vals), dev(offs), Xd, Y=Yd)
    check_product(host(Yd), vals, offs, lay, X, wdt, f"B={B}")
    if B == 1:
        y = plan.spmv(dev(vals), dev(offs), dev(X[:, 0].copy()))
        check_product(host(y), vals, offs, lay, X[:, 0], wdt, "spmv")


@pytest.mark.parametrize("B", [8, 20, 24, 32, 48, 64, 96, 128])
@pytest.mark.parametrize("wx", [("f32", "f32"), ("f16", "f16"), ("f16", "f32")])
def test_spmm_column_widths(darb, B, wx):
    # a lane takes 1, 2, 4 (or 8 fp16) columns depending on B and on the alignment of
    # X's rows: 16-byte rows (ldx = B), rows aligned to 4 columns only (ldx = B + 4:
    # 16 bytes for fp32, 8 for fp16), to 2 columns (ldx = B + 2) or to one.  Every
    # width sums each column in the same order, so all four results are bitwise equal.
    wdt, xdt = {"f32": np.float32, "f16": np.float16}[wx[0]], {"f32": np.float32,
                                                              "f16": np.float16}[wx[1]]
    say(f"spmm column widths B={B} w={wx[0]} x={wx[1]}")
    rng = np.random.default_rng(1000 + B)
    M, N = 400, 1536
    W = rng.standard_normal((M, N)).astype(wdt)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 2, 64)
    X = rng.standard_normal((N, B)).astype(xdt)
    vd, od = dev(vals), dev(offs)
    outs = []
    for pad in (0, 4, 2, 1):
        Xbig = np.zeros((N, B + pad), dtype=xdt)
        Xbig[:, :B] = X
        Xd = dev(Xbig)[:, :B]
        outs.append(host(plan.spmm(vd, od, Xd)))
    check_product(outs[0], vals, offs, lay, X, wdt, f"B={B} aligned")
    for o in outs[1:]:
        assert np.array_equal(o.view(np.uint32), outs[0].view(np.uint32))


@pytest.mark.parametrize("case", ["all_empty_rows", "b_one", "b_wider_than_row", "one_row",
                                  "wide_no_lds", "odd_nblk", "fp16_odd"])
def test_product_edge_cases(darb, case):
    say(f"edge case {case}")
    rng = np.random.default_rng(len(case))
    wdt = np.float16 if case == "fp16_odd" else np.float32
    M, N, bmin, bmax = 50, 300, 1, 128
    d = None
    if case == "all_empty_rows":
        d = np.zeros(M)
    elif case == "b_one":
        d, bmax = np.ones(M), 1
    elif case == "b_wider_than_row":
        M, N = 40, 50
        d = np.zeros(M)
    elif case == "one_row":
        M, N = 1, 1000
    elif case == "wide_no_lds":
        M, N = 64, 20000                # x does not fit the LDS staging buffer
    elif case == "odd_nblk":
        M, N = 33, 333
    elif case == "fp16_odd":
        M, N = 29, 1001
    W = rng.standard_normal((M, N)).astype(wdt)
    if d is None:
        d = rng.integers(0, N + 1, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, float(np.mean(d)), 0, bmin, bmax)
    x = rng.standard_normal(N).astype(wdt if wdt == np.float16 else np.float32)
    y = host(plan.spmv(dev(vals), dev(offs), dev(x)))
    check_product(y, vals, offs, lay, x, wdt, case + " spmv")
    X = rng.standard_normal((N, 5)).astype(np.float32)
    Y = host(plan.spmm(dev(vals), dev(offs), dev(X)))
    check_product(Y, vals, offs, lay, X, wdt, case + " spmm")


@pytest.mark.parametrize("case", ["many_rows", "wide_rows", "wide_batch"])
def test_large_shapes(darb, case):
    # grids of 10^5+ workgroups, x past the LDS staging size with every block size,
    # and a batch spanning several column slabs
    say(f"large shape {case}")
    rng = np.random.default_rng(len(case) + 40)
    B = 5
    if case == "many_rows":
        M, N = 200_000, 48
    elif case == "wide_rows":
        M, N = 24, 100_003
    else:
        M, N, B = 300, 1500, 1000
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = 1.0 / (1 << rng.integers(0, 8, size=M))
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 1, 128)
    x = rng.standard_normal(N).astype(np.float32)
    check_product(host(plan.spmv(dev(vals), dev(offs), dev(x))), vals, offs, lay, x, np.float32,
                  case + " spmv")
    X = rng.standard_normal((N, B)).astype(np.float32)
    check_product(host(plan.spmm(dev(vals), dev(offs), dev(X))), vals, offs, lay, X, np.float32,
                  case + f" spmm B={B}")


@pytest.mark.parametrize("case", [(1024, 4100, "f32", 64), (512, 8200, "f32", 32),
                                  (1024, 4096, "f16", 64), (700, 4100, "f32", 128)])
def test_spmm_wide_batch_short_rows(darb, case):
    # N small enough that a slab of X (32 or 64 columns) fits in LDS, B wide enough
    # for >= 128 slabs and rows in whole steps of 16 weights: the product stages X
    # slabs in LDS (the last case has rows of ragged length and takes the general path);
    # both offset forms take the same path
    N, B, wdt, bmax = case
    wdt = np.float32 if wdt == "f32" else np.float16
    say(f"wide-batch spmm N={N} B={B} w={wdt.__name__} b<={bmax}")
    rng = np.random.default_rng(N + B)
    M = 300
    W = rng.standard_normal((M, N)).astype(wdt)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 1, bmax)
    X = rng.standard_normal((N, B)).astype(np.float32)
    vd, od, Xd = dev(vals), dev(offs), dev(X)
    Y = host(plan.spmm(vd, od, Xd))
    check_product(Y, vals, offs, lay, X, wdt, f"wide B={B}")
    # packed offsets take the same kernel and give the same bits
    Yp = host(plan.spmm_packed(vd, plan.pack_offsets(od), Xd))
    assert np.array_equal(Yp.view(np.uint32), Y.view(np.uint32)), "packed != byte form"


def test_spmv_misaligned_values_uses_scalar_path(darb):
    say("spmv with values/offsets starting at an odd element")
    rng = np.random.default_rng(12)
    M, N = 77, 512
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = rng.integers(0, N, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 4, 64)
    vbig = dev(np.concatenate([[0.0], vals]).astype(np.float32))[1:]
    obig = dev(np.concatenate([[0], offs]).astype(np.uint8))[1:]
    x = rng.standard_normal(N).astype(np.float32)
    y = host(plan.spmv(vbig, obig, dev(x)))
    check_product(y, vals, offs, lay, x, np.float32, "misaligned spmv")


def test_unit_vector_returns_masked_column(darb):
    say("spmv(e_c) == column c of the masked matrix")
    rng = np.random.default_rng(13)
    M, N = 200, 640
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = rng.integers(0, N, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 1, 128)
    Wm = oracle.decode(vals, offs, lay)
    X = np.zeros((N, 8), dtype=np.float32)
    cols = [0, 1, 63, 64, 300, 511, 638, 639]
    for j, c in enumerate(cols):
        X[c, j] = 1.0
    Y = host(plan.spmm(dev(vals), dev(offs), dev(X)))
    assert np.array_equal(Y, Wm[:, cols])


# --------------------------------------------------------------------------------
# the recurrent workload
# --------------------------------------------------------------------------------

def _lstm_case(darb, hidden, seq_len, batch, layers, seed):
    cfg, mats, xs, shp = workloads.make_lstm_inputs(seed=seed, seq_len=seq_len, batch=batch,
                                                    hidden=hidden, layers=layers)
    H, T, Bt = shp["hidden"], shp["seq_len"], shp["batch"]
    masked, dev_layers = [], []
    for (wih, whh) in mats:
        pair_m, pair_d = [], []
        for mi in (wih, whh):
            plan, lay, vals, offs = encode_both(darb, mi.W, mi.row_density, mi.matrix_density,
                                                0, cfg.b_min, cfg.b_max)
            pair_m.append(oracle.decode(vals, offs, lay).astype(np.float64))
            pair_d.append((plan, dev(vals), dev(offs)))
        masked.append(tuple(pair_m))
        dev_layers.append(tuple(pair_d))
    ref, finals = oracle.lstm_forward(masked, xs, H, T, Bt)
    inp = dev(xs)
    for (wih, whh) in dev_layers:
        inp, h, c = darb.lstm_layer(wih, whh, inp, H, T, Bt)
    out = host(inp)
    err = float(np.abs(out - ref).max())
    say(f"  lstm H={H} T={T} B={Bt}: max abs err {err:.3e}")
    assert err <= 2e-3
    assert np.abs(host(c) - finals[-1][1]).max() <= 2e-3
    # the final hidden state is the last step's output
    assert np.array_equal(host(h), out[:, (T - 1) * Bt:])


def test_lstm_small(darb):
    say("lstm small")
    _lstm_case(darb, hidden=64, seq_len=7, batch=3, layers=2, seed=1)


@pytest.mark.parametrize("batch", [1, 8, 40, 200, 300])
def test_lstm_batches(darb, batch):
    # lanes per row from 1 to 64, and a batch past one column slab
    say(f"lstm batch {batch}")
    _lstm_case(darb, hidden=96, seq_len=5, batch=batch, layers=1, seed=batch)


def test_lstm_full_workload(darb):
    say("lstm 2 layers, hidden 1024, T=200, batch 32")
    _lstm_case(darb, hidden=None, seq_len=None, batch=None, layers=None, seed=0)


# --------------------------------------------------------------------------------
# paper-mode plans and the benchmark's output contract
# --------------------------------------------------------------------------------

def test_paper_rounding_mode_end_to_end(darb):
    say("paper rounding mode: plan, encode, products")
    cfg, mi, x, X = _config("lstm_1024")
    plan, lay, vals, offs = encode_both(darb, mi.W, mi.row_density, mi.matrix_density,
                                        darb.ROUND_PAPER, cfg.b_min, cfg.b_max)
    y = host(plan.spmv(dev(vals), dev(offs), dev(x)))
    check_product(y, vals, offs, lay, x, np.float32, "paper-mode spmv")
    X16 = X[:, :1].repeat(16, axis=1) if X.shape[1] < 16 else X[:, :16]
    Y = host(plan.spmm(dev(vals), dev(offs), dev(np.ascontiguousarray(X16))))
    check_product(Y, vals, offs, lay, np.ascontiguousarray(X16), np.float32, "paper-mode spmm")


def test_bench_prints_contract_json(darb, capsys):
    say("bench.py main(): one short run, JSON contract")
    import json

    import bench
    bench.main(["--steps", "3", "--warmup", "1", "--cpu-seconds", "0.2"])
    line = capsys.readouterr().out.strip().splitlines()[-1]
    d = json.loads(line)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
                "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
                "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["value"] > 0
    assert d["roofline"]["bound"] == "hbm" and 0 < d["roofline"]["frac"] < 1.5
    assert d["cpu_baseline"]["kind"] == "oracle" and d["cpu_baseline"]["cores"] >= 1
    assert "workload" in d["config"]


def test_spmv_workgroups_take_several_blocks(darb):
    # 5000 rows of 16 384 columns at b = 8: 1250 blocks of 4 rows (625 of 8 rows with
    # INT8 codes), while x (64 KiB of LDS per workgroup) lets only 2 workgroups per
    # CU fit (512 on 256 CUs), so each workgroup stages x once and loops over several
    # blocks.  Byte, packed and INT8 forms.
    say("spmv with looping workgroups")
    rng = np.random.default_rng(77)
    M, N = 5000, 16384
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = np.full(M, 1.0 / 8)
    plan, lay, vals, offs = encode_both(darb, W, d, 0.125, 0, 1, 128)
    assert int(np.unique(lay.log2b)[0]) == 3
    x = rng.standard_normal(N).astype(np.float32)
    vd, od = dev(vals), dev(offs)
    y = host(plan.spmv(vd, od, dev(x)))
    check_product(y, vals, offs, lay, x, np.float32, "looping spmv")
    packed = plan.pack_offsets(od)
    yp = host(plan.spmv_packed(vd, packed, dev(x)))
    assert np.array_equal(y.view(np.uint32), yp.view(np.uint32))
    q, s = oracle.quantize_i8(vals, lay)
    y8 = host(plan.spmv_i8(dev(q), dev(s), dev(x), packed=packed))
    compare(y8, oracle.spmm_i8(q, s, offs, lay, x), oracle.spmm_i8_absdot(q, s, offs, lay, x),
            1e-5, "looping spmv INT8")


@pytest.mark.parametrize("wdtype", [np.float32, np.float16])
def test_spmv_row_blocks_on_resident_workgroups(darb, wdtype):
    # 4800 rows of 15 360 columns at b = 8, 16, 32: x takes 61 KiB of LDS, so two
    # workgroups fit per CU (512 on 256 CUs) against about 700 row blocks of four
    # waves; the row-block kernel then keeps its workgroups resident and each goes
    # through several blocks of its group, the next block's row index loaded a block
    # ahead.  fp32 and fp16 weights with fp32 x; byte, packed and INT8 forms.
    say(f"spmv row blocks on resident workgroups, {np.dtype(wdtype).name} weights")
    rng = np.random.default_rng(78)
    M, N = 4800, 15360
    W = rng.standard_normal((M, N)).astype(wdtype)
    d = 1.0 / rng.choice([8, 16, 32], size=M)
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 8, 32)
    assert set(np.unique(lay.log2b).tolist()) == {3, 4, 5}
    x = rng.standard_normal(N).astype(np.float32)
    vd, od, xd = dev(vals), dev(offs), dev(x)
    y = host(plan.spmv(vd, od, xd))
    check_product(y, vals, offs, lay, x, wdtype, "row blocks spmv")
    packed = plan.pack_offsets(od)
    yp = host(plan.spmv_packed(vd, packed, xd))
    assert np.array_equal(y.view(np.uint32), yp.view(np.uint32))
    q, s = oracle.quantize_i8(vals, lay)
    for label, kw in (("byte", dict(offsets=od)), ("packed", dict(packed=packed))):
        y8 = host(plan.spmv_i8(dev(q), dev(s), xd, **kw))
        compare(y8, oracle.spmm_i8(q, s, offs, lay, x), oracle.spmm_i8_absdot(q, s, offs, lay, x),
                1e-5, f"row blocks spmv INT8 {label}")


# --------------------------------------------------------------------------------
# special values in x / X: a product reads only its row's kept columns, so inf and
# nan reach exactly the outputs whose kept weights read them (a lane past a row's
# weights, or a masked column, must add nothing, not 0 * inf)
# --------------------------------------------------------------------------------

def _with_specials(rng, X):
    X = X.copy()
    flat = X.reshape(-1)
    idx = rng.choice(flat.size, size=max(6, flat.size // 3000), replace=False)
    flat[idx] = np.array([np.inf, -np.inf, np.nan], dtype=X.dtype)[np.arange(idx.size) % 3]
    return X


def _check_specials(Y, ref, scale, tol, label):
    Y = np.asarray(Y, dtype=np.float64)
    assert np.isnan(ref).any() and np.isinf(ref).any(), label
    assert np.array_equal(np.isnan(Y), np.isnan(ref)), label + ": nan positions differ"
    inf = np.isinf(ref)
    assert np.array_equal(np.isinf(Y), inf), label + ": inf positions differ"
    assert np.array_equal(Y[inf], ref[inf]), label + ": inf signs differ"
    fin = np.isfinite(ref)
    compare(Y[fin], ref[fin], scale[fin], tol, label + " (finite outputs)")


@pytest.mark.parametrize("path", ["spmv", "spmm64", "spmm_wide", "f16_spmm", "int8"])
def test_products_special_values_reach_only_their_rows(darb, path):
    rng = np.random.default_rng({"spmv": 1, "spmm64": 2, "spmm_wide": 3, "f16_spmm": 4,
                                 "int8": 5}[path])
    M, N, B = 300, 2048, {"spmv": 1, "spmm64": 64, "spmm_wide": 4100, "f16_spmm": 16,
                          "int8": 64}[path]
    if path == "spmm_wide":
        N = 1024                                    # X slabs staged in LDS
    wdt = np.float16 if path == "f16_spmm" else np.float32
    say(f"special values in x/X: {path} ({M}x{N}, B={B})")
    W = rng.standard_normal((M, N)).astype(wdt)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = encode_both(darb, W, d, 0.1, 0, 1, 64)
    X = _with_specials(rng, rng.standard_normal((N, B)).astype(wdt))
    if B == 1:
        X = X[:, 0].copy()
    X0 = np.where(np.isfinite(X), X, 0).astype(X.dtype)
    vd, od, Xd = dev(vals), dev(offs), dev(X)
    pk = plan.pack_offsets(od)
    prod = plan.spmv if B == 1 else plan.spmm
    prod_pk = plan.spmv_packed if B == 1 else plan.spmm_packed
    with np.errstate(invalid="ignore", over="ignore"):
        if path == "int8":
            q_ref, s_ref = oracle.quantize_i8(vals, lay)
            q, s = plan.quantize_i8(vd)
            assert np.array_equal(host(q), q_ref) and np.array_equal(
                host(s).view(np.uint32), s_ref.view(np.uint32)), "codes or scales differ"
            ref = oracle.spmm_i8(q_ref, s_ref, offs, lay, X)
            scale = oracle.spmm_i8_absdot(q_ref, s_ref, offs, lay, X0)
            outs = [host(plan.spmm_i8(q, s, Xd, offsets=od)),
                    host(plan.spmm_i8(q, s, Xd, packed=pk))]
        else:
            ref = oracle.spmm(vals, offs, lay, X)
            scale = oracle.spmm_absdot(vals, offs, lay, X0)
            outs = [host(prod(vd, od, Xd)), host(prod_pk(vd, pk, Xd))]
    tol = 2e-3 if wdt == np.float16 else 1e-5
    for o, form in zip(outs, ("byte offsets", "packed offsets")):
        _check_specials(o, ref, scale, tol, f"{path}, {form}")
    assert np.array_equal(np.nan_to_num(outs[0]).view(np.uint32),
                          np.nan_to_num(outs[1]).view(np.uint32)), "forms differ"
