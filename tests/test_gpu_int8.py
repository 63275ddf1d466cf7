"""GPU parity of INT8 retained values (section 4.2's storage accounting assumes INT8
weights; the per-row symmetric scheme is the reading documented on
oracle.quantize_i8).

Codes are integers decided in fp32 by the same correctly rounded operations on both
sides, so they and the scales must equal the oracle's bit for bit.  The products
must match the oracle's fp64 product within 1e-5 of |s_r| * sum |q * x|, and the
byte-offset and packed-offset forms must give the same bits.
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

TOL = 1e-5


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


def quantize_both(darb, plan, lay, vals):
    """GPU and oracle quantisation of the same values; asserts bitwise equality."""
    q_ref, s_ref = oracle.quantize_i8(vals, lay)
    q, s = plan.quantize_i8(dev(vals))
    q, s = host(q), host(s)
    assert np.array_equal(q, q_ref), "codes differ from the oracle"
    assert np.array_equal(s.view(np.uint32), s_ref.view(np.uint32)), "scales differ"
    return q_ref, s_ref


def check_i8_product(Y, q, s, offs, lay, X, label):
    compare(Y, oracle.spmm_i8(q, s, offs, lay, X), oracle.spmm_i8_absdot(q, s, offs, lay, X),
            TOL, label)


def plan_for(darb, W, d, D, bmin, bmax):
    M, N = W.shape
    plan = darb.Plan(M, N, d, D, darb.ROUND_FLOOR, bmin, bmax).upload()
    lay = oracle.plan(N, d, D, oracle.ROUND_FLOOR, bmin, bmax)
    vals, offs = oracle.encode(W, lay)
    return plan, lay, vals, offs


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216"])
def test_config_quantize_and_products(darb, name):
    cfg, mi, x, X = workloads.make_config(name, seed=0)
    say(f"{name}: int8 {cfg.M}x{cfg.N} from {cfg.wdtype}")
    plan, lay, vals, offs = plan_for(darb, mi.W, mi.row_density, mi.matrix_density, cfg.b_min,
                                     cfg.b_max)
    # quantise the values the GPU encode produced (bitwise the oracle's)
    v_gpu, o_gpu = plan.encode(dev(mi.W))
    assert np.array_equal(host(o_gpu), offs)
    q, s = quantize_both(darb, plan, lay, vals)
    qd, sd = dev(q), dev(s)
    packed = plan.pack_offsets(o_gpu)
    y8 = host(plan.spmv_i8(qd, sd, dev(x), offsets=o_gpu))
    yp = host(plan.spmv_i8(qd, sd, dev(x), packed=packed))
    assert np.array_equal(y8.view(np.uint32), yp.view(np.uint32)), "packed spmv differs"
    check_i8_product(y8, q, s, offs, lay, x, f"{name} spmv_i8")
    for B in sorted({X.shape[1], 16, 64}):
        XB = np.random.default_rng(B).standard_normal((cfg.N, B)).astype(X.dtype)
        Y8 = host(plan.spmm_i8(qd, sd, dev(XB), offsets=o_gpu))
        Yp = host(plan.spmm_i8(qd, sd, dev(XB), packed=packed))
        assert np.array_equal(Y8.view(np.uint32), Yp.view(np.uint32)), "packed spmm differs"
        check_i8_product(Y8, q, s, offs, lay, XB, f"{name} spmm_i8 B={B} x={XB.dtype}")


def test_quantize_edge_rows(darb):
    # ties at .5 under both scales, a zero row, rows below / at the overflow threshold,
    # long rows (many lanes' strides), b = 1 rows; fp32 values
    N = 640
    rng = np.random.default_rng(3)
    t = float(oracle.I8_MIN_ABSMAX)
    rows = [
        np.r_[127.0, 2.5, -3.5, 0.5, -0.0, rng.standard_normal(N - 5)],
        np.zeros(N),
        np.r_[t / 2, -t / 4, np.zeros(N - 2)],
        np.r_[t, -t / 2, np.zeros(N - 2)],
        np.r_[-2.0, 1.0, 0.5, np.zeros(N - 3)],
        rng.standard_normal(N) * 1e-30,
        rng.standard_normal(N) * 1e30,
    ]
    W = np.stack(rows).astype(np.float32)
    M = W.shape[0]
    for bmin, bmax in ((1, 1), (2, 8), (1, 128)):
        d = rng.integers(0, N, size=M) / N
        plan, lay, vals, offs = plan_for(darb, W, d, 0.2, bmin, bmax)
        say(f"edge rows b in [{bmin}, {bmax}]")
        quantize_both(darb, plan, lay, vals)


@pytest.mark.parametrize("seed", range(4))
def test_quantize_random_layouts_fp16(darb, seed):
    rng = np.random.default_rng(40 + seed)
    M, N = int(rng.integers(1, 300)), int(rng.integers(1, 5000))
    W = (rng.standard_normal((M, N)) * np.exp(rng.uniform(-8, 4, size=(M, 1)))).astype(np.float16)
    d = rng.integers(0, N + 1, size=M) / N
    plan, lay, vals, offs = plan_for(darb, W, d, 0.1, 1, 128)
    say(f"fp16 random layout {M}x{N}")
    quantize_both(darb, plan, lay, vals)


@pytest.mark.parametrize("B", [1, 2, 3, 4, 8, 16, 24, 32, 33, 64, 65])
@pytest.mark.parametrize("xdt", [np.float32, np.float16])
def test_i8_spmm_batches(darb, B, xdt):
    rng = np.random.default_rng(B + 11)
    M, N = 300, 2048
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = plan_for(darb, W, d, 0.1, 1, 128)
    q, s = quantize_both(darb, plan, lay, vals)
    qd, sd, od = dev(q), dev(s), dev(offs)
    packed = plan.pack_offsets(od)
    X = rng.standard_normal((N, B)).astype(xdt)
    Y8 = host(plan.spmm_i8(qd, sd, dev(X), offsets=od))
    Yp = host(plan.spmm_i8(qd, sd, dev(X), packed=packed))
    assert np.array_equal(Y8.view(np.uint32), Yp.view(np.uint32))
    check_i8_product(Y8, q, s, offs, lay, X, f"spmm_i8 B={B} x={np.dtype(xdt).name}")
    if B == 1:
        y = host(plan.spmv_i8(qd, sd, dev(X[:, 0].copy()), offsets=od))
        check_i8_product(y, q, s, offs, lay, X[:, 0], "spmv_i8")


def test_i8_misaligned_codes_use_element_paths(darb):
    # codes starting at an odd byte force the element-wise paths of both products
    rng = np.random.default_rng(9)
    M, N = 77, 1000
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = rng.integers(0, N, size=M) / N
    plan, lay, vals, offs = plan_for(darb, W, d, 0.1, 2, 128)
    q, s = quantize_both(darb, plan, lay, vals)
    qbig = dev(np.concatenate([[0], q]).astype(np.int8))[1:]
    sd, od = dev(s), dev(offs)
    x = rng.standard_normal(N).astype(np.float32)
    check_i8_product(host(plan.spmv_i8(qbig, sd, dev(x), offsets=od)), q, s, offs, lay, x,
                     "misaligned spmv_i8")
    X = rng.standard_normal((N, 5)).astype(np.float32)
    check_i8_product(host(plan.spmm_i8(qbig, sd, dev(X), offsets=od)), q, s, offs, lay, X,
                     "misaligned spmm_i8")


def test_i8_argument_errors(darb):
    rng = np.random.default_rng(2)
    W = rng.standard_normal((10, 64)).astype(np.float32)
    plan, lay, vals, offs = plan_for(darb, W, np.full(10, 0.25), 0.25, 4, 4)
    q, s = plan.quantize_i8(dev(vals))
    od = dev(offs)
    packed = plan.pack_offsets(od)
    x = dev(rng.standard_normal(64).astype(np.float32))
    y = torch.empty(10, dtype=torch.float32, device="cuda")
    L = darb.lib()
    P = ctypes.c_void_p
    st = P(torch.cuda.current_stream().cuda_stream)
    both = L.darb_spmv_i8(plan.handle, P(q.data_ptr()), P(s.data_ptr()), P(od.data_ptr()),
                          P(packed.data_ptr()), darb.F32, P(x.data_ptr()), P(y.data_ptr()), st)
    assert both == darb.E_INVALID
    no_scales = L.darb_spmv_i8(plan.handle, P(q.data_ptr()), None, P(od.data_ptr()), None,
                               darb.F32, P(x.data_ptr()), P(y.data_ptr()), st)
    assert no_scales == darb.E_INVALID
    no_words = L.darb_spmv_i8(plan.handle, P(q.data_ptr()), P(s.data_ptr()), None, None,
                              darb.F32, P(x.data_ptr()), P(y.data_ptr()), st)
    assert no_words == darb.E_INVALID                      # the plan has packed words
    bad_dtype = L.darb_spmv_i8(plan.handle, P(q.data_ptr()), P(s.data_ptr()), P(od.data_ptr()),
                               None, 7, P(x.data_ptr()), P(y.data_ptr()), st)
    assert bad_dtype == darb.E_DTYPE
    assert L.darb_quantize_i8(plan.handle, 5, P(od.data_ptr()), P(q.data_ptr()),
                              P(s.data_ptr()), st) == darb.E_DTYPE
    with pytest.raises(ValueError):
        plan.spmv_i8(q, s, x)                               # neither offsets nor packed
