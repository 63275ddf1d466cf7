"""GPU parity of the bit-packed offsets (section 4.2: log2 b bits per index).

The pack and unpack kernels are compared bit for bit with the oracle's packing;
the products that read packed offsets must equal the byte-offset products bit
for bit (only the offset source differs) and the oracle within the product
tolerance.
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

TOL = {np.dtype(np.float32): 1e-5, np.dtype(np.float16): 2e-3}


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


def check_product(Y, vals, offs, lay, X, wdtype, label):
    compare(Y, oracle.spmm(vals, offs, lay, X), oracle.spmm_absdot(vals, offs, lay, X),
            TOL[np.dtype(wdtype)], label)


def setup(darb, W, d, D, bmin, bmax):
    M, N = W.shape
    plan = darb.Plan(M, N, d, D, darb.ROUND_FLOOR, bmin, bmax).upload()
    lay = oracle.plan(N, d, D, oracle.ROUND_FLOOR, bmin, bmax)
    vals, offs = oracle.encode(W, lay)
    return plan, lay, vals, offs


def pack_both(darb, plan, lay, offs):
    """GPU pack and unpack against the oracle, bit for bit; returns the packed tensor."""
    ref = oracle.pack_offsets(offs, lay)
    assert plan.packed_words == ref.size
    packed = plan.pack_offsets(dev(offs))
    got = host(packed)[:ref.size].view(np.uint32)
    assert np.array_equal(got, ref), "packed words differ from the oracle"
    back = host(plan.unpack_offsets(dev(ref.view(np.int32)) if ref.size else packed))
    assert np.array_equal(back, offs), "unpacked offsets differ"
    return packed


@pytest.mark.parametrize("name", ["lstm_tiny", "lstm_1024", "gru_1536", "fc_9216"])
def test_config_pack_and_packed_products(darb, name):
    cfg, mi, x, X = workloads.make_config(name, seed=0)
    say(f"{name}: pack {cfg.M}x{cfg.N}")
    plan, lay, vals, offs = setup(darb, mi.W, mi.row_density, mi.matrix_density, cfg.b_min,
                                  cfg.b_max)
    packed = pack_both(darb, plan, lay, offs)
    bits = 32.0 * plan.packed_words / plan.nnz
    say(f"{name}: {plan.packed_words} words, {bits:.2f} bits per index")
    vd, od = dev(vals), dev(offs)
    y8 = host(plan.spmv(vd, od, dev(x)))
    yp = host(plan.spmv_packed(vd, packed, dev(x)))
    assert np.array_equal(y8.view(np.uint32), yp.view(np.uint32)), "spmv packed != byte form"
    check_product(yp, vals, offs, lay, x, mi.W.dtype, f"{name} spmv packed")
    Xd = dev(X)
    Y8 = host(plan.spmm(vd, od, Xd))
    Yp = host(plan.spmm_packed(vd, packed, Xd))
    assert np.array_equal(Y8.view(np.uint32), Yp.view(np.uint32)), "spmm packed != byte form"
    check_product(Yp, vals, offs, lay, X, mi.W.dtype, f"{name} spmm packed B={X.shape[1]}")


@pytest.mark.parametrize("seed", range(6))
def test_random_layouts_every_block_size(darb, seed):
    # every block size 1 ... 128 in one plan, ragged N, group sizes that leave
    # partial runs of 32
    rng = np.random.default_rng(100 + seed)
    M, N = int(rng.integers(8, 120)), int(rng.integers(1, 3000))
    say(f"random layout seed {seed}: {M}x{N}")
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = np.array([1.0 / (1 << int(rng.integers(0, 8))) for _ in range(M)])
    d[rng.random(M) < 0.1] = 0.0
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 1, 128)
    packed = pack_both(darb, plan, lay, offs)
    x = rng.standard_normal(N).astype(np.float32)
    vd, od = dev(vals), dev(offs)
    assert np.array_equal(host(plan.spmv(vd, od, dev(x))),
                          host(plan.spmv_packed(vd, packed, dev(x))))


@pytest.mark.parametrize("B", [1, 2, 3, 4, 8, 16, 33, 64, 65])
@pytest.mark.parametrize("wx", [("f32", "f32"), ("f16", "f16"), ("f16", "f32")])
def test_packed_spmm_batches(darb, B, wx):
    # B <= 4 (fp32) / 8 (fp16) puts one lane on a row, which loads 16 consecutive
    # indices at once (two 8-index windows of the packed form)
    dt = {"f32": np.float32, "f16": np.float16}
    wdt, xdt = dt[wx[0]], dt[wx[1]]
    say(f"packed spmm B={B} w={wx[0]} x={wx[1]}")
    rng = np.random.default_rng(B + 7)
    M, N = 300, 2048
    W = rng.standard_normal((M, N)).astype(wdt)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 1, 128)
    packed = pack_both(darb, plan, lay, offs)
    X = rng.standard_normal((N, B)).astype(xdt)
    vd, od, Xd = dev(vals), dev(offs), dev(X)
    Y8 = host(plan.spmm(vd, od, Xd))
    Yp = host(plan.spmm_packed(vd, packed, Xd))
    assert np.array_equal(Y8.view(np.uint32), Yp.view(np.uint32))
    check_product(Yp, vals, offs, lay, X, wdt, f"packed B={B}")


def test_packed_misaligned_values_scalar_paths(darb):
    # values starting at an odd element force the element-wise (scalar) paths of
    # both products; the packed words are read per weight there
    say("packed products, values at an odd element")
    rng = np.random.default_rng(21)
    M, N = 77, 1000
    W = rng.standard_normal((M, N)).astype(np.float32)
    d = rng.integers(0, N, size=M) / N
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 2, 128)
    packed = pack_both(darb, plan, lay, offs)
    vbig = dev(np.concatenate([[0.0], vals]).astype(np.float32))[1:]
    x = rng.standard_normal(N).astype(np.float32)
    check_product(host(plan.spmv_packed(vbig, packed, dev(x))), vals, offs, lay, x, np.float32,
                  "misaligned spmv packed")
    X = rng.standard_normal((N, 3)).astype(np.float32)
    check_product(host(plan.spmm_packed(vbig, packed, dev(X))), vals, offs, lay, X, np.float32,
                  "misaligned spmm packed")


def _shifted(a: np.ndarray, shift: int):
    """A device copy of `a` starting `shift` elements into its buffer (misaligned)."""
    t = torch.zeros(a.size + shift, dtype=dev(a[:1]).dtype, device="cuda")
    t[shift:].copy_(dev(a))
    return t[shift:]


@pytest.mark.parametrize("case", [(300, 2048, "f32"), (300, 2048, "f16"), (77, 1000, "f32"),
                                  (20000, 2048, "f32"), (300, 2048, "i8")])
def test_spmv_bits_depend_on_the_plan_only(darb, case):
    # a row's lanes and their order follow the plan alone: values, offsets and x
    # aligned or not (vector or element loads, the row-block or the general kernel),
    # byte or packed offsets, one-pass or looping launches (20000 rows) -- same bits
    M, N, kind = case
    say(f"spmv bits across forms and alignments: {M}x{N} {kind}")
    rng = np.random.default_rng(M + N)
    W = rng.standard_normal((M, N)).astype(np.float16 if kind == "f16" else np.float32)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 2, 128)
    packed = plan.pack_offsets(dev(offs))
    x = rng.standard_normal(N).astype(np.float32)
    xs = [dev(x), _shifted(x, 1)]
    if kind == "i8":
        q, s = oracle.quantize_i8(vals, lay)
        ws = [dev(q), _shifted(q, 1)]
        run = lambda w, o, p, xx: plan.spmv_i8(w, dev(s), xx, offsets=o, packed=p)
        ref = oracle.spmm_i8(q, s, offs, lay, x)
        scale = oracle.spmm_i8_absdot(q, s, offs, lay, x)
    else:
        ws = [dev(vals), _shifted(vals, 1)]
        run = lambda w, o, p, xx: plan.spmv(w, o, xx) if p is None else plan.spmv_packed(w, p, xx)
        ref = oracle.spmm(vals, offs, lay, x)
        scale = oracle.spmm_absdot(vals, offs, lay, x)
    outs = {}
    for wi, w in enumerate(ws):
        for xi, xx in enumerate(xs):
            outs[("bytes", wi, xi)] = host(run(w, dev(offs), None, xx))
            outs[("bytes, offsets shifted", wi, xi)] = host(run(w, _shifted(offs, 1), None, xx))
            outs[("packed", wi, xi)] = host(run(w, None, packed, xx))
    first = outs[("bytes", 0, 0)]
    compare(first, ref, scale, 2e-3 if kind == "f16" else 1e-5, f"{case}")
    for key, y in outs.items():
        assert np.array_equal(y.view(np.uint32), first.view(np.uint32)), key


@pytest.mark.parametrize("B", [3, 16, 64])
@pytest.mark.parametrize("kind", ["f32", "f16", "i8"])
def test_spmm_bits_depend_on_the_plan_only(darb, B, kind):
    # the L2-gather SpMM: values and byte offsets aligned or not (vector or element
    # pair loads), packed offsets, X rows padded to any width -- same bits
    M, N = 300, 2048
    say(f"spmm bits across forms and alignments: B={B} {kind}")
    rng = np.random.default_rng(7 * B)
    W = rng.standard_normal((M, N)).astype(np.float16 if kind == "f16" else np.float32)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 2, 128)
    packed = plan.pack_offsets(dev(offs))
    X = rng.standard_normal((N, B)).astype(np.float32)
    if kind == "i8":
        q, sc = oracle.quantize_i8(vals, lay)
        ws, scd = (dev(q), _shifted(q, 1)), dev(sc)
        run = lambda w, o, p, Xd: plan.spmm_i8(w, scd, Xd, offsets=o, packed=p)
        ref = oracle.spmm_i8(q, sc, offs, lay, X)
        scale = oracle.spmm_i8_absdot(q, sc, offs, lay, X)
    else:
        ws = (dev(vals), _shifted(vals, 1))
        run = lambda w, o, p, Xd: (plan.spmm(w, o, Xd) if p is None
                                   else plan.spmm_packed(w, p, Xd))
        ref = oracle.spmm(vals, offs, lay, X)
        scale = oracle.spmm_absdot(vals, offs, lay, X)
    first = None
    for pad in (0, 1):
        Xbig = np.zeros((N, B + pad), dtype=np.float32)
        Xbig[:, :B] = X
        Xd = dev(Xbig)[:, :B]
        for w in ws:
            for label, o, p in (("bytes", dev(offs), None), ("bytes, offsets shifted",
                                 _shifted(offs, 1), None), ("packed", None, packed)):
                y = host(run(w, o, p, Xd))
                if first is None:
                    first = y
                    compare(y, ref, scale, 2e-3 if kind == "f16" else 1e-5, f"B={B} {kind}")
                assert np.array_equal(y.view(np.uint32), first.view(np.uint32)), (pad, label)


@pytest.mark.parametrize("case", [(4100, "f32"), (4098, "f32"), (4100, "f16")])
def test_wide_spmm_bits_depend_on_the_plan_only(darb, case):
    # the LDS-slab SpMM (N = 1024, B >= 4096) is chosen from the plan and B alone:
    # values and byte offsets aligned or not (vector or element loads), packed
    # offsets, X rows padded to any width (staged as vectors or element by element),
    # B not a multiple of 4 -- same bits
    B, kind = case
    M, N = 200, 1024
    say(f"wide spmm bits across forms and alignments: B={B} {kind}")
    rng = np.random.default_rng(B)
    W = rng.standard_normal((M, N)).astype(np.float16 if kind == "f16" else np.float32)
    d = rng.integers(0, N // 3, size=M) / N
    plan, lay, vals, offs = setup(darb, W, d, 0.1, 1, 64)
    packed = plan.pack_offsets(dev(offs))
    X = rng.standard_normal((N, B)).astype(np.float32)
    first = None
    for pad in (0, 4, 2, 1):
        Xbig = np.zeros((N, B + pad), dtype=np.float32)
        Xbig[:, :B] = X
        Xd = dev(Xbig)[:, :B]
        for w in (dev(vals), _shifted(vals, 1)):
            for label, Y in (("bytes", lambda: plan.spmm(w, dev(offs), Xd)),
                             ("bytes, offsets shifted", lambda: plan.spmm(w, _shifted(offs, 1), Xd)),
                             ("packed", lambda: plan.spmm_packed(w, packed, Xd))):
                y = host(Y())
                if first is None:
                    first = y
                    compare(y, oracle.spmm(vals, offs, lay, X),
                            oracle.spmm_absdot(vals, offs, lay, X),
                            2e-3 if kind == "f16" else 1e-5, f"wide B={B} {kind}")
                assert np.array_equal(y.view(np.uint32), first.view(np.uint32)), (pad, label)


def test_packed_all_b_one_has_no_words(darb):
    # b = 1 everywhere: every index is 0, the packed form is empty and the C ABI
    # accepts a NULL packed pointer
    say("packed, b = 1 everywhere (NULL packed)")
    rng = np.random.default_rng(5)
    M, N = 20, 130
    W = rng.standard_normal((M, N)).astype(np.float32)
    plan, lay, vals, offs = setup(darb, W, np.ones(M), 1.0, 1, 1)
    assert plan.packed_words == 0
    L = darb.lib()
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    vd, x = dev(vals), dev(rng.standard_normal(N).astype(np.float32))
    y = torch.empty(M, dtype=torch.float32, device="cuda")
    assert L.darb_spmv_packed(plan.handle, darb.F32, ctypes.c_void_p(vd.data_ptr()), None,
                              darb.F32, ctypes.c_void_p(x.data_ptr()),
                              ctypes.c_void_p(y.data_ptr()), s) == 0
    check_product(host(y), vals, offs, lay, host(x), np.float32, "b=1 spmv packed")
    o = torch.full((plan.nnz,), 7, dtype=torch.uint8, device="cuda")
    assert L.darb_unpack_offsets(plan.handle, None, ctypes.c_void_p(o.data_ptr()), s) == 0
    assert not host(o).any()
    assert L.darb_pack_offsets(plan.handle, ctypes.c_void_p(o.data_ptr()), None, s) == 0


def test_packed_rejects_null_when_words_exist(darb):
    rng = np.random.default_rng(6)
    W = rng.standard_normal((10, 64)).astype(np.float32)
    plan, lay, vals, offs = setup(darb, W, np.full(10, 0.25), 0.25, 4, 4)
    assert plan.packed_words > 0
    L = darb.lib()
    buf = ctypes.c_void_p(dev(vals).data_ptr())
    assert L.darb_spmv_packed(plan.handle, darb.F32, buf, None, darb.F32, buf, buf,
                              None) == darb.E_INVALID
    assert L.darb_pack_offsets(plan.handle, buf, ctypes.c_void_p(buf.value + 2),
                               None) == darb.E_INVALID          # packed not 4-byte aligned
