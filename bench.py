#!/usr/bin/env python3
"""DARB benchmark on one MI355X: SpMV (batch 1) and SpMM (batch 64) over the DARB format.

Workload: the FC-head matrix (W fp32 [4096 x 9216], Laplace weights, 4 % irregular
keep, block sizes 8..128), encoded on the device with BMWM.  The metric is the
products' effective bandwidth and rate: ``value`` is the SpMV's algorithmic bytes
divided by its average kernel time, in GB/s; the SpMM (B = 64) figures and the
whole step's are extra keys.

One step (the timed loop, ``ms_per_step``) is one pass of the whole hot path:
    darb_encode(W)  ->  darb_spmv(x)  ->  darb_spmm(X, B = 64)
Inputs are resident in HBM before any timed region.  To measure HBM rather than
the 256 MB Infinity Cache, every launch reads buffers not touched recently: W
rotates over ``--rotate-w`` copies (151 MB each) and the format and activations
over ``--rotate-fmt`` copies (>= 64, over 540 MB); the products of step i read
the copy encoded several steps earlier (identical contents).

Per-kernel times: for each kernel, at least 256 launches (whatever ``--steps``
says) rotating over the same copies are enqueued behind a sleep kernel, so the
host's enqueue cost cannot starve the GPU, and timed with HIP events on the
launch stream; the average per launch is what the rocprofv3 kernel trace shows
for the same kernel.  The same-size read floor is the fastest of several launch
shapes of a plain read over buffers of the SpMV's size, same rotation.

Prints one JSON line.
"""
import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X published HBM3E bandwidth
# X-row gathers of the SpMM go through each CU's load path at 128 bytes per clock:
# 256 CUs x 128 B x 2.4 GHz
GATHER_PEAK_GBPS = 256 * 128 * 2.4
MIN_LAUNCHES = 256
MIN_ROTATION_BYTES = 512 << 20  # > 2x the 256 MB Infinity Cache

METRIC = "DARB SpMV/SpMM effective GB/s (% of HBM peak) and GFLOP/s, batch 1 & 64"

READ_SHAPES = [(256, 1), (256, 2), (256, 4), (256, 8), (512, 1), (512, 2), (512, 4),
               (1024, 1), (1024, 2), (64, 4), (128, 4)]


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="fc_9216")
    ap.add_argument("--batch", type=int, default=None,
                    help="SpMM batch (default: the workload's own; 64 for fc_9216)")
    ap.add_argument("--rotate-w", type=int, default=4)
    ap.add_argument("--rotate-fmt", type=int, default=64)
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="budget of the oracle timing on the host (0 disables)")
    ap.add_argument("--no-recurrent", action="store_true",
                    help="skip the recurrent-workload figures in the default line")
    ap.add_argument("--seed", type=int, default=0)
    return ap.parse_args(argv)


def step_bytes(M, N, nnz, s_w, s_x, B):
    """Algorithmic bytes of each kernel: the format, x or X and y or Y once each (and
    W once for the encode), the row order and the per-row table."""
    enc = M * N * s_w + nnz * (s_w + 1) + 4 * M
    spmv = nnz * (s_w + 1) + N * s_x + 4 * M + 4 * M
    spmm = nnz * (s_w + 1) + N * B * s_x + 4 * M * B + 4 * M
    return {"encode": enc, "spmv": spmv, "spmm": spmm}


# source file of each measured kernel; its local includes (the public header among them),
# the C-ABI layer that lays out the plan and the compile flags are hashed with it
KERNEL_SOURCES = {"encode": "encode.hip", "pack": "packed.hip", "spmv": "product.hip",
                  "spmm": "product.hip", "spmv_packed": "product.hip",
                  "spmm_packed": "product.hip", "prune": "prune.hip",
                  "quantize_i8": "product_i8.hip", "spmv_i8": "product_i8.hip",
                  "spmv_i8_packed": "product_i8.hip", "spmm_i8_packed": "product_i8.hip"}


def kernel_sha256(kernel):
    """Hash of the sources a kernel is built from, to tell whether stored counters of
    that kernel still apply; None for a kernel with no known source."""
    import hashlib
    import re
    src = KERNEL_SOURCES.get(kernel)
    if src is None:
        return None
    from paper_1911_08020_amd import build as _build
    pkg = os.path.join(ROOT, "paper_1911_08020_amd")
    dirs = (os.path.join(pkg, "csrc"), os.path.join(ROOT, "include"))
    todo, seen = [src, "api.cpp"], {"compile flags": repr(_build.HIPCC_FLAGS).encode()}
    while todo:
        name = todo.pop(0)
        if name in seen:
            continue
        path = next(os.path.join(d, name) for d in dirs if os.path.exists(os.path.join(d, name)))
        with open(path, "rb") as f:
            seen[name] = f.read()
        todo += [m.decode() for m in re.findall(rb'#include\s+"([^"]+)"', seen[name])]
    h = hashlib.sha256()
    for name in sorted(seen):
        h.update(name.encode())
        h.update(seen[name])
    return h.hexdigest()


def stored_traffic(workload, batch):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, for each kernel
    whose sources are unchanged since the counters were taken; {} when the summary is
    missing or was taken on another workload."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.txt")
    if batch != 64 or not os.path.exists(path):
        return {}
    out = {}
    with open(path) as f:
        for ln in f:
            ln = ln.strip()
            if ln.startswith("kernel="):
                kv = dict(t.split("=", 1) for t in ln.split())
                if kv.get("sources_sha256") == kernel_sha256(kv["kernel"]):
                    out[kv["kernel"]] = int(kv["traffic_bytes"])
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(cfg, mi, x, X, seconds, nbytes):
    """The oracle as it stands (plain C, fp64 sums) on the same workload: encode, SpMV
    and SpMM (B = X's columns), each the median of >= 5 runs, on one thread and with
    the rows split over every core this process may use (threads calling the oracle
    on disjoint row ranges; the oracle's arithmetic is unchanged).  A reported
    baseline, not a target."""
    import statistics
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    lay = oracle.plan(cfg.N, mi.row_density, mi.matrix_density, oracle.ROUND_FLOOR,
                      cfg.b_min, cfg.b_max)
    affinity = len(os.sched_getaffinity(0))
    cores = min(affinity, 16)       # the host share of one GPU on the test boxes
    W = np.ascontiguousarray(mi.W)
    v, o = oracle.encode(W, lay)
    ranges = {1: [(0, cfg.M)]}
    step = -(-cfg.M // cores)
    ranges[cores] = [(r, min(cfg.M, r + step)) for r in range(0, cfg.M, step)]
    budget = seconds / 6.0      # per op and thread count

    def run(threads, op):
        rs = ranges[threads]
        pool = ThreadPoolExecutor(max_workers=threads)
        try:
            if op == "encode":
                vv, oo = np.zeros_like(v), np.zeros_like(o)
                fn = lambda r: oracle.encode_rows(W, lay, r[0], r[1], vv, oo)   # noqa: E731
            else:
                act = x if op == "spmv" else X
                Y = np.zeros((cfg.M, 1 if act.ndim == 1 else act.shape[1]), dtype=np.float64)
                fn = lambda r: oracle.spmm_rows(v, o, lay, act, r[0], r[1], Y)   # noqa: E731
            times = []
            t_end = time.perf_counter() + budget
            while len(times) < 5 or (time.perf_counter() < t_end and len(times) < 50):
                t0 = time.perf_counter()
                list(pool.map(fn, rs))
                times.append(time.perf_counter() - t0)
            return statistics.median(times), len(times)
        finally:
            pool.shutdown()

    per_op = {}
    for threads in sorted(ranges):
        for op in ("encode", "spmv", "spmm"):
            t, n = run(threads, op)
            per_op[f"{op}_{threads}t"] = {"median_ms": round(t * 1e3, 3), "runs": n,
                                          "gbps": round(nbytes[op] / t / 1e9, 3)}
    best = per_op[f"spmv_{cores}t"]
    return {"value": best["gbps"], "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"{cfg.name} SpMV (B=1) over the full matrix, rows split over {cores} "
                      f"threads, median of {best['runs']} runs; the oracle's fp64 loops as "
                      f"they stand; CPU: {cpu_model()}",
            "cpu_model": cpu_model(), "affinity_cores": affinity, "per_op": per_op}


class Timer:
    """Average per-launch GPU time of back-to-back launches, HIP events on the launch
    stream.  The launches are enqueued behind a sleep kernel long enough to cover the
    host's enqueue time, so the GPU runs them back to back."""

    def __init__(self, torch, stream):
        self.torch, self.stream = torch, stream
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        torch.cuda._sleep(1 << 20)
        e1.record(stream)
        torch.cuda.synchronize()
        self.cycles_per_us = (1 << 20) / (e0.elapsed_time(e1) * 1e3)

    def __call__(self, fn, args_list, count, host_us_per_call=30.0):
        torch = self.torch
        rc = fn(*args_list[0])                       # first launch loads the code object
        if rc:
            raise RuntimeError(f"launch failed ({rc})")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        torch.cuda._sleep(int(self.cycles_per_us * host_us_per_call * count))
        e0.record(self.stream)
        for i in range(count):
            rc |= fn(*args_list[i % len(args_list)])
        e1.record(self.stream)
        torch.cuda.synchronize()
        if rc:
            raise RuntimeError(f"launch failed ({rc})")
        return e0.elapsed_time(e1) * 1e3 / count


def recurrent_figures(args, with_cpu):
    """The recurrent workload: 2-layer LSTM, hidden 1024, T = 200, batch 32, fp16 DARB
    weights, fp32 state.  One sequence = both layers (darb_lstm_layer each).  The
    weights are encoded once before timing (model load) and stay cache-resident, as
    in a serving loop.  Returns tokens/s, the per-step time of the fused step kernel
    and the two products' times."""
    import ctypes

    import torch

    import paper_1911_08020_amd as darb
    import workloads

    dev = torch.device("cuda", 0)
    cfg, mats, xs, shp = workloads.make_lstm_inputs(seed=args.seed)
    H, T, Bt = shp["hidden"], shp["seq_len"], shp["batch"]
    layers, nnz = [], []
    for (wih, whh) in mats:
        pair = []
        for mi in (wih, whh):
            plan = darb.Plan(4 * H, H, mi.row_density, mi.matrix_density, darb.ROUND_FLOOR,
                             cfg.b_min, cfg.b_max).upload()
            v, o = plan.encode(torch.from_numpy(mi.W).to(dev))
            pair.append((plan, v, o))
            nnz.append(plan.nnz)
        layers.append(tuple(pair))
    x_seq = torch.from_numpy(xs).to(dev)
    hs = [torch.empty((H, T * Bt), dtype=torch.float32, device=dev) for _ in layers]
    hh = [torch.zeros((H, Bt), dtype=torch.float32, device=dev) for _ in layers]
    cc = [torch.zeros((H, Bt), dtype=torch.float32, device=dev) for _ in layers]
    ws = torch.empty(darb.lstm_workspace_floats(H, T, Bt), dtype=torch.float32, device=dev)

    def sequence():
        inp = x_seq
        for l, (wih, whh) in enumerate(layers):
            hh[l].zero_()
            cc[l].zero_()
            darb.lstm_layer(wih, whh, inp, H, T, Bt, h=hh[l], c=cc[l], h_seq=hs[l], workspace=ws)
            inp = hs[l]

    sequence()
    torch.cuda.synchronize()
    ref = hs[-1].clone()
    K = max(3, args.steps // 20)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        sequence()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / K
    assert torch.equal(hs[-1], ref), "sequence output changed across runs"

    stream = torch.cuda.current_stream()
    timer = Timer(torch, stream)
    lib = darb.lib()
    P = ctypes.c_void_p
    Uo = torch.empty((4 * H, T * Bt), dtype=torch.float32, device=dev)
    Go = torch.empty((4 * H, Bt), dtype=torch.float32, device=dev)
    res = {}
    for name, (pl, vv, oo), X, Y, B, reps in (("input_product", layers[0][0], x_seq, Uo, T * Bt, 20),
                                              ("recurrent_product", layers[0][1], hh[0], Go, Bt,
                                               MIN_LAUNCHES)):
        a = [(pl.handle, darb.F16, P(vv.data_ptr()), P(oo.data_ptr()), darb.F32, B,
              P(X.data_ptr()), B, P(Y.data_ptr()), B, P(stream.cuda_stream))]
        us = timer(lib.darb_spmm, a, reps)
        res[name] = {"avg_us": round(us, 3), "batch": B,
                     "gflops": round(2 * pl.nnz * B / (us * 1e-6) / 1e9, 1)}
    # the fused time step: the layer's time minus its input product, over T steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wih, whh = layers[0]
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(3):
        darb.lstm_layer(wih, whh, x_seq, H, T, Bt, h=hh[0], c=cc[0], h_seq=hs[0], workspace=ws)
    e1.record(stream)
    torch.cuda.synchronize()
    layer_us = e0.elapsed_time(e1) * 1e3 / 3
    step_us = (layer_us - res["input_product"]["avg_us"]) / T
    out = {"workload": "lstm2_seq: 2-layer LSTM, hidden 1024, T=200, batch 32, W_ih and W_hh "
                       "[4096 x 1024] fp16 DARB (keep 5 %, b 4..64), fp32 state",
           "tokens_per_s": round(T * Bt / (ms * 1e-3), 1), "ms_per_sequence": round(ms, 4),
           "sequences": K, "us_per_step": round(step_us, 3),
           "gflops": round(sum(2 * n * T * Bt for n in nnz) / (ms * 1e-3) / 1e9, 1),
           "nnz_per_matrix": nnz, "kernels": res}
    if with_cpu:
        import oracle
        masked = []
        for (wih, whh) in layers:
            pair = []
            for (pl, vv, oo) in (wih, whh):
                log2b, row_start, perm = pl.export()
                lay = oracle.layout(pl.N, log2b)
                pair.append(oracle.decode(vv.cpu().numpy(), oo.cpu().numpy(), lay))
            masked.append(tuple(pair))
        from threadpoolctl import threadpool_limits
        cores = len(os.sched_getaffinity(0))
        with threadpool_limits(limits=cores):
            t0 = time.perf_counter()
            oracle.lstm_forward(masked, xs, H, T, Bt)
            el = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(T * Bt / el, 1), "unit": "tokens/s",
                               "cores": cores, "kind": "oracle",
                               "sample": f"one full sequence in {el:.1f} s (numpy fp64 dense "
                                         f"masked products, {cores} BLAS threads)"}
    return out


def bench_lstm(args):
    """``--workload lstm2_seq``: the recurrent workload as the headline."""
    import torch
    torch.cuda.set_device(0)
    r = recurrent_figures(args, with_cpu=args.cpu_seconds > 0)
    out = {
        "metric": "DARB 2-layer LSTM forward tokens/s (hidden 1024, T=200, batch 32)",
        "value": r["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": r["sequences"],
        "warmup": 1, "ms_per_step": r["ms_per_sequence"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic: seeded fp16 weights, exact-k irregular densities, N(0,1) inputs",
        "config": {"workload": r["workload"] + "; step = one forward pass over the sequence",
                   "nnz_per_matrix": r["nnz_per_matrix"]},
        "gflops_step": r["gflops"], "us_per_time_step": r["us_per_step"], "kernels": r["kernels"],
        "roofline": None, "cpu_baseline": r.get("cpu_baseline"),
    }
    print(json.dumps(out), flush=True)


def main(argv=None):
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the DARB path here runs on a single MI355X and has "
              "no multi-GPU mode (rows would shard across GPUs with no communication). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.workload == "lstm2_seq":
        return bench_lstm(args)

    import ctypes

    import numpy as np
    import torch

    import paper_1911_08020_amd as darb
    import workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    cfg, mi, x, X = workloads.make_config(args.workload, seed=args.seed, batch=args.batch)
    B = X.shape[1]
    t0 = time.perf_counter()
    plan = darb.Plan(cfg.M, cfg.N, mi.row_density, mi.matrix_density, darb.ROUND_FLOOR,
                     cfg.b_min, cfg.b_max)
    plan_ms = (time.perf_counter() - t0) * 1e3
    plan.upload()
    wdt = torch.float32 if cfg.wdtype == "f32" else torch.float16
    s_w = 4 if cfg.wdtype == "f32" else 2
    s_x = 4 if cfg.xdtype == "f32" else 2
    RW, RE = args.rotate_w, args.rotate_fmt
    with_spmm = B > 1

    Wd = [torch.from_numpy(mi.W).to(dev) for _ in range(RW)]
    fmt = [plan.empty_format(wdt, dev) for _ in range(RE)]
    xd = [torch.from_numpy(x).to(dev) for _ in range(RE)]
    Xd = [torch.from_numpy(X).to(dev) for _ in range(RE)] if with_spmm else []
    y = torch.empty(cfg.M, dtype=torch.float32, device=dev)
    Y = torch.empty((cfg.M, B), dtype=torch.float32, device=dev)
    for v, o in fmt:
        plan.encode(Wd[0], v, o)
    torch.cuda.synchronize()

    # Pre-bound C-ABI calls: the timed loops only enqueue (argument checks done once
    # by the binding above; the library checks again on every call).
    lib = darb.lib()
    h = plan.handle
    wcode = darb.F32 if cfg.wdtype == "f32" else darb.F16
    xcode = darb.F32 if cfg.xdtype == "f32" else darb.F16
    P = ctypes.c_void_p
    stream = torch.cuda.current_stream()
    sp = P(stream.cuda_stream)
    enc_args = [(h, wcode, P(Wd[i % RW].data_ptr()), cfg.N, P(fmt[i % RE][0].data_ptr()),
                 P(fmt[i % RE][1].data_ptr()), sp) for i in range(RW * RE)]
    spmv_args = [(h, wcode, P(fmt[j][0].data_ptr()), P(fmt[j][1].data_ptr()), xcode,
                  P(xd[j].data_ptr()), P(y.data_ptr()), sp) for j in range(RE)]
    spmm_args = [(h, wcode, P(fmt[j][0].data_ptr()), P(fmt[j][1].data_ptr()), xcode, B,
                  P(Xd[j].data_ptr()), B, P(Y.data_ptr()), B, sp) for j in range(RE)] \
        if with_spmm else []

    def step(i):
        rc = lib.darb_encode(*enc_args[i % (RW * RE)])
        rc |= lib.darb_spmv(*spmv_args[(i + 7) % RE])
        if with_spmm:
            rc |= lib.darb_spmm(*spmm_args[(i + 13) % RE])
        if rc:
            raise RuntimeError(f"DARB call failed: {lib.darb_last_error().decode()}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    y_ref, Y_ref = y.clone(), Y.clone()

    # timed region: exactly K steps between two synchronisations
    K = args.steps
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(K):
        step(args.warmup + i)
    t_enq = time.perf_counter()
    torch.cuda.synchronize()
    t_end = time.perf_counter()
    ms_per_step = (t_end - t_start) * 1e3 / K
    host_us = (t_enq - t_start) * 1e6 / K

    timer = Timer(torch, stream)
    NL = max(K, MIN_LAUNCHES)
    spmv_rot = [spmv_args[(i + 7) % RE] for i in range(RE)]
    avg_us = {"encode": timer(lib.darb_encode, enc_args, NL),
              "spmv": timer(lib.darb_spmv, spmv_rot, NL)}
    if with_spmm:
        avg_us["spmm"] = timer(lib.darb_spmm, [spmm_args[(i + 13) % RE] for i in range(RE)], NL)
    names = ["encode", "spmv", "spmm"] if with_spmm else ["encode", "spmv"]
    nbytes = step_bytes(cfg.M, cfg.N, plan.nnz, s_w, s_x, B)
    flops = {"encode": 0, "spmv": 2 * plan.nnz, "spmm": 2 * plan.nnz * B}
    kernels = {}
    for n in names:
        us = avg_us[n]
        gbps = nbytes[n] / (us * 1e-6) / 1e9
        kernels[n] = {
            "avg_us": round(us, 3), "launches": NL, "bytes": int(nbytes[n]),
            "flops": int(flops[n]), "gbps": round(gbps, 1),
            "frac_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
            "gflops": round(flops[n] / (us * 1e-6) / 1e9, 1),
        }
    assert torch.equal(y.view(torch.int32), y_ref.view(torch.int32)), "SpMV not deterministic"

    # HBM reference reads in the same process: the 4 GiB rate (measured peak) and the
    # fastest of several launch shapes over buffers of the SpMV's size, rotated like
    # the format (same-size floor: launch, ramp and one memory latency included)
    sink = torch.empty(8192, dtype=torch.float32, device=dev)
    big = torch.empty(1 << 30, dtype=torch.float32, device=dev)
    read_peak_us = timer(lib.darb_stream_read, [(P(big.data_ptr()), big.numel() * 4,
                                                 P(sink.data_ptr()), sp)], 5)
    read_peak = big.numel() * 4 / (read_peak_us * 1e-6) / 1e9
    del big
    small_b = nbytes["spmv"] // 16 * 16
    n_small = max(RE, -(-MIN_ROTATION_BYTES // small_b))
    smalls = [torch.empty(small_b // 4, dtype=torch.float32, device=dev) for _ in range(n_small)]
    shapes = {}
    for (th, vp) in READ_SHAPES:
        a = [(P(t.data_ptr()), small_b, th, vp, P(sink.data_ptr()), sp) for t in smalls]
        shapes[f"{th}x{vp}"] = round(timer(lib.darb_stream_read_shape, a, NL), 3)
    del smalls
    best_shape = min(shapes, key=shapes.get)
    floor_us = shapes[best_shape]
    # the same read over the encode's input: the rotated W copies themselves
    w_bytes = (Wd[0].numel() * Wd[0].element_size()) // 16 * 16
    w_read_us = timer(lib.darb_stream_read, [(P(t.data_ptr()), w_bytes, P(sink.data_ptr()), sp)
                                             for t in Wd], max(K // 4, 32))

    # the step DARB starts from, on the device: per-row counts of the k largest
    # magnitudes (radix select over W, several kernels)
    nb_ws = ctypes.c_int64()
    lib.darb_prune_workspace(cfg.M, cfg.N, wcode, ctypes.byref(nb_ws))
    prune_ws = torch.empty(nb_ws.value, dtype=torch.uint8, device=dev)
    counts = torch.empty(cfg.M, dtype=torch.int64, device=dev)
    prune_args = [(cfg.M, cfg.N, wcode, P(Wd[i].data_ptr()), cfg.N, mi.k, P(counts.data_ptr()),
                   P(prune_ws.data_ptr()), nb_ws.value, sp) for i in range(RW)]
    prune_us = timer(lib.darb_prune_counts, prune_args, max(K // 4, 32), host_us_per_call=60.0)
    prune_ok = bool(np.array_equal(counts.cpu().numpy(), mi.mask.sum(axis=1)))
    w_stream = cfg.M * cfg.N * s_w
    w_passes = 1 + 1 / 32 if w_stream >= (64 << 20) else (4 if cfg.wdtype == "f32" else 3)
    prune_ctx = {"avg_us": round(prune_us, 3), "k": mi.k, "passes_over_W": round(w_passes, 3),
                 "bytes": int(w_passes * w_stream),
                 "gbps": round(w_passes * w_stream / (prune_us * 1e-6) / 1e9, 1),
                 "x_of_W_read": round(prune_us / w_read_us, 3),
                 "counts_equal_generator": prune_ok}
    del prune_ws

    # the paper's storage form: offsets bit-packed to log2 b bits (section 4.2), the
    # conversion and both products on it; outputs equal the byte-offset products bit
    # for bit
    packed = [plan.empty_packed(dev) for _ in range(RE)]
    for j in range(RE):
        plan.pack_offsets(fmt[j][1], packed[j])
    torch.cuda.synchronize()
    pack_args = [(h, P(fmt[j][1].data_ptr()), P(packed[j].data_ptr()), sp) for j in range(RE)]
    pk_spmv = [(h, wcode, P(fmt[j][0].data_ptr()), P(packed[j].data_ptr()), xcode,
                P(xd[j].data_ptr()), P(y.data_ptr()), sp) for j in range(RE)]
    pk_spmm = [(h, wcode, P(fmt[j][0].data_ptr()), P(packed[j].data_ptr()), xcode, B,
                P(Xd[j].data_ptr()), B, P(Y.data_ptr()), B, sp) for j in range(RE)] \
        if with_spmm else []
    pw = plan.packed_words
    pk_bytes = {"pack": plan.nnz + 4 * pw,
                "spmv": plan.nnz * s_w + 4 * pw + cfg.N * s_x + 8 * cfg.M,
                "spmm": plan.nnz * s_w + 4 * pw + cfg.N * B * s_x + 4 * cfg.M * B + 4 * cfg.M}
    pk_us = {"pack": timer(lib.darb_pack_offsets, pack_args, NL)}
    lib.darb_spmv_packed(*pk_spmv[(K + args.warmup + 6) % RE])
    torch.cuda.synchronize()
    pk_same = bool(torch.equal(y.view(torch.int32), y_ref.view(torch.int32)))
    pk_us["spmv"] = timer(lib.darb_spmv_packed, pk_spmv, NL)
    if with_spmm:
        pk_us["spmm"] = timer(lib.darb_spmm_packed, pk_spmm, NL)
        lib.darb_spmm_packed(*pk_spmm[0])
        torch.cuda.synchronize()
        pk_same = pk_same and bool(torch.equal(Y.view(torch.int32), Y_ref.view(torch.int32)))
    packed_ctx = {"words": pw, "bits_per_index": round(32.0 * pw / plan.nnz, 3),
                  "format_bytes": plan.nnz * s_w + 4 * pw,
                  "equals_byte_offset_products": pk_same}
    traffic = stored_traffic(args.workload, B)
    for n, us in pk_us.items():
        gbps = pk_bytes[n] / (us * 1e-6) / 1e9
        packed_ctx[n] = {"avg_us": round(us, 3), "bytes": int(pk_bytes[n]), "gbps": round(gbps, 1),
                         "frac_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
                         "traffic_bytes": traffic.get(n if n == "pack" else n + "_packed")}

    # INT8 retained values (section 4.2's storage accounting assumes INT8 weights): the
    # per-row quantisation and both products on INT8 codes, with the packed offsets
    # (the paper's full storage form, 8 + log2 b bits per weight) and with byte offsets
    codes = [torch.empty(plan.nnz, dtype=torch.int8, device=dev) for _ in range(RE)]
    scales = [torch.empty(cfg.M, dtype=torch.float32, device=dev) for _ in range(RE)]
    for j in range(RE):
        plan.quantize_i8(fmt[j][0], codes[j], scales[j])
    torch.cuda.synchronize()
    q_args = [(h, wcode, P(fmt[j][0].data_ptr()), P(codes[j].data_ptr()),
               P(scales[j].data_ptr()), sp) for j in range(RE)]
    i8_spmv = [(h, P(codes[j].data_ptr()), P(scales[j].data_ptr()), None,
                P(packed[j].data_ptr()), xcode, P(xd[j].data_ptr()), P(y.data_ptr()), sp)
               for j in range(RE)]
    i8_spmv_b = [(h, P(codes[j].data_ptr()), P(scales[j].data_ptr()), P(fmt[j][1].data_ptr()),
                  None, xcode, P(xd[j].data_ptr()), P(y.data_ptr()), sp) for j in range(RE)]
    i8_spmm = [(h, P(codes[j].data_ptr()), P(scales[j].data_ptr()), None,
                P(packed[j].data_ptr()), xcode, B, P(Xd[j].data_ptr()), B, P(Y.data_ptr()), B,
                sp) for j in range(RE)] if with_spmm else []
    i8_us = {"quantize": timer(lib.darb_quantize_i8, q_args, NL),
             "spmv_byte_offsets": timer(lib.darb_spmv_i8, i8_spmv_b, NL),
             "spmv": timer(lib.darb_spmv_i8, i8_spmv, NL)}
    lib.darb_spmv_i8(*i8_spmv[(K + args.warmup + 6) % RE])
    torch.cuda.synchronize()
    i8_err = {"spmv": float((y - y_ref).norm() / y_ref.norm())}
    if with_spmm:
        i8_us["spmm"] = timer(lib.darb_spmm_i8, i8_spmm, NL)
        lib.darb_spmm_i8(*i8_spmm[0])
        torch.cuda.synchronize()
        i8_err["spmm"] = float((Y - Y_ref).norm() / Y_ref.norm())
    i8_fmt = plan.nnz + 4 * pw + 4 * cfg.M
    i8_bytes = {"quantize": plan.nnz * (s_w + 1) + 8 * cfg.M,
                "spmv_byte_offsets": 2 * plan.nnz + cfg.N * s_x + 12 * cfg.M,
                "spmv": i8_fmt + cfg.N * s_x + 8 * cfg.M,
                "spmm": i8_fmt + cfg.N * B * s_x + 4 * cfg.M * B + 4 * cfg.M}
    int8_ctx = {"format_bytes": i8_fmt,
                "bits_per_weight": round(8.0 * i8_fmt / plan.nnz, 3),
                "rel_rms_vs_unquantised_product": {n: round(e, 6) for n, e in i8_err.items()}}
    for n, us in i8_us.items():
        gbps = i8_bytes[n] / (us * 1e-6) / 1e9
        tkey = {"quantize": "quantize_i8", "spmv_byte_offsets": "spmv_i8"}.get(n, n + "_i8_packed")
        int8_ctx[n] = {"avg_us": round(us, 3), "bytes": int(i8_bytes[n]), "gbps": round(gbps, 1),
                       "frac_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
                       "traffic_bytes": traffic.get(tkey)}
    del packed, codes, scales

    # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE counters calibrate the
    # HBM-traffic counters of the DARB kernels (same process, same command)
    cp_src = torch.ones(16 << 20, dtype=torch.float32, device=dev)      # 64 MiB
    cp_dst = torch.empty_like(cp_src)
    for _ in range(3):
        darb.stream_copy(cp_dst, cp_src)
    torch.cuda.synchronize()
    del cp_src, cp_dst

    # the SpMV at larger sizes: the same rows tiled t times (t*M rows with the same
    # densities), format copies rotated past the cache.  A single launch pays a fixed
    # start-up and memory latency; these sizes show the rate once that is amortised,
    # for the fp32 byte-offset form and for INT8 codes with packed offsets.
    size_sweep = []
    for t in (1, 4, 16):
        Mt = cfg.M * t
        plan_t = darb.Plan(Mt, cfg.N, np.tile(mi.row_density, t), mi.matrix_density,
                           darb.ROUND_FLOOR, cfg.b_min, cfg.b_max).upload()
        fbytes = plan_t.nnz * (s_w + 1)
        reps = int(max(2, -(-MIN_ROTATION_BYTES // fbytes)))
        Wt = Wd[0].repeat(t, 1)
        fmts = [plan_t.empty_format(wdt, dev) for _ in range(reps)]
        for v_t, o_t in fmts:
            plan_t.encode(Wt, v_t, o_t)
        del Wt
        y_t = torch.empty(Mt, dtype=torch.float32, device=dev)
        sw_args = [(plan_t.handle, wcode, P(v_t.data_ptr()), P(o_t.data_ptr()), xcode,
                    P(xd[0].data_ptr()), P(y_t.data_ptr()), sp) for v_t, o_t in fmts]
        us = timer(lib.darb_spmv, sw_args, max(NL // 4, 64))
        sb = fbytes + cfg.N * s_x + 8 * Mt
        gbps = sb / (us * 1e-6) / 1e9
        entry = {"rows": Mt, "bytes": int(sb), "copies": reps, "avg_us": round(us, 3),
                 "gbps": round(gbps, 1), "frac_of_4GiB_read": round(gbps / read_peak, 4)}
        i8 = []
        for v_t, o_t in fmts:
            q_t, sc_t = plan_t.quantize_i8(v_t)
            i8.append((q_t, sc_t, plan_t.pack_offsets(o_t)))
        del fmts
        sb8 = plan_t.nnz + 4 * plan_t.packed_words + 4 * Mt + cfg.N * s_x + 8 * Mt
        reps8 = int(max(2, -(-MIN_ROTATION_BYTES // sb8)))
        while len(i8) < reps8:
            q_t, sc_t, pk_t = i8[len(i8) % reps]
            i8.append((q_t.clone(), sc_t.clone(), pk_t.clone()))
        i8_args = [(plan_t.handle, P(q_t.data_ptr()), P(sc_t.data_ptr()), None,
                    P(pk_t.data_ptr()), xcode, P(xd[0].data_ptr()), P(y_t.data_ptr()), sp)
                   for q_t, sc_t, pk_t in i8]
        us8 = timer(lib.darb_spmv_i8, i8_args, max(NL // 4, 64))
        entry["int8_packed"] = {"bytes": int(sb8), "copies": len(i8), "avg_us": round(us8, 3),
                                "gbps": round(sb8 / (us8 * 1e-6) / 1e9, 1)}
        size_sweep.append(entry)
        del i8, y_t, plan_t

    # context, not a target: the same masked matrix as a dense matrix through torch
    # (hipBLASLt / rocBLAS) and in CSR (hipSPARSE), rotated like the DARB format
    Wm = plan.decode(*fmt[0])
    dense = [Wm.clone() for _ in range(RW)]
    xs_t = [t.to(Wm.dtype) for t in xd[:16]]
    Xs_t = [t.to(Wm.dtype) for t in Xd[:16]]
    del Wm

    def timed_torch(fn, count):
        for i in range(3):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(count):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / count

    dense_ctx = {"gemv_us": round(timed_torch(
        lambda i: torch.mv(dense[i % RW], xs_t[i % 16]), 64), 3)}
    if with_spmm:
        dense_ctx["gemm_us"] = round(timed_torch(
            lambda i: torch.mm(dense[i % RW], Xs_t[i % 16]), 64), 3)
    if cfg.wdtype == "f32":
        try:
            import warnings
            with warnings.catch_warnings():
                warnings.simplefilter("ignore")      # torch flags sparse CSR as beta
                csr = [dense[0].to_sparse_csr() for _ in range(8)]
            dense_ctx["csr_spmv_us"] = round(timed_torch(
                lambda i: torch.mv(csr[i % 8], xs_t[i % 16]), 64), 3)
            if with_spmm:
                dense_ctx["csr_spmm_us"] = round(timed_torch(
                    lambda i: torch.mm(csr[i % 8], Xs_t[i % 16]), 64), 3)
            del csr
        except RuntimeError as e:          # sparse kernels unavailable in this torch build
            dense_ctx["csr_error"] = str(e)[:120]
    del dense, xs_t, Xs_t

    for n in names:
        kernels[n]["traffic_bytes"] = traffic.get(n)
    ks = kernels["spmv"]
    step_total = sum(nbytes[n] for n in names)
    roofline = {"kernel": "spmv", "bound": "hbm", "achieved": ks["gbps"], "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(ks["gbps"] / HBM_PEAK_GBPS, 4),
                "traffic": traffic.get("spmv"),
                "frac_of_measured_read_peak": round(ks["gbps"] / read_peak, 4),
                "x_of_same_size_read_floor": round(ks["avg_us"] / floor_us, 3)}
    out = {
        "metric": METRIC,
        "value": ks["gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if cfg.wdtype == "f32" else "f16",
        "data": "synthetic: seeded weights of the workload's shape and distribution, "
                "exact-k irregular-magnitude row densities, N(0,1) activations",
        "config": {
            "workload": f"{cfg.name}: W {cfg.wdtype} [{cfg.M} x {cfg.N}] {cfg.dist}, "
                        f"keep {cfg.keep}, block sizes {cfg.b_min}..{cfg.b_max} (floor rule); "
                        f"value = SpMV (B=1) over the encoded matrix; step = encode + SpMV"
                        + (f" + SpMM (B={B})" if with_spmm else ""),
            "M": cfg.M, "N": cfg.N, "nnz": plan.nnz, "spmm_batch": B,
            "bins": {str(1 << b["log2b"]): b["rows"] for b in plan.bins},
            "rotation": {"W_copies": RW, "format_copies": RE,
                         "format_rotation_MB": round(RE * plan.nnz * (s_w + 1) / 1e6, 1)},
        },
        "roofline": roofline,
        "spmv_gflops": ks["gflops"],
        "kernels": kernels,
        "step_gbps": round(step_total / (ms_per_step * 1e-3) / 1e9, 1),
        "gflops_step": round(sum(flops[n] for n in names) / (ms_per_step * 1e-3) / 1e9, 1),
        "hbm_measured": {"stream_read_4GiB_gbps": round(read_peak, 1),
                         "same_size_read_us_by_shape": shapes,
                         "same_size_read_floor_us": floor_us,
                         "same_size_read_floor_shape": best_shape,
                         "same_size_read_floor_gbps": round(small_b / (floor_us * 1e-6) / 1e9, 1),
                         "same_size_rotation": n_small,
                         "stream_read_W_us": round(w_read_us, 3),
                         "stream_read_W_gbps": round(w_bytes / (w_read_us * 1e-6) / 1e9, 1)},
        "encode_frac_of_W_read": round(w_read_us / kernels["encode"]["avg_us"], 4),
        "spmv_size_sweep": size_sweep,
        "packed_offsets": packed_ctx,
        "int8_values": int8_ctx,
        "prune_counts": prune_ctx,
        "dense_masked_context": dense_ctx,
        "host": {"plan_ms": round(plan_ms, 3), "enqueue_us_per_step": round(host_us, 2)},
    }
    if with_spmm:
        km = kernels["spmm"]
        gather = plan.nnz * B * s_x       # every retained weight reads its X row on chip
        g_gbps = gather / (km["avg_us"] * 1e-6) / 1e9
        out["spmm_b64_gbps"] = km["gbps"]
        out["spmm_b64_gflops"] = km["gflops"]
        out["roofline_spmm"] = {"kernel": "spmm", "bound": "gather", "achieved": round(g_gbps, 1),
                                "peak": round(GATHER_PEAK_GBPS, 1), "unit": "GB/s",
                                "frac": round(g_gbps / GATHER_PEAK_GBPS, 4),
                                "gather_bytes": int(gather),
                                "hbm_gbps": km["gbps"],
                                "hbm_frac": km["frac_hbm_peak"],
                                "traffic": traffic.get("spmm")}
    if not args.no_recurrent:
        out["recurrent"] = recurrent_figures(args, with_cpu=False)
    out["cpu_baseline"] = (cpu_baseline(cfg, mi, x, X, args.cpu_seconds, nbytes)
                           if args.cpu_seconds > 0 else None)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
