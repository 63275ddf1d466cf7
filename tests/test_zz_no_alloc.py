"""The pruning entry point that allocates nothing (fixed per-device scratch) against
the one that takes a workspace: the same per-row counts, bit for bit, on two calls
in a row -- the second on a smaller matrix -- through the C ABI."""
import ctypes
import sys

import numpy as np
import pytest

import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def say(*a):
    print(*a, flush=True, file=sys.stderr)


@pytest.mark.parametrize("first,second", [("fc_9216", "lstm_tiny"), ("gru_1536", "lstm_1024")])
def test_noalloc_counts_equal_workspace_call(first, second):
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_1911_08020_amd as darb
    lib = darb.lib()
    P = ctypes.c_void_p
    stream = P(torch.cuda.current_stream().cuda_stream)
    for name in (first, second):
        cfg, mi, _, _ = workloads.make_config(name, seed=0)
        W = torch.from_numpy(mi.W).cuda()
        M, N = W.shape
        code = darb.F32 if W.dtype == torch.float32 else darb.F16
        for k in (mi.k, max(1, mi.k // 3)):
            say(f"no-alloc pruning: {name} {M}x{N} {cfg.wdtype} k={k}")
            ref = darb.prune_counts(W, k)
            got = torch.full((M,), -1, dtype=torch.int64, device="cuda")
            rc = lib.darb_prune_counts_noalloc(M, N, code, P(W.data_ptr()), N, int(k),
                                               P(got.data_ptr()), stream)
            assert rc == 0, lib.darb_last_error().decode()
            torch.cuda.synchronize()
            assert torch.equal(got, ref), name
            assert int(got.sum()) == k
            if k == mi.k:
                assert np.array_equal(got.cpu().numpy(), mi.mask.sum(axis=1))
