"""The allocation-free entry point vcr_crown_bounds_noalloc, called through the C ABI, against
vcr_crown_bounds on the same inputs: two calls in a row (the second smaller, after a larger
one has left its contents in the shared scratch), a different network after that, and a
request whose single input does not fit the scratch.  A context that only ever makes
allocation-free calls never allocates a workspace."""
import ctypes

import numpy as np
import pytest

from tests.gpu_util import gpu_crown, gpu_ctx, log, to_dev
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _noalloc(ctx, x0, eps, C):
    """Direct C-ABI call; returns the status and the outputs (pre-filled with a sentinel)."""
    import torch
    B, m = C.shape[0], C.shape[1]
    lb = torch.full((B, m), 123.0, device="cuda")
    ub = torch.full((B, m), 123.0, device="cuda")
    xd, Cd = to_dev(x0), to_dev(C)
    ctx._stream_sync()
    st = ctx.lib.vcr_crown_bounds_noalloc(ctx.h, ctypes.c_void_p(xd.data_ptr()), B, ctypes.c_float(float(eps)),
                                          ctypes.c_void_p(Cd.data_ptr()), m, ctypes.c_void_p(lb.data_ptr()),
                                          ctypes.c_void_p(ub.data_ptr()))
    torch.cuda.synchronize()
    return st, lb.cpu().numpy(), ub.cpu().numpy()


def _layers(ctx, B):
    import torch
    out = [tuple(t.cpu().numpy() for t in ctx.layer_bounds(r, B)) for r in range(ctx.n_relu)]
    torch.cuda.synchronize()
    return out


def test_noalloc_matches_crown_bounds_two_calls():
    from paper_2606_09377_amd.vcrown import VCR_ERR_OOM, VCR_OK
    wl = make_workload("mlp784x1024x6")
    ref_ctx = gpu_ctx(wl.net)
    ctx = gpu_ctx(wl.net)               # allocation-free calls only
    # first call: 16 inputs (more than fit the scratch at once: the call runs in chunks)
    sel1 = list(range(16))
    st, lb, ub = _noalloc(ctx, wl.x0[sel1], wl.eps, wl.C[sel1])
    assert st == VCR_OK, ctx.lib.vcr_last_error(ctx.h)
    lay = _layers(ctx, len(sel1))
    chunks = ctx.stats()["n_chunks_last_call"]
    rlb, rub, rlay = gpu_crown(ref_ctx, wl, inputs=sel1)
    log("16 inputs: chunks", chunks, "vs", ref_ctx.stats()["n_chunks_last_call"])
    assert chunks > ref_ctx.stats()["n_chunks_last_call"]
    assert np.array_equal(lb, rlb) and np.array_equal(ub, rub)
    for r in range(len(rlay)):
        assert np.array_equal(lay[r][0], rlay[r][0]) and np.array_equal(lay[r][1], rlay[r][1])
    # second call: 3 other inputs, on the scratch the first call filled
    sel2 = [40, 41, 63]
    st, lb2, ub2 = _noalloc(ctx, wl.x0[sel2], wl.eps, wl.C[sel2])
    assert st == VCR_OK, ctx.lib.vcr_last_error(ctx.h)
    rlb2, rub2, _ = gpu_crown(ref_ctx, wl, inputs=sel2)
    assert np.array_equal(lb2, rlb2) and np.array_equal(ub2, rub2)
    # a smaller network in another context on the same GPU
    w1 = make_workload("mlp784x256x2")
    c1, r1 = gpu_ctx(w1.net), gpu_ctx(w1.net)
    st, lb3, ub3 = _noalloc(c1, w1.x0, w1.eps, w1.C)
    assert st == VCR_OK, c1.lib.vcr_last_error(c1.h)
    rlb3, rub3, _ = gpu_crown(r1, w1)
    assert np.array_equal(lb3, rlb3) and np.array_equal(ub3, rub3)
    # the allocation-free contexts never held a workspace
    assert ctx.stats()["peak_workspace_bytes"] == 0 and c1.stats()["peak_workspace_bytes"] == 0
    # one input of the wide MLP needs more than the scratch: rejected, outputs untouched
    w3 = make_workload("mlp3072x8192x4", batch=1)
    c3 = gpu_ctx(w3.net)
    st, lb4, ub4 = _noalloc(c3, w3.x0, w3.eps, w3.C)
    assert st == VCR_ERR_OOM
    assert b"scratch" in c3.lib.vcr_last_error(c3.h)
    assert np.all(lb4 == 123.0) and np.all(ub4 == 123.0)
    assert c3.stats()["peak_workspace_bytes"] == 0
