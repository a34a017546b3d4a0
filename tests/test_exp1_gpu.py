"""GPU parity on the paper's Exp. 1 network shape (Sec. 4.1): one hidden ReLU layer, one
output, the property being the output itself.  The hidden layer is large enough that its
IBP step runs on the matrix cores (two GEMMs, c' = W c + b and r' = |W| r)."""
import os

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from workloads import make_workload

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_exp1_shape_small_every_bound():
    """1024 -> 16384 -> 1 (2^24 first-layer weights): final and hidden bounds of sampled
    inputs of the 64, element by element; IBP bounds too."""
    import torch
    wl = make_workload("exp1_mlp1024x16384x1")
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in range(0, 64, 9):
        rlb, rub, l, u = oracle.crown_one_hidden(wl.net, wl.x0[b], wl.eps, wl.C[b])
        assert_close(lb[b], rlb, f"input {b} lb")
        assert_close(ub[b], rub, f"input {b} ub")
        assert_close(layers[0][0][b], l, f"input {b} hidden l")
        assert_close(layers[0][1][b], u, f"input {b} hidden u")
    il, iu = ctx.ibp_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C))
    torch.cuda.synchronize()
    il, iu = il.cpu().numpy(), iu.cpu().numpy()
    for b in (0, 63):
        rl, ru = oracle.ibp_spec_bounds(wl.net, wl.x0[b], wl.eps, wl.C[b])
        assert_close(il[b], rl, f"input {b} ibp lb")
        assert_close(iu[b], ru, f"input {b} ibp ub")
    # an input alone gives its batch row bit for bit
    lb1, ub1, lay1 = gpu_crown(ctx, wl, inputs=[7])
    assert np.array_equal(lb1[0], lb[7]) and np.array_equal(ub1[0], ub[7])
    assert np.array_equal(lay1[0][0][0], layers[0][0][7])


def test_exp1_full_size():
    """4096 -> 262144 -> 1 at 2048 inputs: stored oracle bounds of inputs 0 and 1 (final
    bounds and sampled hidden neurons), batch invariance, soundness on sampled points."""
    import torch
    g = np.load(os.path.join(GOLDEN, "exp1_mlp4096x262144x1.npz"))
    log("generating the 1.07e9-weight network")
    wl = make_workload("exp1_mlp4096x262144x1")
    ctx = gpu_ctx(wl.net)
    log("gpu run B=2048")
    lb, ub, layers = gpu_crown(ctx, wl)
    idx = g["idx"]
    for b in g["inputs"]:
        assert_close(lb[b], g[f"lb_{b}"], f"input {b} lb")
        assert_close(ub[b], g[f"ub_{b}"], f"input {b} ub")
        assert_close(layers[0][0][b][idx], g[f"l_{b}"], f"input {b} hidden l")
        assert_close(layers[0][1][b][idx], g[f"u_{b}"], f"input {b} hidden u")
    assert np.all(lb <= ub) and np.all(layers[0][0] <= layers[0][1])
    lb1, ub1, _ = gpu_crown(ctx, wl, inputs=[1000])
    assert np.array_equal(lb1[0], lb[1000]) and np.array_equal(ub1[0], ub[1000])
    from tests.pins import box_of
    rng = np.random.default_rng(12)
    W1 = torch.from_numpy(wl.net.nodes[0].W).cuda()
    b1 = torch.from_numpy(wl.net.nodes[0].b).cuda()
    W2 = torch.from_numpy(wl.net.nodes[2].W).cuda()
    b2 = torch.from_numpy(wl.net.nodes[2].b).cuda()
    for b in (0, 2047):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        X = np.concatenate([lo + (hi - lo) * rng.random((256, lo.size)),
                            np.where(rng.random((256, lo.size)) < 0.5, lo, hi)])
        with torch.no_grad():
            h = torch.relu(torch.from_numpy(X.astype(np.float32)).cuda() @ W1.T + b1)
            Y = (h @ W2.T + b2).double().cpu().numpy()[:, 0]
        slack = 1e-4 + 1e-4 * np.abs(Y)
        assert np.all(Y >= lb[b, 0] - slack) and np.all(Y <= ub[b, 0] + slack)
