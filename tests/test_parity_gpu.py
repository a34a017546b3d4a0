"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Bar: |delta| <= 1e-4 + 1e-4 |oracle bound| on final bounds and every intermediate bound;
ReLU classes equal except within that tolerance of zero; bitwise batch invariance."""
import os

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_close, check_input, gpu_crown, gpu_ctx, log, to_dev
from workloads import make_workload, random_mlp

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

SMALL = [
    # (seed, dims, batch, eps): several tiles in every GEMM dimension and ragged tails
    (101, [100, 200, 300, 130, 7], 3, 0.05),
    (102, [33, 257, 129, 65, 5], 5, 0.08),
    (103, [20, 64, 10], 4, 0.1),            # one hidden layer
    (104, [16, 40, 40, 40, 40, 40, 3], 3, 0.1),
    (105, [300, 129, 2], 2, 0.02),          # a single spec row
]


@pytest.mark.parametrize("case", SMALL, ids=lambda c: "x".join(map(str, c[1])))
def test_small_mlps(case):
    seed, dims, B, eps = case
    log("case", case)
    wl = random_mlp(seed, dims, B, eps)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in range(B):
        check_input(wl.net, wl.x0[b], wl.eps, wl.C[b], lb[b], ub[b], [(l[b], u[b]) for l, u in layers],
                    what=f"{dims} input {b}")


def test_single_dense_layer():
    wl = random_mlp(106, [70, 9], 3, 0.05)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = gpu_crown(ctx, wl)
    for b in range(3):
        r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b])
        assert_close(lb[b], r.lb, "lb")
        assert_close(ub[b], r.ub, "ub")


def test_mlp784x256x2():
    wl = make_workload("mlp784x256x2")
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    check_input(wl.net, wl.x0[0], wl.eps, wl.C[0], lb[0], ub[0], [(l[0], u[0]) for l, u in layers], what="C1")


def test_mlp784x1024x6_full_batch_sampled_inputs():
    wl = make_workload("mlp784x1024x6")
    ctx = gpu_ctx(wl.net)
    log("gpu run B=64")
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in (0, 37, 63):
        log("oracle input", b)
        check_input(wl.net, wl.x0[b], wl.eps, wl.C[b], lb[b], ub[b], [(l[b], u[b]) for l, u in layers],
                    what=f"mlp784x1024x6 input {b}")


def test_mlp3072x8192x4_full_batch_golden():
    path = os.path.join(GOLDEN, "mlp3072x8192x4.npz")
    g = np.load(path)
    wl = make_workload("mlp3072x8192x4")
    ctx = gpu_ctx(wl.net)
    log("gpu run B=16 wide")
    lb, ub, layers = gpu_crown(ctx, wl)
    relu_ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    for b in g["inputs"]:
        assert_close(lb[b], g[f"lb_{b}"], f"wide input {b} lb")
        assert_close(ub[b], g[f"ub_{b}"], f"wide input {b} ub")
        for r, i in enumerate(relu_ids):
            assert_close(layers[r][0][b], g[f"l_{b}_{i}"], f"wide input {b} relu {r} l")
            assert_close(layers[r][1][b], g[f"u_{b}_{i}"], f"wide input {b} relu {r} u")


def test_ibp_bounds():
    for seed, dims, B, eps in SMALL[:3]:
        wl = random_mlp(seed, dims, B, eps)
        ctx = gpu_ctx(wl.net)
        lb, ub = ctx.ibp_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C))
        lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
        for b in range(B):
            il, iu = oracle.ibp_spec_bounds(wl.net, wl.x0[b], wl.eps, wl.C[b])
            assert_close(lb[b], il, "ibp lb")
            assert_close(ub[b], iu, "ibp ub")


def test_ibp_bounds_several_tiles():
    """IBP where the batch spans several input tiles (ragged last tile), the outputs several
    64-wide groups, and K splits unevenly over the workgroup's waves; checked against the
    oracle and for batch invariance (bit for bit against the inputs alone)."""
    wl = random_mlp(108, [300, 200, 130, 7], 19, 0.05)
    ctx = gpu_ctx(wl.net)
    lb, ub = ctx.ibp_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C))
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    for b in range(19):
        il, iu = oracle.ibp_spec_bounds(wl.net, wl.x0[b], wl.eps, wl.C[b])
        assert_close(lb[b], il, "ibp lb")
        assert_close(ub[b], iu, "ibp ub")
    for b in (0, 17):
        l1, u1 = ctx.ibp_bounds(to_dev(wl.x0[b:b + 1]), wl.eps, to_dev(wl.C[b:b + 1]))
        assert np.array_equal(l1.cpu().numpy()[0], lb[b]) and np.array_equal(u1.cpu().numpy()[0], ub[b])


def test_eps_zero_is_a_point():
    wl = random_mlp(107, [50, 130, 140, 6], 3, 0.0)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = gpu_crown(ctx, wl)
    from tests.pins import spec_values
    for b in range(3):
        y = spec_values(wl.net, wl.C[b], wl.x0[b][None].astype(np.float64))[0]
        assert_close(lb[b], y, "lb")
        assert_close(ub[b], y, "ub")


def test_batch_invariance_bitwise():
    """One input alone, inside a batch of 64, chunked under a workspace cap, and run to
    run: identical bits."""
    from paper_2606_09377_amd.vcrown import OPT_WORKSPACE_CAP_BYTES
    wl = make_workload("mlp784x1024x6")
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    lb2, ub2, layers2 = gpu_crown(ctx, wl)
    assert np.array_equal(lb, lb2) and np.array_equal(ub, ub2)
    for b in (5, 63):
        lb1, ub1, lay1 = gpu_crown(ctx, wl, inputs=[b])
        assert np.array_equal(lb1[0], lb[b]) and np.array_equal(ub1[0], ub[b])
        for r in range(len(layers)):
            assert np.array_equal(lay1[r][0][0], layers[r][0][b])
            assert np.array_equal(lay1[r][1][0], layers[r][1][b])
    full = ctx.workspace_bytes(64, wl.C.shape[1])
    ctx.set_option(OPT_WORKSPACE_CAP_BYTES, full // 5)
    lb3, ub3, layers3 = gpu_crown(ctx, wl)
    st = ctx.stats()
    assert st["n_chunks_last_call"] > 6, st
    assert np.array_equal(lb3, lb) and np.array_equal(ub3, ub)
    for r in range(len(layers)):
        assert np.array_equal(layers3[r][0], layers[r][0]) and np.array_equal(layers3[r][1], layers[r][1])


def test_gpu_bounds_sound_on_samples():
    """The soundness contract on the GPU's own bounds (with the parity slack)."""
    from tests.pins import box_of, spec_values, vertex_for
    wl = make_workload("mlp784x256x2")
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = gpu_crown(ctx, wl)
    lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
    rng = np.random.default_rng(5)
    X = lo + (hi - lo) * rng.random((100000, lo.size))
    Xc = np.where(rng.random((10000, lo.size)) < 0.5, lo, hi)
    r = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0], keep_A=True)
    Xa = np.concatenate([[vertex_for(a, lo, hi, True) for a in r.A_lower],
                         [vertex_for(a, lo, hi, False) for a in r.A_upper]])
    for P in (X, Xc, Xa):
        Y = spec_values(wl.net, wl.C[0], P)
        slack = 1e-4 + 1e-4 * np.abs(Y)
        assert np.all(Y >= lb[0][None] - slack) and np.all(Y <= ub[0][None] + slack)
