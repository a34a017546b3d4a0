"""GPU parity of alpha-CROWN against the fp64 alpha-CROWN oracle.

At a given set of slopes the bounds and their gradients are deterministic functions of the
slopes, compared element by element; whole optimisation runs are compared evaluation by
evaluation (both sides start from the same slopes), and at the 784-1024x6 MLP's full batch
on sampled inputs, with soundness and batch invariance checked at any size."""
import numpy as np
import pytest

import oracle
from oracle import alpha64
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from workloads import make_workload, random_mlp

pytestmark = pytest.mark.gpu


def _roots(wl, inputs):
    return {b: oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b]) for b in inputs}


def _check_layers_and_classes(ctx, wl, roots):
    """The alpha semantics need the GPU's ReLU classes to be the oracle's: check the
    intermediate bounds and that no oracle bound sits within the tolerance of 0."""
    _, _, layers = gpu_crown(ctx, wl)
    ids = alpha64.relu_ids(wl.net)
    for b, root in roots.items():
        for r, i in enumerate(ids):
            assert_close(layers[r][0][b], root.layer_l[i], f"input {b} relu {i} l")
            assert_close(layers[r][1][b], root.layer_u[i], f"input {b} relu {i} u")
            near = (np.abs(root.layer_l[i]) <= 1e-4 + 1e-4 * np.abs(root.layer_l[i])) | \
                   (np.abs(root.layer_u[i]) <= 1e-4 + 1e-4 * np.abs(root.layer_u[i]))
            assert not near.any(), "a bound in the tolerance band of 0: pick another seed"


def _assert_grad_close(got, ref, what):
    # fp32 gradients a * D: tolerance relative to the row's largest gradient
    scale = 1.0 + np.max(np.abs(ref), axis=-1, keepdims=True)
    bad = np.abs(got - ref) > 1e-4 * scale + 1e-4 * np.abs(ref)
    assert not bad.any(), f"{what}: {bad.sum()} gradients outside tolerance, worst " \
                          f"{np.max(np.abs(got - ref) / (1e-4 * scale + 1e-4 * np.abs(ref)))}"


def small_case(seed=81, dims=(30, 96, 80, 70, 6), B=3, eps=0.06):
    return random_mlp(seed, list(dims), B, eps)


def test_alpha_eval_and_gradient_match_oracle():
    """Random slopes, no step: bounds and gradients element by element."""
    import torch
    wl = small_case()
    ctx = gpu_ctx(wl.net)
    B, m = wl.C.shape[0], wl.C.shape[1]
    roots = _roots(wl, range(B))
    _check_layers_and_classes(ctx, wl, roots)
    n_total = sum(int(np.prod(s)) for s in [oracle.node_shapes(wl.net)[i] for i in alpha64.relu_ids(wl.net)])
    rng = np.random.default_rng(3)
    A0 = rng.random((B, 2 * m, n_total)).astype(np.float32)
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=0, alpha_init=to_dev(A0),
                                        want_grad=True, want_alpha=True)
    torch.cuda.synchronize()
    lb, ub, g = lb.cpu().numpy(), ub.cpu().numpy(), ex["grad"].cpu().numpy()
    for b in range(B):
        al, au = alpha64.split_rows(wl.net, A0[b].astype(np.float64), m)
        rl, ru, gl, gu = alpha64.alpha_bound(wl.net, roots[b], wl.C[b], al, au)
        assert_close(lb[b], rl, f"input {b} lb")
        assert_close(ub[b], ru, f"input {b} ub")
        gref = alpha64.flat_rows(wl.net, gl, gu)
        _assert_grad_close(g[b], gref, f"input {b} gradient")
        # slopes out: the given ones at unstable neurons, CROWN's fixed slope elsewhere
        unst = np.concatenate([alpha64.unstable_mask(roots[b], i) for i in alpha64.relu_ids(wl.net)])
        lam0 = np.concatenate([roots[b].relax[i][0].reshape(-1) for i in alpha64.relu_ids(wl.net)])
        want = np.where(unst[None, :], A0[b], lam0[None, :].astype(np.float32))
        assert np.array_equal(ex["alpha"][b].cpu().numpy(), want)
        log("input", b, "max |grad|", float(np.max(np.abs(gref))))


def test_alpha_trajectory_matches_oracle():
    """Ten Adam steps from the same initial slopes: every evaluation's bounds, the best
    bounds and the final gradients."""
    import torch
    wl = small_case()
    ctx = gpu_ctx(wl.net)
    B, m = wl.C.shape[0], wl.C.shape[1]
    roots = _roots(wl, range(B))
    _check_layers_and_classes(ctx, wl, roots)
    A0 = np.stack([alpha64.flat_rows(wl.net, *alpha64.initial_alpha(wl.net, roots[b], m)) for b in range(B)])
    T = 10
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=T,
                                        alpha_init=to_dev(A0.astype(np.float32)), want_hist=True)
    torch.cuda.synchronize()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    for b in range(B):
        r = alpha64.alpha_crown(wl.net, wl.x0[b], wl.eps, wl.C[b], iters=T, root=roots[b])
        for t in range(T + 1):
            assert_close(lh[t, b], r.lb_hist[t], f"input {b} evaluation {t} lb")
            assert_close(uh[t, b], r.ub_hist[t], f"input {b} evaluation {t} ub")
        assert_close(lb[b].cpu().numpy(), r.lb, f"input {b} best lb")
        assert_close(ub[b].cpu().numpy(), r.ub, f"input {b} best ub")
        assert np.all(r.lb > r.root.lb - 1e-12) and np.any(r.lb > r.root.lb + 1e-3)


def test_alpha_first_evaluation_is_crown_bitwise():
    """CROWN's own slopes give CROWN's bounds bit for bit (same kernels, same order)."""
    import torch
    wl = small_case(seed=82, B=4)
    ctx = gpu_ctx(wl.net)
    lb0, ub0, _ = gpu_crown(ctx, wl)
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=0)
    torch.cuda.synchronize()
    assert np.array_equal(lb.cpu().numpy(), lb0) and np.array_equal(ub.cpu().numpy(), ub0)


def test_alpha_mlp784x1024x6_full_batch():
    """The 784-1024x6 MLP, 64 inputs, 20 steps: oracle parity on sampled inputs, never
    looser than CROWN, sound on sampled points, one input alone equals its batch row."""
    import torch
    from tests.test_conv_gpu import torch_forward
    wl = make_workload("mlp784x1024x6")
    ctx = gpu_ctx(wl.net)
    B, m = wl.C.shape[0], wl.C.shape[1]
    lbc, ubc, _ = gpu_crown(ctx, wl)
    T = 20
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=T, want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    assert np.all(lb >= lbc) and np.all(ub <= ubc)
    log("mean lb gain over CROWN", float(np.mean(lb - lbc)), "mean ub gain", float(np.mean(ubc - ub)))
    for b in (0, 37):
        log("oracle input", b)
        root = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b])
        r = alpha64.alpha_crown(wl.net, wl.x0[b], wl.eps, wl.C[b], iters=T, root=root)
        assert_close(lb[b], r.lb, f"input {b} lb")
        assert_close(ub[b], r.ub, f"input {b} ub")
    from tests.pins import box_of
    rng = np.random.default_rng(11)
    for b in (0, 63):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        X = np.concatenate([lo + (hi - lo) * rng.random((8192, lo.size)),
                            np.where(rng.random((2048, lo.size)) < 0.5, lo, hi)])
        with torch.no_grad():
            y = torch_forward(wl.net, torch.from_numpy(X.astype(np.float32)).cuda())[-1]
            Y = (y.double() @ torch.from_numpy(wl.C[b].astype(np.float64)).cuda().T).cpu().numpy()
        slack = 1e-4 + 1e-4 * np.abs(Y)
        assert np.all(Y >= lb[b][None] - slack) and np.all(Y <= ub[b][None] + slack)
    lb1, ub1, _ = ctx.alpha_crown_bounds(to_dev(wl.x0[5:6]), wl.eps, to_dev(wl.C[5:6]), iters=T)
    assert np.array_equal(lb1.cpu().numpy()[0], lb[5]) and np.array_equal(ub1.cpu().numpy()[0], ub[5])


def test_alpha_chunked_equals_whole():
    """A workspace cap that splits the inputs into chunks gives the same bits."""
    import torch
    from paper_2606_09377_amd.vcrown import OPT_WORKSPACE_CAP_BYTES
    wl = small_case(seed=83, B=6)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=5)
    torch.cuda.synchronize()
    st0 = ctx.stats()
    ctx.set_option(OPT_WORKSPACE_CAP_BYTES, st0["peak_workspace_bytes"] - 1)
    lb2, ub2, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=5)
    torch.cuda.synchronize()
    assert ctx.stats()["n_chunks_last_call"] > st0["n_chunks_last_call"]
    assert np.array_equal(lb.cpu().numpy(), lb2.cpu().numpy()) and np.array_equal(ub.cpu().numpy(), ub2.cpu().numpy())


def test_alpha_rejects_bad_options():
    """Bad options fail with VCR_ERR_ARG before any device work, on both network paths."""
    from paper_2606_09377_amd.vcrown import VcrError
    from tests.test_conv_gpu import small_resnet
    for wl in (small_case(seed=84, B=1), small_resnet(305)):
        ctx = gpu_ctx(wl.net)
        for kw in ({"lr": 0.0}, {"beta1": 1.0}, {"iters": -1}, {"adam_eps": 0.0}):
            with pytest.raises(VcrError, match="ARG"):
                ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), **kw)


def test_alpha_mlp3072x8192x4_bench_size():
    """The wide MLP (8192-wide layers, 99 spec rows), 16 inputs, 5 Adam steps: the batch runs
    its spec-pass steps on the 128 x 128 tile kernel with the alpha-CROWN epilogues, one
    input alone on the 64 x 64 and 32 x 64 tile kernels.  The input alone equals its batch
    row bit for bit at every evaluation, and input 0 matches the stored oracle run (every
    evaluation and the best bounds)."""
    import os
    import torch
    from paper_2606_09377_amd.vcrown import OPT_TIME_GEMM
    g = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mlp3072x8192x4_alpha.npz"))
    T = int(g["iters"])
    wl = make_workload("mlp3072x8192x4")
    ctx = gpu_ctx(wl.net)
    log("alpha B=16 T", T)
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=T, want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    ctx.set_option(OPT_TIME_GEMM, 1)
    log("alpha B=1")
    lb1, ub1, ex1 = ctx.alpha_crown_bounds(to_dev(wl.x0[:1]), wl.eps, to_dev(wl.C[:1]), iters=T, want_hist=True)
    torch.cuda.synchronize()
    assert ctx.stats()["timed_mid_launches"] > 0   # the single input's spec-pass steps
    assert np.array_equal(lb1.cpu().numpy()[0], lb[0]) and np.array_equal(ub1.cpu().numpy()[0], ub[0])
    assert np.array_equal(ex1["lb_hist"].cpu().numpy()[:, 0], lh[:, 0])
    assert np.array_equal(ex1["ub_hist"].cpu().numpy()[:, 0], uh[:, 0])
    for b in g["inputs"]:
        for t in range(T + 1):
            assert_close(lh[t, b], g[f"lb_hist_{b}"][t], f"input {b} evaluation {t} lb")
            assert_close(uh[t, b], g[f"ub_hist_{b}"][t], f"input {b} evaluation {t} ub")
        assert_close(lb[b], g[f"lb_{b}"], f"input {b} best lb")
        assert_close(ub[b], g[f"ub_{b}"], f"input {b} best ub")
        log("input", b, "mean lb gain over CROWN", float(np.mean(g[f"lb_{b}"] - g[f"lb_hist_{b}"][0])))
