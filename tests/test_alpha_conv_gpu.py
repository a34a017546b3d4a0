"""GPU parity of alpha-CROWN on convolutional networks (residual blocks, stride-2
convolutions, flatten into dense layers) against the fp64 alpha-CROWN oracle.

The spec pass relaxes every ReLU with the rows' own slopes and records the coefficients
before each relaxation; the gradient pass evaluates the relaxed network forward from each
row's box vertex (convolutions, the additions of the residual blocks and the dense layers).
At given slopes the bounds and the gradients are compared element by element; optimisation
runs evaluation by evaluation from the same start; the 3x8x8 ResNet at full width (64 and
128 channels, a 512-wide dense layer, 99 spec rows) against a stored oracle run."""
import os

import numpy as np
import pytest

import oracle
from oracle import alpha64
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from tests.test_alpha_gpu import _assert_grad_close, _check_layers_and_classes, _roots
from workloads import make_workload

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _nets():
    from tests.test_conv_gpu import conv_chain, small_resnet
    return [small_resnet(316), conv_chain(314)]


def _n_total(net):
    shapes = oracle.node_shapes(net)
    return sum(int(np.prod(shapes[i])) for i in alpha64.relu_ids(net))


@pytest.mark.parametrize("which", [0, 1])
def test_alpha_conv_eval_and_gradient_match_oracle(which):
    """Random slopes, no step: bounds, gradients and the reported slopes, per input."""
    import torch
    wl = _nets()[which]
    log("net", wl.name)
    ctx = gpu_ctx(wl.net)
    B, m = wl.C.shape[0], wl.C.shape[1]
    roots = _roots(wl, range(B))
    _check_layers_and_classes(ctx, wl, roots)
    n_total = _n_total(wl.net)
    assert n_total == int(ctx.lib.vcr_relu_neurons(ctx.h))
    rng = np.random.default_rng(13 + which)
    A0 = rng.random((B, 2 * m, n_total)).astype(np.float32)
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=0, alpha_init=to_dev(A0),
                                        want_grad=True, want_alpha=True)
    torch.cuda.synchronize()
    lb, ub, g = lb.cpu().numpy(), ub.cpu().numpy(), ex["grad"].cpu().numpy()
    ids = alpha64.relu_ids(wl.net)
    for b in range(B):
        al, au = alpha64.split_rows(wl.net, A0[b].astype(np.float64), m)
        rl, ru, gl, gu = alpha64.alpha_bound(wl.net, roots[b], wl.C[b], al, au)
        assert_close(lb[b], rl, f"{wl.name} input {b} lb")
        assert_close(ub[b], ru, f"{wl.name} input {b} ub")
        gref = alpha64.flat_rows(wl.net, gl, gu)
        _assert_grad_close(g[b], gref, f"{wl.name} input {b} gradient")
        assert np.count_nonzero(gref) > 0
        unst = np.concatenate([alpha64.unstable_mask(roots[b], i).reshape(-1) for i in ids])
        lam0 = np.concatenate([roots[b].relax[i][0].reshape(-1) for i in ids])
        want = np.where(unst[None, :], A0[b], lam0[None, :].astype(np.float32))
        assert np.array_equal(ex["alpha"][b].cpu().numpy(), want)
        log("input", b, "unstable", int(unst.sum()), "max |grad|", float(np.max(np.abs(gref))))


@pytest.mark.parametrize("which", [0, 1])
def test_alpha_conv_trajectory_matches_oracle(which):
    """Eight Adam steps from CROWN's slopes: every evaluation's bounds and the best bounds;
    the optimised bounds improve on CROWN's."""
    import torch
    wl = _nets()[which]
    log("net", wl.name)
    ctx = gpu_ctx(wl.net)
    B, m = wl.C.shape[0], wl.C.shape[1]
    roots = _roots(wl, range(B))
    _check_layers_and_classes(ctx, wl, roots)
    T = 8
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=T, want_hist=True)
    torch.cuda.synchronize()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    for b in range(B):
        r = alpha64.alpha_crown(wl.net, wl.x0[b], wl.eps, wl.C[b], iters=T, root=roots[b])
        for t in range(T + 1):
            assert_close(lh[t, b], r.lb_hist[t], f"{wl.name} input {b} evaluation {t} lb")
            assert_close(uh[t, b], r.ub_hist[t], f"{wl.name} input {b} evaluation {t} ub")
        assert_close(lb[b].cpu().numpy(), r.lb, f"{wl.name} input {b} best lb")
        assert_close(ub[b].cpu().numpy(), r.ub, f"{wl.name} input {b} best ub")
        assert np.any(r.lb > r.root.lb + 1e-4) or np.any(r.ub < r.root.ub - 1e-4)


def test_alpha_conv_first_evaluation_is_crown():
    """CROWN's own slopes give CROWN's bounds bit for bit, and one input alone equals its
    batch row bit for bit after steps."""
    import torch
    for wl in _nets():
        ctx = gpu_ctx(wl.net)
        lb0, ub0, _ = gpu_crown(ctx, wl)
        lb, ub, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=0)
        torch.cuda.synchronize()
        assert np.array_equal(lb.cpu().numpy(), lb0) and np.array_equal(ub.cpu().numpy(), ub0), wl.name
        lb, ub, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=4)
        lb1, ub1, _ = ctx.alpha_crown_bounds(to_dev(wl.x0[1:2]), wl.eps, to_dev(wl.C[1:2]), iters=4)
        torch.cuda.synchronize()
        assert np.array_equal(lb1.cpu().numpy()[0], lb.cpu().numpy()[1]), wl.name
        assert np.array_equal(ub1.cpu().numpy()[0], ub.cpu().numpy()[1]), wl.name


def test_alpha_conv_chunked_equals_whole():
    """A workspace cap that splits the inputs into chunks gives the same bits."""
    import torch
    from paper_2606_09377_amd.vcrown import OPT_WORKSPACE_CAP_BYTES
    from tests.test_conv_gpu import small_resnet
    wl = small_resnet(317, batch=4)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=3)
    torch.cuda.synchronize()
    st0 = ctx.stats()
    ctx.set_option(OPT_WORKSPACE_CAP_BYTES, st0["peak_workspace_bytes"] - 1)
    lb2, ub2, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=3)
    torch.cuda.synchronize()
    assert ctx.stats()["n_chunks_last_call"] > st0["n_chunks_last_call"]
    assert np.array_equal(lb.cpu().numpy(), lb2.cpu().numpy()) and np.array_equal(ub.cpu().numpy(), ub2.cpu().numpy())


def test_alpha_resnet3x8x8_full_width():
    """The 3x8x8 ResNet at full width, both inputs, 5 steps: input 0 against the stored
    oracle run (every evaluation, the best bounds), never looser than CROWN, sound on sampled
    points of the box, and input 1 alone equals its batch row bit for bit."""
    import torch
    from tests.pins import box_of
    from tests.test_conv_gpu import torch_forward
    g = np.load(os.path.join(GOLDEN, "resnet3x8x8_alpha.npz"))
    T = int(g["iters"])
    wl = make_workload("resnet3x8x8")
    ctx = gpu_ctx(wl.net)
    lbc, ubc, _ = gpu_crown(ctx, wl)
    lb, ub, ex = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=T, want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    assert np.all(lb >= lbc) and np.all(ub <= ubc)
    log("mean lb gain over CROWN", float(np.mean(lb - lbc)), "mean ub gain", float(np.mean(ubc - ub)))
    for t in range(T + 1):
        assert_close(lh[t, 0], g["lb_hist_0"][t], f"evaluation {t} lb")
        assert_close(uh[t, 0], g["ub_hist_0"][t], f"evaluation {t} ub")
    assert_close(lb[0], g["lb_0"], "best lb")
    assert_close(ub[0], g["ub_0"], "best ub")
    rng = np.random.default_rng(17)
    for b in range(2):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        X = np.concatenate([lo + (hi - lo) * rng.random((4096, lo.size)),
                            np.where(rng.random((1024, lo.size)) < 0.5, lo, hi)])
        with torch.no_grad():
            y = torch_forward(wl.net, torch.from_numpy(X.astype(np.float32)).cuda())[-1]
            Y = (y.double() @ torch.from_numpy(wl.C[b].astype(np.float64)).cuda().T).cpu().numpy()
        slack = 1e-4 + 1e-4 * np.abs(Y)
        assert np.all(Y >= lb[b][None] - slack) and np.all(Y <= ub[b][None] + slack)
    lb1, ub1, _ = ctx.alpha_crown_bounds(to_dev(wl.x0[1:2]), wl.eps, to_dev(wl.C[1:2]), iters=T)
    torch.cuda.synchronize()
    assert np.array_equal(lb1.cpu().numpy()[0], lb[1]) and np.array_equal(ub1.cpu().numpy()[0], ub[1])
