"""GPU parity of the lower-slope rules and the input scan (options VCR_OPT_LAMBDA_RULE and
VCR_OPT_CHECK_FINITE).

Sec. 2.1 only asks the lower slope of an unstable ReLU to lie in [0, 1]; the library's
default is the adaptive choice, and the option selects zero, one or the upper line's slope
instead.  With every rule the GPU bounds (final and per layer) must match the oracle run
with the same rule, on MLPs, on convolutional nets with residual blocks, and on
branch-and-bound subdomains (whose split neurons get the rule too)."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_classes, assert_close, gpu_crown, gpu_ctx, log, to_dev
from workloads import random_mlp

pytestmark = pytest.mark.gpu
RULES = ("zero", "one", "same_slope")


def _compare_rule(wl, rule, what):
    from paper_2606_09377_amd.vcrown import LAMBDA_RULES, OPT_LAMBDA_RULE
    ctx = gpu_ctx(wl.net)
    ctx.set_option(OPT_LAMBDA_RULE, LAMBDA_RULES[rule])
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in range(wl.x0.shape[0]):
        r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b], lambda_rule=rule)
        assert_close(lb[b], r.lb, f"{what} {rule} input {b} lb")
        assert_close(ub[b], r.ub, f"{what} {rule} input {b} ub")
        for k, i in enumerate(sorted(r.layer_l)):
            assert_close(layers[k][0][b], r.layer_l[i], f"{what} {rule} input {b} relu {k} l")
            assert_close(layers[k][1][b], r.layer_u[i], f"{what} {rule} input {b} relu {k} u")
            assert_classes(layers[k][0][b], layers[k][1][b], r.layer_l[i], r.layer_u[i], f"{what} {rule} relu {k}")
    return lb, ub


@pytest.mark.parametrize("rule", RULES)
def test_lambda_rule_mlp(rule):
    wl = random_mlp(91, [40, 160, 130, 120, 10], 3, 0.05)
    log("mlp rule", rule)
    _compare_rule(wl, rule, "mlp")


@pytest.mark.parametrize("rule", RULES)
def test_lambda_rule_conv(rule):
    from tests.test_conv_gpu import conv_chain, small_resnet
    for wl in (small_resnet(92), conv_chain(93)):
        log("conv rule", rule, wl.name)
        _compare_rule(wl, rule, wl.name)


def test_lambda_rules_differ_and_stay_ordered():
    """The rules give different bounds on a net with unstable neurons (the option reaches the
    kernels); every rule is sound, so none may cut below a sampled value."""
    from paper_2606_09377_amd.vcrown import LAMBDA_RULES, OPT_LAMBDA_RULE
    from tests.pins import box_of
    wl = random_mlp(94, [30, 120, 120, 8], 2, 0.08)
    ctx = gpu_ctx(wl.net)
    out = {}
    for rule in ("adaptive",) + RULES:
        ctx.set_option(OPT_LAMBDA_RULE, LAMBDA_RULES[rule])
        lb, ub, _ = gpu_crown(ctx, wl)
        out[rule] = (lb, ub)
    assert not np.array_equal(out["zero"][0], out["one"][0])
    rng = np.random.default_rng(5)
    for b in range(2):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        X = lo + (hi - lo) * rng.random((4000, lo.size))
        Y = np.stack([wl.C[b].astype(np.float64) @ oracle.forward(wl.net, x)[-1] for x in X])
        for rule, (lb, ub) in out.items():
            assert np.all(Y >= lb[b][None] - 1e-4 - 1e-4 * np.abs(Y)), rule
            assert np.all(Y <= ub[b][None] + 1e-4 + 1e-4 * np.abs(Y)), rule


@pytest.mark.parametrize("rule", ("one", "same_slope"))
def test_lambda_rule_subdomains(rule):
    """Subdomains of one root: the root pass and every split neuron's relaxation follow the
    rule; each domain against the oracle's subdomain bounds with the same rule."""
    from paper_2606_09377_amd.vcrown import LAMBDA_RULES, OPT_LAMBDA_RULE
    from workloads import draw_splits
    wl = random_mlp(95, [30, 96, 80, 70, 6], 1, 0.06)
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0], lambda_rule=rule)
    pool = oracle.unstable_pool(wl.net, root)
    sp = draw_splits(np.random.default_rng(6), pool, 24, 4)
    ctx = gpu_ctx(wl.net)
    ctx.set_option(OPT_LAMBDA_RULE, LAMBDA_RULES[rule])
    lb, ub, _ = gpu_crown(ctx, wl, splits=sp)
    LB, UB = oracle.crown_domains(wl.net, root, wl.C[0], sp, lambda_rule=rule)
    for d in range(sp.n_domains):
        if not np.isfinite(LB[d]).all():
            assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d]))
            continue
        assert_close(lb[d], LB[d], f"{rule} domain {d} lb")
        assert_close(ub[d], UB[d], f"{rule} domain {d} ub")


def test_check_finite_rejects_nan_and_inf():
    """With the scan on, a NaN in x0 or an infinity in C fails the call with VCR_ERR_ARG and
    leaves the outputs untouched; finite inputs pass and give the unscanned call's bits.
    (Non-finite inputs are never sent without the scan.)"""
    import torch
    from paper_2606_09377_amd.vcrown import OPT_CHECK_FINITE, VcrError
    from tests.test_conv_gpu import small_resnet
    for wl in (random_mlp(96, [20, 40, 40, 5], 2, 0.05), small_resnet(97)):
        ctx = gpu_ctx(wl.net)
        lb0, ub0, _ = gpu_crown(ctx, wl)
        ctx.set_option(OPT_CHECK_FINITE, 1)
        lb1, ub1, _ = gpu_crown(ctx, wl)
        assert np.array_equal(lb0, lb1) and np.array_equal(ub0, ub1)
        m = wl.C.shape[1]
        for which in ("x0", "C"):
            x0, C = wl.x0.copy(), wl.C.copy()
            if which == "x0":
                x0[1, 3] = np.nan
            else:
                C[0, 0, 1] = np.inf
            lb = torch.full((2, m), 7.0, device="cuda")
            ub = torch.full((2, m), 7.0, device="cuda")
            for call in ("crown", "ibp"):
                with pytest.raises(VcrError, match="ARG"):
                    if call == "crown":
                        ctx.crown_bounds(to_dev(x0), wl.eps, to_dev(C), out=(lb, ub))
                    else:
                        ctx.ibp_bounds(to_dev(x0), wl.eps, to_dev(C))
            torch.cuda.synchronize()
            assert torch.all(lb == 7.0) and torch.all(ub == 7.0)
