"""Each plausible mistake planted in a copy of the oracle (a dropped term, a wrong sign, a
swapped slope, a transposed or misaligned operand) must make at least one pin fail.
The mistakes are planted in an in-memory copy of the oracle's source, on the CPU."""
import os
import sys
import types

import pytest

from tests import pins, pins_alpha, pins_beta

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")
SRC = os.path.join(ORACLE_DIR, "crown64.py")
SRC_ALPHA = os.path.join(ORACLE_DIR, "alpha64.py")

MUTANTS = {
    "drop_relax_intercept_lower": ("bias = bias + An @ t", "bias = bias"),
    "drop_relax_intercept_upper": ("bias = bias + Ap @ t", "bias = bias"),
    "swap_slopes_lower": ("Az = Ap * lam + An * s", "Az = Ap * s + An * lam"),
    "swap_slopes_upper": ("Az = Ap * s + An * lam", "Az = Ap * lam + An * s"),
    "drop_dense_bias": ("bias = bias + Ai @ _f64(nd.b)", "bias = bias"),
    "drop_conv_bias": ("bias = bias + A4.sum(axis=(2, 3)) @ _f64(nd.b)", "bias = bias"),
    "dense_weight_rows_reversed": ("Ai @ _f64(nd.W))", "Ai @ _f64(nd.W)[::-1])"),
    "ibp_wrong_operand": ("L.append(Wp @ l + Wn @ u + _f64(nd.b))", "L.append(Wp @ l + Wn @ l + _f64(nd.b))"),
    "ibp_conv_wrong_operand": ("L.append(conv2d(l, Wp, nd.stride, nd.pad) + conv2d(u, Wn, nd.stride, nd.pad) + b)",
                               "L.append(conv2d(l, Wp, nd.stride, nd.pad) + conv2d(l, Wn, nd.stride, nd.pad) + b)"),
    "concretize_wrong_vertex": ("np.minimum(A_x * lo, A_x * hi)", "np.minimum(A_x * lo, A_x * lo)"),
    "lambda_rule_flipped": ("np.where(uu > -lu, 1.0, 0.0)", "np.where(uu > -lu, 0.0, 1.0)"),
    "chord_slope_wrong": ("su = uu / (uu - lu)", "su = -lu / (uu - lu)"),
    "chord_intercept_sign": ("t[unstable] = -su * lu", "t[unstable] = su * lu"),
    "add_drops_branch": ('elif nd.op == "add":\n            _accumulate(acc, nd.in0, Ai)\n            _accumulate(acc, nd.in1, Ai)',
                         'elif nd.op == "add":\n            _accumulate(acc, nd.in0, Ai)\n            pass'),
    "conv_transpose_misaligned": ("return out[:, :, pad:pad + h, pad:pad + w]", "return out[:, :, :h, :w]"),
    "conv_transpose_unflipped_stride": ("j:j + stride * (wo - 1) + 1:stride] += contrib",
                                        "j:j + (wo - 1) + 1:1] += contrib"),
    "split_clamps_wrong_side": ("L[i][j] = max(L[i][j], 0.0)", "U[i][j] = max(U[i][j], 0.0)"),
    "box_not_clipped": ("lo = np.maximum(lo, np.float32(clip[0]))", "lo = lo"),
    "intersect_reversed": ("l = np.maximum(l, il)", "l = np.minimum(l, il)"),
    "final_upper_uses_lower_rule": ("Au, bu = backward(net, shapes, relax, out, Cm, zero, upper=True)",
                                    "Au, bu = backward(net, shapes, relax, out, Cm, zero, upper=False)"),
    "direct_affine_upper_wrong": ("concretize(W, b, lo, hi, False), concretize(W, b, lo, hi, True)",
                                  "concretize(W, b, lo, hi, False), concretize(W, b, lo, hi, False)"),
    "infeasible_not_detected": ("if np.any(L[i] > U[i]):", "if False:"),
}


def _mutant(old, new):
    src = open(SRC).read()
    # the mistake is planted everywhere the anchor occurs (the receptive-field sampler repeats
    # some of the full oracle's steps)
    assert src.count(old) >= 1, f"mutation anchor missing: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    sys.modules["oracle_mutant"] = mod          # dataclasses look their module up here
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    mod = _mutant(*MUTANTS[name])
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except Exception:
            return
    pytest.fail(f"mutant {name} passed every pin")


ALPHA_MUTANTS = {
    "alpha_upper_pass_uses_lower_rule": ("        if not upper:\n                bias = bias + An @ t",
                                         "        if True:\n                bias = bias + An @ t"),
    "alpha_grad_branch_swapped": ("on_lam, on_chord_t = a > 0.0, a < 0.0", "on_lam, on_chord_t = a < 0.0, a > 0.0"),
    "alpha_grad_drops_intercept": ("s[None, :] * D + np.where(on_chord_t, t[None, :], 0.0)", "s[None, :] * D"),
    "alpha_grad_wrong_vertex": ("else c[None, :] - sgn * r[None, :]", "else c[None, :] + sgn * r[None, :]"),
    "alpha_no_projection": ("np.clip(a[i] + sign * lr * mhat / (np.sqrt(vhat) + adam_eps), 0.0, 1.0)",
                            "a[i] + sign * lr * mhat / (np.sqrt(vhat) + adam_eps)"),
    "alpha_upper_ascends": ('(("l", al, gl, 1.0), ("u", au, gu, -1.0))', '(("l", al, gl, 1.0), ("u", au, gu, 1.0))'),
    "alpha_best_not_kept": ("best_l = np.where(better_l, lb, best_l)", "best_l = lb"),
    # residual networks: one input of an add dropped in the backward pass, or in the forward
    # evaluation of the gradient
    "alpha_pass_add_drops_branch": ("            add_to(nd.in0, A)\n            add_to(nd.in1, A)",
                                    "            add_to(nd.in0, A)"),
    "alpha_grad_add_drops_skip": ("val[i] = v.reshape(rows, -1) + get(nd.in1).reshape(rows, -1)",
                                  "val[i] = v.reshape(rows, -1)"),
}


def _alpha_mutant(old, new):
    src = open(SRC_ALPHA).read()
    assert src.count(old) >= 1, f"mutation anchor missing: {old!r}"
    mod = types.ModuleType("alpha_mutant")
    sys.modules["alpha_mutant"] = mod
    exec(compile(src.replace(old, new), "alpha_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(ALPHA_MUTANTS))
def test_alpha_mutant_is_caught(name):
    mod = _alpha_mutant(*ALPHA_MUTANTS[name])
    for pin in pins_alpha.ALPHA_PINS:
        try:
            pin(mod)
        except Exception:
            return
    pytest.fail(f"mutant {name} passed every pin")


SRC_BETA = os.path.join(ORACLE_DIR, "beta64.py")
BETA_MUTANTS = {
    "beta_term_dropped": ("A[:, j] += (-S if upper else S) * beta[:, e]", "A[:, j] += 0.0 * beta[:, e]"),
    "beta_term_sign_flipped": ("A[:, j] += (-S if upper else S) * beta[:, e]", "A[:, j] += (S if upper else -S) * beta[:, e]"),
    "beta_grad_sign_flipped": ("gb[:, e] = (-S if upper else S) * D[:, j]", "gb[:, e] = (S if upper else -S) * D[:, j]"),
    "beta_not_projected": ('bl = adam("bl", bl, gbl, 1.0, lr_beta, 0.0, np.inf)', 'bl = adam("bl", bl, gbl, 1.0, lr_beta, -np.inf, np.inf)'),
    "beta_split_sign_ignored": ("(ids[int(r)], int(j), -1.0 if sg > 0 else 1.0)", "(ids[int(r)], int(j), 1.0)"),
    "bab_branches_same_neuron": ("nxt = next((o for o in order if o not in used), None)", "nxt = order[0] if order else None"),
    "bab_keeps_verified": ("if np.all(r.lb > 0.0):\n                pruned += 1", "if False:\n                pruned += 1"),
    # residual networks: an add's coefficients reach one input only; the forward evaluation
    # drops the skip connection
    "beta_add_one_input": ("            add_to(nd.in0, A)\n            add_to(nd.in1, A)",
                           "            add_to(nd.in0, A)"),
    "beta_forward_drops_skip": ("val[i] = v.reshape(rows, -1) + get(nd.in1).reshape(rows, -1)",
                                "val[i] = get(nd.in1).reshape(rows, -1)"),
}


def _beta_mutant(old, new):
    src = open(SRC_BETA).read()
    assert src.count(old) >= 1, f"mutation anchor missing: {old!r}"
    mod = types.ModuleType("beta_mutant")
    sys.modules["beta_mutant"] = mod
    exec(compile(src.replace(old, new), "beta_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(BETA_MUTANTS))
def test_beta_mutant_is_caught(name):
    mod = _beta_mutant(*BETA_MUTANTS[name])
    for pin in pins_beta.BETA_PINS:
        try:
            pin(mod)
        except Exception:
            return
    pytest.fail(f"mutant {name} passed every pin")
