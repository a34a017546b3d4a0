"""Pins for the fp64 oracle: checks against facts the paper and the mathematics fix.

Every pin takes the oracle module as its argument, so the same checks run against the real
oracle (tests/test_oracle_pins.py, all must pass) and against copies of it with a planted
mistake (tests/test_oracle_mutants.py, each mutant must fail at least one pin).

None of these re-types the oracle's formulas.  They use closed forms of special networks,
exact extrema of affine maps attained at box vertices, plain forward evaluation at sampled
points and on dense grids, a linear-programming solve of the triangle relaxation, library
convolutions, and the worked example printed in the paper.
"""
from __future__ import annotations

import json
import os

import numpy as np

from workloads import Net, Node, random_mlp, make_workload

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# --------------------------------------------------------------------------------------
# independent evaluation helpers (not the oracle's code)

def batch_forward(net, X):
    """fp64 forward of many points at once; dense/relu/add/flatten via numpy, conv via torch."""
    X = np.asarray(X, np.float64)
    vals = []
    n = X.shape[0]
    inp = X.reshape((n,) + tuple(net.in_shape))
    get = lambda i: inp if i == -1 else vals[i]  # noqa: E731
    for nd in net.nodes:
        v = get(nd.in0)
        if nd.op == "dense":
            vals.append(v.reshape(n, -1) @ np.asarray(nd.W, np.float64).T + np.asarray(nd.b, np.float64))
        elif nd.op == "conv2d":
            import torch
            out = torch.nn.functional.conv2d(torch.from_numpy(v), torch.from_numpy(np.asarray(nd.W, np.float64)),
                                             torch.from_numpy(np.asarray(nd.b, np.float64)),
                                             stride=nd.stride, padding=nd.pad)
            vals.append(out.numpy())
        elif nd.op == "relu":
            vals.append(np.maximum(v, 0.0))
        elif nd.op == "add":
            vals.append(v + get(nd.in1))
        elif nd.op == "flatten":
            vals.append(v.reshape(n, -1))
    return vals


def spec_values(net, C, X):
    return batch_forward(net, X)[-1].reshape(X.shape[0], -1) @ np.asarray(C, np.float64).T


def box_of(x0, eps, clip):
    # the box definition: float32 x0 -/+ eps, rounded to nearest, clamped to the clip box
    x0 = np.asarray(x0, np.float32)
    lo = (x0 - np.float32(eps)).astype(np.float32)
    hi = (x0 + np.float32(eps)).astype(np.float32)
    if clip is not None:
        lo = np.maximum(lo, np.float32(clip[0]))
        hi = np.minimum(hi, np.float32(clip[1]))
    return lo.astype(np.float64), hi.astype(np.float64)


def vertex_for(a, lo, hi, minimise):
    """Vertex of the box where a . x is minimal (or maximal)."""
    return np.where((a > 0) == minimise, lo, hi)


def assert_sound(lb, ub, Y, slack_rel=1e-9, what=""):
    Y = np.atleast_2d(Y)
    tol = slack_rel * (1.0 + np.abs(Y))
    bad_l = Y < lb[None, :] - tol
    bad_u = Y > ub[None, :] + tol
    assert not bad_l.any(), f"{what}: lower bound violated by {np.max(lb[None, :] - Y)}"
    assert not bad_u.any(), f"{what}: upper bound violated by {np.max(Y - ub[None, :])}"


# --------------------------------------------------------------------------------------
# the pins

def pin_relu_hand_values(o):
    """ReLU relaxation at hand-computed, exactly representable points."""
    lam, s, t = o.relu_relaxation(np.array([-1.0, -2.0, -1.0, 0.0, 0.5, -3.0, -1.0]),
                                  np.array([2.0, 1.0, 1.0, 3.0, 2.0, 0.0, -0.5]))
    np.testing.assert_allclose(lam, [1, 0, 0, 1, 1, 0, 0], atol=0)
    np.testing.assert_allclose(s, [2 / 3, 1 / 3, 1 / 2, 1, 1, 0, 0], rtol=1e-15)
    np.testing.assert_allclose(t, [2 / 3, 2 / 3, 1 / 2, 0, 0, 0, 0], rtol=1e-15)
    # the two lines enclose ReLU on the whole interval, and the upper line is the chord
    for l, u in [(-1.0, 2.0), (-2.0, 1.0), (-1.0, 1.0), (-0.3, 5.0), (-7.0, 0.01)]:
        la, sa, ta = (v[0] for v in o.relu_relaxation(np.array([l]), np.array([u])))
        z = np.linspace(l, u, 2001)
        r = np.maximum(z, 0)
        assert np.all(la * z <= r + 1e-15) and np.all(r <= sa * z + ta + 1e-12)
        assert abs(sa * l + ta) < 1e-12 and abs(sa * u + ta - u) < 1e-12


def _relu_on_input_net():
    return Net((1,), [Node("relu", -1), Node("dense", 0, W=np.ones((1, 1), np.float32),
                                               b=np.zeros(1, np.float32))])


def pin_relu_net_bounds(o):
    """y = ReLU(x) on [-1,2], [-2,1], [-1,1]: CROWN gives [-1,2], [0,1], [0,1]."""
    net = _relu_on_input_net()
    C = np.ones((1, 1), np.float32)
    for x0, eps, want in [(0.5, 1.5, (-1.0, 2.0)), (-0.5, 1.5, (0.0, 1.0)), (0.0, 1.0, (0.0, 1.0))]:
        r = o.crown(net, np.array([x0], np.float32), eps, C, clip=None)
        assert r.lb[0] == want[0] and abs(r.ub[0] - want[1]) < 1e-15, (x0, eps, r.lb, r.ub)


def pin_single_affine(o):
    """One dense layer: IBP and CROWN both give the exact range W x0 + b -/+ eps |W| 1,
    attained at the box vertices."""
    rng = np.random.default_rng(11)
    W = rng.standard_normal((7, 5)).astype(np.float32)
    b = rng.standard_normal(7).astype(np.float32)
    net = Net((5,), [Node("dense", -1, W=W, b=b)])
    x0 = rng.random(5).astype(np.float32)
    eps = np.float32(0.125)           # x0 -/+ eps exact in float32 for x0 in [0,1)? not
    C = np.eye(7, dtype=np.float32)   # always, hence the rounding-level tolerance below
    r = o.crown(net, x0, eps, C, clip=None)
    il, iu = o.ibp_spec_bounds(net, x0, eps, C, clip=None)
    W64, x64 = W.astype(np.float64), x0.astype(np.float64)
    cf_l = W64 @ x64 + b - 0.125 * np.abs(W64).sum(1)
    cf_u = W64 @ x64 + b + 0.125 * np.abs(W64).sum(1)
    for got in (r.lb, il):
        np.testing.assert_allclose(got, cf_l, rtol=1e-6, atol=1e-6)
    for got in (r.ub, iu):
        np.testing.assert_allclose(got, cf_u, rtol=1e-6, atol=1e-6)
    lo, hi = box_of(x0, eps, None)
    for i in range(7):
        vl = vertex_for(W64[i], lo, hi, True)
        vu = vertex_for(W64[i], lo, hi, False)
        assert abs(r.lb[i] - (W64[i] @ vl + b[i])) < 1e-12
        assert abs(r.ub[i] - (W64[i] @ vu + b[i])) < 1e-12


def _all_active_net(seed, dims):
    rng = np.random.default_rng(seed)
    nodes, prev = [], -1
    for i in range(1, len(dims)):
        W = (rng.standard_normal((dims[i], dims[i - 1])) * (0.2 / np.sqrt(dims[i - 1]))).astype(np.float32)
        b = np.full(dims[i], 10.0, np.float32)
        nodes.append(Node("dense", prev, W=W, b=b))
        prev = len(nodes) - 1
        if i < len(dims) - 1:
            nodes.append(Node("relu", prev))
            prev = len(nodes) - 1
    return Net((dims[0],), nodes)


def pin_all_stable(o):
    """An all-active ReLU net is affine on the box, so CROWN is exact: lb = min over the box
    of C W_eff x + const, attained at the vertex chosen by the signs of C W_L...W_1."""
    dims = [6, 9, 8, 7, 4]
    net = _all_active_net(3, dims)
    rng = np.random.default_rng(4)
    x0 = rng.random(6).astype(np.float32)
    eps = np.float32(0.05)
    C = rng.standard_normal((3, 4)).astype(np.float32)
    r = o.crown(net, x0, eps, C)
    for i in r.layer_l:
        assert np.all(r.layer_l[i] > 0), "test net is meant to be all active"
    Weff = C.astype(np.float64)
    for nd in reversed(net.nodes):
        if nd.op == "dense":
            Weff = Weff @ nd.W.astype(np.float64)
    lo, hi = box_of(x0, eps, (0.0, 1.0))
    for k in range(3):
        xl = vertex_for(Weff[k], lo, hi, True)
        xu = vertex_for(Weff[k], lo, hi, False)
        yl = spec_values(net, C, xl[None])[0, k]
        yu = spec_values(net, C, xu[None])[0, k]
        assert abs(r.lb[k] - yl) <= 1e-10 * (1 + abs(yl)), (r.lb[k], yl)
        assert abs(r.ub[k] - yu) <= 1e-10 * (1 + abs(yu)), (r.ub[k], yu)
    # IBP is sound but strictly looser on the same net
    il, iu = o.ibp_spec_bounds(net, x0, eps, C)
    assert np.all(il < r.lb - 1e-9) and np.all(iu > r.ub + 1e-9)


def pin_inactive_layer_constant(o):
    """A layer whose pre-activations are negative on the whole box cuts the input off: the
    output is constant and CROWN returns lb = ub = C f(x0)."""
    net = _all_active_net(5, [6, 9, 8, 4])
    net.nodes[2].b = np.full(8, -100.0, np.float32)     # second hidden layer: all inactive
    x0 = np.random.default_rng(6).random(6).astype(np.float32)
    C = np.eye(4, dtype=np.float32)
    r = o.crown(net, x0, 0.1, C)
    y = spec_values(net, C, x0[None].astype(np.float64))[0]
    np.testing.assert_allclose(r.lb, y, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r.ub, y, rtol=0, atol=1e-12)


def pin_paper_wrapping_example(o):
    """The paper's illustrative example of the wrapping effect (Sec. 3.3.2): CROWN gives
    [-2, 2] for z1 = y1 + y2 with y = W x, x in [-1, 1]^2, while IBP gives [-4, 4]."""
    with open(os.path.join(GOLDEN, "wrapping_example.json")) as f:
        g = json.load(f)
    # as a ReLU network: ReLU(W x + 2) is the identity on the box (pre-activations in
    # [0, 4]), followed by z = [1, 1] h - 4
    W = np.array(g["W"], np.float32)
    net = Net((2,), [Node("dense", -1, W=W, b=np.full(2, 2.0, np.float32)),
                     Node("relu", 0),
                     Node("dense", 1, W=np.ones((1, 2), np.float32), b=np.array([-4.0], np.float32))])
    x0 = np.array(g["x_center"], np.float32)
    C = np.ones((1, 1), np.float32)
    r = o.crown(net, x0, g["x_radius"], C, clip=None)
    il, iu = o.ibp_spec_bounds(net, x0, g["x_radius"], C, clip=None)
    assert (r.lb[0], r.ub[0]) == tuple(g["crown"]), (r.lb, r.ub)
    assert (il[0], iu[0]) == tuple(g["ibp"]), (il, iu)


def pin_wrapping_example_intermediate(o):
    """The same example one layer deeper: z1 = y1 + y2 feeds a ReLU, so its interval is an
    intermediate bound and must be CROWN's exact [-2, 2], not IBP's [-4, 4].  ReLU(z1) =
    ReLU(2 x1) then has the exact range [0, 2]."""
    with open(os.path.join(GOLDEN, "wrapping_example.json")) as f:
        g = json.load(f)
    W = np.array(g["W"], np.float32)
    net = Net((2,), [Node("dense", -1, W=W, b=np.full(2, 2.0, np.float32)),
                     Node("relu", 0),
                     Node("dense", 1, W=np.ones((1, 2), np.float32), b=np.array([-4.0], np.float32)),
                     Node("relu", 2),
                     Node("dense", 3, W=np.ones((1, 1), np.float32), b=np.zeros(1, np.float32))])
    r = o.crown(net, np.array(g["x_center"], np.float32), g["x_radius"], np.ones((1, 1), np.float32), clip=None)
    assert (r.layer_l[3][0], r.layer_u[3][0]) == tuple(g["crown"])
    assert (r.ibp_l[3][0], r.ibp_u[3][0]) == tuple(g["ibp"])
    assert (r.lb[0], r.ub[0]) == (0.0, 2.0), (r.lb, r.ub)


def pin_eps_zero(o):
    """eps = 0: the box is a point and lb = ub = C f(x0)."""
    wl = random_mlp(21, [12, 20, 20, 5], 2, 0.0)
    for b in range(2):
        r = o.crown(wl.net, wl.x0[b], 0.0, wl.C[b])
        y = spec_values(wl.net, wl.C[b], wl.x0[b][None])[0]
        np.testing.assert_allclose(r.lb, y, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r.ub, y, rtol=1e-12, atol=1e-12)


def pin_lp_sandwich(o):
    """One hidden layer: CROWN lb <= (triangle-relaxation LP optimum) <= sampled minimum,
    and the same mirrored for ub."""
    from scipy.optimize import linprog
    for seed, n0, n1 in [(31, 2, 12), (32, 4, 10), (33, 8, 16)]:
        wl = random_mlp(seed, [n0, n1, 3], 1, 0.3)
        net = wl.net
        r = o.crown(net, wl.x0[0], wl.eps, wl.C[0])
        l, u = r.layer_l[1], r.layer_u[1]
        lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
        W1, b1 = net.nodes[0].W.astype(np.float64), net.nodes[0].b.astype(np.float64)
        W2, b2 = net.nodes[2].W.astype(np.float64), net.nodes[2].b.astype(np.float64)
        C = wl.C[0].astype(np.float64)
        # variables v = [x (n0), h (n1)]; z = W1 x + b1 is substituted
        A_ub, b_ub = [], []
        A_eq, b_eq = [], []
        for j in range(n1):
            row_z = np.concatenate([W1[j], np.zeros(n1)])
            e_h = np.zeros(n0 + n1)
            e_h[n0 + j] = 1.0
            if u[j] <= 0:
                A_eq.append(e_h); b_eq.append(0.0)
            elif l[j] >= 0:
                A_eq.append(e_h - row_z); b_eq.append(b1[j])
            else:
                A_ub.append(row_z - e_h); b_ub.append(-b1[j])            # h >= z
                A_ub.append(-e_h); b_ub.append(0.0)                      # h >= 0
                k = u[j] / (u[j] - l[j])
                A_ub.append(e_h - k * row_z); b_ub.append(k * (b1[j] - l[j]))   # h <= k (z - l)
        bounds = [(lo[i], hi[i]) for i in range(n0)] + [(None, None)] * n1
        X = lo + (hi - lo) * np.random.default_rng(seed).random((20000, n0))
        Y = spec_values(net, C, X)
        for k in range(C.shape[0]):
            c = C[k] @ W2
            kw = dict(A_ub=np.array(A_ub) if A_ub else None, b_ub=np.array(b_ub) if b_ub else None,
                      A_eq=np.array(A_eq) if A_eq else None, b_eq=np.array(b_eq) if b_eq else None,
                      bounds=bounds, method="highs")
            lp_min = linprog(np.concatenate([np.zeros(n0), c]), **kw)
            lp_max = linprog(-np.concatenate([np.zeros(n0), c]), **kw)
            assert lp_min.status == 0 and lp_max.status == 0
            lmin = lp_min.fun + C[k] @ b2
            lmax = -lp_max.fun + C[k] @ b2
            assert r.lb[k] <= lmin + 1e-7 * (1 + abs(lmin)), (seed, k, r.lb[k], lmin)
            assert lmin <= Y[:, k].min() + 1e-7 * (1 + abs(lmin))
            assert r.ub[k] >= lmax - 1e-7 * (1 + abs(lmax)), (seed, k, r.ub[k], lmax)
            assert lmax >= Y[:, k].max() - 1e-7 * (1 + abs(lmax))


def pin_soundness(o, net, x0, eps, C, clip=(0.0, 1.0), n_samples=20000, n_corners=2000, seed=0,
                  lambda_rule="adaptive"):
    """The soundness contract (Sec. 2.1.1): no sampled point, random box corner or the
    vertex where a final linear bound is attained lies outside [lb, ub]."""
    r = o.crown(net, x0, eps, C, clip=clip, keep_A=True, lambda_rule=lambda_rule)
    lo, hi = box_of(x0, eps, clip)
    rng = np.random.default_rng(seed)
    X = lo + (hi - lo) * rng.random((n_samples, lo.size))
    Xc = np.where(rng.random((n_corners, lo.size)) < 0.5, lo, hi)
    Xa = np.concatenate([[vertex_for(a, lo, hi, True) for a in r.A_lower],
                         [vertex_for(a, lo, hi, False) for a in r.A_upper]])
    for name, P in (("samples", X), ("corners", Xc), ("A-guided corners", Xa)):
        assert_sound(r.lb, r.ub, spec_values(net, C, P), what=name)
    # every intermediate bound contains the sampled pre-activations
    vals = batch_forward(net, X[:2000])
    for i in r.layer_l:
        z = vals[net.nodes[i].in0].reshape(2000, -1)
        assert np.all(z >= r.layer_l[i] - 1e-9 * (1 + np.abs(z))), f"layer {i} lower"
        assert np.all(z <= r.layer_u[i] + 1e-9 * (1 + np.abs(z))), f"layer {i} upper"
    return r


def pin_soundness_mlps(o):
    wl = make_workload("mlp784x256x2")
    pin_soundness(o, wl.net, wl.x0[0], wl.eps, wl.C[0], n_samples=20000)
    for seed, dims, eps in [(41, [10, 30, 30, 30, 4], 0.08), (42, [5, 40, 3], 0.3)]:
        wl = random_mlp(seed, dims, 1, eps)
        pin_soundness(o, wl.net, wl.x0[0], wl.eps, wl.C[0])


def pin_upper_is_negated_lower(o):
    """ub(C) = -lb(-C): the explicit upper rule mirrors the lower rule exactly."""
    wl = make_workload("mlp784x256x2")
    r1 = o.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    r2 = o.crown(wl.net, wl.x0[0], wl.eps, -wl.C[0])
    assert np.array_equal(r1.ub, -r2.lb) and np.array_equal(r1.lb, -r2.ub)
    net = tiny_resnet(7)
    x0 = np.random.default_rng(8).random(net.n_in).astype(np.float32)
    C = np.random.default_rng(9).standard_normal((3, 5)).astype(np.float32)
    r1 = o.crown(net, x0, 0.02, C)
    r2 = o.crown(net, x0, 0.02, -C)
    assert np.array_equal(r1.ub, -r2.lb) and np.array_equal(r1.lb, -r2.ub)


def pin_grid_bruteforce(o, lambda_rule="adaptive"):
    """2-input nets on a dense 1001 x 1001 grid: lb <= grid min and ub >= grid max."""
    for seed, dims in [(51, [2, 16, 16, 2]), (52, [2, 32, 32, 32, 3])]:
        wl = random_mlp(seed, dims, 1, 0.25)
        C = np.eye(dims[-1], dtype=np.float32)
        r = o.crown(wl.net, wl.x0[0], wl.eps, C, lambda_rule=lambda_rule)
        lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
        g0 = np.linspace(lo[0], hi[0], 1001)
        g1 = np.linspace(lo[1], hi[1], 1001)
        X = np.stack(np.meshgrid(g0, g1, indexing="ij"), -1).reshape(-1, 2)
        Y = spec_values(wl.net, C, X)
        assert_sound(r.lb, r.ub, Y, what=f"grid {dims}")


def tiny_resnet(seed, c=4, hw=6, n_out=5):
    """A small net with every op the conv path has: conv, residual add with a ReLU branch,
    stride-2 conv, flatten, dense, ReLU, dense."""
    rng = np.random.default_rng(seed)

    def cw(co, ci):
        return ((rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2 / (ci * 9))).astype(np.float32),
                (rng.standard_normal(co) * 0.1).astype(np.float32))

    W0, b0 = cw(c, 2)
    W1, b1 = cw(c, c)
    W2, b2 = cw(c, c)
    W3, b3 = cw(2 * c, c)
    n_flat = 2 * c * (hw // 2) * (hw // 2)
    W4 = (rng.standard_normal((8, n_flat)) * np.sqrt(2 / n_flat)).astype(np.float32)
    b4 = (rng.standard_normal(8) * 0.1).astype(np.float32)
    W5 = (rng.standard_normal((n_out, 8)) * np.sqrt(2 / 8)).astype(np.float32)
    b5 = (rng.standard_normal(n_out) * 0.1).astype(np.float32)
    nodes = [Node("conv2d", -1, W=W0, b=b0, stride=1, pad=1),      # 0
             Node("conv2d", 0, W=W1, b=b1, stride=1, pad=1),       # 1
             Node("relu", 1),                                      # 2
             Node("conv2d", 2, W=W2, b=b2, stride=1, pad=1),       # 3
             Node("add", 0, 3),                                    # 4
             Node("conv2d", 4, W=W3, b=b3, stride=2, pad=1),       # 5
             Node("relu", 5),                                      # 6
             Node("flatten", 6),                                   # 7
             Node("dense", 7, W=W4, b=b4),                         # 8
             Node("relu", 8),                                      # 9
             Node("dense", 9, W=W5, b=b5)]                         # 10
    return Net((2, hw, hw), nodes)


def _conv_matrix(W, stride, pad, in_shape):
    """Dense matrix of a bias-free convolution, column k = conv of the k-th basis tensor
    (library convolution)."""
    import torch
    n = int(np.prod(in_shape))
    E = torch.eye(n, dtype=torch.float64).reshape((n,) + tuple(in_shape))
    out = torch.nn.functional.conv2d(E, torch.from_numpy(W.astype(np.float64)), stride=stride, padding=pad)
    return out.reshape(n, -1).T.numpy(), tuple(out.shape[1:])


def pin_conv_library(o):
    """conv2d / conv2d_transpose equal torch's conv2d / conv_transpose2d in fp64."""
    import torch
    rng = np.random.default_rng(61)
    for stride, pad, hw in [(1, 1, 7), (2, 1, 8), (2, 1, 7), (1, 0, 6)]:
        W = rng.standard_normal((5, 3, 3, 3))
        x = rng.standard_normal((3, hw, hw))
        got = o.conv2d(x, W, stride, pad)
        want = torch.nn.functional.conv2d(torch.from_numpy(x[None]), torch.from_numpy(W),
                                          stride=stride, padding=pad)[0].numpy()
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
        A = rng.standard_normal((4,) + want.shape)
        got_t = o.conv2d_transpose(A, W, stride, pad, (hw, hw))
        outpad = hw + 2 * pad - 3 - stride * (want.shape[1] - 1)
        want_t = torch.nn.functional.conv_transpose2d(torch.from_numpy(A), torch.from_numpy(W), stride=stride,
                                                      padding=pad, output_padding=outpad).numpy()
        np.testing.assert_allclose(got_t, want_t, rtol=1e-12, atol=1e-12)


def pin_conv_net_equals_unrolled(o):
    """The same network with every convolution unrolled into its dense matrix gives the
    same CROWN bounds (to 1e-10), and the IBP bounds agree as well."""
    net = tiny_resnet(71)
    shapes = o.node_shapes(net)
    nodes = []
    for i, nd in enumerate(net.nodes):
        if nd.op == "conv2d":
            ins = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
            M, oshape = _conv_matrix(nd.W, nd.stride, nd.pad, ins)
            bb = np.repeat(nd.b.astype(np.float64), oshape[1] * oshape[2])
            nodes.append(Node("dense", nd.in0, W=M, b=bb))
        elif nd.op == "flatten":
            nodes.append(Node("flatten", nd.in0))
        else:
            nodes.append(Node(nd.op, nd.in0, nd.in1, nd.W, nd.b, nd.stride, nd.pad))
    flat = Net((net.n_in,), nodes)
    x0 = np.random.default_rng(72).random(net.n_in).astype(np.float32)
    C = np.random.default_rng(73).standard_normal((4, 5)).astype(np.float32)
    r1 = o.crown(net, x0, 0.03, C)
    r2 = o.crown(flat, x0, 0.03, C)
    np.testing.assert_allclose(r1.lb, r2.lb, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(r1.ub, r2.ub, rtol=1e-10, atol=1e-10)
    for i in r1.layer_l:
        np.testing.assert_allclose(r1.layer_l[i], r2.layer_l[i], rtol=1e-10, atol=1e-10)
        np.testing.assert_allclose(r1.layer_u[i], r2.layer_u[i], rtol=1e-10, atol=1e-10)
    # the conv net's bounds are also sound
    pin_soundness(o, net, x0, 0.03, C, n_samples=3000, n_corners=300)


def pin_residual_closed_form(o):
    """y = x + (W x + b): CROWN is exact, lb = min over the box of (I + W) x + b."""
    rng = np.random.default_rng(81)
    W = (rng.standard_normal((6, 6)) * 0.5).astype(np.float32)
    b = rng.standard_normal(6).astype(np.float32)
    net = Net((6,), [Node("dense", -1, W=W, b=b), Node("add", -1, 0)])
    x0 = rng.random(6).astype(np.float32)
    C = np.eye(6, dtype=np.float32)
    r = o.crown(net, x0, 0.2, C)
    M = np.eye(6) + W.astype(np.float64)
    lo, hi = box_of(x0, 0.2, (0.0, 1.0))
    for k in range(6):
        want_l = M[k] @ vertex_for(M[k], lo, hi, True) + b[k]
        want_u = M[k] @ vertex_for(M[k], lo, hi, False) + b[k]
        assert abs(r.lb[k] - want_l) < 1e-12 and abs(r.ub[k] - want_u) < 1e-12


def pin_bab_invariants(o):
    """Subdomains (Sec. 2.1.1, complete verification): bounds hold on the points of the
    subdomain; splitting a neuron into the state it is already stably in changes nothing;
    contradicting a stable state makes the domain infeasible."""
    from workloads import Splits
    wl = random_mlp(91, [8, 24, 24, 3], 1, 0.15)
    net, x0, C = wl.net, wl.x0[0], wl.C[0]
    root = o.crown(net, x0, wl.eps, C)
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    lo, hi = box_of(x0, wl.eps, wl.clip)
    X = lo + (hi - lo) * np.random.default_rng(92).random((40000, lo.size))
    vals = batch_forward(net, X)
    z0 = batch_forward(net, x0[None].astype(np.float64))
    pool = o.unstable_pool(net, root)
    assert len(pool) >= 6
    rng = np.random.default_rng(93)
    doms = []
    for d in range(12):
        pick = pool[rng.choice(len(pool), 3, replace=False)]
        if d < 4:    # agree with x0's own activation pattern
            sg = [1 if z0[net.nodes[relus[r]].in0][0, j] >= 0 else -1 for r, j in pick]
        else:
            sg = list(rng.choice([-1, 1], 3))
        doms.append((pick[:, 0], pick[:, 1], sg))
    sp = Splits(np.array([d[0] for d in doms], np.int32), np.array([d[1] for d in doms], np.int32),
                np.array([d[2] for d in doms], np.int8))
    LB, UB = o.crown_domains(net, root, C, sp)
    y0 = spec_values(net, C, x0[None].astype(np.float64))[0]
    n_checked = 0
    for d in range(len(doms)):
        if d < 4:
            assert np.all(LB[d] <= y0 + 1e-9) and np.all(UB[d] >= y0 - 1e-9)
        member = np.ones(X.shape[0], bool)
        for r, j, s in zip(*doms[d]):
            z = vals[net.nodes[relus[r]].in0][:, j]
            member &= (z >= 0) if s > 0 else (z <= 0)
        if member.any():
            n_checked += 1
            assert_sound(LB[d], UB[d], spec_values(net, C, X[member]), what=f"domain {d}")
    assert n_checked >= 6
    # stable-state splits are no-ops, bit for bit
    i1 = relus[0]
    act = int(np.nonzero(root.layer_l[i1] > 0)[0][0])
    ina = int(np.nonzero(root.layer_u[i1] < 0)[0][0])
    sp2 = Splits(np.array([[0, 0]], np.int32), np.array([[act, ina]], np.int32), np.array([[1, -1]], np.int8))
    LB2, UB2 = o.crown_domains(net, root, C, sp2)
    assert np.array_equal(LB2[0], root.lb) and np.array_equal(UB2[0], root.ub)
    sp3 = Splits(np.array([[0]], np.int32), np.array([[ina]], np.int32), np.array([[1]], np.int8))
    LB3, UB3 = o.crown_domains(net, root, C, sp3)
    assert np.all(LB3 == np.inf) and np.all(UB3 == -np.inf)


def pin_lambda_rules_sound(o):
    """Every lower slope in [0, 1] is sound: the zero / one / same-slope rules pass the
    sampling and grid checks too."""
    wl = random_mlp(41, [10, 30, 30, 30, 4], 1, 0.08)
    for rule in ("zero", "one", "same_slope"):
        pin_soundness(o, wl.net, wl.x0[0], wl.eps, wl.C[0], n_samples=5000, n_corners=500, lambda_rule=rule)
        pin_grid_bruteforce(o, lambda_rule=rule)


def pin_ibp_sound_and_contains_crown(o):
    """IBP intervals contain all sampled values; CROWN's intermediate bounds computed
    without the IBP intersection are still sound."""
    wl = random_mlp(45, [10, 30, 30, 30, 4], 1, 0.08)
    lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
    L, U = o.ibp(wl.net, lo, hi)
    X = lo + (hi - lo) * np.random.default_rng(46).random((5000, lo.size))
    vals = batch_forward(wl.net, X)
    for i in range(len(wl.net.nodes)):
        v = vals[i].reshape(5000, -1)
        assert np.all(v >= L[i].reshape(-1) - 1e-9) and np.all(v <= U[i].reshape(-1) + 1e-9)
    r = o.crown(wl.net, wl.x0[0], wl.eps, wl.C[0], intersect_ibp=False)
    for i in r.layer_l:
        z = vals[wl.net.nodes[i].in0].reshape(5000, -1)
        assert np.all(z >= r.layer_l[i] - 1e-9) and np.all(z <= r.layer_u[i] + 1e-9)
    il, iu = o.ibp_spec_bounds(wl.net, wl.x0[0], wl.eps, wl.C[0])
    assert_sound(il, iu, spec_values(wl.net, wl.C[0], X), what="ibp spec")


def pin_sampled_equals_full(o):
    """Bounds of selected neurons computed through their receptive fields equal the full
    pass's bounds of those neurons (same arithmetic; the skipped rows only meet zeros)."""
    net = tiny_resnet(75, c=4, hw=8)
    x0 = np.random.default_rng(76).random(net.n_in).astype(np.float32)
    C = np.random.default_rng(77).standard_normal((2, 5)).astype(np.float32)
    full = o.crown(net, x0, 0.05, C)
    relus = sorted(full.layer_l)
    rng = np.random.default_rng(78)
    targets = {relus[1]: rng.choice(full.layer_l[relus[1]].size, 3, replace=False),
               relus[0]: rng.choice(full.layer_l[relus[0]].size, 2, replace=False)}
    got = o.crown_sampled(net, x0, 0.05, targets)
    for i, idx in targets.items():
        gi, gl, gu = got[i]
        pos = np.searchsorted(gi, idx)
        np.testing.assert_allclose(gl[pos], full.layer_l[i][idx], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(gu[pos], full.layer_u[i][idx], rtol=1e-12, atol=1e-12)
    # the receptive field of a second-block neuron does not cover the whole first layer
    assert len(got[relus[0]][0]) < full.layer_l[relus[0]].size


# fastest first (the mutant test stops at the first pin that fails)
def pin_one_hidden_equals_crown(o):
    """The row-block computation for one hidden layer gives the full oracle's bounds (blocks
    smaller than the layer, and a one-output property C = [[1]])."""
    from workloads.gen import mlp_net
    for seed, dims, eps, chunk in [(91, [6, 40, 3], 0.2, 7), (92, [20, 300, 5], 0.05, 64), (93, [64, 2000, 1], 0.01, 300)]:
        if dims[-1] > 1:
            wl = random_mlp(seed, dims, 2, eps)
            net, x0, C = wl.net, wl.x0[0], wl.C[0]
        else:
            rng = np.random.default_rng(seed)
            net = mlp_net(rng, dims)
            x0 = rng.random(dims[0]).astype(np.float32)
            C = np.ones((1, 1), np.float32)
        ref = o.crown(net, x0, np.float32(eps), C)
        lb, ub, l, u = o.crown_one_hidden(net, x0, np.float32(eps), C, chunk=chunk)
        np.testing.assert_allclose(lb, ref.lb, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(ub, ref.ub, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(l, ref.layer_l[1], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(u, ref.layer_u[1], rtol=1e-12, atol=1e-12)


ALL_PINS = [
    pin_one_hidden_equals_crown,
    pin_relu_hand_values, pin_relu_net_bounds, pin_single_affine, pin_paper_wrapping_example,
    pin_wrapping_example_intermediate, pin_all_stable, pin_inactive_layer_constant, pin_eps_zero,
    pin_residual_closed_form, pin_ibp_sound_and_contains_crown, pin_conv_library,
    pin_upper_is_negated_lower, pin_bab_invariants, pin_conv_net_equals_unrolled, pin_sampled_equals_full,
    pin_lp_sandwich,
    pin_soundness_mlps, pin_lambda_rules_sound, pin_grid_bruteforce,
]
