"""Pins for the alpha-CROWN oracle (oracle/alpha64.py): facts the mathematics fixes.

Each pin takes the alpha module as its argument (the real one in tests/test_oracle_pins.py,
copies with a planted mistake in tests/test_oracle_mutants.py).  None re-types the oracle's
formulas:
  * slopes equal to CROWN's own choice reproduce the (separately pinned) CROWN bounds;
  * the gradient agrees with central finite differences of the bound;
  * with one hidden layer the best bound over alpha equals the optimum of the triangle
    relaxation LP (a minimax identity: the LP's inner minimum over x and the maximum over
    the lower slopes can be exchanged), solved by scipy; with more layers every alpha bound
    lies between CROWN's and the LP's;
  * every alpha in [0, 1] gives bounds that contain sampled outputs, box corners and dense
    grids of 2-input networks;
  * the same on networks with residual additions (convolutional and dense): CROWN's slopes
    give CROWN, finite differences, soundness, and with one ReLU layer in a dense residual
    block y = x + W2 ReLU(W1 x + b1) the optimised bound reaches the triangle LP's optimum.
"""
from __future__ import annotations

import numpy as np

from oracle import crown64 as cr
from tests.pins import box_of, spec_values, tiny_resnet
from workloads import Net, Node, margin_spec, random_mlp


def _random_alpha(A, net, root, m, rng):
    al, au = A.initial_alpha(net, root, m)
    return ({i: rng.random(v.shape) for i, v in al.items()}, {i: rng.random(v.shape) for i, v in au.items()})


def triangle_lp(net, root, C, upper):
    """min (or max) of C f(x) over the box with every unstable ReLU replaced by its
    triangle (h >= 0, h >= z, h <= s (z - l)) for the intermediate bounds of `root`,
    solved by scipy's HiGHS.  Variables: x, then (z_k, h_k) per hidden layer."""
    from scipy.optimize import linprog
    dense = [nd for nd in net.nodes if nd.op == "dense"]
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    lo, hi = root.box
    sizes = [lo.size] + [d.W.shape[0] for d in dense[:-1]]
    offs, o = [], lo.size          # offsets of (z_k, h_k)
    for n in sizes[1:]:
        offs.append((o, o + n))
        o += 2 * n
    nv = o
    A_eq, b_eq, A_ub, b_ub = [], [], [], []
    prev = (0, lo.size)            # (offset, width) of h_{k-1} (x for k = 1)
    for k, d in enumerate(dense[:-1]):
        W, b = d.W.astype(np.float64), d.b.astype(np.float64)
        zo, ho = offs[k]
        n = W.shape[0]
        l, u = root.layer_l[relus[k]], root.layer_u[relus[k]]
        for j in range(n):
            row = np.zeros(nv)
            row[zo + j] = 1.0
            row[prev[0]:prev[0] + prev[1]] -= W[j]
            A_eq.append(row); b_eq.append(b[j])                    # z = W h + b
            eh = np.zeros(nv); eh[ho + j] = 1.0
            ez = np.zeros(nv); ez[zo + j] = 1.0
            if u[j] <= 0:
                A_eq.append(eh); b_eq.append(0.0)
            elif l[j] >= 0:
                A_eq.append(eh - ez); b_eq.append(0.0)
            else:
                A_ub.append(ez - eh); b_ub.append(0.0)              # h >= z
                A_ub.append(-eh); b_ub.append(0.0)                  # h >= 0
                s = u[j] / (u[j] - l[j])
                A_ub.append(eh - s * ez); b_ub.append(-s * l[j])    # h <= s (z - l)
        prev = (ho, n)
    WL, bL = dense[-1].W.astype(np.float64), dense[-1].b.astype(np.float64)
    bounds = [(lo[i], hi[i]) for i in range(lo.size)]
    for k, n in enumerate(sizes[1:]):
        l, u = root.layer_l[relus[k]], root.layer_u[relus[k]]
        bounds += [(l[j], u[j]) for j in range(n)] + [(None, None)] * n
    out = []
    for c in np.asarray(C, np.float64):
        obj = np.zeros(nv)
        obj[prev[0]:prev[0] + prev[1]] = c @ WL
        res = linprog(-obj if upper else obj, A_ub=np.array(A_ub) if A_ub else None,
                      b_ub=np.array(b_ub) if b_ub else None, A_eq=np.array(A_eq), b_eq=np.array(b_eq),
                      bounds=bounds, method="highs")
        assert res.status == 0, res.message
        out.append((-res.fun if upper else res.fun) + c @ bL)
    return np.array(out)


def pin_alpha_reduces_to_crown(A):
    """Slopes equal to a fixed CROWN rule give exactly that rule's CROWN bounds."""
    for seed, dims, eps in [(61, [6, 20, 20, 4], 0.2), (62, [10, 30, 25, 30, 5], 0.1)]:
        wl = random_mlp(seed, dims, 1, eps)
        for rule in ("adaptive", "zero", "one"):
            ref = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0], lambda_rule=rule)
            m = wl.C[0].shape[0]
            al, au = A.initial_alpha(wl.net, ref, m)
            lb, ub, _, _ = A.alpha_bound(wl.net, ref, wl.C[0], al, au)
            np.testing.assert_allclose(lb, ref.lb, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ub, ref.ub, rtol=1e-12, atol=1e-12)
        r = A.alpha_crown(wl.net, wl.x0[0], wl.eps, wl.C[0], iters=3)
        np.testing.assert_allclose(r.lb_hist[0], r.root.lb, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r.ub_hist[0], r.root.ub, rtol=1e-12, atol=1e-12)


def pin_alpha_gradient_fd(A):
    """Central finite differences of the bound in single slopes match the gradient."""
    rng = np.random.default_rng(5)
    for seed, dims, eps in [(63, [6, 20, 20, 4], 0.2), (64, [8, 24, 18, 22, 3], 0.15)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        m = wl.C[0].shape[0]
        al, au = _random_alpha(A, wl.net, root, m, rng)
        lb, ub, gl, gu = A.alpha_bound(wl.net, root, wl.C[0], al, au)
        n_checked = 0
        for i in al:
            unst = np.flatnonzero(A.unstable_mask(root, i))
            assert np.all(gl[i][:, ~A.unstable_mask(root, i)] == 0.0)
            for j in rng.choice(unst, size=min(6, unst.size), replace=False) if unst.size else []:
                for q in range(m):
                    for which in ("l", "u"):
                        h = 1e-6
                        a0 = al if which == "l" else au
                        plus = {k: v.copy() for k, v in a0.items()}
                        minus = {k: v.copy() for k, v in a0.items()}
                        plus[i][q, j] += h
                        minus[i][q, j] -= h
                        if which == "l":
                            fp = A.alpha_bound(wl.net, root, wl.C[0], plus, au)[0][q]
                            fm = A.alpha_bound(wl.net, root, wl.C[0], minus, au)[0][q]
                            g = gl[i][q, j]
                        else:
                            fp = A.alpha_bound(wl.net, root, wl.C[0], al, plus)[1][q]
                            fm = A.alpha_bound(wl.net, root, wl.C[0], al, minus)[1][q]
                            g = gu[i][q, j]
                        fd = (fp - fm) / (2 * h)
                        assert abs(fd - g) <= 1e-6 * (1.0 + abs(g)), (seed, i, j, q, which, fd, g)
                        n_checked += 1
        assert n_checked >= 50


def pin_alpha_lp(A):
    """One hidden layer: optimised alpha reaches the triangle LP's optimum from below (and
    never passes it).  Two hidden layers: CROWN <= every alpha bound <= LP optimum."""
    for seed, dims, eps in [(65, [2, 12, 3], 0.3), (66, [4, 10, 3], 0.3), (67, [8, 16, 3], 0.2)]:
        wl = random_mlp(seed, dims, 1, eps)
        r = A.alpha_crown(wl.net, wl.x0[0], wl.eps, wl.C[0], iters=300, lr=0.05)
        lp_lo = triangle_lp(wl.net, r.root, wl.C[0], upper=False)
        lp_hi = triangle_lp(wl.net, r.root, wl.C[0], upper=True)
        tol = 1e-7 * (1 + np.abs(lp_lo))
        assert np.all(r.lb <= lp_lo + tol) and np.all(r.ub >= lp_hi - 1e-7 * (1 + np.abs(lp_hi)))
        gap0_l, gap_l = lp_lo - r.root.lb, lp_lo - r.lb
        gap0_u, gap_u = r.root.ub - lp_hi, r.ub - lp_hi
        assert np.all(gap_l <= 1e-3 * (1 + np.abs(lp_lo)) + 0.02 * gap0_l), (seed, gap_l, gap0_l)
        assert np.all(gap_u <= 1e-3 * (1 + np.abs(lp_hi)) + 0.02 * gap0_u), (seed, gap_u, gap0_u)
    rng = np.random.default_rng(7)
    for seed, dims, eps in [(68, [4, 10, 10, 3], 0.3), (69, [3, 8, 9, 7, 3], 0.4)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        lp_lo = triangle_lp(wl.net, root, wl.C[0], upper=False)
        lp_hi = triangle_lp(wl.net, root, wl.C[0], upper=True)
        m = wl.C[0].shape[0]
        for _ in range(5):
            al, au = _random_alpha(A, wl.net, root, m, rng)
            lb, ub, _, _ = A.alpha_bound(wl.net, root, wl.C[0], al, au)
            assert np.all(lb <= lp_lo + 1e-7 * (1 + np.abs(lp_lo)))
            assert np.all(ub >= lp_hi - 1e-7 * (1 + np.abs(lp_hi)))
        r = A.alpha_crown(wl.net, wl.x0[0], wl.eps, wl.C[0], iters=50, root=root)
        assert np.all(r.lb >= root.lb) and np.all(r.ub <= root.ub)
        assert np.all(r.lb <= lp_lo + 1e-7 * (1 + np.abs(lp_lo)))
        assert np.all(r.ub >= lp_hi - 1e-7 * (1 + np.abs(lp_hi)))


def pin_alpha_sound(A):
    """Random slopes and optimised slopes: sampled points, random corners and dense grids
    of 2-input networks stay inside [lb, ub]."""
    rng = np.random.default_rng(8)
    for seed, dims, eps in [(70, [10, 30, 30, 4], 0.1), (71, [2, 16, 16, 2], 0.4), (72, [2, 24, 20, 3], 0.3)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        m = wl.C[0].shape[0]
        lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
        if lo.size == 2:
            g = np.linspace(0.0, 1.0, 401)
            gx, gy = np.meshgrid(g, g)
            X = np.stack([lo[0] + (hi[0] - lo[0]) * gx.ravel(), lo[1] + (hi[1] - lo[1]) * gy.ravel()], 1)
        else:
            X = np.concatenate([lo + (hi - lo) * rng.random((20000, lo.size)),
                                np.where(rng.random((2000, lo.size)) < 0.5, lo, hi)])
        Y = spec_values(wl.net, wl.C[0], X)
        cands = [_random_alpha(A, wl.net, root, m, rng) for _ in range(3)]
        r = A.alpha_crown(wl.net, wl.x0[0], wl.eps, wl.C[0], iters=40, root=root)
        cands.append((r.alpha_l, r.alpha_u))
        for al, au in cands:
            lb, ub, _, _ = A.alpha_bound(wl.net, root, wl.C[0], al, au)
            assert np.all(Y >= lb[None, :] - 1e-9 * (1 + np.abs(Y))), (seed, np.max(lb[None, :] - Y))
            assert np.all(Y <= ub[None, :] + 1e-9 * (1 + np.abs(Y))), (seed, np.max(Y - ub[None, :]))
        assert np.all(r.lb <= Y.min(axis=0) + 1e-9) and np.all(r.ub >= Y.max(axis=0) - 1e-9)


def pin_alpha_history(A):
    """The result is the best of the evaluated bounds, the first evaluation is CROWN, and
    the slopes returned with it reproduce it."""
    wl = random_mlp(73, [8, 24, 24, 5], 1, 0.15)
    r = A.alpha_crown(wl.net, wl.x0[0], wl.eps, wl.C[0], iters=15)
    np.testing.assert_array_equal(r.lb, r.lb_hist.max(axis=0))
    np.testing.assert_array_equal(r.ub, r.ub_hist.min(axis=0))
    assert np.all(r.lb >= r.root.lb) and np.all(r.ub <= r.root.ub)
    assert np.any(r.lb > r.root.lb + 1e-6)
    lb, ub, _, _ = A.alpha_bound(wl.net, r.root, wl.C[0], r.alpha_l, r.alpha_u)
    np.testing.assert_allclose(lb, r.lb, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ub, r.ub, rtol=1e-12, atol=1e-12)
    for d in (r.alpha_l, r.alpha_u):
        for v in d.values():
            assert np.all((v >= 0.0) & (v <= 1.0))


def _residual_dense(seed, n0=4, hid=10, n_out=3):
    """x -> y = x + W2 ReLU(W1 x + b1) + b2 -> f = W3 y + b3: one ReLU layer with a skip."""
    rng = np.random.default_rng(seed)
    W1 = (rng.standard_normal((hid, n0)) * np.sqrt(2 / n0)).astype(np.float32)
    b1 = (rng.standard_normal(hid) * 0.3).astype(np.float32)
    W2 = (rng.standard_normal((n0, hid)) * np.sqrt(2 / hid)).astype(np.float32)
    b2 = (rng.standard_normal(n0) * 0.1).astype(np.float32)
    W3 = (rng.standard_normal((n_out, n0)) * np.sqrt(2 / n0)).astype(np.float32)
    b3 = (rng.standard_normal(n_out) * 0.1).astype(np.float32)
    nodes = [Node("dense", -1, W=W1, b=b1), Node("relu", 0), Node("dense", 1, W=W2, b=b2),
             Node("flatten", -1), Node("add", 3, 2), Node("dense", 4, W=W3, b=b3)]
    net = Net((n0,), nodes)
    x0 = rng.random((1, n0)).astype(np.float32)
    return net, x0, margin_spec(net, x0)


def _residual_cases():
    out = []
    for seed in (81, 82):
        net = tiny_resnet(seed)
        rng = np.random.default_rng(seed + 100)
        x0 = rng.random((1, int(np.prod(net.in_shape)))).astype(np.float32)
        out.append((net, x0[0], np.float32(0.08), margin_spec(net, x0)[0]))
    net, x0, C = _residual_dense(83)
    out.append((net, x0[0], np.float32(0.25), C[0]))
    return out


def residual_lp(net, root, C, upper):
    """min (or max) of C f(x) over the box for the dense residual block of _residual_dense,
    with the unstable ReLUs replaced by their triangles; variables x, z = W1 x + b1, h."""
    from scipy.optimize import linprog
    W1, b1 = net.nodes[0].W.astype(np.float64), net.nodes[0].b.astype(np.float64)
    W2, b2 = net.nodes[2].W.astype(np.float64), net.nodes[2].b.astype(np.float64)
    W3, b3 = net.nodes[5].W.astype(np.float64), net.nodes[5].b.astype(np.float64)
    lo, hi = root.box
    n0, hid = lo.size, W1.shape[0]
    l, u = root.layer_l[1], root.layer_u[1]
    nv = n0 + 2 * hid
    A_eq, b_eq, A_ub, b_ub = [], [], [], []
    for j in range(hid):
        row = np.zeros(nv)
        row[n0 + j] = 1.0
        row[:n0] = -W1[j]
        A_eq.append(row); b_eq.append(b1[j])
        ez = np.zeros(nv); ez[n0 + j] = 1.0
        eh = np.zeros(nv); eh[n0 + hid + j] = 1.0
        if u[j] <= 0:
            A_eq.append(eh); b_eq.append(0.0)
        elif l[j] >= 0:
            A_eq.append(eh - ez); b_eq.append(0.0)
        else:
            A_ub.append(ez - eh); b_ub.append(0.0)
            A_ub.append(-eh); b_ub.append(0.0)
            s_ = u[j] / (u[j] - l[j])
            A_ub.append(eh - s_ * ez); b_ub.append(-s_ * l[j])
    bounds = [(lo[i], hi[i]) for i in range(n0)] + [(l[j], u[j]) for j in range(hid)] + [(None, None)] * hid
    out = []
    for c in np.asarray(C, np.float64):
        g = c @ W3                      # c f = g (x + W2 h + b2) + c b3
        obj = np.zeros(nv)
        obj[:n0] = g
        obj[n0 + hid:] = g @ W2
        res = linprog(-obj if upper else obj, A_ub=np.array(A_ub) if A_ub else None,
                      b_ub=np.array(b_ub) if b_ub else None, A_eq=np.array(A_eq), b_eq=np.array(b_eq),
                      bounds=bounds, method="highs")
        assert res.status == 0, res.message
        out.append((-res.fun if upper else res.fun) + g @ b2 + c @ b3)
    return np.array(out)


def pin_alpha_residual_nets(A):
    """Residual networks (a conv net with a residual block, a dense residual block): CROWN's
    slopes reproduce CROWN; the gradient matches central finite differences; random and
    optimised slopes stay sound on sampled points and box corners."""
    rng = np.random.default_rng(9)
    for net, x0, eps, C in _residual_cases():
        m = C.shape[0]
        for rule in ("adaptive", "zero", "one"):
            ref = cr.crown(net, x0, eps, C, lambda_rule=rule)
            al, au = A.initial_alpha(net, ref, m)
            lb, ub, _, _ = A.alpha_bound(net, ref, C, al, au)
            np.testing.assert_allclose(lb, ref.lb, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ub, ref.ub, rtol=1e-12, atol=1e-12)
        root = cr.crown(net, x0, eps, C)
        al, au = _random_alpha(A, net, root, m, rng)
        lb, ub, gl, gu = A.alpha_bound(net, root, C, al, au)
        n_checked = 0
        for i in al:
            unst = np.flatnonzero(A.unstable_mask(root, i).reshape(-1))
            for j in rng.choice(unst, size=min(4, unst.size), replace=False) if unst.size else []:
                for q in range(min(m, 3)):
                    for which in ("l", "u"):
                        h = 1e-6
                        a0 = al if which == "l" else au
                        plus = {k: v.copy() for k, v in a0.items()}
                        minus = {k: v.copy() for k, v in a0.items()}
                        plus[i][q, j] += h
                        minus[i][q, j] -= h
                        k = 0 if which == "l" else 1
                        args_p = (plus, au) if which == "l" else (al, plus)
                        args_m = (minus, au) if which == "l" else (al, minus)
                        fd = (A.alpha_bound(net, root, C, *args_p)[k][q] - A.alpha_bound(net, root, C, *args_m)[k][q]) / (2 * h)
                        g = (gl if which == "l" else gu)[i][q, j]
                        assert abs(fd - g) <= 1e-6 * (1.0 + abs(g)), (i, j, q, which, fd, g)
                        n_checked += 1
        assert n_checked >= 12
        lo, hi = box_of(x0, eps, (0.0, 1.0))
        X = np.concatenate([lo + (hi - lo) * rng.random((3000, lo.size)), np.where(rng.random((1000, lo.size)) < 0.5, lo, hi)])
        Y = spec_values(net, C, X)
        r = A.alpha_crown(net, x0, eps, C, iters=20, root=root)
        assert np.all(r.lb >= root.lb) and np.all(r.ub <= root.ub)
        for a_l, a_u in (_random_alpha(A, net, root, m, rng), (r.alpha_l, r.alpha_u)):
            lb, ub, _, _ = A.alpha_bound(net, root, C, a_l, a_u)
            assert np.all(Y >= lb[None, :] - 1e-9 * (1 + np.abs(Y)))
            assert np.all(Y <= ub[None, :] + 1e-9 * (1 + np.abs(Y)))


def pin_alpha_residual_lp(A):
    """A dense residual block with one ReLU layer: the optimised bound reaches the triangle
    LP's optimum (minimax over the slopes) and never passes it."""
    for seed in (84, 85, 87):   # cases where CROWN leaves a gap to the LP
        net, x0, C = _residual_dense(seed, n0=4, hid=12)
        r = A.alpha_crown(net, x0[0], np.float32(0.3), C[0], iters=300, lr=0.05)
        lp_lo = residual_lp(net, r.root, C[0], upper=False)
        lp_hi = residual_lp(net, r.root, C[0], upper=True)
        assert np.all(r.lb <= lp_lo + 1e-7 * (1 + np.abs(lp_lo)))
        assert np.all(r.ub >= lp_hi - 1e-7 * (1 + np.abs(lp_hi)))
        gap0_l, gap_l = lp_lo - r.root.lb, lp_lo - r.lb
        gap0_u, gap_u = r.root.ub - lp_hi, r.ub - lp_hi
        assert np.all(gap_l <= 1e-3 * (1 + np.abs(lp_lo)) + 0.02 * gap0_l), (seed, gap_l, gap0_l)
        assert np.all(gap_u <= 1e-3 * (1 + np.abs(lp_hi)) + 0.02 * gap0_u), (seed, gap_u, gap0_u)
        assert np.any(gap0_l > 1e-3), "the case should leave CROWN a gap to close"


ALPHA_PINS = [pin_alpha_reduces_to_crown, pin_alpha_gradient_fd, pin_alpha_lp, pin_alpha_sound,
              pin_alpha_history, pin_alpha_residual_nets, pin_alpha_residual_lp]
