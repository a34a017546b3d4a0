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
    grids of 2-input networks.
"""
from __future__ import annotations

import numpy as np

from oracle import crown64 as cr
from tests.pins import box_of, spec_values
from workloads import random_mlp


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


ALPHA_PINS = [pin_alpha_reduces_to_crown, pin_alpha_gradient_fd, pin_alpha_lp, pin_alpha_sound,
              pin_alpha_history]
