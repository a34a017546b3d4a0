"""Pins for the beta-CROWN / branch-and-bound oracle (oracle/beta64.py).

Each pin takes the beta module as its argument (the real one in tests/test_oracle_pins.py,
copies with a planted mistake in tests/test_oracle_mutants.py).  None re-types the oracle's
formulas:
  * with beta = 0 and CROWN's slopes the subdomain bounds are the (separately pinned)
    subdomain CROWN bounds;
  * the gradient agrees with central finite differences;
  * with one hidden layer the optimised bound of a subdomain reaches the optimum of the
    triangle LP with the split constraints added (minimax over the slopes and the
    multipliers), solved by scipy, and never passes it;
  * every alpha in [0, 1] and beta >= 0 gives bounds that contain the outputs of sampled
    points satisfying the split constraints;
  * the loop on 2-input networks: it verifies properties that a dense grid confirms with a
    margin, never verifies a property the grid refutes, every bound it computes contains
    the grid points of its subdomain, and its bookkeeping is consistent;
  * the same on networks with residual additions (a convolutional net and a dense residual
    block): beta = 0 gives the subdomain CROWN bounds, finite differences, soundness, and
    with one ReLU layer the split-constrained triangle LP's optimum.
"""
from __future__ import annotations

import numpy as np

from oracle import crown64 as cr
from tests.pins import box_of, spec_values, batch_forward
from tests.pins_alpha import triangle_lp
from workloads import random_mlp
from workloads.gen import Splits


def _domains(order, rng, n, depth):
    out = []
    for _ in range(n):
        pick = rng.choice(len(order), size=depth, replace=False)
        out.append([(order[p][0], order[p][1], int(rng.choice([-1, 1]))) for p in pick])
    return out


def _random_state(B, net, dom, m, rng, scale=0.5):
    rel = B.domain_relaxation(net, dom[0], dom[1])[0]
    al = {i: rng.random((m, rel[i][0].size)) for i in rel}
    au = {i: rng.random((m, rel[i][0].size)) for i in rel}
    return al, au, rng.random((m, len(dom[1]))) * scale, rng.random((m, len(dom[1]))) * scale


def _in_domain(net, X, splits):
    vals = batch_forward(net, X)
    ids = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    ok = np.ones(X.shape[0], bool)
    for r, j, sg in splits:
        z = vals[net.nodes[ids[r]].in0].reshape(X.shape[0], -1)[:, j]
        ok &= (z >= 0) if sg > 0 else (z <= 0)
    return ok


def pin_beta_zero_is_domain_crown(B):
    """beta = 0 with CROWN's slopes: the subdomain CROWN bounds; infeasible stays infeasible."""
    rng = np.random.default_rng(1)
    for seed, dims, eps in [(101, [6, 20, 20, 4], 0.2), (102, [10, 30, 25, 30, 5], 0.1)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        order = B.default_order(wl.net, root)
        m = wl.C[0].shape[0]
        ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
        r_act, j_act = next((r, int(np.flatnonzero(root.layer_l[i] > 0)[0])) for r, i in enumerate(ids)
                            if np.any(root.layer_l[i] > 0))
        # the last two: one split, and an inactive split of a stably active neuron (infeasible)
        doms = _domains(order, rng, 6, 3) + [[order[0] + (1,)], [order[1] + (1,), (r_act, j_act, -1)]]
        sp = Splits(np.array([[s[0] for s in d] + [d[0][0]] * (3 - len(d)) for d in doms], np.int32),
                    np.array([[s[1] for s in d] + [d[0][1]] * (3 - len(d)) for d in doms], np.int32),
                    np.array([[s[2] for s in d] + [d[0][2]] * (3 - len(d)) for d in doms], np.int8))
        LB, UB = cr.crown_domains(wl.net, root, wl.C[0], sp)
        for k, d in enumerate(doms):
            dr = B.domain_relaxation(wl.net, root, d)
            if dr is None:
                assert np.all(np.isinf(LB[k]))
                assert B.beta_crown(wl.net, root, wl.C[0], d, iters=2).feasible is False
                continue
            al = {i: np.tile(dr[0][i][0].reshape(-1), (m, 1)) for i in dr[0]}
            z = np.zeros((m, len(d)))
            lb, ub = B.beta_bound(wl.net, root, wl.C[0], d, al, al, z, z)[:2]
            np.testing.assert_allclose(lb, LB[k], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ub, UB[k], rtol=1e-12, atol=1e-12)
            r = B.beta_crown(wl.net, root, wl.C[0], d, iters=3)
            np.testing.assert_allclose(r.lb_hist[0], LB[k], rtol=1e-12, atol=1e-12)


def pin_beta_gradient_fd(B):
    rng = np.random.default_rng(2)
    n_checked = 0
    for seed, dims, eps in [(103, [6, 20, 20, 4], 0.2), (104, [8, 24, 18, 22, 3], 0.15)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        order = B.default_order(wl.net, root)
        m = wl.C[0].shape[0]
        for d in _domains(order, rng, 4, 3):
            if B.domain_relaxation(wl.net, root, d) is None:
                continue
            al, au, bl, bu = _random_state(B, wl.net, (root, d), m, rng)
            out = B.beta_bound(wl.net, root, wl.C[0], d, al, au, bl, bu)
            gbl, gbu = out[4], out[5]
            h = 1e-6
            for e in range(len(d)):
                for q in range(m):
                    for which, base, g in (("l", bl, gbl), ("u", bu, gbu)):
                        p, mi = base.copy(), base.copy()
                        p[q, e] += h
                        mi[q, e] = max(mi[q, e] - h, 0.0)
                        step = p[q, e] - mi[q, e]
                        args = lambda b: (b, bu) if which == "l" else (bl, b)  # noqa: E731
                        idx = 0 if which == "l" else 1
                        fp = B.beta_bound(wl.net, root, wl.C[0], d, al, au, *args(p))[idx][q]
                        fm = B.beta_bound(wl.net, root, wl.C[0], d, al, au, *args(mi))[idx][q]
                        fd = (fp - fm) / step
                        assert abs(fd - g[q, e]) <= 1e-6 * (1 + abs(g[q, e])), (seed, d, e, q, which, fd, g[q, e])
                        n_checked += 1
            # alpha gradient of one unstable neuron per layer
            gal = out[2]
            for i, a in al.items():
                unst = np.flatnonzero(B.domain_relaxation(wl.net, root, d)[1][i])
                if not unst.size:
                    continue
                j = unst[0]
                p = {k: v.copy() for k, v in al.items()}
                mi = {k: v.copy() for k, v in al.items()}
                p[i][0, j] += 1e-6
                mi[i][0, j] -= 1e-6
                fd = (B.beta_bound(wl.net, root, wl.C[0], d, p, au, bl, bu)[0][0] -
                      B.beta_bound(wl.net, root, wl.C[0], d, mi, au, bl, bu)[0][0]) / 2e-6
                assert abs(fd - gal[i][0, j]) <= 1e-6 * (1 + abs(gal[i][0, j]))
    assert n_checked >= 40


def pin_beta_lp(B):
    """One hidden layer: optimised beta-CROWN reaches the split-constrained triangle LP from
    below; the LP fixes z >= 0 (active) or z <= 0 (inactive) through the clamped bounds."""
    rng = np.random.default_rng(3)
    n_done = 0
    for seed, dims, eps in [(105, [3, 12, 3], 0.3), (106, [6, 14, 3], 0.25)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        order = B.default_order(wl.net, root)
        for d in _domains(order, rng, 4, 2):
            if B.domain_relaxation(wl.net, root, d) is None:
                continue
            clamped = cr.CrownResult(lb=None, ub=None, box=root.box)
            clamped.layer_l = {i: v.copy() for i, v in root.layer_l.items()}
            clamped.layer_u = {i: v.copy() for i, v in root.layer_u.items()}
            ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
            for r, j, sg in d:
                i = ids[r]
                if sg > 0:
                    clamped.layer_l[i][j] = max(clamped.layer_l[i][j], 0.0)
                else:
                    clamped.layer_u[i][j] = min(clamped.layer_u[i][j], 0.0)
            lp_lo = triangle_lp(wl.net, clamped, wl.C[0], upper=False)
            lp_hi = triangle_lp(wl.net, clamped, wl.C[0], upper=True)
            r = B.beta_crown(wl.net, root, wl.C[0], d, iters=400, lr_alpha=0.05, lr_beta=0.05)
            r0 = B.beta_crown(wl.net, root, wl.C[0], d, iters=0)
            tl, tu = 1e-7 * (1 + np.abs(lp_lo)), 1e-7 * (1 + np.abs(lp_hi))
            assert np.all(r.lb <= lp_lo + tl) and np.all(r.ub >= lp_hi - tu), (seed, d)
            assert np.all(lp_lo - r.lb <= 1e-3 * (1 + np.abs(lp_lo)) + 0.03 * (lp_lo - r0.lb)), (seed, d, lp_lo, r.lb, r0.lb)
            assert np.all(r.ub - lp_hi <= 1e-3 * (1 + np.abs(lp_hi)) + 0.03 * (r0.ub - lp_hi)), (seed, d, lp_hi, r.ub, r0.ub)
            n_done += 1
    assert n_done >= 4


def pin_beta_sound(B):
    """Points of the box that satisfy a subdomain's split constraints stay inside its
    bounds for random slopes and multipliers and after optimisation."""
    rng = np.random.default_rng(4)
    for seed, dims, eps in [(107, [6, 24, 24, 4], 0.2), (108, [2, 20, 16, 3], 0.3)]:
        wl = random_mlp(seed, dims, 1, eps)
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        order = B.default_order(wl.net, root)
        m = wl.C[0].shape[0]
        lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
        X = lo + (hi - lo) * rng.random((40000, lo.size))
        for d in _domains(order, rng, 5, 2):
            if B.domain_relaxation(wl.net, root, d) is None:
                continue
            P = X[_in_domain(wl.net, X, d)]
            if len(P) == 0:
                continue
            Y = spec_values(wl.net, wl.C[0], P)
            cands = [_random_state(B, wl.net, (root, d), m, rng, scale=s) for s in (0.5, 3.0)]
            for al, au, bl, bu in cands:
                lb, ub = B.beta_bound(wl.net, root, wl.C[0], d, al, au, bl, bu)[:2]
                assert np.all(Y >= lb[None] - 1e-9 * (1 + np.abs(Y))) and np.all(Y <= ub[None] + 1e-9 * (1 + np.abs(Y)))
            r = B.beta_crown(wl.net, root, wl.C[0], d, iters=30)
            assert np.all(Y >= r.lb[None] - 1e-9 * (1 + np.abs(Y))) and np.all(Y <= r.ub[None] + 1e-9 * (1 + np.abs(Y)))


def _grid(wl, n=301):
    lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
    g = np.linspace(0.0, 1.0, n)
    gx, gy = np.meshgrid(g, g)
    return np.stack([lo[0] + (hi[0] - lo[0]) * gx.ravel(), lo[1] + (hi[1] - lo[1]) * gy.ravel()], 1)


def pin_bab_on_grids(B):
    """2-input networks: properties the grid confirms (with a margin) and that root CROWN
    cannot prove are verified; a property the grid refutes is not; every subdomain bound
    contains the subdomain's grid points; a domain never splits a neuron twice; the round
    log balances."""
    for seed, eps, rounds in [(117, 0.15, 10), (121, 0.15, 10), (122, 0.15, 10)]:
        wl = random_mlp(seed, [2, 16, 16, 3], 1, eps)
        X = _grid(wl)
        Y = spec_values(wl.net, wl.C[0], X)
        assert Y.min() > 0.02
        root = cr.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
        assert root.lb.min() < 0
        res = B.bab(wl.net, wl.x0[0], wl.eps, wl.C[0], batch=8, rounds=rounds, iters=15, root=root)
        assert res.verified, (seed, res.log)
        left = 1
        for (taken, ev, pruned, remaining), kids in zip(res.log, res.children):
            assert ev == 2 * taken and remaining == left - taken + ev - pruned
            left = remaining
            for splits, lb in kids:
                assert len({(r, j) for r, j, _ in splits}) == len(splits)
                inside = _in_domain(wl.net, X, splits)
                if inside.any() and np.all(np.isfinite(lb)):
                    assert np.all(Y[inside] >= lb[None] - 1e-9 * (1 + np.abs(Y[inside])))
    wl = random_mlp(117, [2, 16, 16, 3], 1, 0.4)
    Y = spec_values(wl.net, wl.C[0], _grid(wl))
    assert Y.min() < 0
    res = B.bab(wl.net, wl.x0[0], wl.eps, wl.C[0], batch=8, rounds=6, iters=10)
    assert not res.verified and res.remaining > 0


def _splits_of(doms, S):
    pad = lambda d, k: [s[k] for s in d] + [d[0][k]] * (S - len(d))  # noqa: E731
    return Splits(np.array([pad(d, 0) for d in doms], np.int32), np.array([pad(d, 1) for d in doms], np.int32),
                  np.array([pad(d, 2) for d in doms], np.int8))


def pin_beta_residual_nets(B):
    """Residual networks (a conv net with a residual block, a dense residual block): with
    beta = 0 and CROWN's slopes the subdomain CROWN bounds (an infeasible domain stays
    infeasible); the multiplier and slope gradients match central finite differences; random
    and optimised states stay sound on sampled points that satisfy the splits."""
    from tests.pins_alpha import _residual_cases
    rng = np.random.default_rng(21)
    n_checked = 0
    for net, x0, eps, C in _residual_cases():
        root = cr.crown(net, x0, eps, C)
        order = B.default_order(net, root)
        m = C.shape[0]
        ids = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
        act = [(r, int(np.flatnonzero(root.layer_l[i] > 0)[0])) for r, i in enumerate(ids) if np.any(root.layer_l[i] > 0)]
        doms = _domains(order, rng, 4, 2) + ([[order[0] + (1,), act[0] + (-1,)]] if act else [])
        LB, UB = cr.crown_domains(net, root, C, _splits_of(doms, 2))
        lo, hi = box_of(x0, eps, (0.0, 1.0))
        X = lo + (hi - lo) * rng.random((20000, lo.size))
        for k, d in enumerate(doms):
            dr = B.domain_relaxation(net, root, d)
            if dr is None:
                assert np.all(np.isposinf(LB[k])) and not B.beta_crown(net, root, C, d, iters=1).feasible
                continue
            al0 = {i: np.tile(dr[0][i][0].reshape(-1), (m, 1)) for i in dr[0]}
            z = np.zeros((m, len(d)))
            lb, ub = B.beta_bound(net, root, C, d, al0, al0, z, z)[:2]
            np.testing.assert_allclose(lb, LB[k], rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(ub, UB[k], rtol=1e-12, atol=1e-12)
            al, au, bl, bu = _random_state(B, net, (root, d), m, rng)
            out = B.beta_bound(net, root, C, d, al, au, bl, bu)
            h = 1e-6
            for e in range(len(d)):
                for q in range(min(m, 3)):
                    for which, base, g in (("l", bl, out[4]), ("u", bu, out[5])):
                        p, mi = base.copy(), base.copy()
                        p[q, e] += h
                        mi[q, e] = max(mi[q, e] - h, 0.0)
                        args = (lambda b: (b, bu)) if which == "l" else (lambda b: (bl, b))
                        idx = 0 if which == "l" else 1
                        fd = (B.beta_bound(net, root, C, d, al, au, *args(p))[idx][q] -
                              B.beta_bound(net, root, C, d, al, au, *args(mi))[idx][q]) / (p[q, e] - mi[q, e])
                        assert abs(fd - g[q, e]) <= 1e-6 * (1 + abs(g[q, e])), (d, e, q, which, fd, g[q, e])
                        n_checked += 1
            for i in al:
                unst = np.flatnonzero(dr[1][i])
                if not unst.size:
                    continue
                j = unst[0]
                p = {kk: v.copy() for kk, v in al.items()}
                mi = {kk: v.copy() for kk, v in al.items()}
                p[i][0, j] += 1e-6
                mi[i][0, j] -= 1e-6
                fd = (B.beta_bound(net, root, C, d, p, au, bl, bu)[0][0] -
                      B.beta_bound(net, root, C, d, mi, au, bl, bu)[0][0]) / 2e-6
                assert abs(fd - out[2][i][0, j]) <= 1e-6 * (1 + abs(out[2][i][0, j]))
            P = X[_in_domain(net, X, d)]
            if len(P):
                Y = spec_values(net, C, P)
                r = B.beta_crown(net, root, C, d, iters=15)
                for lb_, ub_ in (out[:2], (r.lb, r.ub)):
                    assert np.all(Y >= lb_[None] - 1e-9 * (1 + np.abs(Y))) and np.all(Y <= ub_[None] + 1e-9 * (1 + np.abs(Y)))
    assert n_checked >= 30


def pin_beta_residual_lp(B):
    """A dense residual block with one ReLU layer: on subdomains, optimised beta-CROWN reaches
    the triangle LP with the split-clamped neuron intervals (a minimax identity over slopes
    and multipliers) and never passes it."""
    from tests.pins_alpha import _residual_dense, residual_lp
    rng = np.random.default_rng(22)
    n_done = 0
    for seed in (84, 85, 87):
        net, x0, C = _residual_dense(seed, n0=4, hid=12)
        root = cr.crown(net, x0[0], np.float32(0.3), C[0])
        order = B.default_order(net, root)
        for d in _domains(order, rng, 3, 2):
            if B.domain_relaxation(net, root, d) is None:
                continue
            clamped = cr.CrownResult(lb=None, ub=None, box=root.box)
            clamped.layer_l = {i: v.copy() for i, v in root.layer_l.items()}
            clamped.layer_u = {i: v.copy() for i, v in root.layer_u.items()}
            for r, j, sg in d:
                if sg > 0:
                    clamped.layer_l[1][j] = max(clamped.layer_l[1][j], 0.0)
                else:
                    clamped.layer_u[1][j] = min(clamped.layer_u[1][j], 0.0)
            try:
                lp_lo = residual_lp(net, clamped, C[0], upper=False)
                lp_hi = residual_lp(net, clamped, C[0], upper=True)
            except AssertionError:   # the splits exclude every point of the box: no LP optimum
                continue
            r = B.beta_crown(net, root, C[0], d, iters=400, lr_alpha=0.05, lr_beta=0.5)
            r0 = B.beta_crown(net, root, C[0], d, iters=0)
            assert np.all(r.lb <= lp_lo + 1e-7 * (1 + np.abs(lp_lo))) and np.all(r.ub >= lp_hi - 1e-7 * (1 + np.abs(lp_hi)))
            assert np.all(lp_lo - r.lb <= 1e-3 * (1 + np.abs(lp_lo)) + 0.03 * (lp_lo - r0.lb)), (seed, d, lp_lo, r.lb, r0.lb)
            assert np.all(r.ub - lp_hi <= 1e-3 * (1 + np.abs(lp_hi)) + 0.03 * (r0.ub - lp_hi)), (seed, d, lp_hi, r.ub, r0.ub)
            n_done += 1
    assert n_done >= 4


BETA_PINS = [pin_beta_zero_is_domain_crown, pin_beta_gradient_fd, pin_beta_lp, pin_beta_sound, pin_bab_on_grids,
             pin_beta_residual_nets, pin_beta_residual_lp]
