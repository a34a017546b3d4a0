"""fp64 CPU oracle for beta-CROWN on branch-and-bound subdomains, and a fixed-batch
branch-and-bound loop, on feed-forward ReLU networks (dense, conv2d, add, flatten).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's CPU-baseline
leg may import this module.  It shares no code with the GPU library.

What it computes (section numbers are the paper's).  Branch-and-bound (Sec. 2.1, complete
verification) splits ReLU neurons into an active (z >= 0) and an inactive (z <= 0) case and
bounds every subdomain.  beta-CROWN (Sec. 2.2, Alpha-Beta-CROWN) puts each split constraint
into the bound propagation with a Lagrange multiplier beta >= 0: writing a split as g <= 0
(g = -z for an active split, g = z for an inactive one), the minimum of f over the
subdomain is at least the minimum over the whole box of f + beta g, and the maximum at most
the maximum of f - beta g.  The multipliers and the lower slopes alpha are optimised
jointly by gradient steps (alpha in [0, 1], beta >= 0).  The loop processes a fixed batch of
domains per round (the paper's force_synchronous mode, Sec. 3.4.4), so every round does a
known amount of work.

Readings where the paper is silent (each is also listed in the design notes):
  * intermediate bounds of every subdomain are the root's full-CROWN bounds with each split
    neuron's own interval clamped (the branch-and-bound batch of the subdomain workload);
  * one beta per (split, specification row, direction), like alpha one slope per
    (neuron, row, direction); both start at CROWN's choice (alpha = adaptive lambda,
    beta = 0); Adam as for alpha-CROWN with its own step size for beta, projection onto
    alpha in [0, 1] and beta >= 0, and each row keeps its best bound;
  * the gradient of a row's bound with respect to beta of split (neuron j, sign) is the
    sign term S = -1 (active) / +1 (inactive) times z_j evaluated forward from the row's
    attaining box vertex through the relaxed network (the same evaluation as alpha's
    gradient); for the upper bound the sign term is -S;
  * the loop: the root is bounded by alpha-CROWN; unverified domains wait in first-in
    first-out order; each round takes up to `batch` of them, splits each on the first
    neuron of a priority order that the domain has not split yet, bounds both children
    with beta-CROWN, and drops the children whose lower bounds are all positive (or that
    are infeasible); the property is verified when no domain is left, unknown when the
    rounds run out or a domain has no neuron left to split.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from oracle import crown64 as cr


def relu_ids(net):
    return [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]


def _check_chain(net):
    for i, nd in enumerate(net.nodes):
        if nd.op not in ("dense", "conv2d", "relu", "add", "flatten"):
            raise ValueError(f"beta-CROWN oracle: unsupported node {nd.op}")
        if not (-1 <= nd.in0 < i) or (nd.op == "add" and not (-1 <= nd.in1 < i)):
            raise ValueError("beta-CROWN oracle: nodes must be in topological order")


def domain_relaxation(net, root, splits):
    """(relaxation dict, unstable masks) of a subdomain; splits = [(relu position, neuron,
    sign)].  None when some clamped interval is empty."""
    rel = cr.apply_splits(net, root, [s[0] for s in splits], [s[1] for s in splits], [s[2] for s in splits])
    if rel is None:
        return None
    unst = {i: (rel[i][2].reshape(-1) > 0.0) for i in rel}   # t > 0 exactly when l < 0 < u
    return rel, unst


def _terms(net, splits):
    ids = relu_ids(net)
    return [(ids[int(r)], int(j), -1.0 if sg > 0 else 1.0) for r, j, sg in splits]


def _pass(net, rel, unst, terms, box, C, alpha, beta, upper):
    """Backward pass from the output with A = C, the rows' slopes and the split terms; the
    coefficients reaching a node along several paths (an add's inputs) are summed before the
    node is expanded.  Returns the bounds, the input coefficients and, per ReLU, the
    coefficients on its output before relaxation."""
    shapes = cr.node_shapes(net)
    A = np.asarray(C, np.float64)
    rows = A.shape[0]
    bias = np.zeros(rows)
    pre = {}
    acc = {len(net.nodes) - 1: A}

    def add_to(node, X):
        acc[node] = acc[node] + X if node in acc else X

    for i in range(len(net.nodes) - 1, -1, -1):
        if i not in acc:
            continue
        A = acc.pop(i)
        nd = net.nodes[i]
        if nd.op == "dense":
            bias = bias + A @ cr._f64(nd.b)
            add_to(nd.in0, A @ cr._f64(nd.W))
        elif nd.op == "conv2d":
            co, ho, wo = shapes[i]
            in_shape = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
            A4 = A.reshape(rows, co, ho, wo)
            bias = bias + A4.sum(axis=(2, 3)) @ cr._f64(nd.b)
            add_to(nd.in0, cr.conv2d_transpose(A4, cr._f64(nd.W), nd.stride, nd.pad, in_shape[1:]).reshape(rows, -1))
        elif nd.op == "relu":
            lam0, s, t = (v.reshape(-1) for v in rel[i])
            lam = np.where(unst[i][None, :], alpha[i], lam0[None, :])
            pre[i] = A.copy()
            Ap, An = np.maximum(A, 0.0), np.minimum(A, 0.0)
            if not upper:
                bias = bias + An @ t
                A = Ap * lam + An * s
            else:
                bias = bias + Ap @ t
                A = Ap * s + An * lam
            # the split constraints' Lagrangian terms on the coefficients of z
            for e, (ri, j, S) in enumerate(terms):
                if ri == i:
                    A[:, j] += (-S if upper else S) * beta[:, e]
            add_to(nd.in0, A)
        elif nd.op == "add":
            add_to(nd.in0, A)
            add_to(nd.in1, A)
        elif nd.op == "flatten":
            add_to(nd.in0, A)
    A = acc.pop(-1) if -1 in acc else np.zeros((rows, int(np.prod(net.in_shape))))
    lo, hi = box
    return cr.concretize(A, bias, lo, hi, upper), A, pre


def _gradient(net, rel, unst, terms, box, A_x, pre, alpha, upper):
    """Gradients with respect to the slopes and the multipliers: the relaxed network
    evaluated forward, node by node, from the attaining box vertex (the multiplier of a
    split on z_j gets its sign term times z_j there)."""
    shapes = cr.node_shapes(net)
    lo, hi = box
    c, r = (lo + hi) / 2.0, (hi - lo) / 2.0
    sgn = np.sign(A_x)
    x = c[None, :] + sgn * r[None, :] if upper else c[None, :] - sgn * r[None, :]
    rows = x.shape[0]
    ga, gb = {}, np.zeros((rows, len(terms)))
    val = {}
    get = lambda i: x if i == -1 else val[i]  # noqa: E731
    for i, nd in enumerate(net.nodes):
        v = get(nd.in0)
        if nd.op == "dense":
            val[i] = v.reshape(rows, -1) @ cr._f64(nd.W).T + cr._f64(nd.b)
        elif nd.op == "conv2d":
            in_shape = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
            x4 = v.reshape((rows,) + tuple(in_shape))
            y = np.stack([cr.conv2d(x4[k], cr._f64(nd.W), nd.stride, nd.pad) for k in range(rows)])
            val[i] = (y + cr._f64(nd.b)[None, :, None, None]).reshape(rows, -1)
        elif nd.op == "relu":
            lam0, s, t = (q.reshape(-1) for q in rel[i])
            lam = np.where(unst[i][None, :], alpha[i], lam0[None, :])
            a, D = pre[i], v.reshape(rows, -1)
            for e, (ri, j, S) in enumerate(terms):
                if ri == i:
                    gb[:, e] = (-S if upper else S) * D[:, j]
            on_lam, on_t = (a < 0.0, a > 0.0) if upper else (a > 0.0, a < 0.0)
            ga[i] = np.where(unst[i][None, :] & on_lam, a * D, 0.0)
            val[i] = np.where(on_lam, lam * D, s[None, :] * D + np.where(on_t, t[None, :], 0.0))
        elif nd.op == "add":
            val[i] = v.reshape(rows, -1) + get(nd.in1).reshape(rows, -1)
        elif nd.op == "flatten":
            val[i] = v.reshape(rows, -1)
    return ga, gb


def beta_bound(net, root, C, splits, alpha_l, alpha_u, beta_l, beta_u):
    """Bounds of C f(x) over one subdomain with the given slopes and multipliers, and their
    gradients: (lb, ub, d lb/d alpha_l, d ub/d alpha_u, d lb/d beta_l, d ub/d beta_u); None
    if the subdomain is infeasible.  alpha_*: {relu id: (m, n)}; beta_*: (m, len(splits))."""
    _check_chain(net)
    dr = domain_relaxation(net, root, splits)
    if dr is None:
        return None
    rel, unst = dr
    terms = _terms(net, splits)
    lb, Al, pl = _pass(net, rel, unst, terms, root.box, C, alpha_l, beta_l, upper=False)
    ub, Au, pu = _pass(net, rel, unst, terms, root.box, C, alpha_u, beta_u, upper=True)
    gal, gbl = _gradient(net, rel, unst, terms, root.box, Al, pl, alpha_l, upper=False)
    gau, gbu = _gradient(net, rel, unst, terms, root.box, Au, pu, alpha_u, upper=True)
    return lb, ub, gal, gau, gbl, gbu


@dataclass
class BetaResult:
    lb: np.ndarray
    ub: np.ndarray
    lb_hist: np.ndarray
    ub_hist: np.ndarray
    feasible: bool = True


def beta_crown(net, root, C, splits, iters=20, lr_alpha=0.1, lr_beta=0.05, beta1=0.9, beta2=0.999,
               adam_eps=1e-8):
    """Jointly optimised alpha, beta bounds of one subdomain (infeasible: lb = +inf,
    ub = -inf)."""
    _check_chain(net)
    C = np.asarray(C, np.float64)
    m = C.shape[0]
    dr = domain_relaxation(net, root, splits)
    if dr is None:
        inf = np.full(m, np.inf)
        return BetaResult(inf, -inf, np.tile(inf, (iters + 1, 1)), np.tile(-inf, (iters + 1, 1)), False)
    rel = dr[0]
    ids = relu_ids(net)
    al = {i: np.tile(rel[i][0].reshape(-1), (m, 1)) for i in ids}
    au = {i: a.copy() for i, a in al.items()}
    bl = np.zeros((m, len(splits)))
    bu = np.zeros((m, len(splits)))
    st = {}
    for key, arr in [(("al", i), al[i]) for i in ids] + [(("au", i), au[i]) for i in ids] + [("bl", bl), ("bu", bu)]:
        st[key] = [np.zeros_like(arr), np.zeros_like(arr)]
    best_l, best_u = np.full(m, -np.inf), np.full(m, np.inf)
    lh, uh = [], []
    for step in range(iters + 1):
        lb, ub, gal, gau, gbl, gbu = beta_bound(net, root, C, splits, al, au, bl, bu)
        lh.append(lb)
        uh.append(ub)
        best_l, best_u = np.maximum(best_l, lb), np.minimum(best_u, ub)
        if step == iters:
            break
        t = step + 1

        def adam(key, x, g, sign, lr, lo, hi):
            mo, ve = st[key]
            mo[...] = beta1 * mo + (1.0 - beta1) * g
            ve[...] = beta2 * ve + (1.0 - beta2) * g * g
            step_ = lr * (mo / (1.0 - beta1 ** t)) / (np.sqrt(ve / (1.0 - beta2 ** t)) + adam_eps)
            return np.clip(x + sign * step_, lo, hi)

        for i in ids:
            al[i] = adam(("al", i), al[i], gal[i], 1.0, lr_alpha, 0.0, 1.0)
            au[i] = adam(("au", i), au[i], gau[i], -1.0, lr_alpha, 0.0, 1.0)
        bl = adam("bl", bl, gbl, 1.0, lr_beta, 0.0, np.inf)
        bu = adam("bu", bu, gbu, -1.0, lr_beta, 0.0, np.inf)
    return BetaResult(best_l, best_u, np.array(lh), np.array(uh))


def default_order(net, root):
    """Split priority: the root's unstable neurons by decreasing chord intercept
    t = -u l / (u - l) (the height of the relaxation triangle), ties by position."""
    cand = []
    for r, i in enumerate(relu_ids(net)):
        l, u = root.layer_l[i], root.layer_u[i]
        for j in np.flatnonzero((l < 0) & (u > 0)):
            cand.append((-(-u[j] * l[j] / (u[j] - l[j])), r, int(j)))
    cand.sort()
    return [(r, j) for _, r, j in cand]


@dataclass
class BabResult:
    verified: bool
    rounds: int
    evaluated: int                         # subdomains bounded (the root not counted)
    remaining: int                         # unverified subdomains left
    log: list = field(default_factory=list)   # per round: (taken, evaluated, pruned, left)
    children: list = field(default_factory=list)   # per round: [(splits, lb)] in order


def bab(net, x0, eps, C, order=None, batch=4, rounds=10, iters=20, lr_alpha=0.1, lr_beta=0.05, root=None):
    """Fixed-batch branch-and-bound on the property C f(x) > 0 (every row) over the
    eps-ball (see the module docstring for the loop)."""
    _check_chain(net)
    if root is None:
        root = cr.crown(net, x0, eps, C)
    order = default_order(net, root) if order is None else [tuple(o) for o in order]
    r0 = beta_crown(net, root, C, [], iters=iters, lr_alpha=lr_alpha, lr_beta=lr_beta)
    res = BabResult(verified=bool(np.all(r0.lb > 0.0)), rounds=0, evaluated=0, remaining=0)
    if res.verified:
        return res
    queue = [()]
    stuck = False
    for rnd in range(rounds):
        if not queue:
            break
        take, queue = queue[:batch], queue[batch:]
        kids = []
        for dom in take:
            used = {(r, j) for r, j, _ in dom}
            nxt = next((o for o in order if o not in used), None)
            if nxt is None:
                stuck = True       # nothing left to split: stays unverified
                queue.append(dom)
                continue
            kids += [dom + ((nxt[0], nxt[1], 1),), dom + ((nxt[0], nxt[1], -1),)]
        pruned = 0
        logged = []
        for k in kids:
            r = beta_crown(net, root, C, list(k), iters=iters, lr_alpha=lr_alpha, lr_beta=lr_beta)
            logged.append((k, r.lb))
            if np.all(r.lb > 0.0):
                pruned += 1
            else:
                queue.append(k)
        res.evaluated += len(kids)
        res.rounds = rnd + 1
        res.log.append((len(take), len(kids), pruned, len(queue)))
        res.children.append(logged)
        if stuck and not kids:
            break
    res.remaining = len(queue)
    res.verified = not queue
    return res
