"""fp64 CPU oracle for alpha-CROWN on feed-forward ReLU chains.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's CPU-baseline
leg may import this module.  It shares no code with the GPU library.

What it computes (section numbers are the paper's): alpha-CROWN (Sec. 2.1) turns the lower
slope lambda of every unstable ReLU neuron into a parameter alpha in [0, 1] and raises the
lower bound (lowers the upper bound) by gradient steps, with no branching.  Every choice of
alpha in [0, 1] gives a sound bound, because alpha*z is below ReLU(z) on any interval.  The
alpha tensors have one slope per (layer, specification row, input, neuron) (Sec. 4.6), so
every bound of every specification row is optimised on its own.

Readings where the paper is silent (each is also listed in the design notes):
  * only the final specification pass is optimised; the intermediate pre-activation bounds
    stay those of full CROWN (IBP-intersected), so the relaxation lines s, t and the
    classes of all neurons are CROWN's;
  * the optimiser is Adam with bias correction (beta1 0.9, beta2 0.999, eps 1e-8, step 0.1
    by default), followed by projection onto [0, 1]; the initial slopes are CROWN's
    adaptive lambda; the result of a run of T steps is, per row, the best bound among the
    T + 1 evaluated slope sets (the initial one included), with its slopes;
  * the gradient at a coefficient that is exactly 0 takes the branch of a negative
    coefficient in the lower pass (upper line, no intercept term) and of a positive one in
    the upper pass, the same as the lines the bound itself uses there; the input vertex
    at a zero input coefficient is the box centre.

How the gradient is obtained: the lower bound of a row is a.x* + beta at the box vertex x*
that minimises it, where a and beta are built by the backward pass.  Differentiating the
backward pass layer by layer shows that d lb / d alpha_j at ReLU k is a_j D_j when the
coefficient a_j on that ReLU's output is positive (0 otherwise), where D_j is the
pre-activation z_j obtained by evaluating the network forward from x* with every ReLU
replaced by the line its coefficient's sign selected (alpha z where a > 0, s z + t where
a < 0, s z where a = 0).  The upper bound is the mirror image (alpha where a < 0, the
maximising vertex).  Networks: dense, conv2d, relu, add and flatten nodes in topological
order (residual blocks included): the backward pass sums the coefficients that reach a node
along every path, and the forward evaluation adds both inputs of an add, so the same
argument holds (the coefficient on h_j is the derivative of the relaxed network's linear
function with respect to h_j).
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
            raise ValueError(f"alpha-CROWN oracle: unsupported node {nd.op}")
        if not (-1 <= nd.in0 < i) or (nd.op == "add" and not (-1 <= nd.in1 < i)):
            raise ValueError("alpha-CROWN oracle: nodes must be in topological order")


def unstable_mask(root, i):
    return (root.layer_l[i] < 0.0) & (root.layer_u[i] > 0.0)


def initial_alpha(net, root, m):
    """CROWN's adaptive lambda for every row: {relu id: (m, n)} for the lower and the upper
    pass."""
    al, au = {}, {}
    for i in relu_ids(net):
        lam = root.relax[i][0].reshape(-1)
        al[i] = np.tile(lam, (m, 1))
        au[i] = np.tile(lam, (m, 1))
    return al, au


def _pass(net, shapes, root, C, alpha, upper):
    """Backward pass from the output with A = C and per-row lower slopes `alpha`.

    Nodes are visited in reverse order; the coefficients that reach a node along several
    paths (the two inputs of an add) are summed before the node is expanded.  Returns the
    bound of every row, the coefficients on the input and, for every ReLU, the coefficient
    rows on its output before relaxation."""
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
            lam0, s, t = (v.reshape(-1) for v in root.relax[i])
            lam = np.where(unstable_mask(root, i).reshape(-1)[None, :], alpha[i], lam0[None, :])
            pre[i] = A.copy()
            Ap, An = np.maximum(A, 0.0), np.minimum(A, 0.0)
            if not upper:
                bias = bias + An @ t
                add_to(nd.in0, Ap * lam + An * s)
            else:
                bias = bias + Ap @ t
                add_to(nd.in0, Ap * s + An * lam)
        elif nd.op == "add":
            add_to(nd.in0, A)
            add_to(nd.in1, A)
        elif nd.op == "flatten":
            # coefficients keep their (C, H, W) order
            add_to(nd.in0, A)
    A = acc.pop(-1) if -1 in acc else np.zeros((rows, int(np.prod(net.in_shape))))
    lo, hi = root.box
    return cr.concretize(A, bias, lo, hi, upper), A, pre


def _gradient(net, shapes, root, A_x, pre, alpha, upper):
    """d bound / d alpha for every ReLU (see the module docstring): the relaxed network
    evaluated forward, node by node, from the attaining box vertex."""
    lo, hi = root.box
    c, r = (lo + hi) / 2.0, (hi - lo) / 2.0
    sgn = np.sign(A_x)
    x = c[None, :] + sgn * r[None, :] if upper else c[None, :] - sgn * r[None, :]
    rows = x.shape[0]
    val = {}
    grad = {}
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
            lam0, s, t = (q.reshape(-1) for q in root.relax[i])
            unst = unstable_mask(root, i).reshape(-1)[None, :]
            lam = np.where(unst, alpha[i], lam0[None, :])
            a = pre[i]
            D = v.reshape(rows, -1)
            if not upper:
                on_lam, on_chord_t = a > 0.0, a < 0.0
            else:
                on_lam, on_chord_t = a < 0.0, a > 0.0
            grad[i] = np.where(unst & on_lam, a * D, 0.0)
            val[i] = np.where(on_lam, lam * D, s[None, :] * D + np.where(on_chord_t, t[None, :], 0.0))
        elif nd.op == "add":
            val[i] = v.reshape(rows, -1) + get(nd.in1).reshape(rows, -1)
        elif nd.op == "flatten":
            val[i] = v.reshape(rows, -1)
    return grad


def alpha_bound(net, root, C, alpha_l, alpha_u):
    """Bounds of C f(x) over the box with the given slopes, and their gradients.

    root: the oracle's full-CROWN result for the input (intermediate bounds, relaxation,
    box).  alpha_l / alpha_u: {relu id: (m, n)} slopes of the lower / upper pass of every
    row (entries of stable neurons are ignored).  Returns lb, ub (m,) and the gradients
    d lb / d alpha_l, d ub / d alpha_u as {relu id: (m, n)}."""
    _check_chain(net)
    shapes = cr.node_shapes(net)
    lb, Al, pre_l = _pass(net, shapes, root, C, alpha_l, upper=False)
    ub, Au, pre_u = _pass(net, shapes, root, C, alpha_u, upper=True)
    gl = _gradient(net, shapes, root, Al, pre_l, alpha_l, upper=False)
    gu = _gradient(net, shapes, root, Au, pre_u, alpha_u, upper=True)
    return lb, ub, gl, gu


@dataclass
class AlphaResult:
    lb: np.ndarray                  # (m,) best lower bound of each row
    ub: np.ndarray                  # (m,) best upper bound of each row
    lb_hist: np.ndarray             # (T + 1, m) lower bound of every evaluation
    ub_hist: np.ndarray             # (T + 1, m)
    alpha_l: dict = field(default_factory=dict)   # slopes of the best lower bound, per row
    alpha_u: dict = field(default_factory=dict)
    grad_l: dict = field(default_factory=dict)    # gradient at the last evaluated slopes
    grad_u: dict = field(default_factory=dict)
    root: object = None


def alpha_crown(net, x0, eps, C, iters=20, lr=0.1, beta1=0.9, beta2=0.999, adam_eps=1e-8,
                clip=(0.0, 1.0), intersect_ibp=True, alpha_init=None, root=None):
    """alpha-CROWN bounds on C f(x) for one input: full CROWN for the intermediate bounds,
    then `iters` projected Adam steps on the slopes of the final pass (ascent on each lower
    bound, descent on each upper bound), keeping each row's best bound."""
    _check_chain(net)
    if root is None:
        root = cr.crown(net, x0, eps, C, clip=clip, intersect_ibp=intersect_ibp)
    C = np.asarray(C, np.float64)
    m = C.shape[0]
    ids = relu_ids(net)
    if alpha_init is None:
        al, au = initial_alpha(net, root, m)
    else:
        al = {i: np.array(alpha_init[0][i], np.float64) for i in ids}
        au = {i: np.array(alpha_init[1][i], np.float64) for i in ids}
    mom = {(d, i): np.zeros_like(al[i]) for d in "lu" for i in ids}
    vel = {(d, i): np.zeros_like(al[i]) for d in "lu" for i in ids}
    lb_hist, ub_hist = [], []
    best_l = np.full(m, -np.inf)
    best_u = np.full(m, np.inf)
    best_al = {i: al[i].copy() for i in ids}
    best_au = {i: au[i].copy() for i in ids}
    gl = gu = None
    for step in range(iters + 1):
        lb, ub, gl, gu = alpha_bound(net, root, C, al, au)
        lb_hist.append(lb)
        ub_hist.append(ub)
        # keep each row's best bound and its slopes
        better_l, better_u = lb > best_l, ub < best_u
        best_l = np.where(better_l, lb, best_l)
        best_u = np.where(better_u, ub, best_u)
        for i in ids:
            best_al[i][better_l] = al[i][better_l]
            best_au[i][better_u] = au[i][better_u]
        if step == iters:
            break
        # Adam: ascent on the lower bounds, descent on the upper bounds, then projection
        t = step + 1
        for d, a, g, sign in (("l", al, gl, 1.0), ("u", au, gu, -1.0)):
            for i in ids:
                mom[d, i] = beta1 * mom[d, i] + (1.0 - beta1) * g[i]
                vel[d, i] = beta2 * vel[d, i] + (1.0 - beta2) * g[i] * g[i]
                mhat = mom[d, i] / (1.0 - beta1 ** t)
                vhat = vel[d, i] / (1.0 - beta2 ** t)
                a[i] = np.clip(a[i] + sign * lr * mhat / (np.sqrt(vhat) + adam_eps), 0.0, 1.0)
    return AlphaResult(lb=best_l, ub=best_u, lb_hist=np.array(lb_hist), ub_hist=np.array(ub_hist),
                       alpha_l=best_al, alpha_u=best_au, grad_l=gl, grad_u=gu, root=root)


def flat_rows(net, per_relu_l, per_relu_u):
    """The GPU library's row layout for one input: rows 0..m-1 the lower pass, m..2m-1 the
    upper pass; columns the ReLU neurons of every ReLU node in node order."""
    ids = relu_ids(net)
    lo = np.concatenate([per_relu_l[i] for i in ids], axis=1)
    up = np.concatenate([per_relu_u[i] for i in ids], axis=1)
    return np.concatenate([lo, up], axis=0)


def split_rows(net, flat, m):
    """Inverse of flat_rows: {relu id: (m, n)} for the lower and the upper pass."""
    shapes = cr.node_shapes(net)
    ids = relu_ids(net)
    al, au, c0 = {}, {}, 0
    for i in ids:
        n = int(np.prod(shapes[i]))
        al[i] = np.asarray(flat[:m, c0:c0 + n], np.float64)
        au[i] = np.asarray(flat[m:, c0:c0 + n], np.float64)
        c0 += n
    return al, au
