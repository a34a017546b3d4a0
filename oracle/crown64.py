"""fp64 CPU oracle for IBP and CROWN bound propagation on feed-forward ReLU networks.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's CPU-baseline
leg may import this module.  It shares no code with the GPU library: it reads the same
seeded arrays (float32 weights, inputs, specifications) and promotes them exactly to
float64.  It is deliberately slow and written to be checked against the paper by eye.

What it computes (section numbers are the paper's):
  * the input set, an L-infinity ball of radius eps around x0 intersected with a clip box
    (Sec. 1.1, local robustness);
  * IBP, the interval step l_y = W+ l_x + W- u_x + b, u_y = W+ u_x + W- l_x + b
    (Sec. 2.1, IBP);
  * the CROWN ReLU relaxation lambda*z <= ReLU(z) <= u/(u-l) (z - l) for unstable neurons
    (Sec. 2.1, CROWN);
  * the CROWN backward pass composing layer weights with the diagonal slope matrices, with
    different slope choices for the lower and the upper branch, giving
    A_L x + b_L <= f(x) <= A_U x + b_U (Sec. 2.1, equation "crown"), then the minimum and
    maximum of those linear functions over the input box;
  * full CROWN: intermediate pre-activation bounds for every ReLU by a backward pass from
    that layer down to the input, each intersected with the IBP bounds;
  * branch-and-bound subdomains that fix ReLUs to the active (z >= 0) or inactive (z <= 0)
    state (Sec. 2.1, complete verification), bounded with the root's intermediate bounds
    and only the split neurons' own intervals clamped;
  * the same full CROWN for one-hidden-layer networks in row blocks of the first weight
    matrix (memory-bounded, for the Exp. 1 network of Sec. 4.1).

Readings where the paper is silent (each is also listed in the design notes):
  * adaptive lower slope: lambda = 1 if u > -l else 0, a tie giving 0;
  * a neuron with u <= 0 is inactive (0, 0, 0); otherwise l >= 0 is active (1, 1, 0);
  * IBP bounds on C f(x) fold C into the last dense layer (C W_L, C b_L);
  * the box is computed in float32 (x0 - eps and x0 + eps rounded to nearest, then
    clamped to the clip box) and promoted to float64;
  * an infeasible subdomain (some l > u after clamping) gets lb = +inf, ub = -inf.

Formulation chosen to differ from a GPU-friendly one wherever the mathematics allows:
IBP uses the W+/W- split (not centre/radius); the upper bound uses the explicit upper rule
(not a negated lower pass); convolutions propagate dense coefficient tensors through an
explicit transposed convolution; the final minimum over the box is taken vertex-wise,
sum_i min(a_i lo_i, a_i hi_i).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "input_box", "node_shapes", "forward", "ibp", "ibp_spec_bounds", "relu_relaxation",
    "conv2d", "conv2d_transpose", "backward", "concretize", "crown", "CrownResult",
    "apply_splits", "crown_domains", "unstable_pool", "support", "crown_sampled", "crown_one_hidden",
]


# --------------------------------------------------------------------------------------
# shapes and plain evaluation

def node_shapes(net):
    """Output shape of every node, in node order."""
    shapes = []
    for nd in net.nodes:
        s = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
        if nd.op == "dense":
            shapes.append((nd.W.shape[0],))
        elif nd.op == "conv2d":
            kh, kw = nd.W.shape[2:]
            shapes.append((nd.W.shape[0], (s[1] + 2 * nd.pad - kh) // nd.stride + 1,
                           (s[2] + 2 * nd.pad - kw) // nd.stride + 1))
        elif nd.op in ("relu", "add"):
            shapes.append(s)
        elif nd.op == "flatten":
            shapes.append((int(np.prod(s)),))
        else:
            raise ValueError(nd.op)
    return shapes


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def conv2d(x, W, stride, pad):
    """Plain 2-D cross-correlation of x (C_in, H, W) with W (C_out, C_in, kh, kw), zero
    padding `pad` on every side; no bias.  out[o, y, x] = sum_{c,i,j} W[o,c,i,j] *
    xpad[c, y*stride + i, x*stride + j]."""
    ci, h, w = x.shape
    co, _, kh, kw = W.shape
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (w + 2 * pad - kw) // stride + 1
    xp = np.zeros((ci, h + 2 * pad, w + 2 * pad))
    xp[:, pad:pad + h, pad:pad + w] = x
    out = np.zeros((co, ho, wo))
    for i in range(kh):
        for j in range(kw):
            patch = xp[:, i:i + stride * (ho - 1) + 1:stride, j:j + stride * (wo - 1) + 1:stride]
            out += np.tensordot(W[:, :, i, j], patch, axes=([1], [0]))
    return out


def conv2d_transpose(A, W, stride, pad, in_hw):
    """Adjoint of `conv2d` for a stack of coefficient rows.

    A is (rows, C_out, H_out, W_out), the coefficients on a convolution's output; the
    result is (rows, C_in, H, W), the coefficients on its input, i.e. the matrix
    transpose of the convolution applied to every row.  Each output position scatters
    A[:, :, y, x] @ W[:, :, i, j] to input position (y*stride + i - pad, x*stride + j - pad);
    positions that fall into the zero padding are dropped."""
    rows, co, ho, wo = A.shape
    _, ci, kh, kw = W.shape
    h, w = in_hw
    hp, wp = h + 2 * pad + stride, w + 2 * pad + stride
    out = np.zeros((rows, ci, hp, wp))
    for i in range(kh):
        for j in range(kw):
            contrib = np.tensordot(A, W[:, :, i, j], axes=([1], [0])).transpose(0, 3, 1, 2)
            out[:, :, i:i + stride * (ho - 1) + 1:stride, j:j + stride * (wo - 1) + 1:stride] += contrib
    return out[:, :, pad:pad + h, pad:pad + w]


def forward(net, x):
    """fp64 network evaluation at one flat input point; returns every node's value."""
    vals = []
    inp = np.asarray(x, dtype=np.float64).reshape(net.in_shape)
    get = lambda i: inp if i == -1 else vals[i]  # noqa: E731
    for nd in net.nodes:
        v = get(nd.in0)
        if nd.op == "dense":
            vals.append(_f64(nd.W) @ v.reshape(-1) + _f64(nd.b))
        elif nd.op == "conv2d":
            vals.append(conv2d(v, _f64(nd.W), nd.stride, nd.pad) + _f64(nd.b)[:, None, None])
        elif nd.op == "relu":
            vals.append(np.maximum(v, 0.0))
        elif nd.op == "add":
            vals.append(v + get(nd.in1))
        elif nd.op == "flatten":
            vals.append(v.reshape(-1))
    return vals


# --------------------------------------------------------------------------------------
# the input set (Sec. 1.1, local robustness in the L-infinity norm)

def input_box(x0, eps, clip=(0.0, 1.0)):
    """Box [lo, hi] = {x : |x - x0|_inf <= eps} intersected with the clip box.  Computed in
    float32 (round to nearest) exactly as the float32 inputs define it, then promoted."""
    x0 = np.asarray(x0, dtype=np.float32)
    e = np.float32(eps)
    lo = (x0 - e).astype(np.float32)
    hi = (x0 + e).astype(np.float32)
    if clip is not None:
        lo = np.maximum(lo, np.float32(clip[0]))
        hi = np.minimum(hi, np.float32(clip[1]))
    return lo.astype(np.float64), hi.astype(np.float64)


# --------------------------------------------------------------------------------------
# IBP (Sec. 2.1): l_y = W+ l + W- u + b, u_y = W+ u + W- l + b

def ibp(net, lo, hi):
    """Interval bounds [l, u] of every node's output over the box [lo, hi] (flat input)."""
    L, U = [], []
    lin = np.asarray(lo, np.float64).reshape(net.in_shape)
    uin = np.asarray(hi, np.float64).reshape(net.in_shape)
    get = lambda i: (lin, uin) if i == -1 else (L[i], U[i])  # noqa: E731
    for nd in net.nodes:
        l, u = get(nd.in0)
        if nd.op == "dense":
            W = _f64(nd.W)
            Wp, Wn = np.maximum(W, 0.0), np.minimum(W, 0.0)
            l, u = l.reshape(-1), u.reshape(-1)
            L.append(Wp @ l + Wn @ u + _f64(nd.b))
            U.append(Wp @ u + Wn @ l + _f64(nd.b))
        elif nd.op == "conv2d":
            W = _f64(nd.W)
            Wp, Wn = np.maximum(W, 0.0), np.minimum(W, 0.0)
            b = _f64(nd.b)[:, None, None]
            L.append(conv2d(l, Wp, nd.stride, nd.pad) + conv2d(u, Wn, nd.stride, nd.pad) + b)
            U.append(conv2d(u, Wp, nd.stride, nd.pad) + conv2d(l, Wn, nd.stride, nd.pad) + b)
        elif nd.op == "relu":
            L.append(np.maximum(l, 0.0))
            U.append(np.maximum(u, 0.0))
        elif nd.op == "add":
            l1, u1 = get(nd.in1)
            L.append(l + l1)
            U.append(u + u1)
        elif nd.op == "flatten":
            L.append(l.reshape(-1))
            U.append(u.reshape(-1))
    return L, U


def ibp_spec_bounds(net, x0, eps, C, clip=(0.0, 1.0)):
    """IBP bounds on C f(x): the last node must be dense; C is folded into it, i.e. the
    interval step is applied to the single affine map (C W_L, C b_L)."""
    last = net.nodes[-1]
    if last.op != "dense":
        raise ValueError("the spec is folded into a final dense layer")
    lo, hi = input_box(x0, eps, clip)
    L, U = ibp(net, lo, hi)
    if last.in0 == -1:
        l, u = lo, hi
    else:
        l, u = L[last.in0].reshape(-1), U[last.in0].reshape(-1)
    Cm = _f64(C)
    W = Cm @ _f64(last.W)
    b = Cm @ _f64(last.b)
    Wp, Wn = np.maximum(W, 0.0), np.minimum(W, 0.0)
    return Wp @ l + Wn @ u + b, Wp @ u + Wn @ l + b


# --------------------------------------------------------------------------------------
# ReLU linear relaxation (Sec. 2.1, CROWN)

def relu_relaxation(l, u, rule="adaptive", override=None):
    """Per-neuron (lam, s, t) with lam*z <= ReLU(z) <= s*z + t on [l, u].

    inactive (u <= 0): (0, 0, 0); active (l >= 0): (1, 1, 0); unstable (l < 0 < u):
    s = u/(u-l), t = -s*l (the chord through (l, 0) and (u, u)) and a lower slope lam in
    [0, 1]: 'adaptive' = 1 if u > -l else 0, 'zero', 'one', or 'same_slope' (= s).
    `override` maps flat neuron index -> lam for unstable neurons (tests only)."""
    l = np.asarray(l, np.float64)
    u = np.asarray(u, np.float64)
    lam = np.zeros_like(l)
    s = np.zeros_like(l)
    t = np.zeros_like(l)
    inactive = u <= 0.0
    active = (l >= 0.0) & ~inactive
    unstable = ~inactive & ~active
    lam[active] = 1.0
    s[active] = 1.0
    lu, uu = l[unstable], u[unstable]
    su = uu / (uu - lu)
    s[unstable] = su
    t[unstable] = -su * lu
    if rule == "adaptive":
        lam[unstable] = np.where(uu > -lu, 1.0, 0.0)
    elif rule == "zero":
        lam[unstable] = 0.0
    elif rule == "one":
        lam[unstable] = 1.0
    elif rule == "same_slope":
        lam[unstable] = su
    else:
        raise ValueError(rule)
    if override:
        flat_l = lam.reshape(-1)
        flat_unst = unstable.reshape(-1)
        for j, v in override.items():
            if flat_unst[j]:
                flat_l[j] = v
    return lam, s, t


# --------------------------------------------------------------------------------------
# CROWN backward pass (Sec. 2.1, equation "crown")

def _accumulate(acc, node, A):
    if node in acc:
        acc[node] = acc[node] + A
    else:
        acc[node] = A


def backward(net, shapes, relax, start, A, bias, upper):
    """Propagate linear coefficients from node `start` down to the network input.

    A (rows, numel(start)) holds coefficients on start's output and `bias` (rows,) the
    constant; together they describe the linear functions A . v_start + bias whose lower
    (upper=False) or upper (upper=True) bound is wanted.  `relax` maps every ReLU node id
    below `start` to its (lam, s, t).  Nodes are visited in reverse node order, so all
    consumers of a node have added their coefficients before the node is expanded.

    Returns (A_x, bias): coefficients on the flat network input and the accumulated
    constant, so that A_x . x + bias bounds the functions for every x in the box."""
    acc = {start: np.asarray(A, np.float64)}
    bias = np.array(bias, dtype=np.float64, copy=True)
    for i in range(start, -1, -1):
        if i not in acc:
            continue
        Ai = acc.pop(i)
        nd = net.nodes[i]
        rows = Ai.shape[0]
        if nd.op == "dense":
            # A . (W h + b) = (A W) . h + A . b
            bias = bias + Ai @ _f64(nd.b)
            _accumulate(acc, nd.in0, Ai @ _f64(nd.W))
        elif nd.op == "conv2d":
            co, ho, wo = shapes[i]
            in_shape = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
            A4 = Ai.reshape(rows, co, ho, wo)
            bias = bias + A4.sum(axis=(2, 3)) @ _f64(nd.b)
            Ain = conv2d_transpose(A4, _f64(nd.W), nd.stride, nd.pad, in_shape[1:])
            _accumulate(acc, nd.in0, Ain.reshape(rows, -1))
        elif nd.op == "relu":
            lam, s, t = (v.reshape(-1) for v in relax[i])
            Ap = np.maximum(Ai, 0.0)
            An = np.minimum(Ai, 0.0)
            if not upper:
                # positive coefficients take the lower line lam*z, negative ones the upper
                # line s*z + t
                bias = bias + An @ t
                Az = Ap * lam + An * s
            else:
                # positive coefficients take the upper line, negative ones the lower line
                bias = bias + Ap @ t
                Az = Ap * s + An * lam
            _accumulate(acc, nd.in0, Az)
        elif nd.op == "add":
            _accumulate(acc, nd.in0, Ai)
            _accumulate(acc, nd.in1, Ai)
        elif nd.op == "flatten":
            _accumulate(acc, nd.in0, Ai)
        else:
            raise ValueError(nd.op)
    A_x = acc.pop(-1) if -1 in acc else np.zeros((A.shape[0], int(np.prod(net.in_shape))))
    return A_x, bias


def concretize(A_x, bias, lo, hi, upper):
    """Minimum (upper=False) or maximum (upper=True) of A_x . x + bias over the box,
    taken coordinate-wise at the minimising / maximising vertex."""
    lo = np.asarray(lo, np.float64).reshape(-1)
    hi = np.asarray(hi, np.float64).reshape(-1)
    if not upper:
        return np.minimum(A_x * lo, A_x * hi).sum(axis=1) + bias
    return np.maximum(A_x * lo, A_x * hi).sum(axis=1) + bias


@dataclass
class CrownResult:
    lb: np.ndarray                       # (m,) lower bounds on C f(x)
    ub: np.ndarray                       # (m,) upper bounds on C f(x)
    layer_l: dict = field(default_factory=dict)   # relu node id -> pre-activation lower bound
    layer_u: dict = field(default_factory=dict)   # relu node id -> pre-activation upper bound
    ibp_l: dict = field(default_factory=dict)     # relu node id -> IBP lower bound of its input
    ibp_u: dict = field(default_factory=dict)
    relax: dict = field(default_factory=dict)     # relu node id -> (lam, s, t)
    A_lower: np.ndarray | None = None    # final coefficients on the input (lower branch)
    A_upper: np.ndarray | None = None
    box: tuple | None = None


def _layer_bounds(net, shapes, relax, z, lo, hi, chunk):
    """CROWN lower/upper bounds of every neuron of node z, from a backward pass per row
    block of the identity."""
    n = int(np.prod(shapes[z]))
    nd = net.nodes[z]
    if nd.op == "dense" and nd.in0 == -1:
        # a single affine map of the input: the backward pass from I ends at A_x = W, bias
        # = b; take it directly instead of multiplying by the identity
        W = _f64(nd.W)
        b = _f64(nd.b)
        return concretize(W, b, lo, hi, False), concretize(W, b, lo, hi, True)
    l = np.empty(n)
    u = np.empty(n)
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        I = np.zeros((r1 - r0, n))
        I[np.arange(r1 - r0), np.arange(r0, r1)] = 1.0
        zero = np.zeros(r1 - r0)
        Al, bl = backward(net, shapes, relax, z, I, zero, upper=False)
        Au, bu = backward(net, shapes, relax, z, I, zero, upper=True)
        l[r0:r1] = concretize(Al, bl, lo, hi, False)
        u[r0:r1] = concretize(Au, bu, lo, hi, True)
    return l, u


def crown(net, x0, eps, C, clip=(0.0, 1.0), intersect_ibp=True, lambda_rule="adaptive",
          lambda_override=None, chunk=256, keep_A=False):
    """Full CROWN bounds on C f(x) for one input x0 (flat) over the clipped eps-ball.

    For every ReLU node in order, its input's pre-activation bounds come from a backward
    pass from that node to the input (intersected with IBP when `intersect_ibp`); the
    relaxation is then fixed, and the final pass runs from the output with A = C.
    `lambda_override` maps relu node id -> {flat neuron: lam} (tests only)."""
    shapes = node_shapes(net)
    lo, hi = input_box(x0, eps, clip)
    IL, IU = ibp(net, lo, hi)
    res = CrownResult(lb=None, ub=None, box=(lo, hi))
    for i, nd in enumerate(net.nodes):
        if nd.op != "relu":
            continue
        z = nd.in0
        if z == -1:
            l, u = lo.copy(), hi.copy()
        else:
            l, u = _layer_bounds(net, shapes, res.relax, z, lo, hi, chunk)
        il, iu = IL[z].reshape(-1) if z >= 0 else lo, IU[z].reshape(-1) if z >= 0 else hi
        if intersect_ibp:
            l = np.maximum(l, il)
            u = np.minimum(u, iu)
        res.layer_l[i], res.layer_u[i] = l, u
        res.ibp_l[i], res.ibp_u[i] = il, iu
        ov = None if lambda_override is None else lambda_override.get(i)
        res.relax[i] = relu_relaxation(l, u, lambda_rule, ov)
    res.lb, res.ub, Al, Au = _final_pass(net, shapes, res.relax, C, lo, hi)
    if keep_A:
        res.A_lower, res.A_upper = Al, Au
    return res


def _final_pass(net, shapes, relax, C, lo, hi):
    out = len(net.nodes) - 1
    Cm = np.asarray(C, np.float64)
    zero = np.zeros(Cm.shape[0])
    Al, bl = backward(net, shapes, relax, out, Cm, zero, upper=False)
    Au, bu = backward(net, shapes, relax, out, Cm, zero, upper=True)
    return concretize(Al, bl, lo, hi, False), concretize(Au, bu, lo, hi, True), Al, Au


# --------------------------------------------------------------------------------------
# branch-and-bound subdomains (Sec. 2.1, complete verification)

def apply_splits(net, root, relu_id, neuron, sign, lambda_rule="adaptive"):
    """Relaxation of one subdomain: the root's intermediate bounds with every split
    neuron's own interval clamped (active: l <- max(l, 0); inactive: u <- min(u, 0)).
    Returns the relaxation dict, or None if some interval became empty (l > u)."""
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    L = {i: root.layer_l[i].copy() for i in relus}
    U = {i: root.layer_u[i].copy() for i in relus}
    for r, j, sg in zip(relu_id, neuron, sign):
        i = relus[int(r)]
        if sg > 0:
            L[i][j] = max(L[i][j], 0.0)
        else:
            U[i][j] = min(U[i][j], 0.0)
    for i in relus:
        if np.any(L[i] > U[i]):
            return None
    return {i: relu_relaxation(L[i], U[i], lambda_rule) for i in relus}


def crown_domains(net, root, C, splits, domains=None, lambda_rule="adaptive"):
    """Final-layer CROWN bounds for each subdomain (lb, ub of shape (D, m)).  Infeasible
    domains get lb = +inf, ub = -inf.  `domains` restricts the evaluation to a subset."""
    shapes = node_shapes(net)
    lo, hi = root.box
    ids = range(splits.n_domains) if domains is None else domains
    m = np.asarray(C).shape[0]
    LB = np.empty((len(ids), m))
    UB = np.empty((len(ids), m))
    for k, d in enumerate(ids):
        rel = apply_splits(net, root, splits.relu_id[d], splits.neuron[d], splits.sign[d], lambda_rule)
        if rel is None:
            LB[k], UB[k] = np.inf, -np.inf
            continue
        LB[k], UB[k], _, _ = _final_pass(net, shapes, rel, C, lo, hi)
    return LB, UB


def unstable_pool(net, root, tau_abs=1e-4, tau_rel=1e-4):
    """(relu_id, neuron) pairs that the root pass finds unstable, excluding neurons whose
    l or u lies within tau = tau_abs + tau_rel*|bound| of zero."""
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    pool = []
    for r, i in enumerate(relus):
        l, u = root.layer_l[i], root.layer_u[i]
        ok = (l < -(tau_abs + tau_rel * np.abs(l))) & (u > tau_abs + tau_rel * np.abs(u))
        for j in np.nonzero(ok)[0]:
            pool.append((r, int(j)))
    return np.asarray(pool, dtype=np.int64).reshape(-1, 2)


# --------------------------------------------------------------------------------------
# bounds of selected neurons without computing whole layers

def support(net, shapes, start, rows_mask):
    """Structural support of a backward pass: for a boolean mask over the neurons of node
    `start` (one row per set entry, all rows together), which neurons of every ReLU node
    below can carry a nonzero coefficient.  Computed by propagating the mask with the
    absolute weights (every entry >= 0, so a sum is nonzero exactly when some path is),
    with every ReLU passed through unchanged.  Returns {relu node id: flat bool mask}."""
    acc = {start: np.asarray(rows_mask, np.float64).reshape(1, -1)}
    out = {}
    for i in range(start, -1, -1):
        if i not in acc:
            continue
        Ai = (acc.pop(i) > 0).astype(np.float64)
        nd = net.nodes[i]
        if nd.op == "dense":
            _accumulate(acc, nd.in0, Ai @ np.abs(_f64(nd.W)))
        elif nd.op == "conv2d":
            co, ho, wo = shapes[i]
            in_shape = tuple(net.in_shape) if nd.in0 == -1 else shapes[nd.in0]
            Ain = conv2d_transpose(Ai.reshape(1, co, ho, wo), np.abs(_f64(nd.W)), nd.stride, nd.pad, in_shape[1:])
            _accumulate(acc, nd.in0, Ain.reshape(1, -1))
        elif nd.op == "relu":
            out[i] = Ai.reshape(-1) > 0
            _accumulate(acc, nd.in0, Ai)
        elif nd.op in ("add",):
            _accumulate(acc, nd.in0, Ai)
            _accumulate(acc, nd.in1, Ai)
        elif nd.op == "flatten":
            _accumulate(acc, nd.in0, Ai)
    return out


def crown_sampled(net, x0, eps, targets, clip=(0.0, 1.0), intersect_ibp=True, chunk=256):
    """Full-CROWN bounds of selected pre-activation neurons, computing at each lower ReLU
    only the neurons the selected rows can reach (their receptive fields).

    targets: {relu node id: array of flat neuron indices}.  The bound of every computed
    neuron is the same sequence of operations as in `crown`: the rows that are not
    computed would only ever be multiplied by exact zeros.  Returns {relu node id:
    (indices, l, u)} for every ReLU node that needed neurons."""
    shapes = node_shapes(net)
    lo, hi = input_box(x0, eps, clip)
    IL, IU = ibp(net, lo, hi)
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    need = {i: np.zeros(int(np.prod(shapes[i])), bool) for i in relus}
    for i, idx in targets.items():
        need[i][np.asarray(idx, np.int64)] = True
    # top-down: the neurons every selected row reaches at the ReLUs below it
    for i in reversed(relus):
        if not need[i].any():
            continue
        z = net.nodes[i].in0
        for k, mask in support(net, shapes, z, need[i]).items():
            need[k] |= mask
    relax = {}
    out = {}
    for i in relus:
        z = net.nodes[i].in0
        n = int(np.prod(shapes[i]))
        idx = np.nonzero(need[i])[0]
        l = np.zeros(n)
        u = np.zeros(n)
        if len(idx):
            nd = net.nodes[z]
            if nd.op == "dense" and nd.in0 == -1:
                W, b = _f64(nd.W)[idx], _f64(nd.b)[idx]
                l[idx], u[idx] = concretize(W, b, lo, hi, False), concretize(W, b, lo, hi, True)
            else:
                for r0 in range(0, len(idx), chunk):
                    sel = idx[r0:r0 + chunk]
                    I = np.zeros((len(sel), n))
                    I[np.arange(len(sel)), sel] = 1.0
                    zero = np.zeros(len(sel))
                    Al, bl = backward(net, shapes, relax, z, I, zero, upper=False)
                    Au, bu = backward(net, shapes, relax, z, I, zero, upper=True)
                    l[sel] = concretize(Al, bl, lo, hi, False)
                    u[sel] = concretize(Au, bu, lo, hi, True)
            if intersect_ibp:
                l[idx] = np.maximum(l[idx], IL[z].reshape(-1)[idx])
                u[idx] = np.minimum(u[idx], IU[z].reshape(-1)[idx])
            out[i] = (idx, l[idx], u[idx])
        # neurons outside the set are never reached; (0, 0) makes them inactive
        relax[i] = relu_relaxation(l, u)
    return out


# --------------------------------------------------------------------------------------
# one hidden layer, processed in row blocks (the paper's Exp. 1 network, Sec. 4.1)

def crown_one_hidden(net, x0, eps, C, clip=(0.0, 1.0), intersect_ibp=True, chunk=8192):
    """Full CROWN for dense -> relu -> dense, the same steps as crown() written for this
    structure so the first weight matrix is promoted to float64 one block of rows at a time
    (the 262144 x 4096 layer would need 8.6 GB per float64 copy).

    The hidden pre-activations are one affine map of the input, so their bounds are the
    exact box range (intersected with the IBP interval W+ l + W- u + b when intersect_ibp);
    the final pass composes C W2, the relaxation and W1 and takes the extremes over the
    box vertex-wise."""
    d1, r1, d2 = net.nodes
    if not (d1.op == "dense" and d1.in0 == -1 and r1.op == "relu" and r1.in0 == 0
            and d2.op == "dense" and d2.in0 == 1 and len(net.nodes) == 3):
        raise ValueError("crown_one_hidden needs dense -> relu -> dense")
    lo, hi = input_box(x0, eps, clip)
    n1 = d1.W.shape[0]
    l = np.empty(n1)
    u = np.empty(n1)
    for r0 in range(0, n1, chunk):
        rows = slice(r0, min(n1, r0 + chunk))
        W = _f64(d1.W[rows])
        b = _f64(d1.b[rows])
        l[rows] = concretize(W, b, lo, hi, False)
        u[rows] = concretize(W, b, lo, hi, True)
        if intersect_ibp:
            Wp, Wn = np.maximum(W, 0.0), np.minimum(W, 0.0)
            l[rows] = np.maximum(l[rows], Wp @ lo + Wn @ hi + b)
            u[rows] = np.minimum(u[rows], Wp @ hi + Wn @ lo + b)
    lam, s, t = relu_relaxation(l, u)
    Cm = _f64(C)
    A = Cm @ _f64(d2.W)
    bias = Cm @ _f64(d2.b)
    Ap, An = np.maximum(A, 0.0), np.minimum(A, 0.0)
    Az_l, bias_l = Ap * lam + An * s, bias + An @ t          # lower: positive -> lower line
    Az_u, bias_u = Ap * s + An * lam, bias + Ap @ t          # upper: positive -> upper line
    n0 = lo.size
    Ax_l, Ax_u = np.zeros((A.shape[0], n0)), np.zeros((A.shape[0], n0))
    for r0 in range(0, n1, chunk):
        rows = slice(r0, min(n1, r0 + chunk))
        W = _f64(d1.W[rows])
        b = _f64(d1.b[rows])
        Ax_l += Az_l[:, rows] @ W
        Ax_u += Az_u[:, rows] @ W
        bias_l = bias_l + Az_l[:, rows] @ b
        bias_u = bias_u + Az_u[:, rows] @ b
    lb = concretize(Ax_l, bias_l, lo, hi, False)
    ub = concretize(Ax_u, bias_u, lo, hi, True)
    return lb, ub, l, u
