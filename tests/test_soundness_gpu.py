"""Soundness of the GPU's own bounds (the contract of Sec. 2.1: a lower bound never exceeds
the true minimum, an upper bound never falls below the true maximum), on the benchmark
workloads at full size.

For each workload, 10^5 points drawn uniformly from the input boxes and 10^4 random box
vertices, split evenly across the batch's inputs, plus per input and spec row two vertices
aimed at the bounds: the one where the gradient of that row at x0 points (lo where the row
increases with x_i, else hi, and the mirror image), and, where the oracle's final linear
bounds are available, the vertex where each of them is attained.  The network is evaluated
at every point by torch's own fp32 linear and convolution routines (independent of the
library); a point passes when lb - tau <= C f(x) <= ub + tau with the parity tolerance
tau = 1e-4 + 1e-4 |C f(x)| (an fp32 bound may sit a rounding above a value it attains).

Branch-and-bound subdomains (the 4096 of the 784-1024x6 MLP): a point belongs to a subdomain
when every split neuron's pre-activation has the split's sign there (kept only when it is
clearly away from 0 in fp32); the subdomain's bounds must hold at its points.  A subdomain
whose splits agree with x0's own activation pattern holds x0."""
import os

import numpy as np
import pytest

import oracle
from tests.gpu_util import gpu_crown, gpu_ctx, log, to_dev
from tests.pins import box_of
from tests.test_conv_gpu import torch_forward
from workloads import make_workload

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
N_SAMPLES, N_CORNERS = 100_000, 10_000


def _spec_values(net, X, Cb):
    """C f(x) at the rows of X (a CUDA float32 tensor), in float64."""
    import torch
    with torch.no_grad():
        y = torch_forward(net, X)[-1]
        return y.double() @ torch.from_numpy(Cb.astype(np.float64)).cuda().T


def _gradient_vertices(net, x0, Cb, lo, hi):
    """Per spec row, the box vertex in the direction that lowers the row (lo where its gradient
    at x0 is positive) and the one that raises it."""
    import torch
    m = Cb.shape[0]
    x = torch.from_numpy(np.repeat(x0[None].astype(np.float32), m, 0)).cuda().requires_grad_(True)
    y = torch_forward(net, x)[-1]
    (y * torch.from_numpy(Cb).cuda()).sum().backward()
    g = x.grad.cpu().numpy()
    low = np.where(g > 0, lo[None], hi[None])
    high = np.where(g > 0, hi[None], lo[None])
    return np.concatenate([low, high]).astype(np.float32)


def _check_points(net, lb, ub, Cb, X, what, chunk=4096):
    import torch
    worst = -np.inf
    for p0 in range(0, X.shape[0], chunk):
        Y = _spec_values(net, X[p0:p0 + chunk], Cb)
        lbt = torch.from_numpy(lb.astype(np.float64)).cuda()[None]
        ubt = torch.from_numpy(ub.astype(np.float64)).cuda()[None]
        slack = 1e-4 + 1e-4 * Y.abs()
        lo_v = (lbt - slack - Y).max().item()
        hi_v = (Y - ubt - slack).max().item()
        worst = max(worst, lo_v, hi_v)
        assert lo_v <= 0.0, f"{what}: C f(x) below the lower bound by {lo_v} beyond the slack"
        assert hi_v <= 0.0, f"{what}: C f(x) above the upper bound by {hi_v} beyond the slack"
    return worst


def _sound_on_workload(name, a_guided=None, alpha_iters=0):
    """T7 on every input of the workload's batch.  a_guided: {input: (n, n0) vertices}.
    alpha_iters > 0: the alpha-CROWN bounds after that many steps (never looser than
    CROWN's) instead of CROWN's."""
    import torch
    wl = make_workload(name)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = gpu_crown(ctx, wl)
    if alpha_iters:
        la, ua, _ = ctx.alpha_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), iters=alpha_iters)
        la, ua = la.cpu().numpy(), ua.cpu().numpy()
        assert np.all(la >= lb) and np.all(ua <= ub)
        log(name, "alpha-CROWN mean gain over CROWN", float(np.mean(la - lb)), float(np.mean(ub - ua)))
        lb, ub = la, ua
    B = wl.x0.shape[0]
    ns, nc = N_SAMPLES // B, N_CORNERS // B
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1234)
    n_points = 0
    for b in range(B):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        lo_t = torch.from_numpy(lo.astype(np.float32)).cuda()
        hi_t = torch.from_numpy(hi.astype(np.float32)).cuda()
        U = torch.rand((ns, lo.size), generator=gen, device="cuda")
        X = lo_t + (hi_t - lo_t) * U
        V = torch.where(torch.rand((nc, lo.size), generator=gen, device="cuda") < 0.5, lo_t, hi_t)
        G = torch.from_numpy(_gradient_vertices(wl.net, wl.x0[b], wl.C[b], lo, hi)).cuda()
        sets = [("samples", X), ("corners", V), ("gradient vertices", G)]
        if a_guided and b in a_guided:
            sets.append(("A-guided vertices", torch.from_numpy(a_guided[b].astype(np.float32)).cuda()))
        for what, P in sets:
            _check_points(wl.net, lb[b], ub[b], wl.C[b], P, f"{name} input {b} {what}")
            n_points += P.shape[0]
    log(name, "points checked", n_points)
    assert n_points >= N_SAMPLES + N_CORNERS - 2 * B


def _a_guided_from_oracle(wl, b):
    r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b], keep_A=True)
    lo, hi = r.box
    return np.concatenate([np.where(r.A_lower > 0, lo[None], hi[None]), np.where(r.A_upper > 0, hi[None], lo[None])])


def test_sound_mlp784x1024x6():
    wl = make_workload("mlp784x1024x6")
    _sound_on_workload("mlp784x1024x6", {b: _a_guided_from_oracle(wl, b) for b in (0, 63)})


def test_sound_mlp3072x8192x4():
    wl = make_workload("mlp3072x8192x4")
    g = np.load(os.path.join(GOLDEN, "mlp3072x8192x4_corners.npz"))
    guided = {}
    n0 = wl.x0.shape[1]
    for b in g["inputs"]:
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        at_lo = np.unpackbits(g[f"lower_at_lo_{b}"], axis=1, count=n0).astype(bool)
        at_hi = np.unpackbits(g[f"upper_at_hi_{b}"], axis=1, count=n0).astype(bool)
        guided[int(b)] = np.concatenate([np.where(at_lo, lo[None], hi[None]), np.where(at_hi, hi[None], lo[None])])
    _sound_on_workload("mlp3072x8192x4", guided)


def test_sound_resnet3x32x32():
    _sound_on_workload("resnet3x32x32")


def test_sound_resnet3x32x32_alpha():
    """alpha-CROWN (20 steps) on the full ResNet: the optimised bounds hold at the sampled
    points, corners and gradient vertices of every input."""
    _sound_on_workload("resnet3x32x32", alpha_iters=20)


def test_sound_bab_subdomains_membership():
    """T12 on the 4096 stored subdomains: points of the root box sorted into subdomains by the
    signs of their split neurons' pre-activations."""
    import torch
    wl = make_workload("bab_mlp784x1024x6")
    sp = np.load(os.path.join(GOLDEN, "bab_mlp784x1024x6_splits.npz"))
    D, S = sp["relu_id"].shape
    ctx = gpu_ctx(wl.net)
    splits = tuple(to_dev(np.ascontiguousarray(sp[k])) for k in ("relu_id", "neuron", "sign"))
    lb, ub = ctx.crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), splits=splits)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy().astype(np.float64), ub.cpu().numpy().astype(np.float64)
    feasible = np.isfinite(lb).all(1)
    pre_ids = [nd.in0 for nd in wl.net.nodes if nd.op == "relu"]
    rid = torch.from_numpy(sp["relu_id"].astype(np.int64)).cuda()
    neu = torch.from_numpy(sp["neuron"].astype(np.int64)).cuda()
    sgn = torch.from_numpy(sp["sign"].astype(np.float64)).cuda()
    lo, hi = box_of(wl.x0[0], wl.eps, wl.clip)
    lo_t = torch.from_numpy(lo.astype(np.float32)).cuda()
    hi_t = torch.from_numpy(hi.astype(np.float32)).cuda()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4321)
    Ct = torch.from_numpy(wl.C[0].astype(np.float64)).cuda()
    lbt, ubt = torch.from_numpy(lb).cuda(), torch.from_numpy(ub).cuda()
    hits = torch.zeros(D, dtype=torch.int64, device="cuda")
    x0_point = torch.from_numpy(wl.x0[0:1]).cuda()
    batches = [x0_point] + [lo_t + (hi_t - lo_t) * torch.rand((2048, lo.size), generator=gen, device="cuda")
                            for _ in range(N_SAMPLES // 2048 + 1)]
    for X in batches:
        with torch.no_grad():
            vals = torch_forward(wl.net, X)
            Y = vals[-1].double() @ Ct.T                                   # (P, m)
            Z = torch.stack([vals[i].double() for i in pre_ids], 1)        # (P, R, n)
        zs = Z[:, rid, neu]                                                # (P, D, S)
        clear = zs.abs() > 1e-5 * (1.0 + zs.abs())
        member = ((zs * sgn[None] > 0) & clear).all(2)                     # (P, D)
        hits += member.sum(0)
        slack = 1e-4 + 1e-4 * Y.abs()                                      # (P, m)
        below = (lbt[None] - slack[:, None] - Y[:, None]).amax(2)          # (P, D)
        above = (Y[:, None] - ubt[None] - slack[:, None]).amax(2)
        bad = member & ((below > 0) | (above > 0))
        assert not bad.any(), f"{int(bad.sum())} (point, subdomain) pairs outside the subdomain bounds"
        # a member point makes its subdomain feasible
        assert not (member.any(0).cpu().numpy() & ~feasible).any()
    hits = hits.cpu().numpy()
    log("subdomains with >= 1 member point:", int((hits > 0).sum()), "of", D, "; member pairs", int(hits.sum()))
    assert (hits > 0).sum() >= 16
