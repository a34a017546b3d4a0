"""GPU parity of beta-CROWN on subdomains and of the branch-and-bound loop against the fp64
oracle (oracle/beta64.py).

Subdomain bounds are compared evaluation by evaluation over an optimisation run; the loop
is run on both sides with the same split order (computed from the oracle's root bounds) and
must take the same decisions round by round.  The chosen networks keep every bound the loop
decides on farther than the parity tolerance from 0, so both sides decide alike."""
import numpy as np
import pytest

import oracle
from oracle import beta64
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from workloads import random_mlp

pytestmark = pytest.mark.gpu


def _split_tensors(doms, S):
    import torch
    D = len(doms)
    r = np.full((D, S), -1, np.int32)
    n = np.zeros((D, S), np.int32)
    g = np.ones((D, S), np.int8)
    for d, dom in enumerate(doms):
        for e, (ri, j, sg) in enumerate(dom):
            r[d, e], n[d, e], g[d, e] = ri, j, sg
    return tuple(torch.from_numpy(a).cuda() for a in (r, n, g))


def _case():
    wl = random_mlp(81, [30, 96, 80, 70, 6], 1, 0.06)
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    return wl, root


def _domains(wl, root):
    order = beta64.default_order(wl.net, root)
    rng = np.random.default_rng(5)
    doms = []
    for depth in (1, 1, 2, 3, 4, 4, 6):
        pick = rng.choice(len(order), size=depth, replace=False)
        doms.append([(order[p][0], order[p][1], int(rng.choice([-1, 1]))) for p in pick])
    ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    r_act, j_act = next((r, int(np.flatnonzero(root.layer_l[i] > 0)[0])) for r, i in enumerate(ids)
                        if np.any(root.layer_l[i] > 0))
    doms.append([order[0][:2] + (1,), (r_act, j_act, -1)])          # infeasible
    doms.append([])                                                  # no split at all
    return doms


def test_beta_subdomains_match_oracle():
    """Ten joint Adam steps on nine subdomains of different depths (unused slots, one
    infeasible, one without splits): every evaluation's bounds and the best ones."""
    import torch
    wl, root = _case()
    ctx = gpu_ctx(wl.net)
    _, _, layers = gpu_crown(ctx, wl)
    for r, i in enumerate(beta64.relu_ids(wl.net)):
        assert_close(layers[r][0][0], root.layer_l[i], f"root relu {i} l")
        assert_close(layers[r][1][0], root.layer_u[i], f"root relu {i} u")
    doms = _domains(wl, root)
    T = 10
    lb, ub, ex = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), _split_tensors(doms, 6), iters=T,
                                       want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    for d, dom in enumerate(doms):
        r = beta64.beta_crown(wl.net, root, wl.C[0], dom, iters=T)
        if not r.feasible:
            assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d]))
            continue
        for t in range(T + 1):
            assert_close(lh[t, d], r.lb_hist[t], f"domain {d} evaluation {t} lb")
            assert_close(uh[t, d], r.ub_hist[t], f"domain {d} evaluation {t} ub")
        assert_close(lb[d], r.lb, f"domain {d} lb")
        assert_close(ub[d], r.ub, f"domain {d} ub")
        if dom:
            log("domain", d, "beta-CROWN gain over CROWN", float(np.min(r.lb - r.lb_hist[0])))


def test_beta_first_evaluation_is_subdomain_crown_bitwise():
    import torch
    wl, root = _case()
    ctx = gpu_ctx(wl.net)
    doms = [d for d in _domains(wl, root) if d]
    sp = _split_tensors(doms, 6)
    lb0, ub0 = ctx.crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), splits=sp)
    lb, ub, _ = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), sp, iters=0)
    torch.cuda.synchronize()
    assert np.array_equal(lb.cpu().numpy(), lb0.cpu().numpy()) and np.array_equal(ub.cpu().numpy(), ub0.cpu().numpy())


@pytest.mark.parametrize("seed,dims,eps,batch,rounds", [
    (117, [2, 16, 16, 3], 0.15, 8, 10),
    (201, [10, 40, 40, 4], 0.04, 4, 5),
    (208, [10, 40, 40, 4], 0.04, 4, 5),
    (208, [10, 40, 40, 4], 0.02, 4, 5),
])
def test_bab_loop_matches_oracle(seed, dims, eps, batch, rounds):
    """Same order, same decisions: verified or not, and per round the subdomains taken,
    bounded, verified and left."""
    wl = random_mlp(seed, dims, 1, eps)
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    order = beta64.default_order(wl.net, root)
    ref = beta64.bab(wl.net, wl.x0[0], wl.eps, wl.C[0], order=order, batch=batch, rounds=rounds, iters=10, root=root)
    lbs = [lb for kids in ref.children for _, lb in kids]
    if lbs:
        closest = min(float(np.min(np.abs(lb))) for lb in lbs)
        assert closest > 1e-3, "a decision within reach of fp32 rounding: pick another case"
    ctx = gpu_ctx(wl.net)
    got = ctx.bab_verify(to_dev(wl.x0), wl.eps, to_dev(wl.C), batch=batch, max_rounds=rounds, iters=10, order=order)
    log(seed, eps, "oracle", ref.verified, ref.log, "gpu", got["verified"], got["log"])
    assert got["verified"] == ref.verified
    assert got["rounds"] == ref.rounds and got["log"] == [tuple(x) for x in ref.log]
    assert got["evaluated"] == ref.evaluated and got["remaining"] == ref.remaining


def test_bab_default_order_is_intercept_order():
    """Without an order the library splits the root's unstable neurons by decreasing chord
    intercept of its own root bounds: the same run as with that order given explicitly."""
    wl = random_mlp(201, [10, 40, 40, 4], 1, 0.04)
    ctx = gpu_ctx(wl.net)
    a = ctx.bab_verify(to_dev(wl.x0), wl.eps, to_dev(wl.C), batch=4, max_rounds=5, iters=10)
    _, _, layers = gpu_crown(ctx, wl)
    cand = []
    for r, (l, u) in enumerate(layers):
        l, u = l[0].astype(np.float64), u[0].astype(np.float64)
        for j in np.flatnonzero((l < 0) & (u > 0)):
            cand.append((-(-u[j] * l[j] / (u[j] - l[j])), r, int(j)))
    order = [(r, j) for _, r, j in sorted(cand, key=lambda t: t[0])]
    b = ctx.bab_verify(to_dev(wl.x0), wl.eps, to_dev(wl.C), batch=4, max_rounds=5, iters=10, order=order)
    assert a == b


def test_beta_deep_domains_one_layer():
    """Subdomains with 12 to 24 splits, most at one ReLU layer (many split columns per lane):
    every evaluation of five Adam steps against the oracle."""
    import torch
    wl, root = _case()
    ctx = gpu_ctx(wl.net)
    order = beta64.default_order(wl.net, root)
    layer1 = [o for o in order if o[0] == 1]
    assert len(layer1) >= 24
    rng = np.random.default_rng(29)
    doms = []
    for depth in (12, 16, 20, 24):
        pick = rng.choice(len(layer1), size=depth, replace=False)
        doms.append([(layer1[p][0], layer1[p][1], int(rng.choice([-1, 1]))) for p in pick])
    doms.append(doms[0] + [(order[0][0], order[0][1], 1)] if order[0][0] != 1 else doms[0][:6])
    T = 5
    lb, ub, ex = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), _split_tensors(doms, 25), iters=T,
                                       want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    for d, dom in enumerate(doms):
        r = beta64.beta_crown(wl.net, root, wl.C[0], dom, iters=T)
        if not r.feasible:
            assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d]))
            continue
        for t in range(T + 1):
            assert_close(lh[t, d], r.lb_hist[t], f"domain {d} evaluation {t} lb")
            assert_close(uh[t, d], r.ub_hist[t], f"domain {d} evaluation {t} ub")
        assert_close(lb[d], r.lb, f"domain {d} lb")
        assert_close(ub[d], r.ub, f"domain {d} ub")


def test_beta_bench_size_batches():
    """beta-CROWN on the 784-1024x6 MLP's stored subdomains (8 splits each) at the sizes the
    branch-and-bound bench runs: 512 subdomains (9216 rows, the 64 x 64 tile kernel with
    split multipliers in its epilogues) and 4096 (73728 rows, the 128 x 128 tile kernel).
    Every evaluation of 5 joint Adam steps on 16 sampled subdomains of each call against the
    oracle; the 512 subdomains are the first of the 4096, and their bounds agree bit for bit
    between the two calls."""
    import os
    import torch
    from paper_2606_09377_amd.vcrown import OPT_TIME_GEMM
    from workloads import make_workload
    wl = make_workload("bab_mlp784x1024x6")
    sp = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "bab_mlp784x1024x6_splits.npz"))
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    ctx = gpu_ctx(wl.net)
    T = 5
    rng = np.random.default_rng(17)
    res = {}
    for D in (512, 4096):
        tens = tuple(to_dev(np.ascontiguousarray(sp[k][:D])) for k in ("relu_id", "neuron", "sign"))
        ctx.set_option(OPT_TIME_GEMM, 1)
        log("beta D", D)
        lb, ub, ex = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), tens, iters=T, want_hist=True)
        torch.cuda.synchronize()
        # the root pass (2048 rows) never reaches the 128 x 128 tile kernel; the spec pass of
        # 4096 subdomains does, that of 512 does not
        n_big = ctx.stats()["timed_gemm_launches"]
        assert (n_big > 0) if D == 4096 else (n_big == 0), (D, n_big)
        lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
        lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
        res[D] = (lb, ub)
        for d in sorted(rng.choice(D, 16, replace=False)):
            dom = [(int(sp["relu_id"][d, e]), int(sp["neuron"][d, e]), int(sp["sign"][d, e])) for e in range(8)]
            r = beta64.beta_crown(wl.net, root, wl.C[0], dom, iters=T)
            if not r.feasible:
                assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d]))
                continue
            for t in range(T + 1):
                assert_close(lh[t, d], r.lb_hist[t], f"D={D} domain {d} evaluation {t} lb")
                assert_close(uh[t, d], r.ub_hist[t], f"D={D} domain {d} evaluation {t} ub")
            assert_close(lb[d], r.lb, f"D={D} domain {d} lb")
            assert_close(ub[d], r.ub, f"D={D} domain {d} ub")
    assert np.array_equal(res[512][0], res[4096][0][:512]) and np.array_equal(res[512][1], res[4096][1][:512])
