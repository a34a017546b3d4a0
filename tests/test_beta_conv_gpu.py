"""GPU parity of branch-and-bound on convolutional networks (residual blocks, stride-2
convolutions, flatten into dense layers): subdomain CROWN bounds, beta-CROWN on subdomains
and the branch-and-bound loop, against the fp64 oracles (oracle/crown64.py for subdomain
CROWN, oracle/beta64.py for beta-CROWN and the loop).

Split neurons are given in each ReLU's (C, H, W) order; the spec pass relaxes them with
their clamped intervals in the transposed-convolution epilogue, adds the multipliers' terms
there, and the gradient pass writes the multipliers' gradients where the convolution forms
the split neuron's value."""
import numpy as np
import pytest

import oracle
from oracle import beta64
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from tests.test_beta_gpu import _split_tensors

pytestmark = pytest.mark.gpu


def _nets(eps=None):
    from tests.test_conv_gpu import conv_chain, small_resnet
    kw = {} if eps is None else {"eps": eps}
    return [small_resnet(316, batch=1, **kw), conv_chain(314, batch=1, **kw)]


def _domains(wl, root, seed):
    """Subdomains of depths 1 to 6 over the root's unstable neurons (every ReLU layer, the
    convolutional ones included), one infeasible (an inactive split of a stably active
    neuron) and one without splits."""
    order = beta64.default_order(wl.net, root)
    rng = np.random.default_rng(seed)
    doms = []
    for depth in (1, 2, 2, 3, 4, 6):
        pick = rng.choice(len(order), size=depth, replace=False)
        doms.append([(order[p][0], order[p][1], int(rng.choice([-1, 1]))) for p in pick])
    ids = beta64.relu_ids(wl.net)
    r_act, j_act = next((r, int(np.flatnonzero(root.layer_l[i] > 0)[0])) for r, i in enumerate(ids)
                        if np.any(root.layer_l[i] > 0))
    doms.append([order[0][:2] + (1,), (r_act, j_act, -1)])
    doms.append([])
    return doms


def _root(wl):
    return oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])


@pytest.mark.parametrize("which", [0, 1])
def test_conv_subdomain_crown_matches_oracle(which):
    """CROWN on subdomains: every domain's bounds against the oracle's subdomain CROWN; the
    infeasible domain reports lb = +inf, ub = -inf."""
    from workloads import Splits
    wl = _nets()[which]
    root = _root(wl)
    doms = [d for d in _domains(wl, root, 7) if d]
    ctx = gpu_ctx(wl.net)
    sp = _split_tensors(doms, 6)
    lb, ub, layers = gpu_crown(ctx, wl, splits=Splits(*(t.cpu().numpy() for t in sp)))
    for r, i in enumerate(beta64.relu_ids(wl.net)):
        assert_close(layers[r][0][0], root.layer_l[i], f"root relu {i} l")
        assert_close(layers[r][1][0], root.layer_u[i], f"root relu {i} u")
    used = [d + [d[0]] * (6 - len(d)) for d in doms]
    ref = Splits(np.array([[s[0] for s in d] for d in used], np.int32), np.array([[s[1] for s in d] for d in used], np.int32),
                 np.array([[s[2] for s in d] for d in used], np.int8))
    LB, UB = oracle.crown_domains(wl.net, root, wl.C[0], ref)
    for d in range(len(doms)):
        if not np.isfinite(LB[d]).all():
            assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d])), f"domain {d}"
            continue
        assert_close(lb[d], LB[d], f"{wl.name} domain {d} lb")
        assert_close(ub[d], UB[d], f"{wl.name} domain {d} ub")
    assert ctx.stats()["invalid_domains"] == 0


@pytest.mark.parametrize("which", [0, 1])
def test_conv_beta_subdomains_match_oracle(which):
    """Six joint Adam steps on eight subdomains of different depths (unused slots, one
    infeasible, one without splits): every evaluation's bounds and the best ones."""
    import torch
    wl = _nets()[which]
    root = _root(wl)
    doms = _domains(wl, root, 8)
    ctx = gpu_ctx(wl.net)
    T = 6
    lb, ub, ex = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), _split_tensors(doms, 6), iters=T,
                                       want_hist=True)
    torch.cuda.synchronize()
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    gained = 0
    for d, dom in enumerate(doms):
        r = beta64.beta_crown(wl.net, root, wl.C[0], dom, iters=T)
        if not r.feasible:
            assert np.all(np.isposinf(lb[d])) and np.all(np.isneginf(ub[d]))
            continue
        for t in range(T + 1):
            assert_close(lh[t, d], r.lb_hist[t], f"{wl.name} domain {d} evaluation {t} lb")
            assert_close(uh[t, d], r.ub_hist[t], f"{wl.name} domain {d} evaluation {t} ub")
        assert_close(lb[d], r.lb, f"{wl.name} domain {d} lb")
        assert_close(ub[d], r.ub, f"{wl.name} domain {d} ub")
        gained += int(np.any(r.lb > r.lb_hist[0] + 1e-4))
    log(wl.name, "domains improved by the steps", gained)
    assert gained > 0


def test_conv_beta_first_evaluation_is_subdomain_crown_bitwise():
    import torch
    for wl in _nets():
        root = _root(wl)
        ctx = gpu_ctx(wl.net)
        sp = _split_tensors([d for d in _domains(wl, root, 9) if d], 6)
        lb0, ub0 = ctx.crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), splits=sp)
        lb, ub, _ = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), sp, iters=0)
        torch.cuda.synchronize()
        assert np.array_equal(lb.cpu().numpy(), lb0.cpu().numpy()), wl.name
        assert np.array_equal(ub.cpu().numpy(), ub0.cpu().numpy()), wl.name


@pytest.mark.parametrize("which,eps,batch,rounds", [(0, 0.004, 4, 4), (1, 0.015, 4, 4)])
def test_conv_bab_loop_matches_oracle(which, eps, batch, rounds):
    """The loop on a residual conv net (verified after pruning four children) and on a conv
    chain (no child verified in four rounds): same order, same decisions round by round."""
    wl = _nets(eps)[which]
    root = _root(wl)
    order = beta64.default_order(wl.net, root)
    ref = beta64.bab(wl.net, wl.x0[0], wl.eps, wl.C[0], order=order, batch=batch, rounds=rounds, iters=10, root=root)
    lbs = [lb for kids in ref.children for _, lb in kids]
    if lbs:
        closest = min(float(np.min(np.abs(lb))) for lb in lbs)
        assert closest > 1e-3, "a decision within reach of fp32 rounding: pick another case"
    ctx = gpu_ctx(wl.net)
    got = ctx.bab_verify(to_dev(wl.x0), wl.eps, to_dev(wl.C), batch=batch, max_rounds=rounds, iters=10, order=order)
    log(wl.name, eps, "oracle", ref.verified, ref.log, "gpu", got["verified"], got["log"])
    assert got["verified"] == ref.verified
    assert got["rounds"] == ref.rounds and got["log"] == [tuple(x) for x in ref.log]
    assert got["evaluated"] == ref.evaluated and got["remaining"] == ref.remaining


def test_beta_resnet3x8x8_full_width():
    """The 3x8x8 ResNet at full width (64 and 128 channels, FC 512, 99 spec rows): six
    subdomains of input 0 with splits across the convolutional and dense ReLU layers, five
    joint Adam steps, against the stored oracle run evaluation by evaluation; the same six
    domains inside a batch of 64 (the others their sign variants) give the same bits."""
    import os
    import torch
    g = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "resnet3x8x8_beta.npz"))
    from workloads import make_workload
    wl = make_workload("resnet3x8x8", batch=1)
    T = int(g["iters"])
    rid, neu, sgn = g["relu_id"], g["neuron"], g["sign"]
    D0 = rid.shape[0]
    ctx = gpu_ctx(wl.net)
    sp = tuple(torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in (rid, neu, sgn))
    lb, ub, ex = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), sp, iters=T, want_hist=True)
    torch.cuda.synchronize()
    lh, uh = ex["lb_hist"].cpu().numpy(), ex["ub_hist"].cpu().numpy()
    for d in range(D0):
        if not bool(g[f"feasible_{d}"]):
            assert np.all(np.isposinf(lb[d].cpu().numpy()))
            continue
        for t in range(T + 1):
            assert_close(lh[t, d], g[f"lb_hist_{d}"][t], f"domain {d} evaluation {t} lb")
            assert_close(uh[t, d], g[f"ub_hist_{d}"][t], f"domain {d} evaluation {t} ub")
    rng = np.random.default_rng(3)
    reps = rng.integers(0, D0, 64 - D0)
    big = [np.concatenate([a, a[reps]]) for a in (rid, neu, sgn)]
    big[2][D0:] = np.where(rng.random(big[2][D0:].shape) < 0.5, -1, 1).astype(np.int8)
    spb = tuple(torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in big)
    lb2, ub2, _ = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), spb, iters=T)
    torch.cuda.synchronize()
    assert np.array_equal(lb2.cpu().numpy()[:D0], lb.cpu().numpy())
    assert np.array_equal(ub2.cpu().numpy()[:D0], ub.cpu().numpy())
    log("64-domain batch: lb range", float(lb2.min()), float(lb2[torch.isfinite(lb2)].max()))


def test_conv_subdomain_edge_cases():
    """Splits on convolutional ReLUs (neurons in (C, H, W) order): splits that restate a
    stable neuron's state are bitwise no-ops, a contradicting split is infeasible, a neuron
    out of range or repeated makes the domain invalid (NaN, counted), and a domain that agrees
    with x0's own activation pattern contains f(x0)."""
    from tests.pins import batch_forward, spec_values
    from workloads import Splits
    wl = _nets()[0]
    net = wl.net
    root = _root(wl)
    ids = beta64.relu_ids(net)
    l0, u0 = root.layer_l[ids[0]], root.layer_u[ids[0]]
    act = np.flatnonzero(l0 > 1e-3)
    ina = int(np.flatnonzero(u0 < -1e-3)[0])
    l1, u1 = root.layer_l[ids[1]], root.layer_u[ids[1]]
    unst = np.flatnonzero((l1 < -1e-3) & (u1 > 1e-3))
    z = batch_forward(net, wl.x0[:1].astype(np.float64))
    zin = z[net.nodes[ids[1]].in0].reshape(-1)
    zsign = [1 if zin[j] >= 0 else -1 for j in unst[:3]]
    n0 = l0.size
    rid = np.array([[0, 0, 0], [0, 1, 1], [0, 1, 1], [1, 1, 1], [1, 1, 0]], np.int32)
    neu = np.array([[act[0], ina, act[1]], [ina, unst[0], unst[1]], [act[0], n0 * 4, unst[0]],
                    list(unst[:3]), [unst[0], unst[0], act[0]]], np.int32)
    sgn = np.array([[1, -1, 1], [1, 1, -1], [1, 1, 1], zsign, [1, -1, 1]], np.int8)
    ctx = gpu_ctx(net)
    lb, ub, _ = gpu_crown(ctx, wl, splits=Splits(rid, neu, sgn))
    assert ctx.stats()["invalid_domains"] == 2
    lbr, ubr, _ = gpu_crown(ctx, wl)
    assert np.array_equal(lb[0], lbr[0]) and np.array_equal(ub[0], ubr[0]), "stable splits must be no-ops"
    assert np.all(lb[1] == np.inf) and np.all(ub[1] == -np.inf)
    for d in (2, 4):
        assert np.all(np.isnan(lb[d])) and np.all(np.isnan(ub[d])), d
    y0 = spec_values(net, wl.C[0], wl.x0[:1].astype(np.float64))[0]
    assert np.all(lb[3] <= y0 + 1e-4) and np.all(ub[3] >= y0 - 1e-4)
    LB, UB = oracle.crown_domains(net, root, wl.C[0], Splits(rid[[3]], neu[[3]], sgn[[3]]))
    assert_close(lb[3], LB[0], "domain 3 lb")
    assert_close(ub[3], UB[0], "domain 3 ub")


def test_conv_beta_chunked_equals_whole():
    """beta-CROWN on 24 subdomains of a residual conv net: a workspace cap that splits the
    domains into chunks gives the same bits."""
    import torch
    from paper_2606_09377_amd.vcrown import OPT_WORKSPACE_CAP_BYTES
    wl = _nets()[0]
    root = _root(wl)
    order = beta64.default_order(wl.net, root)
    rng = np.random.default_rng(12)
    doms = []
    for _ in range(24):
        pick = rng.choice(len(order), size=3, replace=False)
        doms.append([(order[p][0], order[p][1], int(rng.choice([-1, 1]))) for p in pick])
    sp = _split_tensors(doms, 3)
    ctx = gpu_ctx(wl.net)
    lb, ub, _ = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), sp, iters=3)
    torch.cuda.synchronize()
    st0 = ctx.stats()
    ctx.set_option(OPT_WORKSPACE_CAP_BYTES, st0["peak_workspace_bytes"] - 1)
    lb2, ub2, _ = ctx.beta_crown_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C), sp, iters=3)
    torch.cuda.synchronize()
    assert ctx.stats()["n_chunks_last_call"] > st0["n_chunks_last_call"]
    assert np.array_equal(lb.cpu().numpy(), lb2.cpu().numpy()) and np.array_equal(ub.cpu().numpy(), ub2.cpu().numpy())


def test_bab_loop_resnet3x8x8_full_width():
    """The loop on the full-width 3x8x8 ResNet's first input (99 spec rows) at a radius where
    the root is not verified, with the oracle's split order: the same rounds, the same
    children bounded and kept, as the stored oracle run (whose children's lower bounds all
    stay farther than the parity tolerance from 0)."""
    import os
    from workloads import make_workload
    g = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "resnet3x8x8_bab.npz"))
    assert float(np.min(np.abs(g["children_lb"]))) > 1e-3
    wl = make_workload("resnet3x8x8", batch=1, eps=g["eps"])
    order = [tuple(int(v) for v in o) for o in g["order"]]
    ctx = gpu_ctx(wl.net)
    got = ctx.bab_verify(to_dev(wl.x0), wl.eps, to_dev(wl.C), batch=int(g["batch"]), max_rounds=int(g["rounds"]),
                         iters=int(g["iters"]), order=order)
    log("oracle", g["log"].tolist(), "gpu", got["log"])
    assert got["verified"] == bool(g["verified"])
    assert got["log"] == [tuple(int(v) for v in x) for x in g["log"]]
    assert got["evaluated"] == int(g["evaluated"]) and got["remaining"] == int(g["remaining"])
