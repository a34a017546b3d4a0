"""GPU parity of branch-and-bound subdomain bounds (one root input, fixed ReLU splits)."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_close, gpu_crown, gpu_ctx, log, to_dev
from workloads import Splits, draw_splits, make_workload, random_mlp

pytestmark = pytest.mark.gpu


def bab_workload(n_domains=4096):
    wl = make_workload("bab_mlp784x1024x6")
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    pool = oracle.unstable_pool(wl.net, root)
    splits = draw_splits(wl.rng, pool, n_domains, 8)
    return wl, root, splits


def test_bab_4096_domains_sampled():
    log("oracle root pass")
    wl, root, splits = bab_workload()
    ctx = gpu_ctx(wl.net)
    log("gpu run 4096 domains")
    lb, ub, layers = gpu_crown(ctx, wl, splits=splits)
    assert lb.shape == (4096, 9)
    relu_ids = sorted(root.layer_l)
    for r, i in enumerate(relu_ids):
        assert_close(layers[r][0][0], root.layer_l[i], f"root relu {r} l")
        assert_close(layers[r][1][0], root.layer_u[i], f"root relu {r} u")
    rng = np.random.default_rng(17)
    sample = sorted(set(range(8)) | set(rng.choice(4096, 56, replace=False).tolist()) | {4095})
    log("oracle on", len(sample), "domains")
    LB, UB = oracle.crown_domains(wl.net, root, wl.C[0], splits, domains=sample)
    for k, d in enumerate(sample):
        assert_close(lb[d], LB[k], f"domain {d} lb")
        assert_close(ub[d], UB[k], f"domain {d} ub")
    assert ctx.stats()["invalid_domains"] == 0


def test_bab_edge_cases():
    """Stable-state splits are bitwise no-ops, contradicting splits are infeasible, bad
    entries give NaN and are counted, and a domain that agrees with x0 contains f(x0)."""
    wl = random_mlp(201, [60, 140, 150, 5], 1, 0.05)
    net = wl.net
    root = oracle.crown(net, wl.x0[0], wl.eps, wl.C[0])
    relus = sorted(root.layer_l)
    l0, u0 = root.layer_l[relus[0]], root.layer_u[relus[0]]
    acts = np.nonzero(l0 > 1e-3)[0]
    act, act2 = int(acts[0]), int(acts[1])
    ina = int(np.nonzero(u0 < -1e-3)[0][0])
    l1, u1 = root.layer_l[relus[1]], root.layer_u[relus[1]]
    unst = np.nonzero((l1 < -1e-3) & (u1 > 1e-3))[0]
    assert len(unst) >= 3
    from tests.pins import batch_forward
    z = batch_forward(net, wl.x0[:1].astype(np.float64))
    zsign = [1 if z[net.nodes[relus[1]].in0][0, j] >= 0 else -1 for j in unst[:3]]
    S = 3
    rid = np.zeros((7, S), np.int32)
    neu = np.zeros((7, S), np.int32)
    sgn = np.ones((7, S), np.int8)
    # 0: stable-state no-ops
    rid[0], neu[0], sgn[0] = [0, 0, 0], [act, ina, act2], [1, -1, 1]
    # 1: infeasible (active split on a stably inactive neuron)
    rid[1], neu[1], sgn[1] = [0, 1, 1], [ina, unst[0], unst[1]], [1, 1, -1]
    # 2: relu id out of range
    rid[2], neu[2], sgn[2] = [0, 5, 1], [act, 0, unst[0]], [1, 1, 1]
    # 3: agrees with x0's own pattern
    rid[3], neu[3], sgn[3] = [1, 1, 1], unst[:3], zsign
    # 4: duplicate neuron
    rid[4], neu[4], sgn[4] = [1, 1, 0], [unst[0], unst[0], act], [1, -1, 1]
    # 5: sign 0
    rid[5], neu[5], sgn[5] = [1, 1, 1], unst[:3], [1, 0, 1]
    # 6: neuron out of range
    rid[6], neu[6], sgn[6] = [1, 1, 1], [unst[0], 10 ** 6, unst[1]], [1, 1, 1]
    splits = Splits(rid, neu, sgn)
    ctx = gpu_ctx(net)
    lb, ub, _ = gpu_crown(ctx, wl, splits=splits)
    assert ctx.stats()["invalid_domains"] == 4
    lbr, ubr, _ = gpu_crown(ctx, wl)           # the root's own final pass, no splits
    assert np.array_equal(lb[0], lbr[0]) and np.array_equal(ub[0], ubr[0]), "stable splits must be no-ops"
    assert np.all(lb[1] == np.inf) and np.all(ub[1] == -np.inf)
    for d in (2, 4, 5, 6):
        assert np.all(np.isnan(lb[d])) and np.all(np.isnan(ub[d])), d
    from tests.pins import spec_values
    y0 = spec_values(net, wl.C[0], wl.x0[:1].astype(np.float64))[0]
    assert np.all(lb[3] <= y0 + 1e-4) and np.all(ub[3] >= y0 - 1e-4)
    LB, UB = oracle.crown_domains(net, root, wl.C[0], Splits(rid[[1, 3]], neu[[1, 3]], sgn[[1, 3]]))
    assert np.all(LB[0] == np.inf)
    assert_close(lb[3], LB[1], "domain 3 lb")
    assert_close(ub[3], UB[1], "domain 3 ub")
    # with the synchronous check the same call reports the invalid domains as an error
    from paper_2606_09377_amd.vcrown import OPT_SYNC_CHECK, VcrError
    ctx.set_option(OPT_SYNC_CHECK, 1)
    with pytest.raises(VcrError):
        gpu_crown(ctx, wl, splits=splits)


def test_bab_many_splits_per_layer():
    """Forty splits per domain, most of them at one ReLU layer (many per column block and per
    lane), against the oracle on every domain."""
    wl = random_mlp(202, [60, 140, 300, 5], 1, 0.05)
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    pool = oracle.unstable_pool(wl.net, root)
    first, last = pool[pool[:, 0] == 0], pool[pool[:, 0] == 1]
    assert len(first) >= 12 and len(last) >= 40
    rng = np.random.default_rng(23)
    a = draw_splits(rng, last, 256, 40)
    b1, b2 = draw_splits(rng, last, 256, 28), draw_splits(rng, first, 256, 12)
    splits = Splits(np.concatenate([a.relu_id, np.concatenate([b1.relu_id, b2.relu_id], 1)]),
                    np.concatenate([a.neuron, np.concatenate([b1.neuron, b2.neuron], 1)]),
                    np.concatenate([a.sign, np.concatenate([b1.sign, b2.sign], 1)]))
    ctx = gpu_ctx(wl.net)
    log("gpu run 512 domains, 40 splits each")
    lb, ub, _ = gpu_crown(ctx, wl, splits=splits)
    assert ctx.stats()["invalid_domains"] == 0
    LB, UB = oracle.crown_domains(wl.net, root, wl.C[0], splits, domains=list(range(512)))
    for d in range(512):
        assert_close(lb[d], LB[d], f"domain {d} lb")
        assert_close(ub[d], UB[d], f"domain {d} ub")
