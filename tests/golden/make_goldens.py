"""Write the stored oracle results used by the GPU parity tests and the bench.

Calls only the fp64 oracle (oracle/) on the seeded workloads (workloads/).
  * <workload>.npz: the final bounds and every ReLU layer's pre-activation bounds of the
    listed inputs;
  * exp1_mlp4096x262144x1.npz: the paper's Exp. 1 network (one hidden layer of 262144):
    final bounds of the listed inputs and the hidden bounds of sampled neurons, from the
    oracle's row-block computation for one hidden layer;
  * bab_mlp784x1024x6_splits.npz: the branch-and-bound subdomains of that workload, drawn
    from the oracle root pass's unstable neurons (the draw continues the workload's seeded
    generator, so it equals what the tests draw at run time);
  * <workload>_alpha.npz: the alpha-CROWN oracle's run (every evaluation's bounds and the
    best ones) on the listed inputs, from CROWN's own slopes;
  * <workload>_corners.npz: for the listed inputs, the box vertices where each spec row's
    final linear bounds are attained (x_i = lo_i where the oracle's lower-bound coefficient
    on x_i is positive, else hi_i; the mirror image for the upper bound), as sign bits.

  python tests/golden/make_goldens.py [name ...]     (name "bab" for the split file)
"""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from workloads import make_workload  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))

# workload name -> inputs of the full batch to store
GOLDENS = {
    "mlp3072x8192x4": [0, 15],
    "resnet3x16x16": [0, 1],
    "resnet3x8x8": [0, 1],
}

# alpha-CROWN runs: {workload: (inputs, Adam steps)}
ALPHA = {
    "mlp3072x8192x4": ([0], 5),
    "resnet3x8x8": ([0], 5),
}

# beta-CROWN runs on subdomains of input 0: {workload: (domains, splits per domain, Adam steps)}
BETA = {
    "resnet3x8x8": (6, 3, 5),
}

# branch-and-bound loops on input 0: {workload: (eps, batch, rounds, Adam steps)}
BAB = {
    "resnet3x8x8": (1.6 / 255, 2, 3, 5),
}

# A-guided box vertices: {workload: inputs}
CORNERS = {
    "mlp3072x8192x4": [0, 15],
}

# full-size workloads whose bounds are stored for sampled neurons (with every neuron their
# receptive fields reach): {workload: (inputs, {ReLU position: number of target neurons})}
SAMPLED = {
    "resnet3x32x32": ([0], {0: 128, 1: 3, 2: 1}),
}


def tie_count(r, tie=1e-5):
    """Neurons whose adaptive lower slope sits on its tie u = -l (either slope would be a
    correct result there; a stored result must have none)."""
    n = 0
    for i in r.layer_l:
        l, u = r.layer_l[i], r.layer_u[i]
        n += int(np.sum((l < 0) & (u > 0) & (np.abs(u + l) <= tie * (u - l))))
    return n


def make(name, inputs):
    wl = make_workload(name)
    out = {"inputs": np.array(inputs)}
    for b in inputs:
        t = time.time()
        r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b])
        if tie_count(r):
            raise SystemExit(f"{name} input {b}: {tie_count(r)} neurons on the slope tie; pick another seed")
        out[f"lb_{b}"] = r.lb
        out[f"ub_{b}"] = r.ub
        for i in r.layer_l:
            out[f"l_{b}_{i}"] = r.layer_l[i]
            out[f"u_{b}_{i}"] = r.layer_u[i]
        print(f"{name} input {b}: {time.time() - t:.1f} s", flush=True)
    path = os.path.join(HERE, f"{name}.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_sampled(name, inputs, counts):
    wl = make_workload(name)
    relus = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    shapes = oracle.node_shapes(wl.net)
    out = {"inputs": np.array(inputs), "relus": np.array(relus)}
    rng = np.random.default_rng(2024)
    for b in inputs:
        targets = {relus[k]: np.sort(rng.choice(int(np.prod(shapes[relus[k]])), c, replace=False))
                   for k, c in counts.items()}
        t = time.time()
        res = oracle.crown_sampled(wl.net, wl.x0[b], wl.eps, targets)
        for i, (idx, l, u) in res.items():
            out[f"idx_{b}_{i}"] = idx
            out[f"l_{b}_{i}"] = l
            out[f"u_{b}_{i}"] = u
            print(f"{name} input {b} relu {i}: {len(idx)} neurons", flush=True)
        print(f"{name} input {b}: {time.time() - t:.1f} s", flush=True)
    path = os.path.join(HERE, f"{name}_sampled.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


# one-hidden-layer workloads: {workload: (inputs, sampled hidden neurons per input)}
ONE_HIDDEN = {
    "exp1_mlp4096x262144x1": ([0, 1], 4096),
}


def make_one_hidden(name, inputs, n_sample):
    wl = make_workload(name)
    n1 = wl.net.nodes[0].W.shape[0]
    rng = np.random.default_rng(2025)
    idx = np.sort(rng.choice(n1, n_sample, replace=False))
    out = {"inputs": np.array(inputs), "idx": idx}
    for b in inputs:
        t = time.time()
        lb, ub, l, u = oracle.crown_one_hidden(wl.net, wl.x0[b], wl.eps, wl.C[b])
        out[f"lb_{b}"], out[f"ub_{b}"] = lb, ub
        out[f"l_{b}"], out[f"u_{b}"] = l[idx], u[idx]
        print(f"{name} input {b}: {time.time() - t:.1f} s", flush=True)
    path = os.path.join(HERE, f"{name}.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_alpha(name, inputs, iters):
    from oracle import alpha64
    wl = make_workload(name)
    out = {"inputs": np.array(inputs), "iters": np.array(iters)}
    for b in inputs:
        t = time.time()
        r = alpha64.alpha_crown(wl.net, wl.x0[b], wl.eps, wl.C[b], iters=iters)
        out[f"lb_{b}"], out[f"ub_{b}"] = r.lb, r.ub
        out[f"lb_hist_{b}"], out[f"ub_hist_{b}"] = r.lb_hist, r.ub_hist
        print(f"{name} alpha input {b}: {time.time() - t:.1f} s", flush=True)
    path = os.path.join(HERE, f"{name}_alpha.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_beta(name, n_dom, depth, iters):
    """Subdomains of input 0 whose splits mix the ReLU layers (every split on a neuron the
    root finds unstable, one per chosen layer, random signs), each run through the beta-CROWN
    oracle: every evaluation's bounds."""
    from oracle import beta64
    wl = make_workload(name)
    t = time.time()
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    print(f"{name} root: {time.time() - t:.1f} s", flush=True)
    rng = np.random.default_rng(2026)
    ids = beta64.relu_ids(wl.net)
    unst = [np.flatnonzero((root.layer_l[i] < 0) & (root.layer_u[i] > 0)) for i in ids]
    layers = [r for r in range(len(ids)) if unst[r].size]
    rid = np.zeros((n_dom, depth), np.int32)
    neu = np.zeros((n_dom, depth), np.int32)
    sgn = np.zeros((n_dom, depth), np.int8)
    out = {"iters": np.array(iters)}
    for d in range(n_dom):
        chosen = rng.choice(layers, size=depth, replace=False)
        dom = [(int(r), int(rng.choice(unst[r])), int(rng.choice([-1, 1]))) for r in chosen]
        rid[d], neu[d], sgn[d] = [x[0] for x in dom], [x[1] for x in dom], [x[2] for x in dom]
        t = time.time()
        r = beta64.beta_crown(wl.net, root, wl.C[0], dom, iters=iters)
        out[f"feasible_{d}"] = np.array(r.feasible)
        out[f"lb_hist_{d}"], out[f"ub_hist_{d}"] = r.lb_hist, r.ub_hist
        print(f"{name} domain {d} {dom}: {time.time() - t:.1f} s", flush=True)
    out["relu_id"], out["neuron"], out["sign"] = rid, neu, sgn
    path = os.path.join(HERE, f"{name}_beta.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_bab(name, eps, batch, rounds, iters):
    """The oracle's loop on input 0 at the given radius, with its default split order: the
    order, the per-round log and the children's lower bounds."""
    from oracle import beta64
    wl = make_workload(name, batch=1, eps=np.float32(eps))
    t = time.time()
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    order = beta64.default_order(wl.net, root)
    r = beta64.bab(wl.net, wl.x0[0], wl.eps, wl.C[0], order=order, batch=batch, rounds=rounds, iters=iters, root=root)
    lbs = np.array([lb for kids in r.children for _, lb in kids])
    print(f"{name} loop: {time.time() - t:.1f} s, log {r.log}, closest bound to 0 "
          f"{np.min(np.abs(lbs)) if lbs.size else None}", flush=True)
    out = {"eps": np.array(eps, np.float32), "batch": np.array(batch), "rounds": np.array(rounds),
           "iters": np.array(iters), "order": np.array(order, np.int32), "log": np.array(r.log, np.int64),
           "verified": np.array(r.verified), "evaluated": np.array(r.evaluated), "remaining": np.array(r.remaining),
           "children_lb": lbs}
    path = os.path.join(HERE, f"{name}_bab.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_corners(name, inputs):
    wl = make_workload(name)
    out = {"inputs": np.array(inputs)}
    for b in inputs:
        t = time.time()
        r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b], keep_A=True)
        # lower bound: attained at lo where the coefficient is positive; upper: at hi there
        out[f"lower_at_lo_{b}"] = np.packbits(r.A_lower > 0, axis=1)
        out[f"upper_at_hi_{b}"] = np.packbits(r.A_upper > 0, axis=1)
        print(f"{name} corners input {b}: {time.time() - t:.1f} s", flush=True)
    path = os.path.join(HERE, f"{name}_corners.npz")
    np.savez_compressed(path, **out)
    print("wrote", path)


def make_bab_splits():
    from workloads import draw_splits
    wl = make_workload("bab_mlp784x1024x6")
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    pool = oracle.unstable_pool(wl.net, root)
    sp = draw_splits(wl.rng, pool, 4096, 8)
    path = os.path.join(HERE, "bab_mlp784x1024x6_splits.npz")
    np.savez_compressed(path, relu_id=sp.relu_id, neuron=sp.neuron, sign=sp.sign)
    print("wrote", path, "pool", len(pool))


if __name__ == "__main__":
    names = sys.argv[1:] or (list(GOLDENS) + ["bab"] + [f"{k}_sampled" for k in SAMPLED] + list(ONE_HIDDEN)
                             + [f"{k}_alpha" for k in ALPHA] + [f"{k}_corners" for k in CORNERS]
                             + [f"{k}_beta" for k in BETA] + [f"{k}_bab" for k in BAB])
    for n in names:
        if n.endswith("_bab"):
            make_bab(n[:-len("_bab")], *BAB[n[:-len("_bab")]])
        elif n.endswith("_beta"):
            make_beta(n[:-len("_beta")], *BETA[n[:-len("_beta")]])
        elif n.endswith("_alpha"):
            make_alpha(n[:-len("_alpha")], *ALPHA[n[:-len("_alpha")]])
        elif n.endswith("_corners"):
            make_corners(n[:-len("_corners")], CORNERS[n[:-len("_corners")]])
        elif n in ONE_HIDDEN:
            make_one_hidden(n, *ONE_HIDDEN[n])
        elif n == "bab":
            make_bab_splits()
        elif n.endswith("_sampled"):
            make_sampled(n[:-len("_sampled")], *SAMPLED[n[:-len("_sampled")]])
        else:
            make(n, GOLDENS[n])
