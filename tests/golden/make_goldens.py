"""Write the stored oracle results used by the GPU parity tests and the bench.

Calls only the fp64 oracle (oracle/) on the seeded workloads (workloads/).
  * <workload>.npz: the final bounds and every ReLU layer's pre-activation bounds of the
    listed inputs;
  * exp1_mlp4096x262144x1.npz: the paper's Exp. 1 network (one hidden layer of 262144):
    final bounds of the listed inputs and the hidden bounds of sampled neurons, from the
    oracle's row-block computation for one hidden layer;
  * bab_mlp784x1024x6_splits.npz: the branch-and-bound subdomains of that workload, drawn
    from the oracle root pass's unstable neurons (the draw continues the workload's seeded
    generator, so it equals what the tests draw at run time).

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
}

# full-size workloads whose bounds are stored for sampled neurons (with every neuron their
# receptive fields reach): {workload: (inputs, {ReLU position: number of target neurons})}
SAMPLED = {
    "resnet3x32x32": ([0], {0: 128, 1: 3, 2: 1}),
}


def make(name, inputs):
    wl = make_workload(name)
    out = {"inputs": np.array(inputs)}
    for b in inputs:
        t = time.time()
        r = oracle.crown(wl.net, wl.x0[b], wl.eps, wl.C[b])
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
    names = sys.argv[1:] or list(GOLDENS) + ["bab"] + [f"{k}_sampled" for k in SAMPLED] + list(ONE_HIDDEN)
    for n in names:
        if n in ONE_HIDDEN:
            make_one_hidden(n, *ONE_HIDDEN[n])
        elif n == "bab":
            make_bab_splits()
        elif n.endswith("_sampled"):
            make_sampled(n[:-len("_sampled")], *SAMPLED[n[:-len("_sampled")]])
        else:
            make(n, GOLDENS[n])
