"""Write the stored oracle results used by the GPU parity tests and the bench.

Calls only the fp64 oracle (oracle/) on the seeded workloads (workloads/).
  * <workload>.npz: the final bounds and every ReLU layer's pre-activation bounds of the
    listed inputs;
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
    names = sys.argv[1:] or list(GOLDENS) + ["bab"]
    for n in names:
        if n == "bab":
            make_bab_splits()
        else:
            make(n, GOLDENS[n])
