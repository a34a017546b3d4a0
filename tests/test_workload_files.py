"""Stored inputs equal what the seeded generators and the oracle produce at run time."""
import os

import numpy as np

import oracle
from workloads import draw_splits, make_workload

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_stored_bab_splits_match_the_draw():
    wl = make_workload("bab_mlp784x1024x6")
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    pool = oracle.unstable_pool(wl.net, root)
    sp = draw_splits(wl.rng, pool, 4096, 8)
    g = np.load(os.path.join(GOLDEN, "bab_mlp784x1024x6_splits.npz"))
    assert np.array_equal(g["relu_id"], sp.relu_id)
    assert np.array_equal(g["neuron"], sp.neuron)
    assert np.array_equal(g["sign"], sp.sign)
    # every split is on a neuron the root pass finds unstable (outside the tolerance band)
    relus = sorted(root.layer_l)
    for r, j in zip(sp.relu_id.ravel()[:2000], sp.neuron.ravel()[:2000]):
        assert root.layer_l[relus[r]][j] < 0 < root.layer_u[relus[r]][j]
    # distinct within each domain
    keys = sp.relu_id.astype(np.int64) * 100000 + sp.neuron
    assert all(len(set(k)) == sp.per_domain for k in keys)


def test_workload_shapes():
    wl = make_workload("mlp784x1024x6", batch=2)
    assert wl.C.shape == (2, 9, 10) and wl.x0.shape == (2, 784)
    c = np.argmax(wl.C[0] == 1, axis=1)
    assert np.all(c == c[0])
    assert np.all((wl.C[0] == -1).sum(1) == 1)
