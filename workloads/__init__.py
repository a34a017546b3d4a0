"""Seeded synthetic workloads shared by the GPU path's tests, the oracle's tests and the bench.

This package only draws random numbers and builds arrays (network weights, input points,
margin specifications, branch-and-bound split lists).  It contains none of the bound
propagation arithmetic: neither interval propagation nor any linear relaxation.
"""
from .gen import (  # noqa: F401
    Node, Net, Workload, Splits,
    mlp_net, resnet_net, node_shapes, relu_nodes, forward64, margin_spec,
    make_workload, draw_splits, random_mlp, WORKLOADS,
)
