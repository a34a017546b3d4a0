"""Seeded synthetic workloads for batched CROWN bound propagation.

The paper measures on MNIST/CIFAR ReLU classifiers and VNN-COMP models that are not
available here.  These generators stand in for them with arrays of the same shapes and
value distributions: inputs drawn uniformly from [0,1] at image sizes, He-normal weights
N(0, 2/fan_in), biases N(0, 0.01^2), and margin specifications e_c - e_j built from the
predicted class (local robustness, Sec. 1.1 of the paper).

Draw order (fixed, so every consumer regenerates identical arrays from a seed):
  for every parametrised layer in node order: W = standard_normal(shape) * sqrt(2/fan_in),
  then b = standard_normal(n_out) * 0.01, both cast to float32; afterwards the inputs
  X0 = random((B, n0)) cast to float32.  fan_in is d_in for dense layers and C_in*kh*kw
  for convolutions.

Nothing here propagates bounds.  ``forward64`` evaluates the network at points, which is
only needed to pick the predicted class for the margin specification.
"""
from __future__ import annotations

from dataclasses import dataclass, field
import math

import numpy as np

OPS = ("dense", "conv2d", "relu", "add", "flatten")


@dataclass
class Node:
    """One node of a feed-forward ReLU network in topological order.

    op      : 'dense' | 'conv2d' | 'relu' | 'add' | 'flatten'
    in0/in1 : producer node ids; -1 is the network input; in1 only for 'add'
    W, b    : float32; dense W is (d_out, d_in), conv W is (C_out, C_in, kh, kw)
    stride, pad : conv2d only (zero padding on all four sides)
    """
    op: str
    in0: int
    in1: int = -1
    W: np.ndarray | None = None
    b: np.ndarray | None = None
    stride: int = 1
    pad: int = 0


@dataclass
class Net:
    in_shape: tuple          # (n0,) for MLPs, (C, H, W) for convolutional nets
    nodes: list = field(default_factory=list)

    @property
    def n_in(self) -> int:
        return int(np.prod(self.in_shape))


@dataclass
class Splits:
    """Branch-and-bound subdomains: each fixes `per_domain` ReLUs to a state.

    relu_id[d, k] indexes the ReLU nodes in node order, neuron[d, k] is the flat index
    inside that ReLU's tensor, sign[d, k] is +1 (pre-activation >= 0) or -1 (<= 0).
    """
    relu_id: np.ndarray      # (D, S) int32
    neuron: np.ndarray       # (D, S) int32
    sign: np.ndarray         # (D, S) int8

    @property
    def n_domains(self) -> int:
        return int(self.relu_id.shape[0])

    @property
    def per_domain(self) -> int:
        return int(self.relu_id.shape[1])


@dataclass
class Workload:
    name: str
    net: Net
    x0: np.ndarray           # (B, n0) float32
    eps: np.float32
    C: np.ndarray            # (B, m, n_out) float32
    clip: tuple | None = (0.0, 1.0)
    rng: np.random.Generator | None = None   # generator state after the inputs were drawn
    splits: Splits | None = None


def _he_dense(rng, d_out, d_in):
    W = (rng.standard_normal((d_out, d_in)) * math.sqrt(2.0 / d_in)).astype(np.float32)
    b = (rng.standard_normal(d_out) * 0.01).astype(np.float32)
    return W, b


def _he_conv(rng, c_out, c_in, k):
    W = (rng.standard_normal((c_out, c_in, k, k)) * math.sqrt(2.0 / (c_in * k * k))).astype(np.float32)
    b = (rng.standard_normal(c_out) * 0.01).astype(np.float32)
    return W, b


def _he_dense_f32(rng, d_out, d_in, chunk=8192):
    """He-normal weights drawn as float32 normals, row block by row block (the 262144 x 4096
    layer would need 8.6 GB as float64), then the bias as for every other layer."""
    scale = np.float32(math.sqrt(2.0 / d_in))
    W = np.empty((d_out, d_in), np.float32)
    for r0 in range(0, d_out, chunk):
        r1 = min(d_out, r0 + chunk)
        W[r0:r1] = rng.standard_normal((r1 - r0, d_in), dtype=np.float32) * scale
    b = (rng.standard_normal(d_out) * 0.01).astype(np.float32)
    return W, b


def mlp_net(rng, dims) -> Net:
    """ReLU MLP dims[0] -> dims[1] -> ... -> dims[-1]; ReLU after every hidden layer."""
    nodes = []
    prev = -1
    for i in range(1, len(dims)):
        W, b = _he_dense(rng, dims[i], dims[i - 1])
        nodes.append(Node("dense", prev, W=W, b=b))
        prev = len(nodes) - 1
        if i < len(dims) - 1:
            nodes.append(Node("relu", prev))
            prev = len(nodes) - 1
    return Net((dims[0],), nodes)


def resnet_net(rng, in_chw=(3, 32, 32), c1=64, c2=128, fc=512, n_out=100) -> Net:
    """ResNet-style CNN: conv3x3 c1; two residual blocks x + conv(ReLU(conv(x))) at c1;
    stride-2 conv3x3 c2; one residual block at c2; flatten (C,H,W order); FC fc; ReLU;
    FC n_out.  ReLUs sit only inside the residual branches and after the FC layer."""
    C, H, Wd = in_chw
    nodes = []

    def conv(inp, ci, co, stride=1):
        W, b = _he_conv(rng, co, ci, 3)
        nodes.append(Node("conv2d", inp, W=W, b=b, stride=stride, pad=1))
        return len(nodes) - 1

    def block(inp, ch):
        a = conv(inp, ch, ch)
        nodes.append(Node("relu", a))
        r = len(nodes) - 1
        bb = conv(r, ch, ch)
        nodes.append(Node("add", inp, bb))
        return len(nodes) - 1

    z0 = conv(-1, C, c1)
    y = block(z0, c1)
    y = block(y, c1)
    z3 = conv(y, c1, c2, stride=2)
    y = block(z3, c2)
    nodes.append(Node("flatten", y))
    f = len(nodes) - 1
    n_flat = c2 * (H // 2) * (Wd // 2)
    W, b = _he_dense(rng, fc, n_flat)
    nodes.append(Node("dense", f, W=W, b=b))
    nodes.append(Node("relu", len(nodes) - 1))
    W, b = _he_dense(rng, n_out, fc)
    nodes.append(Node("dense", len(nodes) - 1, W=W, b=b))
    return Net(tuple(in_chw), nodes)


def node_shapes(net: Net) -> list:
    """Output shape of every node (validates the node list on the way)."""
    shapes = []

    def shape_of(i):
        return tuple(net.in_shape) if i == -1 else shapes[i]

    for idx, nd in enumerate(net.nodes):
        if nd.op not in OPS:
            raise ValueError(f"node {idx}: unknown op {nd.op!r}")
        if not (-1 <= nd.in0 < idx):
            raise ValueError(f"node {idx}: in0={nd.in0} is not an earlier node")
        s = shape_of(nd.in0)
        if nd.op == "dense":
            if int(np.prod(s)) != nd.W.shape[1] or len(s) != 1:
                raise ValueError(f"node {idx}: dense expects a flat input of {nd.W.shape[1]}, got {s}")
            shapes.append((nd.W.shape[0],))
        elif nd.op == "conv2d":
            if len(s) != 3 or s[0] != nd.W.shape[1]:
                raise ValueError(f"node {idx}: conv2d input {s} does not match W {nd.W.shape}")
            kh, kw = nd.W.shape[2:]
            ho = (s[1] + 2 * nd.pad - kh) // nd.stride + 1
            wo = (s[2] + 2 * nd.pad - kw) // nd.stride + 1
            shapes.append((nd.W.shape[0], ho, wo))
        elif nd.op == "relu":
            shapes.append(s)
        elif nd.op == "add":
            if not (-1 <= nd.in1 < idx) or shape_of(nd.in1) != s:
                raise ValueError(f"node {idx}: add inputs differ in shape")
            shapes.append(s)
        elif nd.op == "flatten":
            shapes.append((int(np.prod(s)),))
    return shapes


def relu_nodes(net: Net) -> list:
    return [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]


def _conv_fwd64(x, W, b, stride, pad):
    ci, h, w = x.shape
    co, _, kh, kw = W.shape
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (w + 2 * pad - kw) // stride + 1
    xp = np.zeros((ci, h + 2 * pad, w + 2 * pad))
    xp[:, pad:pad + h, pad:pad + w] = x
    out = np.zeros((co, ho, wo)) + b[:, None, None]
    for ky in range(kh):
        for kx in range(kw):
            patch = xp[:, ky:ky + stride * (ho - 1) + 1:stride, kx:kx + stride * (wo - 1) + 1:stride]
            out += np.tensordot(W[:, :, ky, kx], patch, axes=([1], [0]))
    return out


def forward64(net: Net, x: np.ndarray) -> np.ndarray:
    """Plain fp64 evaluation of the network at one point (flat input)."""
    vals = []
    inp = np.asarray(x, dtype=np.float64).reshape(net.in_shape)

    def get(i):
        return inp if i == -1 else vals[i]

    for nd in net.nodes:
        v = get(nd.in0)
        if nd.op == "dense":
            vals.append(nd.W.astype(np.float64) @ v.reshape(-1) + nd.b.astype(np.float64))
        elif nd.op == "conv2d":
            vals.append(_conv_fwd64(v, nd.W.astype(np.float64), nd.b.astype(np.float64), nd.stride, nd.pad))
        elif nd.op == "relu":
            vals.append(np.maximum(v, 0.0))
        elif nd.op == "add":
            vals.append(v + get(nd.in1))
        elif nd.op == "flatten":
            vals.append(v.reshape(-1))
    return vals[-1].reshape(-1)


def margin_spec(net: Net, x0: np.ndarray) -> np.ndarray:
    """Per-input margin specification rows e_c - e_j, j ascending, j != c, where c is the
    argmax of the fp64 forward pass (ties to the lowest index).  Returns (B, m, n_out)."""
    out = []
    for x in x0:
        y = forward64(net, x)
        n = y.shape[0]
        c = int(np.argmax(y))
        rows = []
        for j in range(n):
            if j == c:
                continue
            r = np.zeros(n, dtype=np.float32)
            r[c] = 1.0
            r[j] = -1.0
            rows.append(r)
        out.append(np.stack(rows))
    return np.stack(out).astype(np.float32)


def draw_splits(rng, pool, n_domains, per_domain) -> Splits:
    """Draw `per_domain` distinct (relu_id, neuron) pairs per domain uniformly without
    replacement from `pool` (an (P, 2) integer array), with signs +1/-1 at probability 1/2."""
    pool = np.asarray(pool, dtype=np.int64)
    if pool.shape[0] < per_domain:
        raise ValueError("split pool smaller than the number of splits per domain")
    rid = np.empty((n_domains, per_domain), np.int32)
    neu = np.empty((n_domains, per_domain), np.int32)
    sgn = np.empty((n_domains, per_domain), np.int8)
    for d in range(n_domains):
        pick = rng.choice(pool.shape[0], size=per_domain, replace=False)
        rid[d] = pool[pick, 0]
        neu[d] = pool[pick, 1]
        sgn[d] = np.where(rng.integers(0, 2, size=per_domain) == 1, 1, -1)
    return Splits(rid, neu, sgn)


# name -> (builder kind, seed, shape params, batch, eps)
WORKLOADS = {
    # MNIST-sized MLP, one input (runs in seconds on the CPU)
    "mlp784x256x2": dict(kind="mlp", seed=0, dims=[784, 256, 256, 10], batch=1, eps=0.01),
    # MNIST-sized deep MLP, six hidden layers of 1024, 64 inputs
    "mlp784x1024x6": dict(kind="mlp", seed=1, dims=[784] + [1024] * 6 + [10], batch=64, eps=0.015),
    # CIFAR-sized wide MLP, four hidden layers of 8192, 16 inputs, 100 classes
    "mlp3072x8192x4": dict(kind="mlp", seed=2, dims=[3072] + [8192] * 4 + [100], batch=16, eps=2.0 / 255.0),
    # branch-and-bound batch on the 784-1024x6-10 network: one root input, 4096 domains
    "bab_mlp784x1024x6": dict(kind="bab", seed=3, net_seed=1, dims=[784] + [1024] * 6 + [10],
                              batch=1, eps=0.02, n_domains=4096, per_domain=8),
    # the paper's Exp. 1 network (Sec. 4.1): one hidden layer of 262144 on a 4096-dim input,
    # one output, 2048 inputs, eps 0.01; the property is the output itself (C = [[1]]).
    # Weights drawn as float32 normals in row blocks (see _he_dense_f32)
    "exp1_mlp4096x262144x1": dict(kind="exp1", seed=5, dims=[4096, 262144, 1], batch=2048, eps=0.01),
    # the same shape family small enough for the oracle to bound every input
    "exp1_mlp1024x16384x1": dict(kind="exp1", seed=51, dims=[1024, 16384, 1], batch=64, eps=0.01),
    # ResNet-style CNN on 3x32x32, 8 inputs, 100 classes
    "resnet3x32x32": dict(kind="resnet", seed=4, batch=8, eps=1.0 / 255.0),
    # the same topology at 3x16x16 with 32/64 channels, FC 64, 10 classes (small enough for
    # the oracle to compute every bound)
    "resnet3x16x16": dict(kind="resnet", seed=41, batch=2, eps=2.0 / 255.0,
                          arch=dict(in_chw=(3, 16, 16), c1=32, c2=64, fc=64, n_out=10)),
    # the full ResNet's channel widths (64 / 128), FC 512 and 100 classes on a 3x8x8 image,
    # small enough for the oracle to compute every bound
    "resnet3x8x8": dict(kind="resnet", seed=42, batch=2, eps=2.0 / 255.0,
                        arch=dict(in_chw=(3, 8, 8), c1=64, c2=128, fc=512, n_out=100)),
}


def make_workload(name: str, batch: int | None = None, **overrides) -> Workload:
    """Build a named workload.  `batch` truncates the input batch (the first inputs of the
    full draw, so a truncated workload is a prefix of the full one)."""
    cfg = dict(WORKLOADS[name])
    cfg.update(overrides)
    kind = cfg["kind"]
    if kind == "mlp":
        rng = np.random.default_rng(cfg["seed"])
        net = mlp_net(rng, cfg["dims"])
        x0 = rng.random((cfg["batch"], cfg["dims"][0])).astype(np.float32)
    elif kind == "resnet":
        rng = np.random.default_rng(cfg["seed"])
        net = resnet_net(rng, **cfg.get("arch", {}))
        x0 = rng.random((cfg["batch"], net.n_in)).astype(np.float32)
    elif kind == "exp1":
        rng = np.random.default_rng(cfg["seed"])
        d_in, hid, d_out = cfg["dims"]
        W1, b1 = _he_dense_f32(rng, hid, d_in)
        W2, b2 = _he_dense_f32(rng, d_out, hid)
        net = Net((d_in,), [Node("dense", -1, W=W1, b=b1), Node("relu", 0), Node("dense", 1, W=W2, b=b2)])
        x0 = rng.random((cfg["batch"], d_in)).astype(np.float32)
        if batch is not None:
            x0 = x0[:batch]
        C = np.ones((x0.shape[0], 1, 1), np.float32)
        return Workload(name, net, x0, np.float32(cfg["eps"]), C, (0.0, 1.0), rng)
    elif kind == "bab":
        net = mlp_net(np.random.default_rng(cfg["net_seed"]), cfg["dims"])
        rng = np.random.default_rng(cfg["seed"])
        x0 = rng.random(cfg["dims"][0]).astype(np.float32)[None, :]
    else:
        raise ValueError(kind)
    if batch is not None:
        x0 = x0[:batch]
    C = margin_spec(net, x0)
    return Workload(name, net, x0, np.float32(cfg["eps"]), C, (0.0, 1.0), rng)


def random_mlp(seed, dims, batch, eps, clip=(0.0, 1.0), bias_scale=None) -> Workload:
    """Small random MLP workload for tests (same draw order as the named workloads)."""
    rng = np.random.default_rng(seed)
    net = mlp_net(rng, dims)
    if bias_scale is not None:
        for nd in net.nodes:
            if nd.op == "dense":
                nd.b = (nd.b / 0.01 * bias_scale).astype(np.float32)
    x0 = rng.random((batch, dims[0])).astype(np.float32)
    C = margin_spec(net, x0)
    return Workload(f"mlp{seed}", net, x0, np.float32(eps), C, clip, rng)
