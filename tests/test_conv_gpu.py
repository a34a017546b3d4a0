"""GPU parity of CROWN through convolutions, residual blocks and flatten.

Small networks with the ResNet workload's topology (and a plain conv chain with a stride-2
convolution under a ReLU) are compared with the fp64 oracle on every bound; the full-size
ResNet is checked on neurons the oracle can compute one by one, and by properties that
hold at any size."""
import os

import numpy as np
import pytest

import oracle
from tests.gpu_util import assert_classes, assert_close, check_input, gpu_crown, gpu_ctx, log, to_dev
from workloads import Net, Node, Workload, make_workload
from workloads.gen import margin_spec, resnet_net

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def small_resnet(seed, hw=8, c1=32, c2=64, fc=32, n_out=10, batch=2, eps=2 / 255):
    rng = np.random.default_rng(seed)
    net = resnet_net(rng, in_chw=(3, hw, hw), c1=c1, c2=c2, fc=fc, n_out=n_out)
    x0 = rng.random((batch, net.n_in)).astype(np.float32)
    return Workload(f"resnet{hw}", net, x0, np.float32(eps), margin_spec(net, x0))


def conv_chain(seed, batch=2, eps=0.02):
    """conv -> ReLU -> stride-2 conv -> ReLU -> conv -> ReLU -> flatten -> dense -> ReLU ->
    dense, on 3x8x8 (no residual; ReLUs directly after convolutions, one under a stride-2)."""
    rng = np.random.default_rng(seed)

    def cw(co, ci):
        return ((rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2 / (ci * 9))).astype(np.float32),
                (rng.standard_normal(co) * 0.05).astype(np.float32))

    W0, b0 = cw(32, 3)
    W1, b1 = cw(32, 32)
    W2, b2 = cw(64, 32)
    Wd = (rng.standard_normal((40, 64 * 16)) * np.sqrt(2 / 1024)).astype(np.float32)
    bd = (rng.standard_normal(40) * 0.05).astype(np.float32)
    Wo = (rng.standard_normal((6, 40)) * np.sqrt(2 / 40)).astype(np.float32)
    bo = (rng.standard_normal(6) * 0.05).astype(np.float32)
    nodes = [Node("conv2d", -1, W=W0, b=b0, stride=1, pad=1), Node("relu", 0),
             Node("conv2d", 1, W=W1, b=b1, stride=2, pad=1), Node("relu", 2),
             Node("conv2d", 3, W=W2, b=b2, stride=1, pad=1), Node("relu", 4),
             Node("flatten", 5), Node("dense", 6, W=Wd, b=bd), Node("relu", 7), Node("dense", 8, W=Wo, b=bo)]
    net = Net((3, 8, 8), nodes)
    x0 = rng.random((batch, net.n_in)).astype(np.float32)
    return Workload("convchain", net, x0, np.float32(eps), margin_spec(net, x0))


def stem_net(seed, cin, stride, hw, second=True, batch=1, eps=0.02):
    """conv(cin -> 32, stride) -> ReLU [-> conv 32 -> 32 -> ReLU] -> flatten -> dense 12 -> ReLU
    -> dense 4, on cin x hw x hw: the first convolution's transposed step (onto the input) in
    its other shapes: 1, 2 and 4 input channels (4 needs two 32-column blocks), stride 2, and
    whole-image rows larger than one workgroup's source buffer (split into strips)."""
    rng = np.random.default_rng(seed)

    def cw(co, ci):
        return ((rng.standard_normal((co, ci, 3, 3)) * np.sqrt(2 / (ci * 9))).astype(np.float32),
                (rng.standard_normal(co) * 0.05).astype(np.float32))

    W0, b0 = cw(32, cin)
    nodes = [Node("conv2d", -1, W=W0, b=b0, stride=stride, pad=1), Node("relu", 0)]
    h = (hw - 1) // stride + 1
    if second:
        W1, b1 = cw(32, 32)
        nodes += [Node("conv2d", 1, W=W1, b=b1, stride=1, pad=1), Node("relu", 2)]
    nf = 32 * h * h
    Wd = (rng.standard_normal((12, nf)) * np.sqrt(2 / nf)).astype(np.float32)
    bd = (rng.standard_normal(12) * 0.05).astype(np.float32)
    Wo = (rng.standard_normal((4, 12)) * np.sqrt(2 / 12)).astype(np.float32)
    bo = (rng.standard_normal(4) * 0.05).astype(np.float32)
    k = len(nodes)
    nodes += [Node("flatten", k - 1), Node("dense", k, W=Wd, b=bd), Node("relu", k + 1),
              Node("dense", k + 2, W=Wo, b=bo)]
    net = Net((cin, hw, hw), nodes)
    x0 = rng.random((batch, net.n_in)).astype(np.float32)
    return Workload(f"stem{cin}s{stride}x{hw}", net, x0, np.float32(eps), margin_spec(net, x0))


@pytest.mark.parametrize("cin,stride,hw,second", [(1, 2, 10, True), (2, 1, 8, True), (4, 2, 12, True),
                                                  (4, 1, 16, False), (3, 1, 24, False)])
def test_stem_shapes_all_bounds(cin, stride, hw, second):
    wl = stem_net(305, cin, stride, hw, second)
    log("case", wl.name)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    check_input(wl.net, wl.x0[0], wl.eps, wl.C[0], lb[0], ub[0], [(l[0], u[0]) for l, u in layers], what=wl.name)


@pytest.mark.parametrize("make", [lambda: small_resnet(301), lambda: conv_chain(302)], ids=["resnet8", "convchain"])
def test_small_conv_nets_all_bounds(make):
    wl = make()
    log("case", wl.name)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in range(wl.x0.shape[0]):
        log("oracle input", b)
        check_input(wl.net, wl.x0[b], wl.eps, wl.C[b], lb[b], ub[b], [(l[b], u[b]) for l, u in layers],
                    what=f"{wl.name} input {b}")


@pytest.mark.parametrize("hw,c1,c2", [(4, 32, 64), (6, 32, 128), (4, 128, 128)])
def test_windows_larger_than_the_image(hw, c1, c2):
    """Tiny images, where the coefficient windows outgrow the image (up to 15 x 15 windows on a
    4 x 4 image): most window positions lie outside the image, and whole position classes
    have no position inside it for any anchor; with 128 channels before the stride-2
    convolution the windowed steps run on the 128 x 128 tiles.  Every bound of both inputs
    against the oracle."""
    wl = small_resnet(331, hw=hw, c1=c1, c2=c2, fc=16)
    log("case", wl.name, "c1", c1, "c2", c2)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    for b in range(wl.x0.shape[0]):
        log("oracle input", b)
        check_input(wl.net, wl.x0[b], wl.eps, wl.C[b], lb[b], ub[b], [(l[b], u[b]) for l, u in layers],
                    what=f"{wl.name} input {b}")


def test_conv_ibp_bounds():
    wl = small_resnet(303)
    ctx = gpu_ctx(wl.net)
    lb, ub = ctx.ibp_bounds(to_dev(wl.x0), wl.eps, to_dev(wl.C))
    lb, ub = lb.cpu().numpy(), ub.cpu().numpy()
    for b in range(wl.x0.shape[0]):
        il, iu = oracle.ibp_spec_bounds(wl.net, wl.x0[b], wl.eps, wl.C[b])
        assert_close(lb[b], il, "ibp lb")
        assert_close(ub[b], iu, "ibp ub")


def test_conv_batch_invariance_and_chunking():
    from paper_2606_09377_amd.vcrown import OPT_WORKSPACE_CAP_BYTES
    wl = small_resnet(304, batch=4)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    lb1, ub1, lay1 = gpu_crown(ctx, wl, inputs=[2])
    assert np.array_equal(lb1[0], lb[2]) and np.array_equal(ub1[0], ub[2])
    for r in range(len(layers)):
        assert np.array_equal(lay1[r][0][0], layers[r][0][2]) and np.array_equal(lay1[r][1][0], layers[r][1][2])
    full = ctx.workspace_bytes(4, wl.C.shape[1])
    ctx.set_option(OPT_WORKSPACE_CAP_BYTES, full // 3)
    lb3, ub3, _ = gpu_crown(ctx, wl)
    assert ctx.stats()["n_chunks_last_call"] > len(layers) + 1
    assert np.array_equal(lb3, lb) and np.array_equal(ub3, ub)


def torch_forward(net, X):
    """fp32 forward of many points on the GPU with torch's own conv/linear (an evaluation
    independent of the library)."""
    import torch
    n = X.shape[0]
    inp = X.reshape((n,) + tuple(net.in_shape))
    vals = []
    get = lambda i: inp if i == -1 else vals[i]  # noqa: E731
    for nd in net.nodes:
        v = get(nd.in0)
        if nd.op == "dense":
            vals.append(torch.nn.functional.linear(v.reshape(n, -1), to_dev(nd.W), to_dev(nd.b)))
        elif nd.op == "conv2d":
            vals.append(torch.nn.functional.conv2d(v, to_dev(nd.W), to_dev(nd.b), stride=nd.stride, padding=nd.pad))
        elif nd.op == "relu":
            vals.append(torch.relu(v))
        elif nd.op == "add":
            vals.append(v + get(nd.in1))
        elif nd.op == "flatten":
            vals.append(v.reshape(n, -1))
    return vals


def test_resnet3x16x16_all_bounds_golden():
    g = np.load(os.path.join(GOLDEN, "resnet3x16x16.npz"))
    wl = make_workload("resnet3x16x16")
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    relu_ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    for b in g["inputs"]:
        assert_close(lb[b], g[f"lb_{b}"], f"input {b} lb")
        assert_close(ub[b], g[f"ub_{b}"], f"input {b} ub")
        for r, i in enumerate(relu_ids):
            assert_close(layers[r][0][b], g[f"l_{b}_{i}"], f"input {b} relu {r} l")
            assert_close(layers[r][1][b], g[f"u_{b}_{i}"], f"input {b} relu {r} u")


def test_resnet3x8x8_full_width_all_bounds_golden():
    """The full ResNet's channel widths (64 and 128), FC 512 and 100 classes on a 3x8x8
    image: every intermediate bound of all four ReLU layers, every ReLU class and all 99
    spec rows of both inputs against the stored oracle results.  Its 128-channel
    convolutions run the transposed convolution on 128 x 128 tiles (with and without the
    ReLU relaxation in the epilogue) in the FC 512 and spec passes."""
    g = np.load(os.path.join(GOLDEN, "resnet3x8x8.npz"))
    wl = make_workload("resnet3x8x8")
    assert wl.net.nodes[-1].W.shape == (100, 512)
    ctx = gpu_ctx(wl.net)
    lb, ub, layers = gpu_crown(ctx, wl)
    relu_ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    assert len(relu_ids) == 4
    for b in g["inputs"]:
        assert_close(lb[b], g[f"lb_{b}"], f"input {b} lb")
        assert_close(ub[b], g[f"ub_{b}"], f"input {b} ub")
        for r, i in enumerate(relu_ids):
            rl, ru = g[f"l_{b}_{i}"], g[f"u_{b}_{i}"]
            assert_close(layers[r][0][b], rl, f"input {b} relu {r} l")
            assert_close(layers[r][1][b], ru, f"input {b} relu {r} u")
            assert_classes(layers[r][0][b], layers[r][1][b], rl, ru, f"input {b} relu {r}")
            log("input", b, "relu", r, "unstable (oracle)", int(np.sum((rl < 0) & (ru > 0))))
    # one input alone gives its batch row bit for bit
    lb1, ub1, _ = gpu_crown(ctx, wl, inputs=[1])
    assert np.array_equal(lb1[0], lb[1]) and np.array_equal(ub1[0], ub[1])


def test_resnet3x32x32_full_size():
    """The full ResNet workload (8 inputs): the oracle's bounds of sampled neurons and every
    neuron their receptive fields reach; soundness of the spec bounds on sampled points and
    box corners; one input alone equals its row of the batch bit for bit."""
    import torch
    g = np.load(os.path.join(GOLDEN, "resnet3x32x32_sampled.npz"))
    wl = make_workload("resnet3x32x32")
    ctx = gpu_ctx(wl.net)
    log("gpu run B=8")
    lb, ub, layers = gpu_crown(ctx, wl)
    relu_ids = [i for i, nd in enumerate(wl.net.nodes) if nd.op == "relu"]
    n_checked = 0
    for b in g["inputs"]:
        for r, i in enumerate(relu_ids):
            key = f"idx_{b}_{i}"
            if key not in g:
                continue
            idx = g[key]
            assert_close(layers[r][0][b][idx], g[f"l_{b}_{i}"], f"input {b} relu {r} l")
            assert_close(layers[r][1][b][idx], g[f"u_{b}_{i}"], f"input {b} relu {r} u")
            n_checked += len(idx)
    log("sampled neurons checked", n_checked)
    assert n_checked > 1000
    for r in range(len(layers)):
        assert np.all(layers[r][0] <= layers[r][1])
    assert np.all(lb <= ub)
    # soundness on samples and corners (fp32 forward; slack = parity tolerance)
    from tests.pins import box_of
    rng = np.random.default_rng(9)
    for b in (0, 5):
        lo, hi = box_of(wl.x0[b], wl.eps, wl.clip)
        X = lo + (hi - lo) * rng.random((2048, lo.size))
        Xc = np.where(rng.random((1024, lo.size)) < 0.5, lo, hi)
        for P in (X, Xc):
            with torch.no_grad():
                y = torch_forward(wl.net, torch.from_numpy(P.astype(np.float32)).cuda())[-1]
                Y = (y.double() @ torch.from_numpy(wl.C[b].astype(np.float64)).cuda().T).cpu().numpy()
            slack = 1e-4 + 1e-4 * np.abs(Y)
            assert np.all(Y >= lb[b][None] - slack), np.max(lb[b][None] - Y)
            assert np.all(Y <= ub[b][None] + slack), np.max(Y - ub[b][None])
    lb1, ub1, lay1 = gpu_crown(ctx, wl, inputs=[3])
    assert np.array_equal(lb1[0], lb[3]) and np.array_equal(ub1[0], ub[3])
    for r in range(len(layers)):
        assert np.array_equal(lay1[r][0][0], layers[r][0][3])
