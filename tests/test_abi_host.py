"""The C-ABI library on the host: it loads, exports every function include/vcrown.h
declares, and validates networks and arguments (a validation-only context, no GPU)."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

from workloads import Net, Node, make_workload, random_mlp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="session")
def vc():
    import paper_2606_09377_amd.vcrown as vc
    if not os.path.exists(vc.LIB_PATH):
        from paper_2606_09377_amd import build
        build.build()
    vc.load_library()
    return vc


def test_exports_every_header_symbol(vc):
    syms = vc.header_symbols()
    assert len(syms) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", vc.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [s for s in syms if s not in exported]
    assert not missing, missing
    lib = vc.load_library()
    for s in syms:
        assert hasattr(lib, s)
    assert lib.vcr_abi_version() == vc.ABI_VERSION == 3


def _buf(n, dtype=np.float32):
    # 64-byte aligned host buffer standing in for a device pointer (never dereferenced:
    # the validation-only context stops before any device work)
    raw = np.zeros(n + 16, dtype=dtype)
    off = (-raw.ctypes.data % 64) // raw.itemsize
    return raw[off:off + n]


def test_validation_context_checks_networks(vc):
    ctx = vc.Ctx(-1)
    wl = random_mlp(1, [20, 30, 5], 1, 0.1)
    ctx.load_net(wl.net)
    bad = Net((20,), [Node("dense", 0, W=wl.net.nodes[0].W, b=wl.net.nodes[0].b)])
    with pytest.raises(vc.VcrError) as e:
        ctx.load_net(bad)
    assert e.value.status == vc.VCR_ERR_ARG
    relu_last = Net((20,), [wl.net.nodes[0], Node("relu", 0)])
    with pytest.raises(vc.VcrError) as e:
        ctx.load_net(relu_last)
    assert e.value.status == vc.VCR_ERR_ARG
    add_bad = Net((20,), [wl.net.nodes[0], Node("add", 0, -1), wl.net.nodes[2]])
    with pytest.raises(vc.VcrError) as e:
        ctx.load_net(add_bad)
    assert e.value.status == vc.VCR_ERR_SHAPE


def test_conv_networks_are_reported_unsupported(vc):
    from tests.pins import tiny_resnet
    ctx = vc.Ctx(-1)
    with pytest.raises(vc.VcrError) as e:
        ctx.load_net(tiny_resnet(1))
    assert e.value.status == vc.VCR_ERR_UNSUPPORTED


def test_alpha_on_conv_networks_is_planned(vc):
    """Residual and plain convolutional nets load in a validation-only context, and
    alpha-CROWN on them gets past planning (the slope layout and the gradient pass) to the
    device stage, VCR_ERR_STATE; bad options are still VCR_ERR_ARG.  So do CROWN and
    beta-CROWN on subdomains and the branch-and-bound loop."""
    from tests.test_conv_gpu import conv_chain, small_resnet
    for wl in (small_resnet(1), conv_chain(2)):
        ctx = vc.Ctx(-1)
        ctx.load_net(wl.net)
        lib = ctx.lib
        shapes = oracle_shapes(wl.net)
        n_total = sum(int(np.prod(shapes[i])) for i, nd in enumerate(wl.net.nodes) if nd.op == "relu")
        assert lib.vcr_relu_neurons(ctx.h) == n_total
        B, m = wl.C.shape[0], wl.C.shape[1]
        x, C, lb, ub = _buf(B * wl.net.n_in), _buf(wl.C.size), _buf(B * m), _buf(B * m)
        p = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731
        for lr, want in ((0.1, vc.VCR_ERR_STATE), (0.0, vc.VCR_ERR_ARG)):
            o = vc.VcrAlphaOpts(3, lr, 0.9, 0.999, 1e-8, None, None, None, None, None)
            st = lib.vcr_alpha_crown_bounds(ctx.h, p(x), B, ctypes.c_float(0.01), p(C), m, ctypes.byref(o), p(lb),
                                            p(ub))
            assert st == want, (wl.name, lr, lib.vcr_last_error(ctx.h))
        # subdomains of one input: CROWN, beta-CROWN and the loop are planned as well
        D = 8
        rid, neu, sg = _buf(D * 2, np.int32), _buf(D * 2, np.int32), _buf(D * 2, np.int8)
        sp = vc.VcrSplits(D, 2, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)
        dl, du = _buf(D * m), _buf(D * m)
        st = lib.vcr_crown_bounds(ctx.h, p(x), 1, ctypes.c_float(0.01), p(C), m, ctypes.byref(sp), p(dl), p(du))
        assert st == vc.VCR_ERR_STATE, (wl.name, lib.vcr_last_error(ctx.h))
        bo = vc.VcrBetaOpts(3, 0.1, 0.05, 0.9, 0.999, 1e-8, None, None)
        st = lib.vcr_beta_crown_bounds(ctx.h, p(x), ctypes.c_float(0.01), p(C), m, ctypes.byref(sp), ctypes.byref(bo),
                                       p(dl), p(du))
        assert st == vc.VCR_ERR_STATE, (wl.name, lib.vcr_last_error(ctx.h))
        res = vc.VcrBabResult()
        ob = vc.VcrBabOpts(4, 3, bo, None, None, 0)
        st = lib.vcr_bab_verify(ctx.h, p(x), ctypes.c_float(0.01), p(C), m, ctypes.byref(ob), ctypes.byref(res), None)
        assert st == vc.VCR_ERR_STATE, (wl.name, lib.vcr_last_error(ctx.h))
        wsb = ctypes.c_uint64(0)
        assert lib.vcr_workspace_bytes(ctx.h, 1, m, D, ctypes.byref(wsb)) == vc.VCR_OK and wsb.value > 0


def oracle_shapes(net):
    from workloads.gen import node_shapes
    return node_shapes(net)


def _call(vc, ctx, B, eps, m, n0, n_out, splits=None, x0=None, C=None, lb=None, ub=None):
    lib = ctx.lib
    x0 = _buf(B * n0) if x0 is None else x0
    C = _buf(B * m * n_out) if C is None else C
    rows = splits.n_domains if splits is not None else B
    lb = _buf(max(rows, 1) * m) if lb is None else lb
    ub = _buf(max(rows, 1) * m) if ub is None else ub
    p = lambda a: ctypes.c_void_p(a.ctypes.data) if a is not None else None  # noqa: E731
    sp = ctypes.byref(splits) if splits is not None else None
    return lib.vcr_crown_bounds(ctx.h, p(x0), B, ctypes.c_float(eps), p(C), m, sp, p(lb), p(ub))


def test_argument_validation(vc):
    ctx = vc.Ctx(-1)
    wl = random_mlp(2, [20, 30, 30, 5], 1, 0.1)
    lib = ctx.lib
    null = ctypes.c_void_p()
    # before a network is loaded
    assert _call(vc, ctx, 1, 0.1, 4, 20, 5) == vc.VCR_ERR_STATE
    ctx.load_net(wl.net)
    assert _call(vc, ctx, 2, 0.1, 4, 20, 5) == vc.VCR_ERR_STATE      # valid: stops before device work
    assert b"validation-only" in lib.vcr_last_error(ctx.h)
    assert _call(vc, ctx, 0, 0.1, 4, 20, 5) == vc.VCR_ERR_ARG
    assert _call(vc, ctx, 1, -0.1, 4, 20, 5) == vc.VCR_ERR_ARG
    assert _call(vc, ctx, 1, float("nan"), 4, 20, 5) == vc.VCR_ERR_ARG
    assert _call(vc, ctx, 1, float("inf"), 4, 20, 5) == vc.VCR_ERR_ARG
    assert _call(vc, ctx, 1, 0.1, 0, 20, 5) == vc.VCR_ERR_ARG
    x = _buf(40)
    assert lib.vcr_crown_bounds(ctx.h, null, 1, ctypes.c_float(0.1), ctypes.c_void_p(x.ctypes.data), 4, None,
                                ctypes.c_void_p(x.ctypes.data), ctypes.c_void_p(x.ctypes.data)) == vc.VCR_ERR_ARG
    mis = _buf(64)
    assert lib.vcr_crown_bounds(ctx.h, ctypes.c_void_p(mis.ctypes.data + 4), 1, ctypes.c_float(0.1),
                                ctypes.c_void_p(mis.ctypes.data), 1, None, ctypes.c_void_p(mis.ctypes.data),
                                ctypes.c_void_p(mis.ctypes.data)) == vc.VCR_ERR_ARG
    rid, neu, sg = _buf(8, np.int32), _buf(8, np.int32), _buf(8, np.int8)
    sp = vc.VcrSplits(4, 2, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)
    assert _call(vc, ctx, 1, 0.1, 4, 20, 5, splits=sp) == vc.VCR_ERR_STATE
    assert _call(vc, ctx, 2, 0.1, 4, 20, 5, splits=sp) == vc.VCR_ERR_ARG   # splits need B == 1
    sp0 = vc.VcrSplits(0, 2, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)
    assert _call(vc, ctx, 1, 0.1, 4, 20, 5, splits=sp0) == vc.VCR_ERR_ARG
    spn = vc.VcrSplits(4, 2, None, neu.ctypes.data, sg.ctypes.data)
    assert _call(vc, ctx, 1, 0.1, 4, 20, 5, splits=spn) == vc.VCR_ERR_ARG
    assert lib.vcr_set_option(ctx.h, 99, 1.0) == vc.VCR_ERR_ARG
    assert lib.vcr_set_option(ctx.h, vc.OPT_WORKSPACE_CAP_BYTES, -1.0) == vc.VCR_ERR_ARG
    assert lib.vcr_set_option(ctx.h, vc.OPT_CLIP_LO, float("nan")) == vc.VCR_ERR_ARG
    assert lib.vcr_create(-2, ctypes.byref(ctypes.c_void_p())) == vc.VCR_ERR_ARG


def test_planner_chunks_under_a_workspace_cap(vc):
    """Workspace grows with the batch; under a cap the inputs are processed in chunks (the
    plan is reported by the validation-only context); below the minimum plan: OOM."""
    ctx = vc.Ctx(-1)
    wl = make_workload("mlp784x1024x6", batch=1)
    ctx.load_net(wl.net)
    w1, w64 = ctx.workspace_bytes(1, 9), ctx.workspace_bytes(64, 9)
    assert w64 > 32 * w1 > 0
    # the A ping-pong buffers of 64 inputs: 2 x (64 * 2048 rows) x 1024 floats
    assert w64 >= 2 * 64 * 2048 * 1024 * 4
    assert _call(vc, ctx, 64, 0.015, 9, 784, 10) == vc.VCR_ERR_STATE
    assert ctx.stats()["n_chunks_last_call"] == 5 + 1        # 5 intermediate layers, 1 spec pass
    ctx.set_option(vc.OPT_WORKSPACE_CAP_BYTES, w64 // 4)
    assert _call(vc, ctx, 64, 0.015, 9, 784, 10) == vc.VCR_ERR_STATE
    n = ctx.stats()["n_chunks_last_call"]
    assert n >= 5 * 4 + 1, n
    ctx.set_option(vc.OPT_WORKSPACE_CAP_BYTES, 1 << 20)
    assert _call(vc, ctx, 64, 0.015, 9, 784, 10) == vc.VCR_ERR_OOM
    ctx.set_option(vc.OPT_WORKSPACE_CAP_BYTES, 0)
    # the wide MLP holds its A matrices whole: 2 x (16 * 16384 rows) x 8192 floats
    wl3 = make_workload("mlp3072x8192x4", batch=1)
    ctx.load_net(wl3.net)
    assert ctx.workspace_bytes(16, 99) >= 2 * 16 * 16384 * 8192 * 4
    # subdomains: 4096 domains x 18 rows in one chunk
    ctx.load_net(wl.net)
    assert ctx.workspace_bytes(1, 9, 4096) >= 2 * 4096 * 18 * 1024 * 4


def test_alpha_beta_bab_argument_validation(vc):
    """alpha-CROWN, beta-CROWN and the branch-and-bound loop check their options before any
    device work (a validation-only context then reports VCR_ERR_STATE)."""
    ctx = vc.Ctx(-1)
    wl = random_mlp(3, [20, 30, 30, 5], 1, 0.1)
    ctx.load_net(wl.net)
    lib = ctx.lib
    assert lib.vcr_relu_neurons(ctx.h) == 60
    x, C, lb, ub = _buf(20), _buf(4 * 5), _buf(4), _buf(4)
    p = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731

    def alpha(**kw):
        o = vc.VcrAlphaOpts(kw.get("iters", 5), kw.get("lr", 0.1), kw.get("b1", 0.9), kw.get("b2", 0.999),
                            kw.get("eps", 1e-8), None, None, None, kw.get("lh"), kw.get("uh"))
        return lib.vcr_alpha_crown_bounds(ctx.h, p(x), 1, ctypes.c_float(0.1), p(C), 4, ctypes.byref(o), p(lb), p(ub))

    assert alpha() == vc.VCR_ERR_STATE
    for kw in ({"iters": -1}, {"lr": 0.0}, {"lr": float("inf")}, {"b1": 1.0}, {"b2": -0.1}, {"eps": 0.0},
               {"lh": lb.ctypes.data}):
        assert alpha(**kw) == vc.VCR_ERR_ARG, kw
    assert lib.vcr_alpha_crown_bounds(ctx.h, p(x), 1, ctypes.c_float(0.1), p(C), 4, None, p(lb), p(ub)) == vc.VCR_ERR_ARG

    rid, neu, sg = _buf(8, np.int32), _buf(8, np.int32), _buf(8, np.int8)
    sp = vc.VcrSplits(4, 2, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)

    def beta(splits=sp, **kw):
        o = vc.VcrBetaOpts(kw.get("iters", 5), kw.get("la", 0.1), kw.get("lb", 0.05), 0.9, 0.999, 1e-8, None, None)
        s = ctypes.byref(splits) if splits is not None else None
        return lib.vcr_beta_crown_bounds(ctx.h, p(x), ctypes.c_float(0.1), p(C), 4, s, ctypes.byref(o), p(lb), p(ub))

    assert beta() == vc.VCR_ERR_STATE
    assert beta(splits=None) == vc.VCR_ERR_ARG
    assert beta(la=0.0) == vc.VCR_ERR_ARG and beta(lb=-1.0) == vc.VCR_ERR_ARG and beta(iters=-2) == vc.VCR_ERR_ARG
    assert beta(splits=vc.VcrSplits(0, 2, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)) == vc.VCR_ERR_ARG

    def bab(batch=4, rounds=3, order=None):
        bo = vc.VcrBetaOpts(5, 0.1, 0.05, 0.9, 0.999, 1e-8, None, None)
        o = vc.VcrBabOpts(batch, rounds, bo, None, None, 0)
        keep = None
        if order is not None:
            keep = (np.array([a for a, _ in order], np.int32), np.array([b for _, b in order], np.int32))
            o.order_relu, o.order_neuron, o.order_len = keep[0].ctypes.data, keep[1].ctypes.data, len(order)
        res = vc.VcrBabResult()
        return lib.vcr_bab_verify(ctx.h, p(x), ctypes.c_float(0.1), p(C), 4, ctypes.byref(o), ctypes.byref(res), None)

    assert bab() == vc.VCR_ERR_STATE
    assert bab(order=[(0, 3), (1, 29)]) == vc.VCR_ERR_STATE
    assert bab(batch=0) == vc.VCR_ERR_ARG and bab(rounds=-1) == vc.VCR_ERR_ARG
    assert bab(order=[(2, 0)]) == vc.VCR_ERR_ARG and bab(order=[(1, 30)]) == vc.VCR_ERR_ARG


def test_option_values_and_round_limit(vc):
    """The lambda rule takes the four VCR_LAMBDA_* values only; CHECK_FINITE is a flag; the
    branch-and-bound loop rejects more rounds than a subdomain has split slots (one split
    per round) before any device work."""
    ctx = vc.Ctx(-1)
    wl = random_mlp(3, [20, 30, 30, 5], 1, 0.1)
    ctx.load_net(wl.net)
    for v in vc.LAMBDA_RULES.values():
        ctx.set_option(vc.OPT_LAMBDA_RULE, v)
    for v in (-1, 4, 0.5):
        with pytest.raises(vc.VcrError) as e:
            ctx.set_option(vc.OPT_LAMBDA_RULE, v)
        assert e.value.status == vc.VCR_ERR_ARG
    ctx.set_option(vc.OPT_CHECK_FINITE, 1)
    ctx.set_option(vc.OPT_CHECK_FINITE, 0)
    lib = ctx.lib
    x, C = _buf(20), _buf(4 * 5)
    p = lambda a: ctypes.c_void_p(a.ctypes.data)  # noqa: E731

    def bab(rounds):
        bo = vc.VcrBetaOpts(5, 0.1, 0.05, 0.9, 0.999, 1e-8, None, None)
        o = vc.VcrBabOpts(4, rounds, bo, None, None, 0)
        res = vc.VcrBabResult()
        return lib.vcr_bab_verify(ctx.h, p(x), ctypes.c_float(0.1), p(C), 4, ctypes.byref(o), ctypes.byref(res), None)

    assert bab(vc.MAX_SPLITS) == vc.VCR_ERR_STATE
    assert bab(vc.MAX_SPLITS + 1) == vc.VCR_ERR_ARG
    assert "max_rounds" in lib.vcr_last_error(ctx.h).decode()
    # per_domain beyond the split slots
    rid, neu, sg = _buf(4 * 65, np.int32), _buf(4 * 65, np.int32), _buf(4 * 65, np.int8)
    sp = vc.VcrSplits(4, vc.MAX_SPLITS + 1, rid.ctypes.data, neu.ctypes.data, sg.ctypes.data)
    assert _call(vc, ctx, 1, 0.1, 4, 20, 5, splits=sp) == vc.VCR_ERR_ARG
