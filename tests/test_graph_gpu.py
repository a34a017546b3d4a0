"""HIP graph replay (VCR_OPT_GRAPH): every replay equals the ordinary call bit for bit,
with other work and synchronisations between replays; changing an argument re-records."""
import numpy as np
import pytest

from tests.gpu_util import gpu_ctx, to_dev
from tests.test_conv_gpu import small_resnet
from workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("which", ["mlp", "resnet"])
def test_graph_replays_match_eager(which):
    import torch
    from paper_2606_09377_amd.vcrown import OPT_GRAPH
    wl = make_workload("mlp784x256x2", batch=1) if which == "mlp" else small_resnet(305, batch=2)
    ctx = gpu_ctx(wl.net)
    x0, C = to_dev(wl.x0), to_dev(wl.C)
    B, m = wl.C.shape[0], wl.C.shape[1]
    ref_lb, ref_ub = ctx.crown_bounds(x0, wl.eps, C)
    torch.cuda.synchronize()
    ref_lb, ref_ub = ref_lb.cpu().numpy(), ref_ub.cpu().numpy()
    ctx.set_option(OPT_GRAPH, 1)
    lb = torch.empty((B, m), dtype=torch.float32, device="cuda")
    ub = torch.empty((B, m), dtype=torch.float32, device="cuda")
    other_x = to_dev(np.clip(wl.x0 + 0.01, 0, 1).astype(np.float32))
    ctx2 = gpu_ctx(wl.net)
    for rep in range(4):
        lb.fill_(np.nan)
        ub.fill_(np.nan)
        ctx.crown_bounds(x0, wl.eps, C, out=(lb, ub))     # rep 0 records, later reps replay
        torch.cuda.synchronize()
        assert np.array_equal(lb.cpu().numpy(), ref_lb), rep
        assert np.array_equal(ub.cpu().numpy(), ref_ub), rep
        # other eager work between replays: another context's ordinary call and a torch op
        ctx2.crown_bounds(other_x, wl.eps, C)
        (x0 * 2.0).sum()
        torch.cuda.synchronize()
    # a changed argument records a new graph, whose replays are right too
    lb_o, ub_o = ctx2.crown_bounds(other_x, wl.eps, C)
    torch.cuda.synchronize()
    for rep in range(2):
        ctx.crown_bounds(other_x, wl.eps, C, out=(lb, ub))
        torch.cuda.synchronize()
        assert np.array_equal(lb.cpu().numpy(), lb_o.cpu().numpy())
    ctx.set_option(OPT_GRAPH, 0)
    lb2, ub2 = ctx.crown_bounds(x0, wl.eps, C)
    torch.cuda.synchronize()
    assert np.array_equal(lb2.cpu().numpy(), ref_lb)
