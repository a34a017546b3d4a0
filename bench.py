"""Throughput of batched full-CROWN bound evaluation on one MI355X.

A step is one vcr_crown_bounds call over one batch of seeded synthetic inputs that are
already resident in HBM: the IBP pass, every intermediate layer's backward A-matrix pass,
the ReLU relaxations and the final spec pass.  Default workload: the wide ReLU MLP
3072-8192x4-100 (the width of the paper's Table 4 at h = 8192), 16 inputs, eps = 2/255,
99 margin rows per input, with its 8192 x 8192 A matrices held whole (146.6 TFLOP per call).

Prints one JSON line with the throughput (inputs/s), the dominant kernel's roofline
(the backward-step fp32 MFMA GEMM, timed with HIP events on the stream it runs on) and the
fp64 CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
KERNEL_SOURCES = {"k_gemm": "gemm.hip", "k_convt": "conv.hip", "k_gemm_small": "gemm.hip", "k_gemm_mid": "gemm.hip"}
KERNEL_DESC = {"k_gemm": "k_gemm (dense A.W step, fp32 v_mfma_f32_32x32x2f32)",
               "k_convt": "k_convt (transposed-conv implicit GEMM, fp32 v_mfma_f32_32x32x2f32)",
               "k_gemm_small": "k_gemm_small (dense A.W step on 32x64 tiles, fp32 v_mfma_f32_32x32x2f32)",
               "k_gemm_mid": "k_gemm_mid (dense A.W step on 64x64 tiles, fp32 v_mfma_f32_32x32x2f32)"}


def source_hash(kernel):
    path = os.path.join(ROOT, "paper_2606_09377_amd", "csrc", KERNEL_SOURCES[kernel])
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_for(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed PMC runs, if they were taken on the
    current kernel source; else None."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    k = t.get("kernels", {}).get(kernel)
    if not k or k.get("source_sha") != source_hash(kernel):
        return None
    w = k.get("workloads", {}).get(workload)
    return None if w is None else w.get("bytes_per_launch")


def host_info():
    """The host the oracle runs on: CPU model, logical CPUs and numpy's BLAS thread pools."""
    import threadpoolctl
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    pools = [{k: p.get(k) for k in ("user_api", "internal_api", "num_threads", "version", "threading_layer")}
             for p in threadpoolctl.threadpool_info()]
    return {"cpu_model": model, "cpu_count": os.cpu_count(), "threadpool_info": pools}


def _threads():
    import threadpoolctl
    return int(max((p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()), default=1))


def cpu_baseline(wl, budget_s, alpha_iters=0):
    """The fp64 oracle, as it stands, on the first inputs of the same batch until the time
    budget is used (at least one input); with alpha_iters the alpha-CROWN oracle."""
    import oracle
    from oracle import alpha64
    t0 = time.perf_counter()
    n = 0
    while n < wl.x0.shape[0]:
        if alpha_iters:
            alpha64.alpha_crown(wl.net, wl.x0[n], wl.eps, wl.C[n], iters=alpha_iters)
        elif wl.name.startswith("exp1_"):
            # one hidden layer: the oracle's row-block form (the full-matrix form needs ~40 GB)
            oracle.crown_one_hidden(wl.net, wl.x0[n], wl.eps, wl.C[n])
        else:
            oracle.crown(wl.net, wl.x0[n], wl.eps, wl.C[n])
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "inputs/s", "cores": _threads(), "kind": "oracle",
            "sample": f"first {n} of the {wl.x0.shape[0]} inputs of the same batch, {dt:.1f} s", **host_info()}


def cpu_baseline_sampled(wl, budget_s, chunk, alpha_iters=0):
    """One input of the wide MLP or the full ResNet takes the fp64 oracle minutes to hours,
    so its time per input is estimated from a timed sample of the oracle's own steps on
    input 0: the box, the IBP pass and a first ReLU on an affine map of the input run whole;
    for every other ReLU layer and for the spec rows, chunks of `chunk` rows go through the
    oracle's backward pass and concretization (lower and upper), as the oracle processes
    them, until that layer's share of the budget is used, and the per-row time is scaled to
    the layer's row count.  The cost of a row does not depend on the relaxation values, so
    the sample uses the IBP bounds' relaxation.  With alpha_iters, the alpha-CROWN oracle's
    evaluation (both bounds and their gradients) of a chunk of spec rows is timed as well and
    scaled to all spec rows and the alpha_iters + 1 evaluations."""
    import oracle
    net = wl.net
    shapes = oracle.node_shapes(net)
    t0 = time.perf_counter()
    lo, hi = oracle.input_box(wl.x0[0], wl.eps, wl.clip)
    IL, IU = oracle.ibp(net, lo, hi)
    relus = [i for i, nd in enumerate(net.nodes) if nd.op == "relu"]
    relax = {i: oracle.relu_relaxation(IL[net.nodes[i].in0].reshape(-1), IU[net.nodes[i].in0].reshape(-1))
             for i in relus}
    total = time.perf_counter() - t0
    parts = [f"box and IBP {total:.1f} s"]
    starts = [(net.nodes[i].in0, int(np.prod(shapes[net.nodes[i].in0]))) for i in relus]
    starts.append((len(net.nodes) - 1, wl.C.shape[1]))
    per_layer = max(budget_s / len(starts), 0.5)
    for k, (z, n_rows) in enumerate(starts):
        n = int(np.prod(shapes[z]))
        nd = net.nodes[z]
        t0 = time.perf_counter()
        if k < len(relus) and nd.op == "dense" and nd.in0 == -1:
            # the oracle bounds an affine map of the input directly from W, b
            W, b = nd.W.astype(np.float64), nd.b.astype(np.float64)
            oracle.concretize(W, b, lo, hi, False)
            oracle.concretize(W, b, lo, hi, True)
            dt = time.perf_counter() - t0
            total += dt
            parts.append(f"node {z} (affine map of the input) whole in {dt:.1f} s")
            continue
        done = 0
        while done < n_rows and (done == 0 or time.perf_counter() - t0 < per_layer):
            rows = min(chunk, n_rows - done)
            if k == len(relus):
                A = wl.C[0][done:done + rows].astype(np.float64)
            else:
                A = np.zeros((rows, n))
                A[np.arange(rows), np.arange(done, done + rows)] = 1.0
            zero = np.zeros(rows)
            for up in (False, True):
                Ax, bx = oracle.backward(net, shapes, relax, z, A, zero, upper=up)
                oracle.concretize(Ax, bx, lo, hi, up)
            done += rows
        dt = time.perf_counter() - t0
        total += dt / done * n_rows
        parts.append(f"{done}/{n_rows} rows of node {z} in {dt:.1f} s")
    if alpha_iters:
        from types import SimpleNamespace
        from oracle import alpha64
        root = SimpleNamespace(relax={i: tuple(v.reshape(shapes[i]) for v in relax[i]) for i in relus},
                               layer_l={i: IL[net.nodes[i].in0] for i in relus},
                               layer_u={i: IU[net.nodes[i].in0] for i in relus}, box=(lo, hi))
        rows = min(chunk, wl.C.shape[1])
        al, au = alpha64.initial_alpha(net, root, rows)
        t0 = time.perf_counter()
        alpha64.alpha_bound(net, root, wl.C[0][:rows], al, au)
        dt = time.perf_counter() - t0
        total += dt / rows * wl.C.shape[1] * (alpha_iters + 1)
        parts.append(f"one alpha-CROWN evaluation with gradients of {rows}/{wl.C.shape[1]} spec rows in {dt:.1f} s, "
                     f"scaled to {alpha_iters + 1} evaluations")
    return {"value": 1.0 / total, "unit": "inputs/s", "cores": _threads(), "kind": "oracle",
            "sample": f"estimated from timed steps of input 0 ({chunk}-row chunks), scaled to each layer's rows: "
                      + "; ".join(parts) + f"; {total:.0f} s per input", **host_info()}


def cpu_baseline_bab(wl, sp, budget_s):
    """The fp64 oracle on the same subdomains: its root pass, then domains until the time
    budget is used; reported as domains/s of the domain evaluations plus the root pass."""
    import oracle
    from workloads import Splits
    splits = Splits(sp["relu_id"], sp["neuron"], sp["sign"])
    t0 = time.perf_counter()
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    t_root = time.perf_counter() - t0
    n = 0
    t1 = time.perf_counter()
    while n < splits.n_domains and time.perf_counter() - t0 < budget_s:
        oracle.crown_domains(wl.net, root, wl.C[0], splits, domains=range(n, n + 16))
        n += 16
    t_dom = time.perf_counter() - t1
    total = t_root + t_dom * splits.n_domains / n
    return {"value": splits.n_domains / total, "unit": "domains/s", "cores": _threads(), "kind": "oracle",
            "sample": f"root pass ({t_root:.1f} s) + first {n} of {splits.n_domains} domains ({t_dom:.1f} s), "
                      f"domain time scaled to all domains", **host_info()}


# workloads whose oracle time per input is estimated from a timed sample (row chunk size):
# the oracle's own 256-row chunks for the wide MLP, 16 rows of the ResNet's dense coefficient
# tensors (up to 65536 columns per row)
SAMPLED_BASELINE = {"mlp3072x8192x4": 256, "resnet3x32x32": 16}

BAB_ROUNDS, BAB_ITERS = 10, 20


def cpu_baseline_bab_loop(wl, batch, budget_s):
    """The oracle's beta-CROWN on the subdomains the loop bounds first (the same loop, with
    the oracle's own split order), until the time budget is used; subdomains per second."""
    import oracle
    from oracle import beta64
    root = oracle.crown(wl.net, wl.x0[0], wl.eps, wl.C[0])
    order = beta64.default_order(wl.net, root)
    t0 = time.perf_counter()
    n, frontier = 0, [()]
    while frontier and time.perf_counter() - t0 < budget_s:
        kids = []
        for dom in frontier[:batch]:
            used = {(r, j) for r, j, _ in dom}
            nxt = next(o for o in order if o not in used)
            kids += [dom + ((nxt[0], nxt[1], 1),), dom + ((nxt[0], nxt[1], -1),)]
        frontier = []
        for k in kids:
            r = beta64.beta_crown(wl.net, root, wl.C[0], list(k), iters=BAB_ITERS)
            n += 1
            if not np.all(r.lb > 0.0):
                frontier.append(k)
            if time.perf_counter() - t0 >= budget_s:
                break
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "domains/s", "cores": _threads(), "kind": "oracle",
            "sample": f"beta-CROWN ({BAB_ITERS} steps) on the first {n} subdomains of the same loop, {dt:.1f} s",
            **host_info()}


def bench_bab_loop(args):
    import torch
    from paper_2606_09377_amd import Ctx
    from paper_2606_09377_amd.vcrown import OPT_TIME_GEMM
    from workloads import make_workload
    conv = args.workload.startswith("resnet")
    if not (args.workload.startswith("bab_") or conv):
        print("--bab-loop runs on a bab_ workload (its root input and property) or on a ResNet's first input",
              file=sys.stderr)
        sys.exit(2)
    wl = make_workload(args.workload)
    ctx = Ctx(0)
    ctx.load_net(wl.net)
    x0 = torch.from_numpy(wl.x0[:1]).cuda()
    C = torch.from_numpy(wl.C[:1]).cuda()

    def step():
        return ctx.bab_verify(x0, wl.eps, C, batch=args.bab_loop, max_rounds=BAB_ROUNDS, iters=BAB_ITERS)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ctx.set_option(OPT_TIME_GEMM, 1)
    t0 = time.perf_counter()
    results = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = ctx.stats()
    ctx.set_option(OPT_TIME_GEMM, 0)
    res = results[-1]
    assert all(r == res for r in results), "the loop is deterministic"
    domains = res["evaluated"] * args.steps
    kinds = ("conv",) if conv else ("gemm", "small", "mid")
    launches = sum(st[f"timed_{k}_launches"] for k in kinds)
    gms = sum(st[f"timed_{k}_ms"] for k in kinds)
    gfl = sum(st[f"timed_{k}_flops"] for k in kinds)
    achieved = gfl / (gms / 1e3) / 1e12 if gms > 0 else None
    rec = {
        "metric": "CROWN bound evals/sec (inputs or BaB domains) at 1 GPU; % fp32 MFMA peak",
        "value": domains / dt,
        "unit": "domains/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": dt / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": args.workload, "mode": "branch-and-bound loop", "batch": args.bab_loop,
                   "rounds": BAB_ROUNDS, "eps": float(wl.eps), "spec_rows": int(wl.C.shape[1]),
                   "method": f"alpha-CROWN root, beta-CROWN subdomains ({BAB_ITERS} joint Adam steps)"},
        "roofline": {"bound": "mfma",
                     "kernel": KERNEL_DESC["k_convt"] if conv else "k_gemm and k_gemm_small (dense A.W steps, fp32 MFMA)",
                     "achieved": achieved,
                     "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_FP32_MFMA_TFLOPS if achieved else None,
                     "traffic": None if conv else traffic_for("k_gemm", args.workload), "launches_timed": launches,
                     "avg_launch_ms": gms / launches if launches else None,
                     "flops_per_launch": gfl / launches if launches else None,
                     "share_of_step": gms / 1e3 / dt if launches else None},
        "bab": {k: res[k] for k in ("verified", "rounds", "evaluated", "remaining", "root_min_lb", "worst_lb", "log")},
    }
    if args.cpu_budget > 0 and not conv:
        rec["cpu_baseline"] = cpu_baseline_bab_loop(wl, args.bab_loop, args.cpu_budget)
    elif conv:
        rec["cpu_baseline"] = None
        rec["cpu_baseline_note"] = "the oracle's root pass alone exceeds the CPU budget on this ResNet"
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mlp3072x8192x4")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time (0: skip)")
    ap.add_argument("--alpha-iters", type=int, default=0,
                    help="alpha-CROWN with this many Adam steps on the final pass (0: CROWN)")
    ap.add_argument("--bab-loop", type=int, default=0, metavar="BATCH",
                    help="run the fixed-batch branch-and-bound loop (10 rounds, beta-CROWN bounds) with this batch "
                         "on the bab_ workload's root input or a ResNet's first input; value = subdomains bounded "
                         "per second")
    ap.add_argument("--graph", action="store_true",
                    help="replay the call as a recorded HIP graph (the roofline then comes from a "
                         "second timed pass without the graph)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB three times (HBM counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.rand(n, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    if args.bab_loop:
        return bench_bab_loop(args)

    if args.alpha_iters and (args.workload.startswith("bab_") or args.workload.startswith("exp1_")):
        print("--alpha-iters runs on the input-batch workloads (MLPs and ResNets)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_09377_amd import Ctx
    from paper_2606_09377_amd.vcrown import OPT_TIME_GEMM
    from workloads import make_workload

    wl = make_workload(args.workload)
    B, m = wl.C.shape[0], wl.C.shape[1]
    ctx = Ctx(0)
    ctx.load_net(wl.net)
    x0 = torch.from_numpy(wl.x0).cuda()
    C = torch.from_numpy(wl.C).cuda()
    splits = None
    units, unit = B, "inputs/s"
    if args.workload.startswith("bab_"):
        # subdomains drawn once from the oracle root pass (stored with the tests)
        sp = np.load(os.path.join(ROOT, "tests", "golden", f"{args.workload}_splits.npz"))
        splits = tuple(torch.from_numpy(np.ascontiguousarray(sp[k])).cuda() for k in ("relu_id", "neuron", "sign"))
        units, unit = splits[0].shape[0], "domains/s"
    lb = torch.empty((units, m), dtype=torch.float32, device="cuda")
    ub = torch.empty((units, m), dtype=torch.float32, device="cuda")

    def step():
        if args.alpha_iters:
            ctx.alpha_crown_bounds(x0, wl.eps, C, iters=args.alpha_iters, out=(lb, ub))
        else:
            ctx.crown_bounds(x0, wl.eps, C, splits=splits, out=(lb, ub))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    flops_call = ctx.stats()["gemm_flops_last_call"]
    if args.graph:
        from paper_2606_09377_amd.vcrown import OPT_GRAPH
        ctx.set_option(OPT_GRAPH, 1)
        step()          # records the graph
        torch.cuda.synchronize()
    else:
        ctx.set_option(OPT_TIME_GEMM, 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    if args.graph:
        ctx.set_option(OPT_GRAPH, 0)
        ctx.set_option(OPT_TIME_GEMM, 1)
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
    st = ctx.stats()
    ctx.set_option(OPT_TIME_GEMM, 0)
    assert np.all(np.isfinite(lb.cpu().numpy()))
    extra = {}
    if splits is not None:
        # the root pass alone (one input, no subdomains), to report domains/s without it
        rl = torch.empty((1, m), dtype=torch.float32, device="cuda")
        ru = torch.empty((1, m), dtype=torch.float32, device="cuda")
        ctx.crown_bounds(x0, wl.eps, C, out=(rl, ru))
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(args.steps):
            ctx.crown_bounds(x0, wl.eps, C, out=(rl, ru))
        torch.cuda.synchronize()
        root_ms = (time.perf_counter() - t1) / args.steps * 1e3
        extra = {"root_pass_ms": root_ms,
                 "domains_per_s_without_root": units / ((dt / args.steps * 1e3 - root_ms) / 1e3)}

    ms_step = dt / args.steps * 1e3
    value = units * args.steps / dt
    timed = {"k_gemm": (st["timed_gemm_launches"], st["timed_gemm_ms"], st["timed_gemm_flops"]),
             "k_convt": (st["timed_conv_launches"], st["timed_conv_ms"], st["timed_conv_flops"]),
             "k_gemm_small": (st["timed_small_launches"], st["timed_small_ms"], st["timed_small_flops"]),
             "k_gemm_mid": (st["timed_mid_launches"], st["timed_mid_ms"], st["timed_mid_flops"])}

    def roofline(kernel):
        launches, ms, fl = timed[kernel]
        achieved = fl / (ms / 1e3) / 1e12 if ms > 0 else None
        return {"bound": "mfma", "kernel": KERNEL_DESC[kernel],
                "achieved": achieved, "peak": PEAK_FP32_MFMA_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_FP32_MFMA_TFLOPS if achieved else None,
                "traffic": traffic_for(kernel, args.workload),
                "launches_timed": launches,
                "avg_launch_ms": ms / launches if launches else None,
                "flops_per_launch": fl / launches if launches else None,
                "share_of_step": ms / args.steps / ms_step if launches else None}

    dominant = max(timed, key=lambda k: timed[k][1])
    other = sorted((k for k in timed if k != dominant and timed[k][0] > 0), key=lambda k: -timed[k][1])
    rec = {
        "metric": "CROWN bound evals/sec (inputs or BaB domains) at 1 GPU; % fp32 MFMA peak",
        "value": value,
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "batch": B, "eps": float(wl.eps), "spec_rows": m,
                   "domains": units if splits is not None else None,
                   "layers": [int(wl.net.nodes[0].W.shape[1])] + [int(nd.W.shape[0]) for nd in wl.net.nodes
                                                                   if nd.op == "dense"],
                   "method": (f"alpha-CROWN ({args.alpha_iters} projected Adam steps on the final pass, "
                              "full-CROWN intermediate bounds)") if args.alpha_iters
                   else "full CROWN (IBP-intersected intermediate bounds)"},
        "roofline": roofline(dominant),
        "call_mfma_frac": flops_call / (ms_step / 1e3) / (PEAK_FP32_MFMA_TFLOPS * 1e12),
        "graph_replay": bool(args.graph),
        "gemm_flops_per_step": flops_call,
        "device_memory": {"net_bytes": st["net_bytes"], "workspace_peak_bytes": st["peak_workspace_bytes"]},
    }
    if other:
        rec["roofline_other"] = [roofline(k) for k in other]
    rec.update(extra)
    if args.cpu_budget > 0 and args.workload in SAMPLED_BASELINE:
        rec["cpu_baseline"] = cpu_baseline_sampled(wl, args.cpu_budget, SAMPLED_BASELINE[args.workload],
                                                   args.alpha_iters)
    elif args.cpu_budget > 0 and splits is None:
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget, args.alpha_iters)
    elif args.cpu_budget > 0:
        rec["cpu_baseline"] = cpu_baseline_bab(wl, sp, args.cpu_budget)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
