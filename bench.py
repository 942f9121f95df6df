#!/usr/bin/env python3
"""Benchmark of the CPDP reconcile hot path on one MI355X.

One timed step = one CPDP period over the workload: K-1 local momentum-SGD
steps and one fused reconcile (gradient mean, synchronized optimizer step,
parameter mean, SlowMo, copy-back), with the cadence decided on the host.
All state and the K per-step gradient buffers are resident in HBM before the
timed region starts (gradients stand in for the backward pass and are reused
period to period: the kernels' cost does not depend on the values).

Prints one JSON line.  value = replica-parameter updates per second over the
whole period (W * P * K / t_period).  The reconcile and local-step kernels are
also reported on their own (replica-params/s, algorithmic GB/s, fraction of
the 8 TB/s HBM peak), each kernel's duration measured with HIP events on the
stream it runs on.  cpu_baseline times the CPU oracle on a bounded sample of
the same workload on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published
MALL_EVICT_BYTES = 512 << 20  # twice the 256 MB MALL


def _code_only(text: str) -> str:
    """Source text without its comments and with whitespace runs collapsed:
    an edit to a comment or to the layout does not change a kernel."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    """Hash of the code that decides what the kernels read and write: the
    kernel translation units with their launch shapes and dispatch, the
    shared device code and the launch interface, comments and layout
    ignored.  (Host validation in cpdp_api.cpp does not change a kernel's
    traffic.)"""
    from paper_2607_21224_amd.build import KERNEL_HEADERS, KERNEL_SOURCES
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_21224_amd", "csrc")
    for f in (*KERNEL_SOURCES, *KERNEL_HEADERS):
        h.update(f.encode() + b"\0")
        h.update(_code_only(open(os.path.join(csrc, f)).read()).encode())
    return h.hexdigest()[:16]


def recorded_traffic(kernel: str, workload: str, variant: str = ""):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, or None when the kernel source changed since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}{variant}_pmc.txt")
    if not os.path.exists(path):
        return None
    m = re.search(r"^TRAFFIC_JSON: (\{.*\})$", open(path).read(), re.M)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


# optimizer descriptors of --optimizer, as bench.py passes them to the GPU path
OPTIMIZERS = {"sgd_wd": dict(kind="sgd", weight_decay=5e-4),
              "adamw": dict(kind="adamw", lr=5e-4, momentum=0.9, beta2=0.999, eps=1e-8,
                            weight_decay=0.05)}


def _oracle_slice(w, start: int, n: int, budget_s: float, method: str = "cpdp",
                  optimizer: str = "sgd") -> dict:
    """Whole periods of the oracle on coordinates [start, start + n) (mod P)
    until budget_s has elapsed, for the strategy and optimizer being
    benchmarked; returns counts and per-kind times."""
    import numpy as np
    import oracle
    from synth import gen

    idx = (start + np.arange(n)) % w.P
    f = lambda x: float(np.float32(x))  # noqa: E731
    lr, mu, beta, alpha = f(w.lr), f(w.mu), f(w.beta), f(w.alpha)
    th0 = gen.theta0(42, idx, w.theta_sigma).astype(np.float64)
    grads = [gen.grads(42, s, w.W, idx, w.grad_sigma, w.outlier_rate)
             for s in range(1, w.K + 1)]
    if w.grad_dt == "bf16":  # the stored bf16 values are the input
        grads = [gen.bf16_round(g) for g in grads]
    grads = [g.astype(np.float64) for g in grads]
    st = oracle.state_init(th0, w.W, w.param_dt, w.mom_dt)
    mom2 = np.zeros((w.W, n))
    o = OPTIMIZERS.get(optimizer)
    if o is None:
        make = None
    elif o["kind"] == "sgd":
        make = lambda t: oracle.sgd(lr, mu, f(o["weight_decay"]))  # noqa: E731
    else:
        make = lambda t: oracle.adamw(f(o["lr"]), f(o["momentum"]), f(o["beta2"]),  # noqa: E731
                                      f(o["eps"]), f(o["weight_decay"]), t)
    out = {"periods": 0, "rec_s": 0.0, "rec_n": 0, "loc_s": 0.0, "loc_n": 0}
    t_global = 0
    t0 = time.perf_counter()
    while True:
        for s in range(1, w.K + 1):
            t_global += 1
            g = grads[s - 1]
            sync = method == "ddp" or oracle.is_sync_step(s, w.K)
            c0 = time.perf_counter()
            if make is not None:
                if sync:
                    oracle.sync_opt(st, method, g, make(t_global), beta, alpha, mom2)
                else:
                    oracle.local_step_opt(st, g, make(t_global), mom2)
            elif not sync:
                oracle.local_step(st, g, lr, mu)
            elif method == "cpdp":
                oracle.reconcile(st, g, lr, mu, beta, alpha)
            elif method == "localsgd":
                oracle.localsgd_sync(st, g, lr, mu)
            else:
                oracle.ddp_step(st, g, lr, mu)
            dt = time.perf_counter() - c0
            key = "rec" if sync else "loc"
            out[key + "_s"] += dt
            out[key + "_n"] += 1
        out["periods"] += 1
        out["elapsed"] = time.perf_counter() - t0
        if out["elapsed"] >= budget_s:
            return out


def cpu_baseline(w, budget_s: float = 10.0, n_coords: int = 1 << 18,
                 parallel_budget_s: float = 5.0, method: str = "cpdp",
                 optimizer: str = "sgd") -> dict:
    """The oracle as it stands on the first n_coords coordinates of the
    workload (coordinates are independent), repeating whole periods until
    budget_s has elapsed, on one thread.  A second leg runs the same oracle
    on one independent coordinate slice per thread (ctypes releases the GIL),
    with as many threads as this process may use, capped at 16."""
    from concurrent.futures import ThreadPoolExecutor

    n = min(n_coords, w.P)
    r = _oracle_slice(w, 0, n, budget_s, method, optimizer)
    el = r["elapsed"]
    scale = w.P / n  # per-call seconds extrapolated to the whole workload
    out = {"value": w.W * n * w.K * r["periods"] / el, "unit": "replica-params/s",
           "cores": 1, "kind": "oracle",
           "sample": f"first {n} of {w.P} coordinates of {w.name}, W={w.W}, "
                     f"{r['periods']} periods of K={w.K} steps ({method}, {optimizer}), "
                     f"fp64 C oracle, 1 thread, "
                     f"{el:.1f} s",
           "s_per_reconcile_full_P": round(r["rec_s"] / max(r["rec_n"], 1) * scale, 4),
           "s_per_local_step_full_P": (round(r["loc_s"] / r["loc_n"] * scale, 4)
                                       if r["loc_n"] else None),
           "extrapolated": w.P > n}
    if parallel_budget_s > 0:
        threads = max(1, min(16, len(os.sched_getaffinity(0))))
        with ThreadPoolExecutor(threads) as ex:
            t0 = time.perf_counter()
            parts = list(ex.map(lambda k: _oracle_slice(w, k * n, n, parallel_budget_s,
                                                        method, optimizer),
                                range(threads)))
            wall = time.perf_counter() - t0
        done = sum(p["periods"] for p in parts)
        out["parallel"] = {"value": w.W * n * w.K * done / wall, "unit": "replica-params/s",
                           "cores": threads,
                           "sample": f"{threads} threads, each on its own {n}-coordinate "
                                     f"slice, {done} periods in {wall:.1f} s"}
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100, help="timed CPDP periods")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="r50_100")
    ap.add_argument("--method", default="cpdp", choices=["cpdp", "localsgd", "ddp"],
                    help="synchronisation strategy (Sec. 5.3); cpdp is the paper's method")
    ap.add_argument("--optimizer", default="sgd", choices=["sgd", "sgd_wd", "adamw"],
                    help="per-replica optimizer (Table 3): sgd = momentum SGD of the "
                         "workload; sgd_wd adds weight decay 5e-4; adamw = AdamW "
                         "(lr 5e-4, betas 0.9/0.999, eps 1e-8, weight decay 0.05)")
    ap.add_argument("--graph", action="store_true",
                    help="also replay the period as a captured HIP graph and time that: "
                         "with the scalars baked in (plain SGD) and with the scalars read "
                         "from a device step table (any optimizer); removes per-launch "
                         "host overhead, matters for small P")
    ap.add_argument("--plan", action="store_true",
                    help="hold the model as one allocation per (replica, tensor), as a "
                         "framework does, and drive it through a multi-tensor plan "
                         "(ResNet-50 / ViT-S tensor lists) instead of the flat buffer")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--grad-dtype", default="f32", choices=["f32", "bf16"],
                    help="gradient storage of the flat momentum-SGD path (bf16 halves the "
                         "gradient bytes; parameters keep the workload's type)")
    ap.add_argument("--mom-dtype", default="f32", choices=["f32", "bf16"],
                    help="momentum storage of the flat momentum-SGD path")
    ap.add_argument("--row-align-bytes", type=int, default=0,
                    help="round each replica row up to a multiple of this many bytes "
                         "(0 = the workload's default of 1 MiB)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the CPDP path runs on exactly one GPU; sharding the "
              "reconcile over several GPUs is not implemented "
              f"(asked for --gpus {args.gpus})", file=sys.stderr)
        return 2

    import torch
    from paper_2607_21224_amd.state import CpdpState, Hyper, Optimizer
    from synth import WORKLOADS
    from synth import device as sdev

    w = WORKLOADS[args.workload]
    if args.grad_dtype != "f32" or args.mom_dtype != "f32":
        if args.plan or args.graph or args.optimizer != "sgd":
            raise SystemExit("--grad-dtype / --mom-dtype bf16 run the flat momentum-SGD path "
                             "only (no --plan, --graph or --optimizer)")
        import dataclasses
        w = dataclasses.replace(w, grad_dt=args.grad_dtype, mom_dt=args.mom_dtype)
    if args.row_align_bytes:
        import dataclasses
        assert args.row_align_bytes % 256 == 0
        w = dataclasses.replace(w, row_align_bytes=args.row_align_bytes)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)  # default priority

    adamw = args.optimizer == "adamw"
    if args.plan and args.graph:
        raise SystemExit("--graph captures the flat-buffer path; drop --plan")
    st = None if args.plan else CpdpState(w.W, w.P, w.ld, w.K, w.param_dt, device=dev,
                                          grad_dt=w.grad_dt, mom_dt=w.mom_dt, adamw=adamw)
    h = Hyper.fp32(w.lr, w.mu, w.beta, w.alpha)
    with torch.cuda.stream(stream):
        th = torch.empty(w.P, dtype=torch.float32, device=dev)
        sdev.fill_theta0(th, w.P, 42, w.theta_sigma, stream=stream)
        if w.param_dt == "bf16":
            th = th.to(torch.bfloat16)
        grads = []
        for s in range(1, w.K + 1):
            g = torch.empty((w.W, w.ld), dtype=torch.float32, device=dev)
            sdev.fill_grads(g, w.P, 42, s, w.grad_sigma, w.outlier_rate, stream=stream)
            if w.grad_dt == "bf16":
                g = g.to(torch.bfloat16)  # round to nearest even
            grads.append(g)
        opt = None
        if args.optimizer != "sgd":
            o = dict(OPTIMIZERS[args.optimizer])
            kind = o.pop("kind")
            if kind == "sgd":  # the workload's learning rate and momentum, plus decay
                o.update(lr=h.lr, momentum=h.mu)
            opt = Optimizer(kind, **o)
        multi = None
        if args.plan:
            from paper_2607_21224_amd.multi import CpdpMultiState
            numels = [x for _, x in w.tensors]
            offs = [0]
            for x in numels:
                offs.append(offs[-1] + x)
            multi = CpdpMultiState(w.W, numels, w.K, w.param_dt, adamw, device=dev)
            multi.init([th[offs[t]:offs[t + 1]] for t in range(len(numels))], stream=stream)
            # one gradient set (step 1's) serves every step: the kernels' cost does not
            # depend on the values, and per-step copies would add traffic to the period
            for i in range(w.W):
                for t in range(len(numels)):
                    multi.grads[i][t][:numels[t]].copy_(grads[0][i, offs[t]:offs[t + 1]])
            if opt is None:
                opt = Optimizer("sgd", h.lr, h.mu)
        elif opt is None:
            st.init(th, stream=stream)
        else:
            st.init_opt(th, opt, stream=stream)
        # copy-kernel ceiling on a 4 GiB buffer pair (also the counter calibration)
        n_copy = 1 << 30
        csrc = torch.ones(n_copy, dtype=torch.float32, device=dev)
        cdst = torch.empty_like(csrc)
    torch.cuda.synchronize()

    def period(evs=None):
        for s in range(1, w.K + 1):
            e0 = e1 = None
            if evs is not None:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
            if multi is not None:
                kind = multi.step(s, opt, h.beta, h.alpha, 0, stream, method=args.method)
            elif opt is None:
                kind = st.step(s, grads[s - 1], h, 0, stream, method=args.method)
            else:
                kind = st.step_opt(s, grads[s - 1], opt, h.beta, h.alpha, 0, stream,
                                   method=args.method)
            if evs is not None:
                e1.record(stream)
                evs.append((kind, e0, e1))

    for _ in range(args.warmup):
        period()
    torch.cuda.synchronize()

    evs = []
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for _ in range(args.steps):
        period(evs)
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps

    dur = {"reconcile": [], "local": []}
    for kind, e0, e1 in evs:
        dur[kind].append(e0.elapsed_time(e1))
    sync_kernel = {"cpdp": "reconcile", "localsgd": "localsgd_sync", "ddp": "ddp_step"}[args.method]
    rec_ms = sum(dur["reconcile"]) / len(dur["reconcile"])
    loc_ms = sum(dur["local"]) / len(dur["local"]) if dur["local"] else None

    def spread(xs):
        xs = sorted(xs)
        return {"median_ms": round(xs[len(xs) // 2], 5), "min_ms": round(xs[0], 5),
                "max_ms": round(xs[-1], 5), "launches": len(xs)}

    # copy ceiling
    for _ in range(3):
        sdev.copy_f32(cdst, csrc, n_copy, stream=stream)
    c0 = torch.cuda.Event(enable_timing=True)
    c1 = torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    reps = 10
    for _ in range(reps):
        sdev.copy_f32(cdst, csrc, n_copy, stream=stream)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * 4 * n_copy * reps / (c0.elapsed_time(c1) * 1e-3) / 1e9

    def time_replays(graph):
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        g0 = torch.cuda.Event(enable_timing=True)
        g1 = torch.cuda.Event(enable_timing=True)
        g0.record()
        for _ in range(args.steps):
            graph.replay()
        g1.record()
        torch.cuda.synchronize()
        return g0.elapsed_time(g1) / args.steps

    graph_ms = graph_table_ms = None
    if args.graph:
        from paper_2607_21224_amd.state import StepTable
        if opt is None:
            # scalars baked into the graph (plain momentum SGD)
            graph, _ = st.capture_period(grads, h, method=args.method)
            graph_ms = time_replays(graph)
        # scalars from a device step table: every replay takes the next K entries
        topt = opt if opt is not None else Optimizer("sgd", h.lr, h.mu)
        n_entries = w.K * (args.warmup + args.steps)
        table = StepTable([(topt, st.opt_step + 1 + i, h.beta, h.alpha)
                           for i in range(n_entries)], device=dev)
        graph, _ = st.capture_steps(grads, table, method=args.method)
        graph_table_ms = time_replays(graph)
        assert table.position() == n_entries

    # cold variant for working sets the 256 MB MALL can hold: a 512 MB scratch
    # write (untimed, same stream) before every timed launch evicts the state
    cold = None
    if w.sync_bytes(args.method, adamw) < MALL_EVICT_BYTES:
        scratch = torch.empty(MALL_EVICT_BYTES // 4, dtype=torch.float32, device=dev)
        cev = []
        with torch.cuda.stream(stream):
            for rep in range(max(args.steps // 2, 5)):
                for s in range(1, w.K + 1):
                    scratch.fill_(float(rep))
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    if multi is not None:
                        kind = multi.step(s, opt, h.beta, h.alpha, 0, stream, method=args.method)
                    elif opt is None:
                        kind = st.step(s, grads[s - 1], h, 0, stream, method=args.method)
                    else:
                        kind = st.step_opt(s, grads[s - 1], opt, h.beta, h.alpha, 0, stream,
                                           method=args.method)
                    e1.record(stream)
                    cev.append((kind, e0, e1))
        torch.cuda.synchronize()
        del scratch
        cd = {"reconcile": [], "local": []}
        for kind, e0, e1 in cev:
            cd[kind].append(e0.elapsed_time(e1))
        cold = {"scratch_bytes_between_launches": MALL_EVICT_BYTES}
        for kind, name, nb in (("reconcile", sync_kernel, w.sync_bytes(args.method, adamw)),
                               ("local", "local_step", w.local_step_bytes(adamw))):
            if cd[kind]:
                med = sorted(cd[kind])[len(cd[kind]) // 2]
                cold[name] = {"median_ms": round(med, 5),
                              "GB_per_s": round(nb / (med * 1e-3) / 1e9, 1),
                              "frac_of_hbm_peak": round(nb / (med * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                              "launches": len(cd[kind])}

    rec_bytes = w.sync_bytes(args.method, adamw)
    loc_bytes = w.local_step_bytes(adamw)
    rec_gbps = rec_bytes / (rec_ms * 1e-3) / 1e9
    wp = w.W * w.P

    variant = "" if (args.method, args.optimizer) == ("cpdp", "sgd") else \
        f"_{args.method}_{args.optimizer}"
    if w.grad_dt == "bf16":
        variant += "_bf16grads"
    if w.mom_dt == "bf16":
        variant += "_bf16mom"
    if args.plan:
        variant += "_plan"

    def roofline(kernel, nbytes, ms):
        ach = nbytes / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                "traffic": recorded_traffic(kernel, w.name, variant),
                "kernel": kernel, "bytes_per_launch": nbytes,
                "avg_launch_ms": round(ms, 5),
                "frac_of_copy_ceiling": round(ach / copy_gbps, 4)}

    out = {
        "metric": "reconcile replica-params/s and achieved HBM GB/s (% of MI355X peak)",
        "value": wp * w.K / (ms_per_step * 1e-3),
        "unit": "replica-params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": ("f32" if (w.param_dt, w.grad_dt, w.mom_dt) == ("f32", "f32", "f32") else
                  f"{w.param_dt} params, {w.grad_dt} grads, {w.mom_dt} mom, f32 u/anchor"),
        "data": "synthetic",
        "config": {"workload": f"{w.name}: W={w.W} replicas, P={w.P} ({w.param_dt} params"
                               f"{', bf16 grads' if w.grad_dt == 'bf16' else ''}"
                               f"{', bf16 momentum' if w.mom_dt == 'bf16' else ''}), "
                               f"K={w.K}, lr={w.lr}, mu={w.mu}, beta={w.beta}, alpha={w.alpha}",
                   "W": w.W, "P": w.P, "ld": w.ld, "K": w.K, "grad_dt": w.grad_dt,
                   "mom_dt": w.mom_dt,
                   "method": args.method, "optimizer": args.optimizer,
                   "layout": (f"multi-tensor plan: {len(w.tensors)} tensors x {w.W} replicas, "
                              "one allocation each; step 1's gradients every step"
                              if args.plan else "flat buffer, one row per replica"),
                   "step": (f"{w.K} DDP steps (K=1 schedule), same gradients as a CPDP period"
                            if args.method == "ddp" else
                            f"one period: {w.K - 1} local steps + 1 {sync_kernel}")},
        "method": args.method,
        "sync_kernel": sync_kernel,
        sync_kernel: {"replica_params_per_s": wp / (rec_ms * 1e-3),
                      "GB_per_s": round(rec_gbps, 1),
                      "frac_of_hbm_peak": round(rec_gbps / HBM_PEAK_GBPS, 4),
                      "ms": round(rec_ms, 5), **spread(dur["reconcile"])},
        "local_step": None if loc_ms is None else {
            "replica_params_per_s": wp / (loc_ms * 1e-3),
            "GB_per_s": round(loc_bytes / (loc_ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(loc_bytes / (loc_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "ms": round(loc_ms, 5), **spread(dur["local"])},
        "roofline": roofline(sync_kernel, rec_bytes, rec_ms),
        "roofline_local_step": None if loc_ms is None else roofline("local_step", loc_bytes, loc_ms),
        "graph_replay": None if graph_ms is None else {
            "ms_per_step": round(graph_ms, 5),
            "replica_params_per_s": wp * w.K / (graph_ms * 1e-3)},
        "graph_replay_step_table": None if graph_table_ms is None else {
            "ms_per_step": round(graph_table_ms, 5),
            "replica_params_per_s": wp * w.K / (graph_table_ms * 1e-3)},
        "cold": cold,
        "copy_ceiling_GBps": round(copy_gbps, 1),
        "wall_s_timed_region": round(wall, 4),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_budget,
                                           parallel_budget_s=args.cpu_budget / 2,
                                           method=args.method, optimizer=args.optimizer)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
