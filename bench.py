#!/usr/bin/env python3
"""Benchmark of the CPDP reconcile hot path on one MI355X.

One timed step = one CPDP period over the workload: K-1 local momentum-SGD
steps and one fused reconcile (gradient mean, synchronized optimizer step,
parameter mean, SlowMo, copy-back), with the cadence decided on the host.
All state and the K per-step gradient buffers are resident in HBM before the
timed region starts (gradients stand in for the backward pass and are reused
period to period: the kernels' cost does not depend on the values).

Prints one JSON line.  value = replica-params/s of the synchronisation kernel
(W * P / t_reconcile for CPDP), the kernel the metric names; the whole period's
rate (W * P * K / t_period) is reported beside it.  The reconcile and
local-step kernels are each reported with replica-params/s, algorithmic GB/s
and the fraction of the 8 TB/s HBM peak, their durations measured with HIP
events on the stream they run on.  cpu_baseline times the CPU oracle on a
bounded sample of the same workload on this host.
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


def cpu_threads() -> dict:
    """Host cores the parallel oracle leg may use: the CPUs in this process's
    affinity set, capped by the CPU share the environment grants the job
    (OMP_NUM_THREADS, when set), with the counts behind the choice."""
    affinity = len(os.sched_getaffinity(0))
    share = os.environ.get("OMP_NUM_THREADS", "")
    cap = int(share) if share.isdigit() and int(share) > 0 else None
    used = min(affinity, cap) if cap else affinity
    return {"threads": max(1, used), "host_cpu_count": os.cpu_count(),
            "affinity_cpus": affinity, "omp_num_threads": cap}


def cpu_baseline(w, budget_s: float = 10.0, n_coords: int = 1 << 18,
                 parallel_budget_s: float = 5.0, method: str = "cpdp",
                 optimizer: str = "sgd") -> dict:
    """The oracle as it stands on bounded samples of the workload
    (coordinates are independent), repeating whole periods of the strategy
    and optimizer being benchmarked.  value is the oracle's rate on the
    synchronisation step the metric names (W * coordinates / seconds spent in
    it), summed over one independent n_coords slice per host thread on every
    core this job may use (cpu_threads(); ctypes releases the GIL during each
    oracle call).  A single-thread leg on the first n_coords coordinates
    gives the per-core rate and the per-call times extrapolated to the full P;
    both legs also report the whole-period rate."""
    from concurrent.futures import ThreadPoolExecutor

    n = min(n_coords, w.P)

    def rates(r):
        return (w.W * n * r["rec_n"] / r["rec_s"], w.W * n * w.K * r["periods"] / r["elapsed"])

    r = _oracle_slice(w, 0, n, budget_s, method, optimizer)
    scale = w.P / n  # per-call seconds extrapolated to the whole workload
    sync_rate, period_rate = rates(r)
    single = {"value": sync_rate, "unit": "replica-params/s", "cores": 1,
              "period_replica_params_per_s": period_rate,
              "sample": f"first {n} of {w.P} coordinates of {w.name}, W={w.W}, "
                        f"{r['periods']} periods of K={w.K} steps ({method}, {optimizer}), "
                        f"fp64 C oracle, 1 thread, {r['elapsed']:.1f} s",
              "s_per_reconcile_full_P": round(r["rec_s"] / max(r["rec_n"], 1) * scale, 4),
              "s_per_local_step_full_P": (round(r["loc_s"] / r["loc_n"] * scale, 4)
                                          if r["loc_n"] else None),
              "extrapolated": w.P > n}
    if parallel_budget_s <= 0:
        return {**single, "kind": "oracle"}
    ct = cpu_threads()
    threads = ct["threads"]
    with ThreadPoolExecutor(threads) as ex:
        t0 = time.perf_counter()
        parts = list(ex.map(lambda k: _oracle_slice(w, k * n, n, parallel_budget_s,
                                                    method, optimizer),
                            range(threads)))
        wall = time.perf_counter() - t0
    done = sum(p["periods"] for p in parts)
    return {"value": sum(rates(p)[0] for p in parts), "unit": "replica-params/s",
            "cores": threads, "kind": "oracle",
            "period_replica_params_per_s": w.W * n * w.K * done / wall,
            "sample": f"{threads} threads, each running whole periods of K={w.K} steps "
                      f"({method}, {optimizer}) of the fp64 C oracle on its own "
                      f"{n}-coordinate slice of {w.name} (W={w.W}); {done} periods in "
                      f"{wall:.1f} s; value sums each thread's rate over the time it spent "
                      f"in the synchronisation step",
            **{k: v for k, v in ct.items() if k != "threads"},
            "single_thread": single}


def sync_shape_rows(st, grads, method: str, adamw: bool):
    """The rows the synchronisation kernel of ``method`` reads and writes on
    the flat state, for the traffic-shape kernels, in the fixed table layout
    both take (gradient rows, then each replica's optimizer state and
    parameters, then the SlowMo state and anchor; LocalSGD: each replica's
    gradient, optimizer state and parameters).  Rows the kernel updates are
    written back in place; LocalSGD's anchor is written only."""
    from synth.device import ShapeRow
    W, ld = st.W, st.ld
    rows = [] if method == "localsgd" else [ShapeRow(grads, i * ld) for i in range(W)]
    for i in range(W):
        if method == "localsgd":
            rows.append(ShapeRow(grads, i * ld))
        rows.append(ShapeRow(st.mom, i * ld, write=True))
        if adamw:
            rows.append(ShapeRow(st.mom2, i * ld, write=True))
        rows.append(ShapeRow(st.params, i * ld, write=True))
    if method == "cpdp":
        rows += [ShapeRow(st.slow_mom, write=True), ShapeRow(st.anchor, write=True)]
    elif method == "localsgd":
        rows.append(ShapeRow(st.anchor, read=False))
    return rows


def time_launches(fn, stream, reps: int = 10, warmup: int = 3) -> float:
    """Average milliseconds of fn(stream) over reps back-to-back launches,
    HIP events on that stream."""
    import torch
    for _ in range(warmup):
        fn(stream)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def shape_probe(w, only=None, reps: int = 10) -> dict:
    """Bandwidth ceilings of traffic shapes, measured with the no-arithmetic
    shape kernel (synth/synth.hip) on fresh buffers sized like workload w:
      reconcile_rows*   the reconcile's exact rows in the library's layout
                        (W rows per family at stride ld) and its block shape
                        (64 threads), plain block order; blocks dealt to XCDs
                        in contiguous eighths; read batches of 16 instead of
                        8; blocks of 128 ... 1024 threads;
      reconcile_order   the same rows loaded and stored in the library's own
                        order (replica batches of 4, parameter stores last);
      reconcile_tile<T> the same rows and bytes in a coordinate-tile-major
                        layout: tile t holds coordinates [tT, (t+1)T) of every
                        row back to back (g_0..g_{W-1}, m_0, th_0, ..., u, a);
      <n>R<m>W          one row of P fp32 coordinates per stream: n rows read,
                        m written (in place on read rows first, then
                        write-only rows);
      full_*            read only, write only and copy over 4 GiB buffers.
    Returns {"workload", "results": [...]}; prints one line per shape to
    stderr as it finishes."""
    import torch
    from paper_2607_21224_amd.state import CpdpState
    from synth import device as sdev
    from synth.device import SYNC_ORDER_W, ShapePass, ShapeRow, ShapeSyncPass

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream(device=dev)
    W, P = w.W, w.P
    out = []

    def run(name, make_pass, note=""):
        if only and name not in only:
            return
        sp = make_pass()
        ms = time_launches(sp.launch, stream, reps)
        gbps = sp.bytes / (ms * 1e-3) / 1e9
        rec = {"name": name, "read_rows": sp.n_rd,
               "written_rows": sum(r.write for r in sp.keep_rows) + sp.n_wo,
               "bytes": sp.bytes, "ms": round(ms, 5), "GB_per_s": round(gbps, 1),
               "frac_of_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4), "note": note}
        out.append(rec)
        print(f"shape {name}: {gbps:.1f} GB/s ({ms:.4f} ms)", file=sys.stderr, flush=True)
        del sp

    # the reconcile's rows in the library's layout
    st = CpdpState(W, P, w.ld, w.K, w.param_dt, device=dev)
    st.params.zero_(); st.mom.zero_(); st.slow_mom.zero_(); st.anchor.zero_()
    g = torch.zeros((W, w.ld), dtype=torch.float32, device=dev)
    rows = sync_shape_rows(st, g, "cpdp", False)
    run("reconcile_rows", lambda: ShapePass(rows, P))
    if W in SYNC_ORDER_W:
        run("reconcile_order", lambda: ShapeSyncPass(rows, P, "cpdp", False, W),
            "the library's own load and store order (parameter stores last)")
    run("reconcile_rows_xcd", lambda: ShapePass(rows, P, xcd=True),
        "blocks in contiguous eighths per XCD")
    run("reconcile_rows_batch16", lambda: ShapePass(rows, P, batch=16))
    for th in (128, 256, 512, 1024):
        run(f"reconcile_rows_t{th}", lambda: ShapePass(rows, P, threads=th),
            f"blocks of {th} threads ({4 * th} coordinates)")
    del st, g, rows
    torch.cuda.empty_cache()

    # coordinate-tile-major layouts of the same rows (fp32 state only)
    if w.param_dt == "f32":
        R = 3 * W + 2
        written = [False] * W + [True] * (2 * W) + [True, True]
        for T in (1024, 2048, 4096):
            name = f"reconcile_tile{T}"
            if only and name not in only:
                continue
            tiles = (P + T - 1) // T
            buf = torch.zeros(tiles * R * T, dtype=torch.float32, device=dev)
            trows = [ShapeRow(buf, r * T, write=written[r]) for r in range(R)]
            run(name, lambda: ShapePass(trows, P, tile=T, tile_stride=R * T * 4),
                f"tiles of {T} coordinates, {R} row segments each")
            del buf, trows
            torch.cuda.empty_cache()

    # one row per stream
    ld = (P + (1 << 18) - 1) // (1 << 18) * (1 << 18)  # 1 MiB rows
    for n_inplace, n_ro, n_wo in ((0, 1, 0), (0, 0, 1), (0, 1, 1), (2, 1, 0), (1, 25, 0),
                                  (8, 0, 0), (18, 8, 0), (10, 16, 0), (1, 0, 17)):
        n = n_inplace + n_ro + n_wo
        name = f"{n_inplace + n_ro}R{n_inplace + n_wo}W"
        if only and name not in only:
            continue
        buf = torch.zeros((n, ld), dtype=torch.float32, device=dev)
        srows = ([ShapeRow(buf, i * ld, write=True) for i in range(n_inplace)] +
                 [ShapeRow(buf, (n_inplace + i) * ld) for i in range(n_ro)] +
                 [ShapeRow(buf, (n_inplace + n_ro + i) * ld, read=False) for i in range(n_wo)])
        run(name, lambda: ShapePass(srows, P),
            f"{n_inplace} in place, {n_ro} read only, {n_wo} write only")
        del buf, srows
        torch.cuda.empty_cache()

    # full size: 4 GiB streams
    n_big = 1 << 30
    if not only or any(x.startswith("full_") for x in only):
        a = torch.zeros(n_big, dtype=torch.float32, device=dev)
        b = torch.zeros(n_big, dtype=torch.float32, device=dev)
        for xcd in (0, 1):
            sfx = "_xcd" if xcd else ""
            run("full_read" + sfx, lambda: ShapePass([ShapeRow(a)], n_big, xcd=bool(xcd)))
            run("full_write" + sfx,
                lambda: ShapePass([ShapeRow(b, read=False)], n_big, xcd=bool(xcd)))
            run("full_copy" + sfx,
                lambda: ShapePass([ShapeRow(a), ShapeRow(b, read=False)], n_big, xcd=bool(xcd)))
        if not only or "full_copy_kernel" in only:
            ms = time_launches(lambda s: sdev.copy_f32(b, a, n_big, stream=s), stream, reps)
            gbps = 8 * n_big / (ms * 1e-3) / 1e9
            out.append({"name": "full_copy_kernel", "read_rows": 1, "written_rows": 1,
                        "bytes": 8 * n_big, "ms": round(ms, 5), "GB_per_s": round(gbps, 1),
                        "frac_of_hbm_peak": round(gbps / HBM_PEAK_GBPS, 4),
                        "note": "synth_copy_f32, the bench's copy ceiling"})
            print(f"shape full_copy_kernel: {gbps:.1f} GB/s", file=sys.stderr, flush=True)
        del a, b
    return {"shape_probe": w.name, "W": W, "P": P, "ld": w.ld, "reps": reps, "results": out}


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
    ap.add_argument("--shape-probe", action="store_true",
                    help="instead of the benchmark, measure the bandwidth ceilings of "
                         "traffic shapes with the no-arithmetic shape kernel: the "
                         "reconcile's rows in the library's layout and in coordinate-"
                         "tile-major layouts, single-row stream mixes, 4 GiB streams")
    ap.add_argument("--shape-only", default="",
                    help="comma-separated shape names of --shape-probe to run")
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
    if args.shape_probe:
        only = [x for x in args.shape_only.split(",") if x]
        print(json.dumps(shape_probe(w, only)), flush=True)
        return 0
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

    # copy ceiling: the faster of the plain copy kernel and the shape kernel's
    # one-read / one-write stream over the same 4 GiB buffers (the latter has
    # measured 1-3 % faster), each as the best of three batches of launches
    from synth.device import ShapePass, ShapeRow
    copy_pass = ShapePass([ShapeRow(csrc), ShapeRow(cdst, read=False)], n_copy)
    copies = {"synth_copy_f32": lambda s: sdev.copy_f32(cdst, csrc, n_copy, stream=s),
              "shape_1r1w": copy_pass.launch}
    copy_each = {k: 2 * 4 * n_copy / (min(time_launches(f, stream) for _ in range(3)) * 1e-3) / 1e9
                 for k, f in copies.items()}
    copy_gbps = max(copy_each.values())
    del copy_pass, csrc, cdst

    # traffic-shape ceiling: the synchronisation kernel's exact rows streamed
    # with no arithmetic (in place, the state keeps its bits), in two orders:
    # each batch of 8 rows written back right after it is read, and the
    # library's own order.  The ceiling is the faster, each order timed as the
    # best of three batches of launches.
    shape = None
    if multi is None:
        from synth.device import SYNC_ORDER_W, ShapePass, ShapeSyncPass
        srows = sync_shape_rows(st, grads[-1], args.method, adamw)
        passes = {"batched_in_place": ShapePass(srows, w.P)}
        if w.W in SYNC_ORDER_W:
            passes["library_order"] = ShapeSyncPass(srows, w.P, args.method, adamw, w.W)
        orders = {}
        for name, sp in passes.items():
            assert sp.bytes == w.sync_bytes(args.method, adamw), (sp.bytes, w.sync_bytes(args.method, adamw))
            ms = min(time_launches(sp.launch, stream) for _ in range(3))
            orders[name] = (sp.bytes / (ms * 1e-3) / 1e9, ms)
        best = max(orders, key=lambda k: orders[k][0])
        shape = {"GBps": orders[best][0], "ms": orders[best][1], "order": best,
                 "orders_GBps": {k: round(v[0], 1) for k, v in orders.items()},
                 "rows": f"{sp.n_rd} read ({sum(r.write for r in sp.keep_rows)} written back in "
                         f"place), {sp.n_wo} write-only"}
        del passes, srows

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

    roof_sync = roofline(sync_kernel, rec_bytes, rec_ms)
    if shape is not None:
        roof_sync["shape_ceiling_GBps"] = round(shape["GBps"], 1)
        roof_sync["frac_of_shape_ceiling"] = round(rec_gbps / shape["GBps"], 4)

    out = {
        "metric": "reconcile replica-params/s and achieved HBM GB/s (% of MI355X peak)",
        "value": wp / (rec_ms * 1e-3),
        "unit": "replica-params/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "period_replica_params_per_s": wp * w.K / (ms_per_step * 1e-3),
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
        "roofline": roof_sync,
        "roofline_local_step": None if loc_ms is None else roofline("local_step", loc_bytes, loc_ms),
        "graph_replay": None if graph_ms is None else {
            "ms_per_step": round(graph_ms, 5),
            "replica_params_per_s": wp * w.K / (graph_ms * 1e-3)},
        "graph_replay_step_table": None if graph_table_ms is None else {
            "ms_per_step": round(graph_table_ms, 5),
            "replica_params_per_s": wp * w.K / (graph_table_ms * 1e-3)},
        "cold": cold,
        "copy_ceiling_GBps": round(copy_gbps, 1),
        "copy_ceiling_streams_GBps": {k: round(v, 1) for k, v in copy_each.items()},
        "shape_ceiling": None if shape is None else {
            "GB_per_s": round(shape["GBps"], 1), "ms": round(shape["ms"], 5),
            "kernel": "synth shape kernels: the same rows, loads and in-place stores, no "
                      "arithmetic, in two orders (the faster one is the ceiling)",
            "order": shape["order"], "orders_GB_per_s": shape["orders_GBps"],
            "rows": shape["rows"]},
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
