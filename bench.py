#!/usr/bin/env python3
"""Benchmark of the DualGCN aggregation path on one MI355X.

A step is one pass of the whole path over one synthetic workload, inputs
already resident in HBM:
  c1        SpMM                                  (F = 16)
  c2,c3,c4  dual-metric partition + SpMM          (F = 64 / 128 / 128)
  c5        partition + 2 GCN layers, each X W on the bf16 matrix cores then SpMM,
            ReLU between (256 -> 128 -> 64)
Metric: edge-features per second, GE/s = sum over the step's SpMMs of nnz F / step time.

The JSON line also carries
  roofline      the SpMM kernel (dominant HBM kernel) against 8 TB/s: algorithmic bytes
                B_min = 4(n+1) + 8 nnz + 4 n F (X once) + 4 n F (Y) + 4 n (perm) per
                launch over its mean duration, timed with HIP events on its stream;
  cpu_baseline  the CPU oracle timed on a bounded sample of the same workload;
  phases        mean milliseconds of partition / X W / SpMM inside the timed steps.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "SpMM GE/s (nnz·F/s) and achieved HBM GB/s vs peak, 1×MI355X"


def spmm_bytes(n, nnz, F):
    return 4 * (n + 1) + 8 * nnz + 4 * n * F + 4 * n * F + 4 * n


def xw_bytes(n, fin, fout):
    return 4 * n * fin + 4 * n * fout


def cpu_baseline(cfg, g, X, weights, budget_s=12.0):
    """Time the oracle on a bounded random sample and scale to one whole step."""
    import numpy as np
    import oracle
    w = cfg
    gen = np.random.default_rng(7)
    rp = g.rowptr.astype(np.int64)
    t_total = 0.0
    parts = []
    # walks: sample nodes, scale by n / sample
    if w.name != "c1":
        ns = min(g.n, 20000)
        nodes = gen.choice(g.n, ns, replace=False).astype(np.int32)
        t0 = time.perf_counter()
        oracle.density_sums(g, 0, w.walks, w.steps, nodes)
        dt = time.perf_counter() - t0
        t_total += dt * g.n / ns
        parts.append(f"walks of {ns} nodes")
        # keys, exact threshold and sort: on the full node count with sampled-size keys
        S = gen.integers(w.walks, w.walks * (w.steps + 1) + 1, g.n).astype(np.uint32)
        t0 = time.perf_counter()
        K = oracle.hybrid_keys(S, oracle.degrees(g), w.walks)
        S1, S2 = oracle.moments(K)
        oracle.threshold_key(g.n, S1, S2)
        np.lexsort((np.arange(g.n), K))
        t_total += time.perf_counter() - t0
        parts.append("keys/threshold/sort of all nodes")
    # per layer: X W on sampled rows (scaled by n / rows) and the SpMM of sampled rows
    # (scaled by nnz / sampled nnz); the SpMM input of a GCN layer is a stand-in of
    # the same shape (the first F_out columns of X)
    layers = w.layers if w.is_gcn else ((None, w.F),)
    for li, (fin, fout) in enumerate(layers):
        rows = gen.choice(g.n, min(g.n, 4000), replace=False).astype(np.int32)
        nnz_s = int((rp[rows + 1] - rp[rows]).sum())
        if fin is not None:
            xin = np.ascontiguousarray(X[rows, :fin])
            t0 = time.perf_counter()
            oracle.xw(xin, weights[li])
            t_total += (time.perf_counter() - t0) * g.n / rows.size
            T = np.ascontiguousarray(X[:, :fout])
        else:
            T = X
        t0 = time.perf_counter()
        oracle.spmm(g, T, rows)
        t_total += (time.perf_counter() - t0) * g.nnz / max(nnz_s, 1)
        del T
        parts.append(f"layer {li}: SpMM of {rows.size} rows ({nnz_s} nnz)"
                     + (f", X W of {rows.size} rows" if fin is not None else ""))
    ge = g.nnz * sum(fo for _, fo in layers)
    return {"value": ge / t_total / 1e9, "unit": "GE/s", "cores": 1, "kind": "oracle",
            "sample": "single-threaded C oracle; " + "; ".join(parts) +
                      "; each part scaled to the whole workload",
            "est_step_s": round(t_total, 3)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=os.environ.get("DUALGCN_BENCH_CONFIG", "c5"))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--spmm-reps", type=int, default=20)
    ap.add_argument("--mode", choices=["full", "spmm"], default="full",
                    help="spmm: one partition, then only the SpMM launches (for counter runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 1 GiB device to device (a dispatch of known traffic)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2609_01983_amd as dg
    from graphgen import configs

    w = configs.WORKLOADS[args.config]
    t0 = time.time()
    g = configs.load_graph(w.name)
    X = configs.load_features(w.name)
    weights = configs.load_weights(w.name)
    print(f"[bench] {w.name}: n={g.n} nnz={g.nnz} maxdeg={g.max_degree()} F={w.F} "
          f"inputs {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    dev = torch.device("cuda:0")
    rowptr = torch.from_numpy(g.rowptr).to(dev)
    col = torch.from_numpy(g.col).to(dev)
    val = torch.from_numpy(g.val).to(dev)
    Xd = torch.from_numpy(X).to(dev)
    Wd = [torch.from_numpy(W).to(dev) for W in weights]
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    if args.copy_calibration:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)                     # reads 1 GiB, writes 1 GiB
        torch.cuda.synchronize()
        del src, dst
        print("[bench] copy calibration: 1073741824 bytes read + written", file=sys.stderr,
              flush=True)
    if args.mode == "spmm":
        F_spmm = w.layers[0][1] if w.is_gcn else w.F
        plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
        Xs = Xd[:, :F_spmm].contiguous() if w.is_gcn else Xd
        Ys = torch.empty_like(Xs)
        times = []
        for _ in range(args.spmm_reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            dg.spmm(plan, Xs, Ys)
            b.record(stream)
            times.append((a, b))
        torch.cuda.synchronize()
        ms = [a.elapsed_time(b) for a, b in times]
        print(json.dumps({"mode": "spmm", "config": w.name, "F": F_spmm,
                          "ms": [round(x, 4) for x in ms],
                          "bytes_min": spmm_bytes(g.n, g.nnz, F_spmm)}), flush=True)
        plan.destroy()
        return

    if w.is_gcn:
        fouts = [fo for _, fo in w.layers]
        Hs = [torch.empty((g.n, fo), dtype=torch.float32, device=dev) for fo in fouts]
        ws_bytes = max(4 * g.n * fo + 2 * fi * fo + 256 for fi, fo in w.layers)
    else:
        Y = torch.empty_like(Xd)

    ev = lambda: torch.cuda.Event(enable_timing=True)
    phase_ms = {"partition": [], "xw_spmm": [], "spmm": []}
    kernel_ms = []

    plan_holder = {}

    def step(timed):
        e0, e1 = ev(), ev()
        e0.record(stream)
        plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
        e1.record(stream)
        if plan_holder.get("plan") is not None:
            plan_holder["plan"].destroy()
        plan_holder["plan"] = plan
        if w.name == "c1":
            e0.record(stream)   # c1 is one SpMM per step; the partition is not part of it
        if w.is_gcn:
            x = Xd
            layer_ev = []
            for li, (fin, fout) in enumerate(w.layers):
                a, b = ev(), ev()
                a.record(stream)
                dg.gcn_layer(plan, x, Wd[li], relu=li < len(w.layers) - 1, Y=Hs[li],
                             workspace=ws)
                b.record(stream)
                layer_ev.append((a, b))
                x = Hs[li]
            if timed:
                torch.cuda.synchronize()
                phase_ms["partition"].append(e0.elapsed_time(e1))
                phase_ms["xw_spmm"].append(sum(a.elapsed_time(b) for a, b in layer_ev))
        else:
            a, b = ev(), ev()
            a.record(stream)
            dg.spmm(plan, Xd, Y)
            b.record(stream)
            if timed:
                torch.cuda.synchronize()
                if w.name != "c1":
                    phase_ms["partition"].append(e0.elapsed_time(e1))
                phase_ms["spmm"].append(a.elapsed_time(b))

    if w.is_gcn:
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)

    if w.name == "c1":
        plan_holder["plan"] = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks,
                                      walk_len=w.steps)

        def step(timed):  # noqa: F811 -- c1: one SpMM per step on a fixed plan
            a, b = ev(), ev()
            a.record(stream)
            dg.spmm(plan_holder["plan"], Xd, Y)
            b.record(stream)
            if timed:
                torch.cuda.synchronize()
                phase_ms["spmm"].append(a.elapsed_time(b))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed * 1e3 / args.steps

    # SpMM kernel alone on the last plan, HIP events on its stream (the roofline figure)
    plan = plan_holder["plan"]
    F_spmm = w.layers[0][1] if w.is_gcn else w.F
    Xs = torch.randn((g.n, F_spmm), dtype=torch.float32, device=dev) if w.is_gcn else Xd
    Ys = torch.empty_like(Xs)
    for _ in range(3):
        dg.spmm(plan, Xs, Ys)
    for _ in range(args.spmm_reps):
        a, b = ev(), ev()
        a.record(stream)
        dg.spmm(plan, Xs, Ys)
        b.record(stream)
        kernel_ms.append((a, b))
    torch.cuda.synchronize()
    spmm_ms = float(np.mean([a.elapsed_time(b) for a, b in kernel_ms]))
    info = plan.info()

    ge_per_step = g.nnz * (sum(fo for _, fo in w.layers) if w.is_gcn else w.F)
    value = ge_per_step / (ms_per_step * 1e-3) / 1e9
    bmin = spmm_bytes(g.n, g.nnz, F_spmm)
    achieved = bmin / (spmm_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "GE/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+bf16mfma" if w.is_gcn else "f32",
        "data": "synthetic (seeded generators, no datasets)",
        "config": {"workload": w.desc, "name": w.name, "n": g.n, "nnz": g.nnz,
                   "max_degree": g.max_degree(), "F": w.F, "walks_per_node": w.walks,
                   "walk_len": w.steps, "layers": [list(l) for l in w.layers],
                   "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "kernel": f"spmm_dual_kernel (F={F_spmm})",
                     "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                     "bytes_per_launch": bmin, "ms_per_launch": round(spmm_ms, 4),
                     "spmm_ge_s": round(g.nnz * F_spmm / (spmm_ms * 1e-3) / 1e9, 2)},
        "phases_ms": {k: round(float(np.mean(v)), 4) for k, v in phase_ms.items() if v},
        "plan": {"n_sparse": info["n_sparse"], "n_dense": info["n_dense"],
                 "kstar": info["kstar"], "n_split_rows": info["n_split_rows"],
                 "n_split_parts": info["n_split_parts"]},
    }
    if not args.no_cpu_baseline:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(w, g, X, weights)
        print(f"[bench] cpu baseline {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    plan.destroy()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
