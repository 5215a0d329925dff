#!/usr/bin/env python3
"""Benchmark of the DualGCN aggregation path on one MI355X.

A step is one pass of the whole path over one synthetic workload, inputs
already resident in HBM:
  c1        SpMM                                  (F = 16)
  c2,c3,c4  dual-metric partition + SpMM          (F = 64 / 128 / 128)
  c5        partition + 2 GCN layers (256 -> 128 -> 64); each layer is the update
            X W on the bf16 matrix cores then the SpMM, ReLU after layer 1; layer 1's
            update does not depend on the partition and runs on a second stream
            while the partition is built; layer 1 writes its output in bfloat16, which
            layer 2's update reads (bit-identical to a float32 intermediate)
Metric: edge-features per second, GE/s = sum over the step's SpMMs of nnz F / step time.

The JSON line also carries
  roofline      the dominant kernel, the F=128 SpMM (the F=64 one for c2, F=16 for c1),
                against 8 TB/s: algorithmic bytes
                B_min = 4(n+1) + 8 nnz + 4 n F (X once) + 4 or 2 n F (Y, float32 or
                bfloat16) + 4 n (order)
                per launch over its mean duration, timed with HIP events on its
                stream around every launch of it inside the timed steps;
                `traffic` is the bytes per launch from the rocprofv3 FETCH_SIZE /
                WRITE_SIZE summary under profiles/, copy-calibrated.  These counters see
                the memory side of the L2s (Infinity Cache hits included), so they are
                fabric bytes, an upper bound on HBM bytes; null when the kernel or plan
                sources, the workload or its graph differ from those of the counters;
  bandwidth     copy and read rates of a plain streaming kernel measured in the same run
                (what the memory system delivers, next to the nominal 8 TB/s);
  cpu_baseline  the CPU oracle, single-threaded, timed on a bounded sample of the same
                workload (each part's sample fraction stated), with the same oracle on
                all host cores as context;
  paper_context the paper's own speedups (RTX 3090), context only;
  phases_ms     mean milliseconds of each phase inside the timed steps;
  partition_alone_ms  (GCN workloads) median of three partitions built alone after the
                timed steps: inside a step the partition runs beside layer 1's update.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "SpMM GE/s (nnz·F/s) and achieved HBM GB/s vs peak, 1×MI355X"
COUNTER_SUMMARY = os.path.join(ROOT, "profiles", "spmm_c5_hbm_counters.md")
# the counted bytes of the SpMM depend on its kernels and on the plan the partition builds
# (processing order, tasks, split rows)
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2609_01983_amd", "csrc", f)
                  for f in ("spmm.hip", "partition.hip", "arw.hip", "internal.h")]
# The paper's own results (abstract, Sec. 4.1-4.2): average SpMM kernel speedups over
# three baselines on its 12 datasets.  Other hardware and workloads: context only.
PAPER_CONTEXT = {"speedup_vs_cusparse": 2.53, "speedup_vs_gnnadvisor": 3.8,
                 "speedup_vs_accel": 2.13, "range_full_dualgcn": [1.48, 6.4],
                 "hardware": "NVIDIA RTX 3090, Ubuntu 20.04, CUDA/NVCC 12.0",
                 "timing": "kernel time only (transfers and CPU preprocessing excluded)",
                 "workloads": "12 real graphs, F = 16..128 (not available here)",
                 "note": "context only: relative speedups on other hardware, not a target"}


def spmm_bytes(n, nnz, F, ybytes=4):
    """B_min of one SpMM launch: row pointers, (column, value) pairs, X once, Y once, order."""
    return 4 * (n + 1) + 8 * nnz + 4 * n * F + ybytes * n * F + 4 * n


def fused_bytes(n, nnz, F_in, F_out):
    """B_min of one aggregation fused with the next update: row pointers, (column, value)
    pairs, X once, T (float32, F_out wide) once, order; W is negligible."""
    return 4 * (n + 1) + 8 * nnz + 4 * n * F_in + 4 * n * F_out + 4 * n


def gather_classes(info, n, F):
    """Does an SpMM of F-wide rows on this plan read cold rows non-temporally?  The
    library's rule: the plan marked its cold columns, the rows fill whole lines (F > 16),
    and the operand is larger than the 256 MiB memory-side cache and below 4 GiB."""
    return bool(info.get("cold_marked")) and F > 16 and 4 * n * F <= 0xFFFFFFFF and 4 * n * F > (256 << 20)


def kernel_source_hash():
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def counter_traffic(workload, kernel, run=None, path=None):
    """Bytes per launch of `kernel` from the committed counter summary, if it was taken on
    the same sources, workload and graph.  `run` holds the run's graph_sha256, F_in, F_out,
    walks_per_node and walk_len; every one must match the summary's line of that name."""
    path = path or COUNTER_SUMMARY
    if not os.path.exists(path):
        return None, "no counter summary"
    text = open(path).read()
    m_w = re.search(r"^workload: (\S+)", text, re.M)
    m_k = re.search(r"^kernel: (.+)$", text, re.M)
    m_t = re.search(r"^traffic_bytes_per_launch: (\d+)", text, re.M)
    m_h = re.search(r"^kernel_source_sha256: ([0-9a-f]{64})", text, re.M)
    if not (m_w and m_t and m_h) or m_w.group(1) != workload:
        return None, "no counters for this workload"
    if not m_k or m_k.group(1).strip() != kernel:
        return None, "no counters for this kernel"
    if m_h.group(1) != kernel_source_hash():
        return None, "kernel or plan sources changed since the counters were taken"
    for key, want in (run or {}).items():
        m = re.search(rf"^{key}: (\S+)", text, re.M)
        if not m or m.group(1) != str(want):
            return None, f"counters taken with another {key}"
    return int(m_t.group(1)), ("rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated: memory-side "
                               "fabric bytes (Infinity Cache hits included), an upper bound on "
                               "HBM bytes")


def _grow(fn, total, first, budget_s):
    """Runs fn(size) on samples of growing size until one takes >= budget_s (or covers
    `total`); returns (seconds, size) of the last run."""
    size = min(first, total)
    while True:
        t0 = time.perf_counter()
        fn(size)
        dt = time.perf_counter() - t0
        if dt >= budget_s or size >= total:
            return dt, size
        size = min(total, max(size * 2, int(size * budget_s / max(dt, 1e-3) * 1.2)))


def host_cores():
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def _on_threads(fn, items, threads):
    """fn over chunks of `items` on `threads` worker threads (the oracle's C calls release the
    interpreter lock); returns the wall time."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    chunks = [c for c in np.array_split(items, threads * 4) if c.size]
    t0 = time.perf_counter()
    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(fn, chunks))
    return time.perf_counter() - t0


def cpu_baseline(w, g, X, weights, part_budget_s=2.5):
    """Times the oracle on bounded random samples of each part of one step and scales every
    part to the whole workload by its sample fraction (stated per part).  The same samples
    are also run on all host cores (the single-threaded oracle on chunks from worker
    threads), as context."""
    import numpy as np
    import oracle
    gen = np.random.default_rng(7)
    threads = max(1, min(16, host_cores()))
    parts = []

    def part(name, unit, size, total, dt, dt_mt):
        parts.append({"part": name, "sample": int(size), "total": int(total), "unit": unit,
                      "fraction": round(size / total, 6), "seconds": round(dt, 4),
                      "seconds_all_cores": round(dt_mt, 4),
                      "est_seconds": round(dt * total / size, 4),
                      "est_seconds_all_cores": round(dt_mt * total / size, 4)})

    if w.name != "c1":
        order = gen.permutation(g.n).astype(np.int32)
        dt, ns = _grow(lambda s: oracle.density_sums(g, 0, w.walks, w.steps, order[:s]),
                       g.n, 2000, part_budget_s)
        dt_mt = _on_threads(lambda c: oracle.density_sums(g, 0, w.walks, w.steps, c),
                            order[:ns], threads)
        part("walks (density sums)", "nodes", ns, g.n, dt, dt_mt)
        # keys, threshold and sort of every node: plain numpy and Python integers, whole
        # (sums of the right size stand in for the walks' S)
        S = gen.integers(w.walks, w.walks * (w.steps + 1) + 1, g.n).astype(np.uint32)
        t0 = time.perf_counter()
        K = oracle.hybrid_keys(S, oracle.degrees(g), w.walks)
        S1, S2 = oracle.moments(K)
        oracle.threshold_key(g.n, S1, S2)
        np.lexsort((np.arange(g.n), K))
        dt = time.perf_counter() - t0
        part("keys, threshold and sort (stand-in S)", "nodes", g.n, g.n, dt, dt)
    rp = np.asarray(g.rowptr, dtype=np.int64)
    layers = w.layers if w.is_gcn else ((None, w.F),)
    for li, (fin, fout) in enumerate(layers):
        rows_all = gen.permutation(g.n).astype(np.int32)
        if fin is not None:
            Wl = weights[li]
            # the layer's input has the shape of X's first fin columns (a stand-in)
            Xin = X if fin == X.shape[1] else np.ascontiguousarray(X[:, :fin])
            dt, nr = _grow(lambda s: oracle.xw(Xin, Wl, rows_all[:s]), g.n, 500,
                           part_budget_s / 2)
            dt_mt = _on_threads(lambda c: oracle.xw(Xin, Wl, c), rows_all[:nr], threads)
            del Xin
            part(f"layer {li + 1}: X W (stand-in input)", "rows", nr, g.n, dt, dt_mt)
            T = np.ascontiguousarray(X[:, :fout])   # a stand-in of the layer's SpMM input shape
        else:
            T = X
        nnz_of = {}

        def run_spmm(s):
            rows = rows_all[:s]
            nnz_of[s] = int((rp[rows + 1] - rp[rows]).sum())
            oracle.spmm(g, T, rows)

        dt, nr = _grow(run_spmm, g.n, 500, part_budget_s / 2)
        dt_mt = _on_threads(lambda c: oracle.spmm(g, T, c), rows_all[:nr], threads)
        part(f"layer {li + 1}: SpMM" if w.is_gcn else "SpMM", "entries", nnz_of[nr], g.nnz,
             dt, dt_mt)
        del T
    ge = g.nnz * sum(fo for _, fo in layers)
    est = sum(p["est_seconds"] for p in parts)
    est_mt = sum(p["est_seconds_all_cores"] for p in parts)
    measured = sum(p["seconds"] for p in parts)
    desc = "; ".join(f"{p['part']}: {p['sample']} of {p['total']} {p['unit']} "
                     f"({100 * p['fraction']:.2f}%)" for p in parts)
    return {"value": ge / est / 1e9, "unit": "GE/s", "cores": 1, "kind": "oracle",
            "sample": "single-threaded C oracle on random samples of the same workload, each part "
                      "scaled to the whole by its sample fraction: " + desc,
            "measured_cpu_seconds": round(measured, 3), "est_step_s": round(est, 3),
            "parts": parts,
            "all_cores": {"value": ge / est_mt / 1e9, "unit": "GE/s", "cores": threads,
                          "est_step_s": round(est_mt, 3),
                          "how": f"the same oracle on {threads} threads over node and row chunks "
                                 "of the same samples (context)"}}


def bandwidth(dg, torch, dev, stream, gib=2, reps=5):
    """Copy and read rates of dualgcn_bandwidth_probe over `gib` GiB (median of reps)."""
    import numpy as np
    src = torch.ones((gib << 28,), dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    out = {}
    for name, kind, moved in (("copy", dg.PROBE_COPY, 2), ("read", dg.PROBE_READ, 1)):
        ms = []
        for _ in range(reps + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            dg.bandwidth_probe(kind, src, dst)
            b.record(stream)
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        t = float(np.median(ms[1:]))
        out[f"{name}_GBps"] = round(moved * src.numel() * 4 / (t * 1e-3) / 1e9, 1)
    del src, dst
    out["bytes"] = gib << 30
    out["how"] = ("dualgcn_bandwidth_probe: copy counts bytes read + written, read the bytes "
                  "read; median of %d" % reps)
    out["frac_of_peak"] = {"copy": round(out["copy_GBps"] / PEAK_HBM_GBS, 4),
                           "read": round(out["read_GBps"] / PEAK_HBM_GBS, 4)}
    return out


# Partition variants of the ablation: the paper's dual metric, its degree-only analogue
# (the baseline partitioning of the paper's DualGCN_0 experiment), density only, and a
# single path for every row, the adaptive weight (each metric's share of the spread) and
# the balanced weight (both terms of H spread alike, so that density can move the split).
ABLATION = [("dual-metric alpha=1/2", (1, 2), "auto"),
            ("dual-metric adaptive alpha", (0xFFFFFFFF, 1024), "auto"),
            ("dual-metric balanced alpha", (0xFFFFFFFE, 1024), "auto"),
            ("degree only alpha=0", (0, 1), "auto"),
            ("density only alpha=1", (1, 1), "auto"),
            ("all rows sparse path", (1, 2), "sparse"),
            ("all rows dense path", (1, 2), "dense")]


def block_stats(g, perm, K, np, blocks=1024):
    """Partition-quality statistics of the paper's objective (Sec. 3.2): cut the sorted order
    into `blocks` contiguous blocks and report the work imbalance max/avg of the blocks'
    entries (Theorem 2's measure) and the sum of the within-block variances of H (in
    key units, and as a share of blocks x the variance of all keys), next to the same for
    blocks of consecutive node ids."""
    deg = np.diff(g.rowptr.astype(np.int64))
    Kf = K.astype(np.float64)
    total_var = float(Kf.var())
    out = {}
    for name, order in (("sorted", perm.astype(np.int64)), ("node_id", np.arange(g.n))):
        edges = np.linspace(0, g.n, blocks + 1).astype(np.int64)
        work = np.add.reduceat(deg[order], edges[:-1])
        kk = Kf[order]
        s1 = np.add.reduceat(kk, edges[:-1])
        s2 = np.add.reduceat(kk * kk, edges[:-1])
        cnt = np.diff(edges)
        var = s2 / cnt - (s1 / cnt) ** 2
        within = float(np.maximum(var, 0).sum())
        out[name] = {"imbalance_max_over_avg": round(float(work.max() / work.mean()), 2),
                     "sum_block_var_K": within,
                     # unit-free: the share of the key's variance left inside the blocks
                     # (comparable across weights alpha, whose keys have other units)
                     "within_block_var_share": round(within / (blocks * total_var), 6)
                                               if total_var > 0 else 0.0}
    out["blocks"] = blocks
    return out


def ablation(args, w, g, dg, torch, np, rowptr, col, val, Xd, F_dom, stream, ev):
    """Times partition and the dominant SpMM for each variant; prints one JSON line each."""
    X = Xd if not w.is_gcn else torch.randn((g.n, F_dom), dtype=torch.float32, device=Xd.device,
                                            generator=torch.Generator(device=Xd.device).manual_seed(0))
    Y = torch.empty(X.shape, dtype=torch.bfloat16 if w.is_gcn else torch.float32, device=X.device)
    for name, alpha, force in ABLATION:
        part_ms, spmm_ms = [], []
        for rep in range(args.warmup + args.steps):
            a, b = ev(), ev()
            a.record(stream)
            plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps,
                           alpha=alpha, force_mode=force)
            b.record(stream)
            c, d = ev(), ev()
            c.record(stream)
            dg.spmm(plan, X, Y, relu=w.is_gcn, out_bf16=w.is_gcn)
            d.record(stream)
            torch.cuda.synchronize()
            if rep >= args.warmup:
                part_ms.append(a.elapsed_time(b))
                spmm_ms.append(c.elapsed_time(d))
            info = plan.info()
            if rep == args.warmup + args.steps - 1:
                plan_perm, _, plan_K = plan.export()
            plan.destroy()
        ms = float(np.mean(spmm_ms))
        stats = block_stats(g, plan_perm, plan_K, np)
        print(json.dumps({"ablation": name, "workload": w.name, "F": F_dom,
                          "alpha": [info["alpha_num"], info["alpha_den"]],
                          "force_mode": force, "n_sparse": info["n_sparse"],
                          "n_dense": info["n_dense"], "kstar": info["kstar"],
                          "partition_ms": round(float(np.mean(part_ms)), 4),
                          "spmm_ms": round(ms, 4), "block_stats": stats,
                          "spmm_ge_s": round(g.nnz * F_dom / (ms * 1e-3) / 1e9, 2),
                          "spmm_hbm_frac_bmin": round(spmm_bytes(g.n, g.nnz, F_dom, 2 if w.is_gcn else 4)
                                                      / (ms * 1e-3) / (PEAK_HBM_GBS * 1e9), 4),
                          "walks_per_node": w.walks, "walk_len": w.steps}), flush=True)


def train(args, w, g, dg, torch, np, rowptr, col, val, Xd, Wd, stream, ev):
    """GCN training steps on one plan (the partition is amortised over the epochs, Sec. 3.2):
    forward with bfloat16 intermediates, softmax cross-entropy on 10% labeled rows,
    backward (A^T = A: the same plan), SGD on every weight.  One JSON line."""
    from graphgen import dense
    if not w.is_gcn:
        raise SystemExit("--mode train needs a GCN workload")
    dev = Xd.device
    L = len(w.layers)
    C = w.layers[-1][1]
    labels = torch.from_numpy(dense.labels(g.n, C, seed=0, labeled_fraction=0.1)).to(dev)
    scale = 1.0 / max(1, int((labels >= 0).sum().item()))
    plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
    # The loss gradient is zero on unlabeled rows, so the last layer's backward aggregation
    # A^T G = A G (A symmetric) only needs the entries whose column is labeled: a second
    # plan of that column-restricted matrix, built once like the first (labels are fixed).
    plan_lab, nnz_lab = None, None
    if not args.full_backward:
        keep = (labels >= 0)[col.long()]
        cum = torch.cat([torch.zeros(1, dtype=torch.int64, device=dev), torch.cumsum(keep.long(), 0)])
        rowptr_lab = cum[rowptr.long()].to(torch.int32)
        col_lab, val_lab = col[keep].contiguous(), val[keep].contiguous()
        nnz_lab = int(col_lab.numel())
        plan_lab = dg.Plan(rowptr_lab, col_lab, val_lab, seed=0, walks_per_node=w.walks,
                           walk_len=w.steps)
        del keep, cum
    # Likewise the loss reads the last layer's output on labeled rows only: a plan of the
    # row-restricted matrix (unlabeled rows empty, so their outputs are zeros) serves it.
    plan_out, nnz_out = None, None
    if not args.full_forward:
        deg = (rowptr[1:] - rowptr[:-1]).long() * (labels >= 0).long()
        rowptr_out = torch.cat([torch.zeros(1, dtype=torch.int64, device=dev),
                                torch.cumsum(deg, 0)]).to(torch.int32)
        keep = torch.repeat_interleave(labels >= 0, (rowptr[1:] - rowptr[:-1]).long())
        col_out, val_out = col[keep].contiguous(), val[keep].contiguous()
        nnz_out = int(col_out.numel())
        plan_out = dg.Plan(rowptr_out, col_out, val_out, seed=0, walks_per_node=w.walks,
                           walk_len=w.steps)
        del keep, deg
    # Both consumers of the input features (layer 1's update and its weight gradient) round
    # them to bfloat16 (nearest-even) before the matrix cores; the features do not change
    # between epochs, so one bfloat16 copy, made once like the plans, halves what both read
    # and gives the same bits (torch's conversion is nearest-even too).
    X_in = Xd if args.x_fp32 else Xd.to(torch.bfloat16)
    Ws = [W.clone() for W in Wd]
    T = [torch.empty((g.n, fo), dtype=torch.float32, device=dev) for _, fo in w.layers]
    H = [torch.empty((g.n, fo), dtype=torch.bfloat16 if li < L - 1 else torch.float32, device=dev)
         for li, (_, fo) in enumerate(w.layers)]
    G = torch.empty((g.n, C), dtype=torch.float32, device=dev)
    loss = torch.empty(dg.LOSS_SLOTS, dtype=torch.float64, device=dev)
    dT = [torch.empty((g.n, fo), dtype=torch.bfloat16, device=dev) for _, fo in w.layers]
    dH = [torch.empty((g.n, fo), dtype=torch.float32, device=dev) for _, fo in w.layers[:-1]]
    dW = [torch.empty_like(W) for W in Ws]
    ws = torch.empty(max(dg.weight_grad_workspace_bytes(g.n, fi, fo) for fi, fo in w.layers),
                     dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()

    def step():
        marks = {}

        def mark(name, fn):
            a, b = ev(), ev()
            a.record(stream)
            fn()
            b.record(stream)
            marks.setdefault(name, []).append((a, b))

        inp = [X_in] + H[:-1]
        for li in range(L):
            fplan = plan_out if (li == L - 1 and plan_out is not None) else plan
            if li == 0 or args.unfused:
                mark("forward_update", lambda: dg.update(inp[li], Ws[li], T[li]))
            if li < L - 1 and not args.unfused:
                # aggregation fused with the next layer's update; H[li] is kept for the backward
                mark("forward_spmm", lambda: dg.spmm_update(fplan, T[li], Ws[li + 1], T[li + 1],
                                                            relu=True, H=H[li]))
            else:
                mark("forward_spmm", lambda: dg.spmm(fplan, T[li], H[li], relu=li < L - 1,
                                                     out_bf16=li < L - 1))
        mark("loss", lambda: dg.softmax_xent(H[-1], labels, scale, G, loss))
        grad = G
        for li in range(L - 1, -1, -1):
            bplan = plan_lab if (li == L - 1 and plan_lab is not None) else plan
            mark("backward_spmm", lambda: dg.spmm(bplan, grad, dT[li], out_bf16=True))
            if li > 0:          # dX before the step changes W
                mark("backward_data", lambda: dg.backward_data(dT[li], Ws[li], H[li - 1], dH[li - 1]))
            mark("weight_grad_sgd", lambda: dg.weight_grad(inp[li], dT[li], dW[li], args.lr, Ws[li], ws))
            if li > 0:
                grad = dH[li - 1]
        return marks

    losses = []
    for _ in range(args.warmup):
        step()
        losses.append(loss[0].item())
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    all_marks = []
    for _ in range(args.steps):
        all_marks.append(step())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    losses.append(loss[0].item())
    phases = {}
    for m in all_marks:
        for k, v in m.items():
            phases[k] = phases.get(k, 0.0) + sum(a.elapsed_time(b) for a, b in v)
    ms = elapsed * 1e3 / args.steps
    aggregated = 2 * g.nnz * sum(fo for _, fo in w.layers)      # forward + backward SpMMs
    print(json.dumps({"mode": "train", "workload": w.desc, "config": w.name, "n": g.n,
                      "nnz": g.nnz, "layers": w.layers, "steps": args.steps, "warmup": args.warmup,
                      "ms_per_step": round(ms, 4),
                      "spmm_ge_s": round(aggregated / (ms * 1e-3) / 1e9, 1),
                      "phases_ms": {k: round(v / args.steps, 4) for k, v in phases.items()},
                      "labeled_rows": int((labels >= 0).sum().item()), "lr": args.lr,
                      "loss_first": losses[0], "loss_last": losses[-1],
                      "last_backward": ("column-restricted plan of the labeled rows, nnz %d" % nnz_lab
                                        if plan_lab is not None else "full plan"),
                      "last_forward": ("row-restricted plan of the labeled rows, nnz %d" % nnz_out
                                       if plan_out is not None else "full plan"),
                      "fused_update": not args.unfused,
                      "input_features": "float32" if args.x_fp32 else "bfloat16 copy made once",
                      "note": "partition built once before the timed steps (amortised over epochs)"}),
          flush=True)
    plan.destroy()
    for p in (plan_lab, plan_out):
        if p is not None:
            p.destroy()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default=os.environ.get("DUALGCN_BENCH_CONFIG", "c5"))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--spmm-reps", type=int, default=20)
    ap.add_argument("--mode", choices=["full", "spmm", "train", "planio"], default="full",
                    help="spmm: one partition, then only the dominant SpMM launches (for counter "
                         "runs); train: GCN training steps on one plan (forward, loss, backward, SGD)")
    ap.add_argument("--cold", action="store_true",
                    help="--mode spmm: write 512 MiB between launches so that every launch starts "
                         "with caches that hold none of its data")
    ap.add_argument("--lr", type=float, default=0.5, help="SGD step of --mode train")
    ap.add_argument("--pipeline", action="store_true",
                    help="GCN workloads: build the next step's partition on a second stream while "
                         "this step's updates and SpMMs run")
    ap.add_argument("--full-forward", action="store_true",
                    help="--mode train: compute the last layer's output on every row instead of "
                         "the labeled rows the loss reads")
    ap.add_argument("--full-backward", action="store_true",
                    help="--mode train: aggregate the loss gradient with the full plan instead of "
                         "the plan restricted to labeled columns")
    ap.add_argument("--unfused", action="store_true",
                    help="GCN steps: layer 1's aggregation and layer 2's update as two calls "
                         "(by default one, dualgcn_spmm_update); --mode spmm: time the plain SpMM")
    ap.add_argument("--x-fp32", action="store_true",
                    help="--mode train: layer 1's update and weight gradient read the float32 "
                         "features (by default a bfloat16 copy made once, with the same results)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 1 GiB device to device (a dispatch of known traffic)")
    ap.add_argument("--ablation", action="store_true",
                    help="time partition + dominant SpMM for each partition variant (one JSON line each)")
    ap.add_argument("--walks", type=int, default=None, help="walks per node (default: the workload's)")
    ap.add_argument("--walk-len", type=int, default=None, help="steps per walk (default: the workload's)")
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
    if args.walks is not None or args.walk_len is not None:
        import dataclasses
        w = dataclasses.replace(w, walks=args.walks or w.walks, steps=args.walk_len or w.steps)
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
    F_dom = w.layers[0][1] if w.is_gcn else w.F      # width of the dominant SpMM
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
        plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
        Xs = torch.randn((g.n, F_dom), dtype=torch.float32, device=dev) if w.is_gcn else Xd
        fused_w = not args.unfused and w.is_gcn and len(w.layers) > 1
        if fused_w:
            F_next = w.layers[1][1]
            Ys = torch.empty((g.n, F_next), dtype=torch.float32, device=dev)
        else:
            Ys = torch.empty(Xs.shape, dtype=torch.bfloat16 if w.is_gcn else torch.float32, device=dev)
        # --cold: 512 MiB written between launches (outside the timed events), so that
        # neither the L2s nor the 256 MiB MALL hold anything of the previous launch
        flush = torch.empty(1 << 27, dtype=torch.float32, device=dev) if args.cold else None
        times = []
        for _ in range(args.spmm_reps):
            if flush is not None:
                flush.fill_(float(len(times)))
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            if fused_w:
                dg.spmm_update(plan, Xs, Wd[1], Ys, relu=True)
            else:
                dg.spmm(plan, Xs, Ys, relu=w.is_gcn, out_bf16=w.is_gcn)
            b.record(stream)
            times.append((a, b))
        torch.cuda.synchronize()
        ms = [a.elapsed_time(b) for a, b in times]
        print(json.dumps({"mode": "spmm", "config": w.name, "F": F_dom, "fused_update": fused_w,
                          "caches": "cold" if args.cold else "warm",
                          "ms": [round(x, 4) for x in ms], "median_ms": round(float(np.median(ms)), 4),
                          "bytes_min": (fused_bytes(g.n, g.nnz, F_dom, F_next) if fused_w else
                                        spmm_bytes(g.n, g.nnz, F_dom, 2 if w.is_gcn else 4))}),
              flush=True)
        plan.destroy()
        return

    ev = lambda: torch.cuda.Event(enable_timing=True)
    if args.mode == "train":
        train(args, w, g, dg, torch, np, rowptr, col, val, Xd, Wd, stream, ev)
        return
    if args.mode == "planio":
        # partition against save + load of the same plan (wall clock, synchronised)
        times = {"partition": [], "save": [], "load": []}
        for rep in range(args.warmup + args.steps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            blob = plan.save()
            t2 = time.perf_counter()
            loaded = dg.Plan.load(rowptr, col, val, blob)
            torch.cuda.synchronize()
            t3 = time.perf_counter()
            if rep >= args.warmup:
                times["partition"].append(t1 - t0)
                times["save"].append(t2 - t1)
                times["load"].append(t3 - t2)
            loaded.destroy()
            plan.destroy()
        print(json.dumps({"mode": "planio", "config": w.name, "saved_bytes": len(blob),
                          **{k + "_ms": round(float(np.mean(v)) * 1e3, 3) for k, v in times.items()}}),
              flush=True)
        return
    if args.ablation:
        ablation(args, w, g, dg, torch, np, rowptr, col, val, Xd, F_dom, stream, ev)
        return
    if w.is_gcn:
        # every layer but the last writes its output in bfloat16: the next update rounds its
        # input to bfloat16 anyway, so the final output is bit-identical (tested)
        Ts = [torch.empty((g.n, fo), dtype=torch.float32, device=dev) for _, fo in w.layers]
        Hs = [torch.empty((g.n, fo), dtype=torch.bfloat16 if li < len(w.layers) - 1 else torch.float32,
                          device=dev) for li, (_, fo) in enumerate(w.layers)]
    else:
        Y = torch.empty_like(Xd)
    holder = {"plan": None}
    if w.name == "c1":      # c1 is one SpMM per step on a fixed plan
        holder["plan"] = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks,
                                 walk_len=w.steps)

    side = torch.cuda.Stream(device=dev)    # default priority, like the main stream
    pipelined = args.pipeline and w.is_gcn
    if pipelined:
        # the partition of step k + 1 is built on the side stream while step k's updates and
        # SpMMs run; the first one is built before the warm-up
        holder["next"] = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks,
                                 walk_len=w.steps, stream=side)

    fused = not args.unfused and w.is_gcn

    def layers(plan, marks, first):
        """Layers `first`.. of the GCN on the main stream (layer 1's update, if first > 0,
        is already in Ts[0]).  With `fused`, a layer's aggregation and the next layer's
        update are one call that never stores the layer's output."""
        for li in range(first, len(w.layers)):
            fout = w.layers[li][1]
            if li > 0 and not fused:
                a, b = ev(), ev()
                a.record(stream)
                dg.update(Hs[li - 1], Wd[li], Ts[li])
                b.record(stream)
                marks[f"update_{li + 1}"] = [(a, b)]
            last = li == len(w.layers) - 1
            a, b = ev(), ev()
            a.record(stream)
            if fused and not last:
                dg.spmm_update(plan, Ts[li], Wd[li + 1], Ts[li + 1], relu=True)
            else:
                dg.spmm(plan, Ts[li], Hs[li], relu=not last, out_bf16=not last)
            b.record(stream)
            marks[f"spmm_{li + 1}_F{fout}"] = [(a, b)]

    def step_pipelined():
        marks = {}
        plan = holder["next"]
        a, b = ev(), ev()
        a.record(stream)
        dg.update(Xd, Wd[0], Ts[0])
        b.record(stream)
        marks["update_1"] = [(a, b)]
        layers(plan, marks, 0)
        a, b = ev(), ev()
        a.record(side)
        holder["next"] = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks,
                                 walk_len=w.steps, stream=side)
        b.record(side)
        marks["partition"] = [(a, b)]
        if holder["plan"] is not None:
            holder["plan"].destroy()              # waits for this step's work
        holder["plan"] = plan
        return marks

    def step():
        """Enqueues one step; returns {phase: [(start, end) events]}."""
        if pipelined:
            return step_pipelined()
        marks = {}
        if w.is_gcn:
            # layer 1's update needs no plan: it runs on a second stream while the
            # partition is built, once the previous step is done with its buffers
            side.wait_stream(stream)
            a, b = ev(), ev()
            a.record(side)
            dg.update(Xd, Wd[0], Ts[0], stream=side)
            b.record(side)
            marks["update_1"] = [(a, b)]
            upd1_done = b
        if w.name != "c1":
            a, b = ev(), ev()
            a.record(stream)
            plan = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
            b.record(stream)
            marks["partition"] = [(a, b)]
            if holder["plan"] is not None:
                holder["plan"].destroy()
            holder["plan"] = plan
        plan = holder["plan"]
        if w.is_gcn:
            stream.wait_event(upd1_done)
            layers(plan, marks, 0)
        else:
            a, b = ev(), ev()
            a.record(stream)
            dg.spmm(plan, Xd, Y)
            b.record(stream)
            marks[f"spmm_1_F{w.F}"] = [(a, b)]
        return marks

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    all_marks = []
    t_start = time.perf_counter()
    for _ in range(args.steps):
        all_marks.append(step())
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed * 1e3 / args.steps

    phases = {}
    for marks in all_marks:
        for k, lst in marks.items():
            phases.setdefault(k, []).extend(a.elapsed_time(b) for a, b in lst)
    dom_key = f"spmm_1_F{F_dom}"
    spmm_ms = float(np.mean(phases[dom_key]))
    info = holder["plan"].info()
    if holder.get("next") is not None:
        holder["next"].destroy()

    ge_per_step = g.nnz * (sum(fo for _, fo in w.layers) if w.is_gcn else w.F)
    value = ge_per_step / (ms_per_step * 1e-3) / 1e9
    lpr = min(64, max(1, 1 << max(0, (F_dom - 1).bit_length() - 2)))
    cp = "true" if gather_classes(info, g.n, F_dom) else "false"
    if fused:
        # the dominant kernel is layer 1's aggregation with layer 2's update fused in: it
        # writes T (float32, F_next wide) instead of the layer's output
        F_next = w.layers[1][1]
        out_bytes = 4 * g.n * F_next
        bmin = fused_bytes(g.n, g.nnz, F_dom, F_next)
        kname = f"spmm_xw_kernel<{lpr}, {cp}>"
        kdesc = f"{kname} (F={F_dom} -> {F_next}, ReLU, fused update)"
    else:
        out_bytes = (2 if w.is_gcn else 4) * g.n * F_dom   # every layer but the last: bfloat16
        bmin = spmm_bytes(g.n, g.nnz, F_dom, 2 if w.is_gcn else 4)
        kname = f"spmm_dual_kernel<{lpr}, 4, {'true' if w.is_gcn else 'false'}, {cp}>"
        kdesc = f"{kname} (F={F_dom}{', ReLU, bfloat16 output' if w.is_gcn else ''})"
    achieved = bmin / (spmm_ms * 1e-3) / 1e9
    run_keys = {"graph_sha256": g.sha256()[:16], "F_in": F_dom,
                "F_out": w.layers[1][1] if fused else F_dom,
                "walks_per_node": w.walks, "walk_len": w.steps}
    traffic, traffic_src = counter_traffic(w.name, kname, run_keys)
    roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
            "kernel": kdesc,
            "bytes_per_launch": bmin, "ms_per_launch": round(spmm_ms, 4),
            "launches_timed": len(phases[dom_key]),
            "traffic_unit": "bytes per launch", "traffic_source": traffic_src,
            "gather_bytes_per_launch": 4 * (g.n + 1) + 8 * g.nnz + 4 * g.nnz * F_dom
                                       + out_bytes + 4 * g.n,
            "spmm_ge_s": round(g.nnz * F_dom / (spmm_ms * 1e-3) / 1e9, 2)}
    if traffic is not None:
        # the counted bytes over the same launch time: the rate at which the kernel moves data
        # through the memory side of the L2s (Infinity Cache hits included), where B_min counts
        # every X row once.  Not a roofline fraction: it counts bytes the kernel need not move.
        roof["fabric_GBps"] = round(traffic / (spmm_ms * 1e-3) / 1e9, 1)
        roof["fabric_unit"] = ("memory-side fabric bytes per second (FETCH_SIZE + WRITE_SIZE, "
                               "Infinity Cache hits included, copy-calibrated)")
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
                   "seed": 0, "graph_sha256": g.sha256()[:16],
                   "parallelism": "single GPU",
                   "fused_update": bool(fused),
                   "steps_overlap": ("partition of the next step beside this step's updates and SpMMs"
                                     if pipelined else "layer-1 update beside the partition")},
        "roofline": roof,
        "bandwidth": None,
        "host_cores": host_cores(),
        "paper_context": PAPER_CONTEXT,
        "phases_ms": {k: round(float(np.mean(v)), 4) for k, v in phases.items()},
        "plan": {"n_sparse": info["n_sparse"], "n_dense": info["n_dense"],
                 "kstar": info["kstar"], "n_tasks": info["n_tasks"],
                 "n_split_rows": info["n_split_rows"], "n_split_parts": info["n_split_parts"]},
    }
    if w.name == "c4":
        # the workload names a hub degree above 10^5; the seeded R-MAT draw reaches a little less
        out["config"]["max_degree_stated"] = "> 1e5"
        out["config"]["max_degree_note"] = (f"the generated graph's largest row has {g.max_degree()} "
                                            "entries, below the stated > 1e5")
    holder["plan"].destroy()
    if w.is_gcn and not pipelined:
        # inside the step the partition shares the memory fabric with layer 1's update;
        # built alone (after the timed steps, outside them) it shows its own cost
        alone = []
        for _ in range(3):
            a, b = ev(), ev()
            a.record(stream)
            pl = dg.Plan(rowptr, col, val, seed=0, walks_per_node=w.walks, walk_len=w.steps)
            b.record(stream)
            torch.cuda.synchronize()
            alone.append(a.elapsed_time(b))
            pl.destroy()
        out["partition_alone_ms"] = round(float(np.median(alone)), 4)
    out["bandwidth"] = bandwidth(dg, torch, dev, stream)
    if not args.no_cpu_baseline:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(w, g, X, weights)
        print(f"[bench] cpu baseline {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
