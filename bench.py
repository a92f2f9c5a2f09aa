"""Benchmark: one partition's DIGEST GCN rounds on one MI355X.

A step is one round r of Algorithm 1 for the partition: every layer's
forward (with the pull / push the schedule asks for in that round), the loss
head, and every layer's backward, all in libdigest.so, replayed from HIP
graphs with inputs resident in HBM.  Default workload: the
OGB-Products-shaped synthetic graph (2,450,000 nodes in 8 blocks,
partition 0 with 306,250 owned rows, GCN 100 -> 256 -> 256 -> 47, sync
interval 10), the largest workload that one GPU holds as one partition.

    python bench.py [--steps K] [--warmup W] [--config NAME] [--sync N]

Prints one JSON line: whole-round throughput in GTEPS (aggregation edges of
the forward and backward per round / time), the roofline of the dominant
kernel (from a second, instrumented pass with HIP events on the launch
stream; its algorithmic bytes and flops come from the library's own launch
plan, digest_profile_model) and the CPU oracle timed on a bounded sample on
this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from types import SimpleNamespace

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GCN layer fwd+bwd GTEPS on one partition; % of HBM / MFMA roofline"
METRIC_GAT = "GAT layer fwd+bwd GTEPS on one partition; % of HBM / MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
# Edges of the single-thread oracle sample per round (a leading block of the
# partition's rows), so that one sampled round takes a few seconds.
CPU_SAMPLE_EDGES = 2_000_000
# Edges per round above which the all-core oracle leg also runs on a row
# sample (a whole round of the largest partitions takes minutes on a host).
CPU_FULL_ROUND_EDGES = 100_000_000


def measured_traffic(workload, key):
    """(bytes per launch, source) of `key` from the committed counter
    summary: L2-to-fabric bytes (rocprofv3 FETCH_SIZE + WRITE_SIZE, each
    scaled by a plain copy kernel of known size; Infinity Cache hits are
    included, so this is not HBM traffic alone).  (None, reason) when there
    is no summary for this kernel or the kernel sources changed since.
    The summaries of a workload are profiles/<workload>_*traffic.txt, one
    kernel (or a list of launches of one kernel) each."""
    import glob
    found = None
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", f"{workload}_*traffic.txt"))):
        kv = {}
        for line in open(path):
            line = line.split("#", 1)[0].strip()
            if "=" in line:
                k, v = line.split("=", 1)
                kv[k.strip()] = v.strip()
        if key in [k.strip() for k in kv.get("kernel", "").split(",")]:
            found = (os.path.relpath(path, ROOT), kv)
            break
    if found is None:
        return None, f"no counter summary of {key} for {workload}"
    rel, kv = found
    from paper_2206_00057_amd.pmc import kernel_source_hash
    sha = kernel_source_hash()
    if kv.get("source_sha") != sha:
        return None, f"{rel} was taken on kernel sources {kv.get('source_sha')}, now {sha}"
    return (float(kv["traffic_bytes_per_launch"]),
            f"{rel}: rocprofv3 FETCH_SIZE+WRITE_SIZE (L2-fabric bytes, Infinity Cache hits "
            f"included), kernel sources {sha}")


def row_sample(part, rows):
    """The first `rows` owned rows of a partition as a partition of their
    own: the same CSR rows, every column that is not one of those rows
    becoming a halo node (ascending id)."""
    rows = min(int(rows), int(part.n_own))
    indptr = np.ascontiguousarray(part.indptr[:rows + 1])
    nnz = int(indptr[-1])
    indices = np.ascontiguousarray(part.indices[:nnz])
    owned = np.ascontiguousarray(part.owned[:rows])
    halo = np.setdiff1d(np.unique(indices), owned)
    return SimpleNamespace(indptr=indptr, indices=indices,
                           values=np.ascontiguousarray(part.values[:nnz]), owned=owned,
                           halo=halo, n_own=rows, n_halo=int(halo.shape[0]),
                           nnz_in=int(np.isin(indices, owned).sum()), nnz=nnz)


def round_edges(part, L, gat):
    """Aggregation edges of one round: GCN forward nnz per layer plus the
    transposed backward's nnz_in for layers >= 2; GAT 2 nnz per layer."""
    return 2 * L * part.nnz if gat else L * part.nnz + (L - 1) * part.nnz_in


def cpu_rounds(cfg, g, part, X, Ws, y, K, budget_s, atts=None):
    """The oracle as it stands, timed on whole rounds of `part` (GCN layers,
    or GAT layers when atts are given) until budget_s has passed (at least
    one round).  Returns (rounds, seconds, threads)."""
    import oracle
    L = cfg.layers
    op = oracle.OraclePartition(g.n, part.indptr, part.indices, part.values, part.owned,
                                part.halo, cfg.widths)
    # stale store levels: synthetic values on the rows this partition pulls
    stores = [X]
    for l in range(1, L):
        st = np.zeros((g.n, cfg.widths[l]), np.float32)
        st[part.halo] = np.maximum(np.random.default_rng(70 + l).standard_normal(
            (part.halo.shape[0], cfg.widths[l]), dtype=np.float32), 0)
        stores.append(st)
    for lev in range(L):
        op.pull(lev, stores[lev])
    x = X[part.owned]
    y = y[:part.n_own]
    t0 = time.perf_counter()
    rounds = 0
    while True:
        rounds += 1
        do_pull, do_push = oracle.sync_period(K, rounds)
        h, outs = x, []
        for l in range(1, L + 1):
            if do_pull and l >= 2:
                op.pull(l - 1, stores[l - 1])
            act = oracle.RELU if l < L else oracle.IDENTITY
            if atts is not None:
                outs.append((h, op.gat_forward(l, h, Ws[l - 1], atts[l - 1], act)))
            else:
                outs.append((h, op.forward(l, h, Ws[l - 1], act)))
            h = outs[-1][1]
            if do_push and l < L:
                op.push(l, h, stores[l])
        _, dh = oracle.softmax_xent(h, y)
        for l in range(L, 0, -1):
            act = oracle.RELU if l < L else oracle.IDENTITY
            if atts is not None:
                _, _, dh = op.gat_backward(l, outs[l - 1][0], Ws[l - 1], atts[l - 1],
                                           outs[l - 1][1], dh, act, want_dh_in=l > 1)
            else:
                _, dh = op.backward(l, outs[l - 1][0], Ws[l - 1], outs[l - 1][1], dh, act,
                                    want_dh_in=l > 1)
        if time.perf_counter() - t0 >= budget_s:
            break
    return rounds, time.perf_counter() - t0, oracle.num_threads()


def cpu_baseline(cfg, g, part, X, Ws, y, K, budget_s, atts=None):
    """The oracle on this host's cores: whole rounds of the partition on
    every thread (of a leading row sample when a round is too large to time
    in seconds), and a smaller leading row sample on one thread."""
    import oracle
    gat = atts is not None
    L = cfg.layers
    full = SimpleNamespace(**{k: getattr(part, k) for k in
                              ("indptr", "indices", "values", "owned", "halo", "n_own",
                               "n_halo")}, nnz=int(part.indptr[-1]),
                           nnz_in=int(np.isin(part.indices, part.owned).sum()))
    e_full = round_edges(full, L, gat)

    def leg(target_edges, budget):
        if e_full <= target_edges:
            smp, what = full, f"whole rounds of the partition ({full.n_own:,} rows)"
        else:
            rows = max(1, int(full.n_own * target_edges / e_full))
            smp = row_sample(full, rows)
            what = (f"whole rounds of its first {smp.n_own:,} owned rows as a partition "
                    f"({smp.n_halo:,} halo rows)")
        nr, secs, thr = cpu_rounds(cfg, g, smp, X, Ws, y, K, budget, atts)
        e = round_edges(smp, L, gat)
        return {"value": e * nr / secs / 1e9, "unit": "GTEPS", "cores": thr, "kind": "oracle",
                "sample": f"{nr} x {e:,} edges: {what}, {secs:.1f}s, float64 oracle, "
                          f"{thr} thread{'s' if thr != 1 else ''}"}

    out = leg(CPU_FULL_ROUND_EDGES, budget_s)
    threads = out["cores"]
    oracle.set_num_threads(1)
    try:
        one = leg(CPU_SAMPLE_EDGES, budget_s / 2)
    finally:
        oracle.set_num_threads(threads)
    out["single_thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample")}
    return out


# What each synthetic workload stands in for (the datasets of the paper's
# experiments, Table 3 of the appendix).
WORKLOADS = {
    "tiny": "small block graph",
    "medium": "Flickr-shaped graph",
    "dense": "Reddit-shaped graph",
    "large": "OGB-Products-shaped graph",
    "halo": "OGB-Products-shaped graph, random 1/16 partition",
}


def workload_name(cfg, K, model, n, st):
    """Workload key and sync interval first, then the shape; under 120
    characters."""
    parts = "16" if cfg.partition == "perm" else str(cfg.blocks)
    head = f"{cfg.name}, K={K}: {WORKLOADS[cfg.name]}, N={n:,}, part 0 of {parts}"
    tail = f"{model.upper()} {'-'.join(map(str, cfg.widths))}"
    full = f"{head} ({st['n_own']:,} own, {st['n_halo']:,} halo), {tail}"
    return full if len(full) < 120 else f"{head}, {tail}"[:119]


def train_bench(args):
    """Algorithm 1 over every subgraph of the workload's graph on this GPU:
    whole rounds (all subgraphs' forward, loss and backward, scheduled
    pulls/pushes, parameter averaging) replayed from HIP graphs."""
    import torch

    from paper_2206_00057_amd import synth
    from paper_2206_00057_amd.train import DigestTrainer

    cfg = synth.CONFIGS[args.config]
    K = args.sync or cfg.sync_periods[-1 if args.config == "halo" else 0]
    t0 = time.time()
    g = synth.make_graph(cfg)
    M = synth.num_partitions(cfg)
    parts = [synth.make_partition(cfg, g, m) for m in range(M)]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    X, y, Ws = synth.features(cfg), synth.labels(cfg), synth.weights(cfg)
    gat = args.model == "gat"
    atts = [dev(a) for a in synth.attentions(cfg)] if gat else None
    tr = DigestTrainer(g.n, parts, cfg.widths, dev(X), dev(y), [dev(w) for w in Ws],
                       args.lr, K, grad_exchange=args.grad_exchange, model=args.model, atts=atts)
    print(f"[bench] training {cfg.name}: {M} subgraphs, inputs {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    tr.init_stores()
    tr.capture()
    for r in range(1, args.warmup + 1):
        tr.replay(r)
    torch.cuda.synchronize()
    first_loss = tr.mean_loss()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for r in range(args.warmup + 1, args.warmup + args.steps + 1):
        tr.replay(r)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    out = {
        "metric": f"DIGEST {args.model.upper()} training GTEPS, all subgraphs of the graph on one GPU",
        "value": round(tr.edges_per_round * args.steps / (ms * 1e-3) / 1e9, 4), "unit": "GTEPS",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms / args.steps, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{cfg.name}, K={K}, all {M} subgraphs: {WORKLOADS[cfg.name]}, "
                               f"{args.model.upper()} {'-'.join(map(str, cfg.widths))}, "
                               f"exchange {args.grad_exchange}",
                   "lr": args.lr,
                   "n_global": g.n, "subgraphs": M, "widths": list(cfg.widths),
                   "edges_per_round": tr.edges_per_round, "launch": "hip-graph replay"},
        "loss": {"after_warmup": round(first_loss, 6), "last": round(tr.mean_loss(), 6)},
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="large", choices=tuple(WORKLOADS))
    ap.add_argument("--sync", type=int, default=0, help="sync interval (default: the workload's)")
    ap.add_argument("--eager", action="store_true", help="launch eagerly instead of graph replay")
    ap.add_argument("--overlap-io", action="store_true",
                    help="pulls and pushes on a second stream next to the layers")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="before the rounds, copy a float32 buffer of this many MiB once "
                         "(a plain copy kernel of known size for counter calibration)")
    ap.add_argument("--model", default="gcn", choices=("gcn", "gat"),
                    help="layer type: the GCN layer of Eq. 5 or the GAT layer over stale halo "
                         "rows")
    ap.add_argument("--train", action="store_true",
                    help="Algorithm 1 rounds over every subgraph of the graph instead of one")
    ap.add_argument("--lr", type=float, default=0.1, help="SGD learning rate for --train")
    ap.add_argument("--grad-exchange", default="none", choices=("none", "fresh", "stale"),
                    help="--train: exchange the halo gradients P_out^T D W^T between "
                         "subgraphs (same round or one round late)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one partition on one GPU; runs on more than one GPU are not "
              "implemented (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    if args.train:
        return train_bench(args)

    import torch

    from paper_2206_00057_amd import digest as D
    from paper_2206_00057_amd import step, synth

    cfg = synth.CONFIGS[args.config]
    K = args.sync or cfg.sync_periods[-1 if args.config == "halo" else 0]
    t0 = time.time()
    g = synth.make_graph(cfg)
    part = synth.make_partition(cfg, g, 0)
    st = synth.shape_stats(cfg, g, part)
    X, Ws, y = synth.features(cfg), synth.weights(cfg), synth.labels(cfg)[part.owned]
    print(f"[bench] workload {cfg.name}: {st} (inputs {time.time() - t0:.1f}s)",
          file=sys.stderr, flush=True)

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    L = cfg.layers
    dX, dWs, dy = dev(X), [dev(w) for w in Ws], dev(y)
    gat = args.model == "gat"
    atts = synth.attentions(cfg) if gat else None
    datts = [dev(a) for a in atts] if gat else None
    # stores initialised by one full-graph forward at the initial weights (library, no halo)
    full = step.GpuPartition(g.n, synth.extract_partition(g, np.arange(g.n)), cfg.widths,
                             model=args.model, atts=datts)
    full.forward(dX, dWs)
    stores = [dX] + [full.H[l].clone() for l in range(1, L)]
    del full
    torch.cuda.synchronize()
    gp = step.GpuPartition(g.n, part, cfg.widths, overlap_io=args.overlap_io, model=args.model,
                           atts=datts)
    x_own = dev(X[part.owned])
    gp.pull_all(stores)
    if args.calibration_copy_mib:
        n_cal = args.calibration_copy_mib * (1 << 20) // 4
        src_cal = torch.ones(n_cal, device="cuda")
        dst_cal = torch.empty_like(src_cal)
        torch.cuda.synchronize()
        dst_cal.copy_(src_cal)
        torch.cuda.synchronize()
        del src_cal, dst_cal

    def run(r):
        if args.eager:
            gp.round(r, K, x_own, dWs, stores, dy)
        else:
            gp.replay(r, K)

    if not args.eager:
        gp.capture(K, x_own, dWs, stores, dy)
    for r in range(1, args.warmup + 1):
        run(r)
    torch.cuda.synchronize()
    # an event after every round (enqueued, no host wait) also gives the
    # median round time beside the mean
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    rounds = range(args.warmup + 1, args.warmup + args.steps + 1)
    ev[0].record()
    for i, r in enumerate(rounds):
        run(r)
        ev[i + 1].record()
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[-1])
    ms_median = float(np.median([ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]))
    if gat:   # per layer: the forward aggregation and the transposed one of the backward
        edges = 2 * L * st["nnz"]
    else:
        edges = sum(st["nnz"] + (st["nnz_in"] if l > 1 else 0) for l in range(1, L + 1))
    value = edges * args.steps / (ms * 1e-3) / 1e9
    print(f"[bench] timed {args.steps} rounds: {ms:.3f} ms", file=sys.stderr, flush=True)

    # instrumented pass over the same rounds: per-kernel durations from HIP
    # events, with every kernel on the caller's stream (no weight gradient
    # on the library's side stream), so that each duration is the kernel's
    # own and not shared with a concurrent one
    D.digest_profile_enable(gp.p, True)
    side_env = os.environ.get("DIGEST_SIDE_STREAM")
    os.environ["DIGEST_SIDE_STREAM"] = "0"
    try:
        for r in rounds:
            gp.round(r, K, x_own, dWs, stores, dy)
        prof = D.digest_profile_read(gp.p)
    finally:
        if side_env is None:
            del os.environ["DIGEST_SIDE_STREAM"]
        else:
            os.environ["DIGEST_SIDE_STREAM"] = side_env
    D.digest_profile_enable(gp.p, False)
    # algorithmic bytes / flops / entries of each launch, from the library's plan
    model = D.digest_profile_model(gp.p, D.MODEL_GAT if gat else D.MODEL_GCN)
    kernels = {}
    for key, (tot_ms, n_l) in prof.items():
        entry = {"launches": n_l, "avg_us": 1e3 * tot_ms / n_l, "total_ms": tot_ms}
        if key in model:
            b, f, e = model[key]
            entry["gbs"] = b / (entry["avg_us"] * 1e-6) / 1e9
            if f:
                entry["tflops"] = f / (entry["avg_us"] * 1e-6) / 1e12
            if e:   # aggregation kernels: entries of the sparse operand per second
                entry["gteps"] = e / (entry["avg_us"] * 1e-6) / 1e9
        kernels[key] = entry
    pp_ms = sum(v["total_ms"] for k, v in kernels.items()
                if k.startswith(("pull_gather.", "push_scatter."))) / args.steps
    dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
    d = kernels[dom]
    b_l, f_l, _ = model.get(dom, (0.0, 0.0, 0))
    mfma_roof = {"bound": "mfma", "achieved": round(d.get("tflops", 0.0), 3),
                 "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(d.get("tflops", 0.0) / FP32_MFMA_PEAK_TFLOPS, 4)}
    hbm_roof = {"bound": "hbm", "achieved": round(d["gbs"], 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(d["gbs"] / HBM_PEAK_GBS, 4)}
    # the bound is the resource whose roofline time is the longer one; a
    # kernel that both gathers and multiplies (the fused passes) reports the
    # other as "secondary"
    mfma_bound = bool(f_l) and f_l / max(b_l, 1.0) > (FP32_MFMA_PEAK_TFLOPS * 1e12 /
                                                       (HBM_PEAK_GBS * 1e9))
    roof = dict(mfma_roof if mfma_bound else hbm_roof)
    if f_l and b_l:
        roof["secondary"] = hbm_roof if mfma_bound else mfma_roof
    traffic, traffic_source = measured_traffic(cfg.name, dom)
    if traffic:   # the rate at which the kernel moves L2-fabric bytes
        roof["traffic_rate_gbs"] = round(traffic / (d["avg_us"] * 1e-6) / 1e9, 1)
    roof.update({"traffic": traffic, "traffic_source": traffic_source, "kernel": dom,
                 "algorithmic_bytes_per_launch": b_l, "algorithmic_flops_per_launch": f_l,
                 "avg_launch_us": round(d["avg_us"], 3),
                 "achieved_basis": "algorithmic (compulsory) bytes or flops of one launch / "
                                   "its mean HIP-event duration on the launch stream"})

    cpu = None
    if not args.no_cpu:
        t_cpu = time.time()
        cpu = cpu_baseline(cfg, g, part, X, Ws, y, K, args.cpu_seconds, atts)
        print(f"[bench] cpu baseline {time.time() - t_cpu:.1f}s", file=sys.stderr, flush=True)

    out = {
        "metric": METRIC_GAT if gat else METRIC, "value": round(value, 4), "unit": "GTEPS",
        "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms / args.steps, 5),
        "ms_per_step_median": round(ms_median, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": workload_name(cfg, K, args.model, g.n, st),
            "n_global": g.n, "n_own": st["n_own"], "n_halo": st["n_halo"],
            "n_boundary": st["n_boundary"], "nnz": st["nnz"], "nnz_in": st["nnz_in"],
            "widths": list(cfg.widths), "sync_interval": K, "edges_per_step": edges,
            "launch": "eager" if args.eager else "hip-graph replay",
            "pull_push": "overlapped on a second stream" if args.overlap_io else "in line",
        },
        # the scheduled pulls and pushes of the timed rounds, per round (from
        # the instrumented pass), and the rate with them taken out of the
        # round time: edges over the forward and backward alone
        "pull_push_ms_per_step": round(pp_ms, 5),
        "gteps_excluding_pull_push": (None if args.overlap_io else
                                      round(edges / ((ms / args.steps - pp_ms) * 1e-3) / 1e9, 4)),
        "roofline": roof,
        "cpu_baseline": cpu,
        # per (kernel, layer): HIP-event durations of an instrumented eager
        # pass over the same rounds, every kernel on the caller's stream
        "kernels": {k: {kk: (round(vv, 3) if isinstance(vv, float) else vv)
                        for kk, vv in v.items()} for k, v in kernels.items()},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
