"""Benchmark: one partition's DIGEST GCN rounds on one MI355X.

A step is one round r of Algorithm 1 for the partition: every layer's
forward (with the pull / push the schedule asks for in that round), the loss
head, and every layer's backward, all in libdigest.so, replayed from HIP
graphs with inputs resident in HBM.  Default workload: the Flickr-shaped
synthetic graph (90,000 nodes in 8 blocks, partition 0, GCN 500 -> 256 -> 7,
sync interval 10).

    python bench.py [--steps K] [--warmup W] [--config NAME] [--sync N]

Prints one JSON line: whole-round throughput in GTEPS (aggregation edges of
the forward and backward per round / time), the roofline of the dominant
kernel (from a second, instrumented pass with HIP events on the launch
stream) and the CPU oracle timed on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GCN layer fwd+bwd GTEPS on one partition; % of HBM / MFMA roofline"
METRIC_GAT = "GAT layer fwd+bwd GTEPS on one partition; % of HBM / MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix


def transform_first(l, widths, st):
    """Mirror of the library's choice for the identity (last) layer: the
    cheaper order under its cost model of gathered bytes and GEMM flops."""
    if l != len(widths) - 1:
        return False
    di, do = widths[l - 1], widths[l]
    n, R, nnz, nnz_in = st["n_own"], st["n_own"] + st["n_halo"], st["nnz"], st["nnz_in"]
    gather, flops = 7.0e12, 80.0e12
    dgrad = l > 1
    af = ((nnz * di + (nnz_in * min(di, do) if dgrad else 0)) * 4.0 / gather
          + 2.0 * n * di * do * (3.0 if dgrad else 2.0) / flops)
    tf = (2.0 * nnz * do * 4.0 / gather
          + (4.0 * R * di * do + (2.0 * n * di * do if dgrad else 0.0)) / flops)
    return tf < af


def loss_group(C):
    """Mirror of the library's lanes per row of the loss head."""
    return 8 if C <= 8 else (16 if C <= 64 else (32 if C <= 128 else 64))


def splitk(M, N, K):
    """Mirror of the library's split-K plan: (splits, rows per split)."""
    tiles = max(1, -(-M // 64) * -(-N // 64))
    cap = min(256, max(1, K // 256))
    lo = max(1, min(-(-768 // tiles), cap))

    def realise(want):
        chunk = -(-K // want)
        chunk = -(-chunk // 32) * 32 or 32
        return max(1, -(-K // chunk)), chunk

    def fill(sp):
        wg = tiles * sp
        return wg / (-(-wg // 256) * 256)

    best = realise(lo)
    for want in range(lo + 1, min(cap, 2 * lo) + 1):
        cand = realise(want)
        if fill(cand[0]) > fill(best[0]) + 1e-9:
            best = cand
    return best


def tf_slices(n, nh, di, do):
    """Mirror of the library's slice plan for the transform-first dW."""
    if do <= 16:
        R = n + nh
        target = max(1, 2048 // -(-di // 64))
        chunk = max(32, -(-R // target))
        chunk = -(-chunk // 32) * 32
        return max(1, -(-R // chunk))
    return splitk(di, do, n)[0] + (splitk(di, do, nh)[0] if nh else 0)


def launch_model_gat(st, widths):
    """Algorithmic bytes, flops and aggregation entries of one launch of each
    GAT (kernel kind, layer): every operand row read once, every output
    written once (R = owned + halo rows)."""
    n, nh, nnz = st["n_own"], st["n_halo"], st["nnz"]
    R = n + nh
    L = len(widths) - 1
    m = {}

    def put(kind, l, b, f=0.0, e=0):
        m[f"{kind}.l{l}"] = (float(b), float(f), int(e))

    for l in range(1, L + 1):
        di, do = widths[l - 1], widths[l]
        put("gat_transform", l, 4 * (R * di + di * do + R * do), 2.0 * R * di * do)
        put("gat_scores", l, 4 * (R * do + 2 * do + 2 * R), 4.0 * R * do)
        put("gat_softmax", l, 4 * (n + 1) + 16 * nnz + 4 * n)
        put("gat_aggregate", l, 4 * (n + 1) + 8 * nnz + 4 * R * do + 4 * n * do, e=nnz)
        put("gat_edge_grad", l, 4 * (n + 1) + 12 * nnz + 12 * n * do + 4 * R * do + 8 * R + 4 * n,
            e=nnz)
        put("gat_transpose_edges", l, 20 * nnz)
        put("gat_aggregate_transposed", l,
            4 * (R + 1) + 8 * nnz + 4 * n * do + 4 * R * do + 4 * R + 4 * n + 8 * do, e=nnz)
        put("gat_score_sums", l, 4 * (R + 1) + 8 * nnz + 4 * n + 4 * R)
        put("gat_score_grad", l, 8 * R + 4 * nh)
        put("gat_datt", l, 4 * (R * do + 2 * R + 2 * do), 4.0 * R * do)
        put("gat_dw", l, 4 * (R * di + R * do + di * do), 2.0 * R * di * do)
        put("splitk_reduce_dw", l, 4 * (tf_slices(n, nh, di, do) + 1) * di * do)
        if l > 1:
            put("gat_dgrad", l, 4 * (n * do + di * do + n * di), 2.0 * n * di * do)
    put("softmax_xent", L, 4 * (2 * n * widths[-1] + n))
    put("loss_mean", L, 4 * -(-n // (4 * (64 // loss_group(widths[-1])))) + 4)
    for lev in range(L):
        put("pull_gather", lev, 8.0 * nh * widths[lev] + 4 * nh)
    for lev in range(1, L):
        put("push_scatter", lev, 8.0 * st["n_boundary"] * widths[lev] + 8 * st["n_boundary"])
    return m


def launch_model(st, widths):
    """Algorithmic bytes and flops of one launch of each (kernel kind, layer).

    Keys follow the library's instrumentation: "kind.lN" with N the layer
    (the level for pull/push, L for the loss head).  The layer order
    (aggregate-first or transform-first) follows the library's rule.
    """
    n, nh, nnz, nnz_in, nb = st["n_own"], st["n_halo"], st["nnz"], st["nnz_in"], st["n_boundary"]
    L = len(widths) - 1
    m = {}

    def put(kind, l, b, f=0.0, e=0):
        m[f"{kind}.l{l}"] = (float(b), float(f), int(e))

    for l in range(1, L + 1):
        di, do = widths[l - 1], widths[l]
        relu = l < L
        if transform_first(l, widths, st):
            R = n + nh
            put("gemm_fwd_relu", l, 4 * (R * di + di * do + R * do), 2.0 * R * di * do)
            put("spmm_fwd", l, 4 * (n + 1) + 8 * nnz + 4 * R * do + 4 * n * do, e=nnz)
            fused = l > 1 and do <= 16 and di <= 1024 and di % 4 == 0
            put("spmm_bwd_transposed", l, 4 * (R + 1) + 8 * nnz + 4 * n * do + 4 * R * do
                + (4 * (n * di + di * do) if fused else 0), e=nnz)
            put("gemm_dw_splitk", l, 4 * (R * di + R * do), 2.0 * R * di * do)
            put("splitk_reduce_dw", l, 4 * (tf_slices(n, nh, di, do) + 1) * di * do)
            if l > 1 and not fused:
                put("gemm_dgrad", l, 4 * (n * do + di * do + n * di), 2.0 * n * di * do)
            continue
        put("spmm_fwd", l, 4 * (n + 1) + 8 * nnz + 4 * (n + nh) * di + 4 * n * di, e=nnz)
        put("gemm_fwd_relu", l, 4 * (n * di + di * do + n * do), 2.0 * n * di * do)
        put("gemm_dw_splitk", l, 4 * (n * di + n * do * (2 if relu else 1) + di * do),
            2.0 * n * di * do)
        s = splitk(di, do, n)[0]
        if s > 1:
            put("splitk_reduce_dw", l, 4 * (s + 1) * di * do)
        if l > 1:
            narrow = (not relu) and do < di
            w = do if narrow else di
            put("spmm_bwd_transposed", l, 4 * (n + 1) + 8 * nnz_in + 8 * n * w, e=nnz_in)
            put("gemm_dgrad", l, 4 * (n * do * (1 if narrow or not relu else 2) + di * do + n * di),
                2.0 * n * di * do)
    put("softmax_xent", L, 4 * (2 * n * widths[-1] + n))
    put("loss_mean", L, 4 * -(-n // (4 * (64 // loss_group(widths[-1])))) + 4)
    for lev in range(L):
        put("pull_gather", lev, 8.0 * nh * widths[lev] + 4 * nh)
    for lev in range(1, L):
        put("push_scatter", lev, 8.0 * nb * widths[lev] + 8 * nb)
    return m


def measured_traffic(workload, key):
    """HBM bytes per launch of `key` from the committed counter summary, or
    None when there is none for this kernel or the kernels changed since."""
    path = os.path.join(ROOT, "profiles", f"{workload}_hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if "=" in line:
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    from paper_2206_00057_amd.pmc import kernel_source_hash
    if kv.get("kernel") != key or kv.get("source_sha") != kernel_source_hash():
        return None
    return float(kv["traffic_bytes_per_launch"])


def cpu_baseline(cfg, g, part, X, Ws, y, K, budget_s, atts=None):
    """The oracle as it stands, timed on this host's cores on whole rounds
    (GCN layers, or GAT layers when atts are given)."""
    import oracle
    L = cfg.layers
    op = oracle.OraclePartition(g.n, part.indptr, part.indices, part.values, part.owned,
                                part.halo, cfg.widths)
    stores = [X] + [np.maximum(np.random.default_rng(70 + l).standard_normal(
        (g.n, cfg.widths[l]), dtype=np.float32), 0) for l in range(1, L)]
    for lev in range(L):
        op.pull(lev, stores[lev])
    x = X[part.owned]
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
        "config": {"workload": f"{cfg.name}: all {M} subgraphs, {args.model.upper()}, "
                               f"Algorithm 1 rounds with "
                               f"sync interval {K}, SGD lr {args.lr}, halo-gradient "
                               f"exchange {args.grad_exchange}",
                   "n_global": g.n, "subgraphs": M, "widths": list(cfg.widths),
                   "edges_per_round": tr.edges_per_round, "launch": "hip-graph replay"},
        "loss": {"after_warmup": round(first_loss, 6), "last": round(tr.mean_loss(), 6)},
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="medium")
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

    # instrumented pass over the same rounds: per-kernel durations from HIP events
    D.digest_profile_enable(gp.p, True)
    for r in rounds:
        gp.round(r, K, x_own, dWs, stores, dy)
    prof = D.digest_profile_read(gp.p)
    D.digest_profile_enable(gp.p, False)
    model = launch_model_gat(st, cfg.widths) if gat else launch_model(st, cfg.widths)
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
    if f_l and f_l / max(b_l, 1.0) > FP32_MFMA_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        roof = {"bound": "mfma", "achieved": round(d["tflops"], 3), "peak": FP32_MFMA_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(d["tflops"] / FP32_MFMA_PEAK_TFLOPS, 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(d["gbs"], 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(d["gbs"] / HBM_PEAK_GBS, 4)}
    roof.update({"traffic": measured_traffic(cfg.name, dom), "kernel": dom,
                 "algorithmic_bytes_per_launch": b_l, "algorithmic_flops_per_launch": f_l,
                 "avg_launch_us": round(d["avg_us"], 3)})

    cpu = None
    if not args.no_cpu:
        import oracle
        nr, secs, cores = cpu_baseline(cfg, g, part, X, Ws, y, K, args.cpu_seconds, atts)
        cpu = {"value": edges * nr / secs / 1e9, "unit": "GTEPS", "cores": cores, "kind": "oracle",
               "sample": f"{nr} whole rounds of the same partition (forward, loss, backward, "
                         f"scheduled pull/push) in {secs:.1f}s, float64 oracle, {cores} threads"}
        # the same oracle on one thread, beside the all-core figure
        oracle.set_num_threads(1)
        nr1, secs1, _ = cpu_baseline(cfg, g, part, X, Ws, y, K, args.cpu_seconds / 2, atts)
        oracle.set_num_threads(cores)
        cpu["single_thread"] = {
            "value": edges * nr1 / secs1 / 1e9, "unit": "GTEPS", "cores": 1,
            "sample": f"{nr1} whole rounds in {secs1:.1f}s, float64 oracle, 1 thread"}

    out = {
        "metric": METRIC_GAT if gat else METRIC, "value": round(value, 4), "unit": "GTEPS",
        "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms / args.steps, 5),
        "ms_per_step_median": round(ms_median, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name}: synthetic block graph, N={g.n:,}, partition 0 "
                         f"({st['n_own']:,} owned + {st['n_halo']:,} halo rows), "
                         f"{args.model.upper()} {'->'.join(map(str, cfg.widths))}, "
                         f"sync interval {K}"),
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
        "kernels": {k: {kk: (round(vv, 3) if isinstance(vv, float) else vv)
                        for kk, vv in v.items()} for k, v in kernels.items()},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
