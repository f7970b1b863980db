"""Benchmark: heterogeneous mini-batch generation on one MI355X.

One step = one mini-batch through the whole path, in one library call
(hg_sample_blocks_gather): multi-hop per-edge-type fanout sampling, per-hop
compaction into relabelled blocks, and the gather of the input frontier's
features for every node type that has them (DistDGLv2, arXiv 2112.15345,
Sec. 3.2 and Sec. 4.2).  Graph, features and seeds are resident in HBM before
the timed region.

Prints one JSON line.  `value` is sampled edges per second over whole steps;
the gathered feature rate, per-stage times, the roofline of the dominant
kernel and the CPU oracle's rate on a bounded sample ride along.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
HOST_LINK_PEAK_GBS = 64.0  # PCIe 5.0 x16, one direction

# Measured HBM traffic of the gather launches of one bundle of the default
# run (academic workload, bundles of 32, 128 warm-up + 320 timed mini-batches):
# FETCH_SIZE and WRITE_SIZE from two rocprofv3 --pmc passes, scaled by what the
# counters read for a 1 GiB device copy (profiles/gather_academic_traffic.md).
# Counter collection runs one dispatch at a time, so a bundle's gather moves
# the same bytes with or without worker streams; the figure is valid only for
# the gather source, the workload, the batches and the bundle size it was
# measured on.
GATHER_TRAFFIC = {"source_sha256_16": "307d950537d4b4f1", "workload": 2, "steps": 320,
                  "warmup": 128, "bundle": 32, "bytes_per_launch": 7975580490.4}


# Measured HBM traffic of a whole mini-batch on the default batches (academic
# workload, bundles of 32, 128 warm-up + 320 timed mini-batches): FETCH_SIZE and
# WRITE_SIZE of every dispatch of this library's kernels (graph creation's
# check aside), scaled as above, summed over the run and divided by its 451
# mini-batches (the bundled ones and the three single calls after the timed
# region).  Valid only for the kernel and runtime sources it was measured on.
STEP_TRAFFIC = {"sources_sha256_16": "4bc3bcef9182dd15", "workload": 2, "steps": 320, "warmup": 128,
                "bundle": 32, "bytes_per_step": 348.96e6}


def kernel_sources_digest():
    import hashlib
    d = os.path.join(ROOT, "paper_2112_15345_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".hpp")) or f == "hg_runtime.cpp":
            h.update(f.encode())
            h.update(open(os.path.join(d, f), "rb").read())
    return h.hexdigest()[:16]


def measured_step_traffic(args):
    t = STEP_TRAFFIC
    if args.host_features or (kernel_sources_digest(), args.workload, args.steps, args.warmup,
                              args.bundle) != (t["sources_sha256_16"], t["workload"],
                                               t["steps"], t["warmup"], t["bundle"]):
        return None
    return t["bytes_per_step"]


def measured_gather_traffic(args):
    import hashlib
    src = os.path.join(ROOT, "paper_2112_15345_amd", "csrc", "hg_gather.hip")
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    t = GATHER_TRAFFIC
    if (digest, args.workload, args.steps, args.warmup, args.bundle) != (
            t["source_sha256_16"], t["workload"], t["steps"], t["warmup"], t["bundle"]):
        return None
    return t["bytes_per_launch"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(gen, wl, first_batch, budget_s=12.0, max_batches=32):
    """The oracle, single-threaded, on the host cores: whole mini-batches
    (sampling, compaction, gather) of the same workload until ~budget_s."""
    import oracle
    t0 = time.perf_counter()
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False)
    log(f"oracle host copy ready in {time.perf_counter() - t0:.1f}s")
    fan = wl.fanout_matrix()
    edges = 0
    rows = 0
    nbytes = 0
    spent = 0.0
    nb = 0
    for b in range(first_batch, first_batch + max_batches):
        seeds = __import__("workloads").seeds_per_type(wl, b)
        t = time.perf_counter()
        res = host.sample_blocks(seeds, fan, b)
        for ti, (n, feat, row_bytes) in enumerate(host.ntypes):
            if feat is not None:
                x = host.gather(ti, res["input"][ti])
                rows += x.shape[0]
                nbytes += x.nbytes
        spent += time.perf_counter() - t
        edges += sum(v[3].size for v in res["edges"].values())
        nb += 1
        if spent >= budget_s:
            break
    return {"value": edges / spent, "unit": "sampled edges/s", "cores": 1, "kind": "oracle",
            "sample": f"{nb} whole mini-batches (batches {first_batch}..{first_batch + nb - 1}: "
                      f"sampling, compaction, gather of {rows} rows) in {spent:.2f} s",
            "gathered_GBps": nbytes / spent / 1e9}


def pipeline_name(args):
    return f"{args.workers} worker streams" if args.workers else "direct calls"


def drive_units(args, g, n_batches, direct, submit, account, gather):
    """Warm-up then timed units of --bundle batch indices (first, last): with
    --workers 0, direct(first, last) returns the unit's Blocks; otherwise
    submit(pipe, first, last) queues the unit on a pipeline of --workers
    worker streams (at most --depth, default 2 x workers x bundle, mini-batches
    outstanding) and the Blocks come back in order.  account(blocks) runs on
    every timed mini-batch.  Returns the timed region's wall time."""
    import torch

    import paper_2112_15345_amd as hg

    B = max(1, args.bundle)
    units = [(b, min(b + B, args.warmup)) for b in range(0, args.warmup, B)]
    timed = [(b, min(b + B, n_batches)) for b in range(args.warmup, n_batches, B)]
    if args.workers == 0:
        for u in units:
            direct(*u)
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for u in timed:
            for blocks in direct(*u):
                account(blocks)
                del blocks
        torch.cuda.synchronize()
        return time.perf_counter() - t_start
    depth = max(args.depth or 2 * args.workers * B, B)
    pipe = hg.Pipeline(g, workers=args.workers, capacity=depth, gather=gather)
    queue = units + timed
    # no timed unit is submitted before the timed region starts
    state = {"next": 0, "outstanding": 0, "limit": len(units)}

    def submit_more():
        while state["next"] < state["limit"]:
            first, last = queue[state["next"]]
            if state["outstanding"] + (last - first) > depth:
                break
            submit(pipe, first, last)
            state["outstanding"] += last - first
            state["next"] += 1

    def take(first, last):
        out = []
        for _ in range(last - first):
            out.append(pipe.next())
            state["outstanding"] -= 1
        submit_more()
        return out

    submit_more()
    for u in units:
        take(*u)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    state["limit"] = len(queue)
    submit_more()
    for u in timed:
        for blocks in take(*u):
            account(blocks)
            del blocks
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    pipe.close()
    return elapsed


def link_main(args, wl, gen, g):
    """Edge-seeded (link-prediction) mini-batches: targets of one forward
    relation, their endpoints as seeds, one negative per target, targets and
    their reverse edges excluded, the paper's link-prediction fanouts [25, 15]
    per hop, every featured type gathered.  Bundles of --bundle mini-batches
    (hg_sample_edge_blocks_bundle), made by --workers pipeline workers or by
    direct calls on one stream."""
    import torch

    import paper_2112_15345_amd as hg
    import workloads as W

    dev = g.device
    rev_et, rev_eid = W.reverse_maps(gen)
    exclude = hg.HG_EXCLUDE_REVERSE if rev_et is not None else hg.HG_EXCLUDE_SELF
    link_et = gen.etype_names.index("cites") if "cites" in gen.etype_names else 0
    fan = [[k] * g.R for k in W.LINK_FANOUTS]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}
    n_batches = args.warmup + args.steps
    targets = [[None if x is None else torch.as_tensor(x, device=dev)
                for x in W.link_targets(gen, b, link_et)] for b in range(n_batches)]

    kw = dict(n_neg=W.LINK_NEG, exclude=exclude, rev_etype=rev_et, rev_eid=rev_eid)

    def direct(first, last):
        return g.sample_edge_bundle([targets[b] for b in range(first, last)], fan,
                                    list(range(first, last)), gather=feat_types, **kw)

    def submit(pipe, first, last):
        pipe.submit_edge_bundle([targets[b] for b in range(first, last)], fan,
                                list(range(first, last)), **kw)

    totals = [0, 0, 0]

    def account(blocks):
        totals[0] += blocks.total_edges()
        for t in feat_types:
            n = blocks.num_input_nodes(t)
            totals[1] += n
            totals[2] += n * row_bytes[t]

    elapsed = drive_units(args, g, n_batches, direct, submit, account, feat_types)
    edges, rows, gbytes = totals
    result = {
        "metric": "sampled edges/s + gathered feature GB/s per mini-batch (1 GPU), % of HBM peak",
        "value": edges / elapsed, "unit": "sampled edges/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic (seeded generator shaped like the paper's workloads)",
        "config": {"workload": wl.name + f"; link prediction: {W.LINK_BATCH} target edges of "
                               f"'{gen.etype_names[link_et]}', {W.LINK_NEG} negative each, "
                               f"exclusion {exclude}, fanout {list(W.LINK_FANOUTS)}",
                   "workload_index": args.workload, "task": "link",
                   "parallelism": "single GPU", "pipeline": pipeline_name(args),
                   "bundle": max(1, args.bundle)},
        "gathered_GBps": gbytes / elapsed / 1e9,
        "sampled_edges_per_step": edges / args.steps,
        "gathered_rows_per_step": rows / args.steps,
    }
    print(json.dumps(result), flush=True)


def layers_main(args, wl, gen, g):
    """Layer-wise (LADIES) mini-batches: the workload's seeds, 512 draws per
    node type in each of two hops, every featured type gathered.  Bundles of
    --bundle mini-batches (hg_sample_layers_bundle), made by --workers
    pipeline workers or by direct calls on one stream."""
    import torch

    import workloads as W

    dev = g.device
    sizes = [[k] * g.T for k in W.LAYER_SIZES]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}
    n_batches = args.warmup + args.steps
    seeds = [[None if s is None else torch.as_tensor(s, device=dev)
              for s in W.seeds_per_type(wl, b)] for b in range(n_batches)]

    def direct(first, last):
        return g.sample_layers_bundle([seeds[b] for b in range(first, last)], sizes,
                                      list(range(first, last)), gather=feat_types)

    def submit(pipe, first, last):
        pipe.submit_layers_bundle([seeds[b] for b in range(first, last)], sizes,
                                  list(range(first, last)))

    totals = [0, 0, 0]

    def account(blocks):
        totals[0] += blocks.total_edges()
        for t in feat_types:
            n = blocks.num_input_nodes(t)
            totals[1] += n
            totals[2] += n * row_bytes[t]

    elapsed = drive_units(args, g, n_batches, direct, submit, account, feat_types)
    edges, rows, gbytes = totals
    result = {
        "metric": "kept edges/s + gathered feature GB/s per layer-wise mini-batch (1 GPU)",
        "value": edges / elapsed, "unit": "kept edges/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic (seeded generator shaped like the paper's workloads)",
        "config": {"workload": wl.name + f"; layer-wise (LADIES): {list(W.LAYER_SIZES)} draws "
                               f"per node type per hop",
                   "workload_index": args.workload, "task": "layers",
                   "parallelism": "single GPU", "pipeline": pipeline_name(args),
                   "bundle": max(1, args.bundle)},
        "gathered_GBps": gbytes / elapsed / 1e9,
        "kept_edges_per_step": edges / args.steps,
        "gathered_rows_per_step": rows / args.steps,
    }
    if not args.no_cpu_baseline:
        import oracle
        host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False)
        spent = 0.0
        cedges = nb = 0
        for b in range(args.warmup, n_batches):
            t = time.perf_counter()
            res = host.sample_layers(W.seeds_per_type(wl, b), sizes, b)
            for ti, (n, feat, _) in enumerate(host.ntypes):
                if feat is not None:
                    host.gather(ti, res["input"][ti])
            spent += time.perf_counter() - t
            cedges += sum(v[3].size for v in res["edges"].values())
            nb += 1
            if spent >= 10.0:
                break
        result["cpu_baseline"] = {
            "value": cedges / spent, "unit": "kept edges/s", "cores": 1, "kind": "oracle",
            "sample": f"{nb} whole layer-wise mini-batches (batches {args.warmup}.."
                      f"{args.warmup + nb - 1}: sampling, compaction, gather) in {spent:.2f} s"}
    print(json.dumps(result), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=320)
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed mini-batches first (default: two bundles per worker, or "
                         "two bundles with direct calls), so that every worker's workspace "
                         "and memory pool have grown before the timed region")
    ap.add_argument("--workload", type=int, default=2,
                    help="1 tiny, 2 academic (default), 3 billion-share, 4 knowledge graph, "
                         "5 gather-heavy academic")
    ap.add_argument("--workers", type=int, default=None,
                    help="pipeline worker threads (own streams); 0 = direct calls on one "
                         "stream (default 2)")
    ap.add_argument("--bundle", type=int, default=None,
                    help="mini-batches per launch sequence (the *_bundle calls, 1..32; "
                         "default 32)")
    ap.add_argument("--depth", type=int, default=0,
                    help="mini-batches outstanding in the pipeline (default 2 x workers x "
                         "bundle)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after warm-up (untimed), copy this many MiB device to device "
                         "once: a copy of known size for scaling memory counters")
    ap.add_argument("--host-features", action="store_true",
                    help="feature tables in pinned host memory, gathered over the host link "
                         "(zero-copy); the gather rate then includes that link")
    ap.add_argument("--task", choices=("vertex", "link", "layers"), default="vertex",
                    help="vertex: mini-batches from seed vertices (the default); link: "
                         "edge-seeded link-prediction mini-batches "
                         "(hg_sample_edge_blocks_bundle); layers: layer-wise LADIES "
                         "mini-batches (hg_sample_layers_bundle)")
    args = ap.parse_args()
    if args.workers is None:
        args.workers = 2
    if args.bundle is None:
        args.bundle = 32
    if args.warmup is None:
        args.warmup = 2 * max(args.workers, 1) * max(1, args.bundle)
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2112_15345_amd as hg
    import workloads as W

    wl = W.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    t0 = time.perf_counter()
    gen = W.make_graph(wl, device=dev, feat_device="cpu" if args.host_features else None)
    if args.host_features:
        gen.feats = [None if f is None else
                     torch.empty(f.shape, dtype=f.dtype, pin_memory=True).copy_(f)
                     for f in gen.feats]
    torch.cuda.synchronize()
    log(f"generated '{wl.name}' in {time.perf_counter() - t0:.1f}s")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)),
                 [(s, d, ip, ix) for s, d, ip, ix in gen.etypes], device=dev)
    if args.task == "link":
        return link_main(args, wl, gen, g)
    if args.task == "layers":
        return layers_main(args, wl, gen, g)
    fan = wl.fanout_matrix()
    n_batches = args.warmup + args.steps
    seeds = [[None if s is None else torch.as_tensor(s, device=dev)
              for s in W.seeds_per_type(wl, b)] for b in range(n_batches)]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}

    if args.copy_calibration_mb > 0:
        # a copy of known size, untimed, for scaling the memory counters
        src = torch.ones(args.copy_calibration_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.copy_calibration_mb} MiB done")
        del src, dst

    # HIP events recorded by the gather kernels themselves (on their stream)
    hip_events = hg.HipEvents(2 * args.steps)
    events = {args.warmup + i: (hip_events.events[2 * i], hip_events.events[2 * i + 1])
              for i in range(args.steps)}
    gather_rec = []
    B = max(1, args.bundle)
    # units of work: bundles of B consecutive mini-batches (warm-up and timed
    # mini-batches never share a bundle); a unit's events time its gather
    units = [list(range(b, min(b + B, args.warmup))) for b in range(0, args.warmup, B)]
    timed_units = [list(range(b, min(b + B, n_batches)))
                   for b in range(args.warmup, n_batches, B)]

    def account(unit, blist, totals=None):
        """Bookkeeping of a returned unit; gather bytes and events of timed ones."""
        rows_all = {t: 0 for t in feat_types}
        for blocks in blist:
            e = blocks.total_edges()
            if totals is not None:
                totals[0] += e
            for t in feat_types:
                n = blocks.num_input_nodes(t)
                rows_all[t] += n
                if totals is not None:
                    totals[1] += n
                    totals[2] += n * row_bytes[t]
        if unit[0] in events:
            gather_rec.append((events[unit[0]][0], events[unit[0]][1], rows_all))

    def unit_events(unit):
        return events.get(unit[0])

    totals = [0, 0, 0]
    if args.workers == 0:
        # direct calls on the current stream, one per unit
        def run(unit):
            if len(unit) == 1:
                b = unit[0]
                return [g.sample_blocks(seeds[b], fan, b, gather=feat_types,
                                        events=unit_events(unit))]
            return g.sample_bundle([seeds[b] for b in unit], fan, unit, gather=feat_types,
                                   events=unit_events(unit))

        for u in units:
            account(u, run(u))
        torch.cuda.synchronize()
        log(f"warm-up done (direct calls, bundles of {B})")
        t_start = time.perf_counter()
        for u in timed_units:
            blist = run(u)
            account(u, blist, totals)
            del blist
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
    else:
        # the pipeline: units generated ahead by worker threads, each on its
        # own stream, returned in order; at most `depth` mini-batches outstanding
        depth = max(args.depth or 2 * args.workers * B, B)
        pipe = hg.Pipeline(g, workers=args.workers, capacity=depth, gather=feat_types)
        queue = units + timed_units
        # no timed unit is submitted before the timed region starts
        state = {"next": 0, "outstanding": 0, "limit": len(units)}

        def submit_more():
            while (state["next"] < state["limit"] and
                   state["outstanding"] + len(queue[state["next"]]) <= depth):
                u = queue[state["next"]]
                pipe.submit_bundle([seeds[b] for b in u], fan, u, events=unit_events(u))
                state["outstanding"] += len(u)
                state["next"] += 1

        def take(unit):
            blist = []
            for _ in unit:
                blist.append(pipe.next())
                state["outstanding"] -= 1
            submit_more()
            return blist

        submit_more()
        for u in units:
            account(u, take(u))
        torch.cuda.synchronize()
        log(f"warm-up done ({args.workers} workers, bundles of {B}, depth {depth})")
        t_start = time.perf_counter()
        state["limit"] = len(queue)
        submit_more()
        for u in timed_units:
            blist = take(u)
            account(u, blist, totals)
            del blist
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
        pipe.close()
    edges, rows, gbytes = totals
    ms_per_step = elapsed / args.steps * 1e3

    # context for the roofline: the same gather with nothing else on the GPU
    # (a few direct calls after the timed region, untimed)
    iso = hg.HipEvents(2)
    iso_ms, iso_bytes = 0.0, 0
    for b in range(min(3, n_batches)):
        torch.cuda.synchronize()
        blocks = g.sample_blocks(seeds[b], fan, b, gather=feat_types,
                                 events=(iso.events[0], iso.events[1]))
        iso_ms += iso.elapsed_ms(iso.events[0], iso.events[1])
        iso_bytes += sum(blocks.num_input_nodes(t) *
                         (row_bytes[t] if args.host_features else 2 * row_bytes[t] + 8)
                         for t in feat_types)
        del blocks
    iso_gbps = iso_bytes / (iso_ms / 1e3) / 1e9 if iso_ms > 0 else 0.0

    # context for the peak: a plain 1 GiB device-to-device copy (torch's copy
    # kernel), read + write bytes over its time, best of 5 (untimed region)
    copy_gbps = None
    if not args.host_features:
        src = torch.ones(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        best = None
        for _ in range(6):
            c0.record()
            dst.copy_(src)
            c1.record()
            c1.synchronize()
            ms = c0.elapsed_time(c1)
            best = ms if best is None else min(best, ms)
        copy_gbps = 2 * src.numel() / (best / 1e3) / 1e9
        del src, dst

    # gather kernel (one launch per step for all feature types): algorithmic
    # bytes per row = read its id (8) + read the row + write the row
    g_ms = sum(hip_events.elapsed_ms(e0, e1) for e0, e1, _ in gather_rec)
    g_alg = sum(n * (2 * row_bytes[t] + 8) for _, _, rows_t in gather_rec
                for t, n in rows_t.items())
    g_achieved = g_alg / (g_ms / 1e3) / 1e9 if g_ms > 0 else 0.0
    if args.host_features:
        # the rows cross the host link once; that link is the roof
        g_alg = sum(n * row_bytes[t] for _, _, rows_t in gather_rec for t, n in rows_t.items())
        g_achieved = g_alg / (g_ms / 1e3) / 1e9 if g_ms > 0 else 0.0
    log(f"{args.steps} steps: {ms_per_step:.3f} ms/step, gather {g_ms / len(gather_rec):.4f} "
        f"ms/launch, {g_achieved:.0f} GB/s algorithmic")

    peak = HOST_LINK_PEAK_GBS if args.host_features else HBM_PEAK_GBS
    result = {
        "metric": "sampled edges/s + gathered feature GB/s per mini-batch (1 GPU), % of HBM peak",
        "value": edges / elapsed,
        "unit": "sampled edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic (seeded generator shaped like the paper's workloads)",
        "config": {"workload": wl.name, "workload_index": args.workload,
                   "seeds_per_batch": wl.batch, "fanouts_per_hop": list(wl.fanouts),
                   "node_types": len(gen.num_nodes), "edge_types": g.R,
                   "edges_in_graph": int(sum(ix.numel() for _, _, _, ix in gen.etypes)),
                   "parallelism": "single GPU",
                   "features": "pinned host memory" if args.host_features else "HBM",
                   "bundle": max(1, args.bundle),
                   "pipeline": (f"{args.workers} worker streams" if args.workers
                                else "direct calls")},
        "gathered_GBps": gbytes / elapsed / 1e9,
        "sampled_edges_per_step": edges / args.steps,
        "gathered_rows_per_step": rows / args.steps,
        "gather_kernel_ms_per_step": g_ms / args.steps,
        "roofline": {"bound": "host link" if args.host_features else "hbm",
                     "kernel": "k_gather_multi (feature gather, all types)",
                     "achieved": g_achieved, "peak": peak, "unit": "GB/s",
                     "frac": g_achieved / peak,
                     "traffic": None if args.host_features else measured_gather_traffic(args),
                     "algorithmic_bytes_per_launch": g_alg / max(len(gather_rec), 1),
                     "avg_launch_us": g_ms / max(len(gather_rec), 1) * 1e3,
                     "overlap": ("the gather launches of a bundle share the GPU with other "
                                 "workers' sampling kernels; isolated_* is the same gather "
                                 "with nothing else running") if args.workers > 1 else "none",
                     "isolated_achieved": iso_gbps,
                     "isolated_frac": iso_gbps / peak,
                     "device_copy_GBps": copy_gbps},
    }
    step_bytes = measured_step_traffic(args)
    if step_bytes is not None:
        # every kernel of the step together: counted HBM bytes per mini-batch
        # over the wall time per mini-batch
        rate = step_bytes / (ms_per_step / 1e3) / 1e9
        result["step_hbm"] = {"bytes_per_step": step_bytes, "achieved": rate, "unit": "GB/s",
                              "frac": rate / HBM_PEAK_GBS,
                              "of_device_copy": rate / copy_gbps if copy_gbps else None}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(gen, wl, first_batch=args.warmup)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
