"""Benchmark: heterogeneous mini-batch generation on one MI355X.

One step = one mini-batch through the whole path: multi-hop per-edge-type
fanout sampling, per-hop compaction into relabelled blocks, and the gather of
the input frontier's features for every node type that has them (DistDGLv2,
arXiv 2112.15345, Sec. 3.2 and Sec. 4.2).  Graph, features and seeds are
resident in HBM before the timed region.  Mini-batches run in bundles of
--bundle (hg_sample_blocks_bundle), made by --workers pipeline worker streams
or, with --workers 0, by direct calls on one stream.

The default workload is the billion-edge single-GPU share (workload 3: 92M
vertices, 1.2B edges, fanout [15, 10, 5], 4096 seeds).  Prints one JSON line:
`value` is sampled edges per second over whole steps; beside it the gathered
feature rate, the per-step spread, every stage's device time (from HIP events
carried by the stages' own kernel launches), the HBM rates of sampling and
compaction (algorithmic bytes and counted bytes), the sampler's random-key
rate against the vector-ALU roof, the roofline of the dominant kernel, the
oracle on every host core, and an element-wise check of timed mini-batches
against the oracle.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]
                    [--workers N] [--bundle B] [--task vertex|link|layers]
    python bench.py --mode philox      # the sampler's key loop alone
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

# The vector-ALU roof of the sampler's random keys.  MI355X: 256 CUs x 4 SIMDs
# x 16 lanes at 2.4 GHz = 39.3e12 32-bit lane operations per second (a wave64
# instruction occupies its SIMD for 4 cycles).  One Philox4x32-10 call of the
# sampler (counter (g, 0, hop, etype), the lane-independent parts of rounds 0
# and 1 in scalar registers) is 37 vector instructions (18 v_mad_u64_u32, 15
# v_bitop3_b32, 4 v_xor_b32) and gives 4 keys.  The key-loop kernel of
# --mode philox and the sampler's hub loop add 3 per call (min, min3, compare:
# the candidate test); both loops are counted and branched on by the scalar
# unit.
VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
PHILOX_VALU_PER_CALL = 37
PHILOX_LOOP_VALU_PER_CALL = 40
PHILOX_HUB_VALU_PER_CALL = 40
PHILOX_PEAK_KEYS = VALU_LANE_OPS * 4 / PHILOX_VALU_PER_CALL

# Per-workload defaults (workers, bundle, steps): the launch that gives each
# workload its best throughput on one MI355X.
DEFAULTS = {1: (2, 32, 320), 2: (3, 32, 384), 3: (3, 2, 40), 4: (3, 4, 96), 5: (3, 8, 96)}

# HBM bytes counted by rocprofv3 (FETCH_SIZE x 2.000 + WRITE_SIZE x 1.000, the
# factors a 1 GiB device copy gives) per mini-batch and per launch (the gather's:
# per bundle, all its launches), and the L2
# hit rates (TCC_HIT / (TCC_HIT + TCC_MISS)), for the kernel sources and
# launch they were measured on (profiles/ holds the runs; every dispatch of
# the run, probe, warm-up and profile pass included, over its mini-batches).  Keyed
# by a digest of the kernel and runtime sources, the workload and the bundle
# size; any other run reports them as null.
COUNTER_TRAFFIC = [
    {"sources": "56dfd8cef016cf90", "workload": 3, "bundle": 2, "task": "vertex",
     "sample_compact": 556421428, "k_sample_per_launch": 113970779,
     "gather": 176148581, "gather_per_launch": 352297162,
     "sample_compact_l2_hit_rate": 0.5455, "gather_l2_hit_rate": 0.3312},
    {"sources": "56dfd8cef016cf90", "workload": 2, "bundle": 32, "task": "vertex",
     "sample_compact": 76145261, "k_sample_per_launch": 553555963,
     "gather": 249191661, "gather_per_launch": 7974133152,
     "sample_compact_l2_hit_rate": 0.727, "gather_l2_hit_rate": 0.3327},
]


def kernel_sources_digest():
    """A digest of the kernel and runtime sources' code: comments and
    whitespace are left out, so that editing a comment keeps measured
    counters valid while any change to the code drops them."""
    import hashlib
    import re
    d = os.path.join(ROOT, "paper_2112_15345_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".hpp", ".cpp")):
            text = open(os.path.join(d, f), encoding="utf-8").read()
            text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
            text = re.sub(r"//[^\n]*", " ", text)
            h.update(f.encode())
            h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def counter_traffic(workload, bundle, task="vertex"):
    digest = kernel_sources_digest()
    for t in COUNTER_TRAFFIC:
        if (t["sources"], t["workload"], t["bundle"], t.get("task", "vertex")) == (
                digest, workload, bundle, task):
            return t
    return None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_info():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def pipeline_name(args):
    return f"{args.workers} worker streams" if args.workers else "direct calls"


def percentiles(xs):
    import numpy as np
    if not xs:
        return None, None, None
    a = np.asarray(xs, dtype=np.float64)
    return tuple(float(np.percentile(a, q)) for q in (10, 50, 90))


# ---------------------------------------------------------------------------
# Units of work: warm-up and timed

def make_units(args, B):
    """Warm-up and timed units (lists of batch indices).  Every unit size the
    timed region uses is warmed up first, twice per worker stream, so that no
    bundle graph, workspace or pool growth happens while timing; the warm-up
    runs at least --warmup mini-batches.  Timed batches follow the warm-up."""
    K = args.steps
    timed_sizes = [B] * (K // B) + ([K % B] if K % B else [])
    per_size = 2 * max(args.workers, 1)
    warm_sizes = []
    for size in sorted(set(timed_sizes), reverse=True):
        warm_sizes += [size] * per_size
    while sum(warm_sizes) < args.warmup:
        warm_sizes.append(B)
    units, b = [], 0
    for size in warm_sizes:
        units.append(list(range(b, b + size)))
        b += size
    warm_n = b
    timed = []
    for size in timed_sizes:
        timed.append(list(range(b, b + size)))
        b += size
    return units, timed, warm_n


def run_units(args, g, units, timed, direct, submit, account):
    """Runs the warm-up units, then the timed ones between two device
    synchronisations.  direct(unit) returns the unit's Blocks (--workers 0);
    submit(pipe, unit) queues it on a pipeline of --workers streams (at most
    --depth mini-batches outstanding; no timed unit is submitted before the
    clock starts).  account(unit, blocks, t) runs on every returned timed unit
    with the host time it came back.  Returns the timed region's wall time."""
    import torch

    import paper_2112_15345_amd as hg

    if args.workers == 0:
        for u in units:
            direct(u)
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for u in timed:
            account(u, direct(u), time.perf_counter() - t_start)
        torch.cuda.synchronize()
        return time.perf_counter() - t_start
    B = max(len(u) for u in timed + units)
    depth = max(args.depth or 2 * args.workers * B, B)
    pipe = hg.Pipeline(g, workers=args.workers, capacity=depth, gather=args.gather_types)
    queue = units + timed
    state = {"next": 0, "outstanding": 0, "limit": len(units)}

    def submit_more():
        while (state["next"] < state["limit"] and
               state["outstanding"] + len(queue[state["next"]]) <= depth):
            u = queue[state["next"]]
            submit(pipe, u)
            state["outstanding"] += len(u)
            state["next"] += 1

    def take(u):
        out = []
        for _ in u:
            out.append(pipe.next())
            state["outstanding"] -= 1
        submit_more()
        return out

    submit_more()
    for u in units:
        take(u)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    state["limit"] = len(queue)
    submit_more()
    for u in timed:
        blist = take(u)
        account(u, blist, time.perf_counter() - t_start)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    pipe.close()
    return elapsed


# ---------------------------------------------------------------------------
# The vertex-seeded mini-batch (the default task)

def stage_bytes_model(g, nd, ns, ne, n_batches=1):
    """Algorithmic HBM bytes of sampling and compaction for n_batches
    mini-batches (nd, ns, ne summed over them), per stage.  Per hop, with D
    frontier vertices, P (vertex, edge type) pairs, S kept edges, U new
    vertices and R edge types per mini-batch: 8 D (read the frontier) + 16 P
    (indptr pairs) + 8 S (read the kept sources) + 8 (P + R) (block CSC) + 16 S
    (edge ID and the two local IDs) + 8 (D + U) (source lists).  The counting
    pass reads the frontier and the indptr pairs; the sampler reads the kept
    sources and writes the block CSC, the edge IDs and the destination IDs;
    the compaction writes the source lists; the relabel writes the source
    IDs."""
    out = {name: 0 for name in ("count", "sample", "select", "compact", "relabel")}
    R = g.R * n_batches
    for h in range(nd.shape[0]):
        D = int(nd[h].sum())
        U = int(ns[h].sum()) - D
        P = sum(int(nd[h, d]) for (_, d, _, _) in g.etypes)
        S = int(ne[h].sum())
        out["count"] += 8 * D + 16 * P
        out["sample"] += 8 * S + 8 * (P + R) + 12 * S
        out["compact"] += 8 * (D + U)
        out["relabel"] += 4 * S
    return out


# Timed units that carry events on a memory-bound dominant stage: one in
# ROOF_EVERY (the sampler's and the gather's launches carry them in every unit).
ROOF_EVERY = 8

# The kernels behind each stage, for the roofline of the dominant one.
STAGE_KERNELS = {
    "count": "k_count_scan (the counting pass: in-degree and kept count of every (vertex, "
             "edge type) pair, the sampler's work lists, one single-pass scan)",
    "select": "k_hub_finish (the K smallest candidates of every hub)",
    "compact": "k_bits_count, k_bits_scan, k_bits_assign (the new frontier: reached marks "
               "ranked into local IDs and source lists)",
    "relabel": "k_relabel (the source local ID of every kept edge)",
}


def blocks_equal(a, b, H, T, R, feat_types):
    """Every block array and every gathered feature byte of two results."""
    import torch
    for h in range(H):
        for t in range(T):
            na, sa = a.nodes(h, t)
            nb, sb = b.nodes(h, t)
            if na != nb or not torch.equal(sa, sb):
                return False
        for e in range(R):
            for x, y in zip(a.edges(h, e), b.edges(h, e)):
                if x.dtype != y.dtype or not torch.equal(x, y):
                    return False
    for t in feat_types:
        if not torch.equal(a.features(t).view(torch.uint8), b.features(t).view(torch.uint8)):
            return False
    return True


def oracle_check(args, wl, gen, fan, kept, cpu, timed, recompute):
    """Every timed mini-batch (or the first --check-batches of them) against
    the oracle's OpenMP build (the same oracle.c on every host core): every
    block array must equal the oracle's and the gathered feature bytes the
    rows of the oracle's input frontier.  The timed region keeps only its
    first results (a whole run's gathered rows would not fit), so each timed
    unit is made again after the clock, with the same bundles, seeds and
    sampling seeds; the results the timed region kept must equal those made
    again, bit for bit.  The oracle's time over the first batches, up to
    --cpu-budget seconds, is the CPU baseline."""
    import numpy as np
    import torch

    import oracle
    import workloads as W

    t0 = time.perf_counter()
    host_nt = [(n, None) for n in gen.num_nodes]
    host = oracle.HostGraph(host_nt, gen.host_etypes(), check=False, lib=oracle.load_omp())
    log(f"oracle host copy of the graph in {time.perf_counter() - t0:.1f}s")
    threads = oracle.threads(host.lib)
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    H, T, R = len(fan), len(gen.num_nodes), len(gen.etypes)
    kept_map = dict(kept)
    n_timed = sum(len(u) for u in timed)
    limit = n_timed if args.check_batches < 0 else min(args.check_batches, n_timed)
    spent, edges, timed_b, checked, bad, same = 0.0, 0, [], [], [], []
    for u in timed:
        if len(checked) >= limit:
            break
        blist = recompute(u)
        for b, blocks in zip(u, blist):
            if len(checked) >= limit:
                break
            ok = True
            if b in kept_map:
                same.append(b)
                if not blocks_equal(kept_map[b], blocks, H, T, R, feat_types):
                    ok = False
                    log(f"batch {b}: the timed result and the one made again differ")
            seeds = W.seeds_per_type(wl, b)
            t = time.perf_counter()
            ref = host.sample_blocks(seeds, fan, b)
            dt = time.perf_counter() - t
            if cpu and spent < args.cpu_budget:
                spent += dt
                edges += sum(v[3].size for v in ref["edges"].values())
                timed_b.append(b)
            for h in range(H):
                for ti in range(T):
                    n_dst, sg = blocks.nodes(h, ti)
                    if n_dst != ref["nodes"][(h, ti)][0] or \
                            not np.array_equal(sg.cpu().numpy(), ref["nodes"][(h, ti)][1]):
                        ok = False
                for e in range(R):
                    for x, y in zip(blocks.edges(h, e), ref["edges"][(h, e)]):
                        xn = x.cpu().numpy()
                        if xn.dtype != y.dtype or not np.array_equal(xn, y):
                            ok = False
            for ti in feat_types:
                f = gen.feats[ti]
                ids = torch.as_tensor(ref["input"][ti], device=f.device)
                got = blocks.features(ti)
                want = f.index_select(0, ids).to(got.device)
                if not torch.equal(got.view(torch.uint8), want.view(torch.uint8)):
                    ok = False
            checked.append(b)
            if not ok:
                bad.append(b)
            log(f"oracle batch {b}: {'equal' if ok else 'DIFFERENT'} "
                f"({dt:.1f}s on {threads} threads)")
            del ref
        del blist
    parity = {"batches": checked, "of_timed": n_timed, "equal": not bad, "different": bad,
              "timed_results_equal_remade": same,
              "what": "every block array (frontiers, source lists, CSC, COO local IDs, edge "
                      "IDs) and every gathered feature byte, element by element; the timed "
                      "units are made again after the clock (same bundles, seeds and "
                      "sampling seeds) and the results the timed region kept equal them bit "
                      "for bit"}
    base = None
    if cpu and timed_b:
        # the plain (one-thread) build too, when a mini-batch fits the budget
        # on one core (the OpenMP time times its threads bounds it from above)
        per_batch = spent / len(timed_b)
        if per_batch * threads <= args.cpu_budget:
            plain = oracle.HostGraph(host_nt, [(a, b_, ip, ix) for a, b_, ip, ix in host.etypes],
                                     check=False, lib=oracle.load())
            s_spent, s_edges, s_b = 0.0, 0, []
            for b in timed_b:
                t = time.perf_counter()
                ref = plain.sample_blocks(W.seeds_per_type(wl, b), fan, b)
                s_spent += time.perf_counter() - t
                s_edges += sum(v[3].size for v in ref["edges"].values())
                s_b.append(b)
                if s_spent >= args.cpu_budget:
                    break
            single = {"value": s_edges / s_spent if s_spent > 0 else None,
                      "unit": "sampled edges/s", "cores": 1,
                      "sample": f"{len(s_b)} of the same mini-batches, the plain build"}
        else:
            single = {"value": None, "cores": 1,
                      "sample": f"not run: one mini-batch would take up to "
                                f"{per_batch * threads:.0f} s on one core"}
        base = {"value": edges / spent if spent > 0 else None, "unit": "sampled edges/s",
                "cores": threads, "kind": "oracle",
                "sample": f"{len(timed_b)} whole timed mini-batches (batches {timed_b[0]}.."
                          f"{timed_b[-1]}) of the same workload, about {args.cpu_budget:.0f} s "
                          f"of CPU work: sampling and compaction by the OpenMP build of the "
                          f"oracle (pairs, relabel and gather loops on every host core), "
                          f"{edges} sampled edges in {spent:.2f} s; the feature gather is "
                          f"checked on the GPU against the oracle's input frontier rather than "
                          f"timed on the host",
                "single_thread": single,
                **host_info()}
    return parity, base


def vertex_main(args, wl, gen, g):
    import numpy as np
    import torch

    import paper_2112_15345_amd as hg
    import workloads as W

    dev = g.device
    fan = wl.fanout_matrix()
    H = len(fan)
    B = max(1, args.bundle)
    units, timed, warm_n = make_units(args, B)
    n_batches = warm_n + args.steps
    seeds = [[None if s is None else torch.as_tensor(s, device=dev)
              for s in W.seeds_per_type(wl, b)] for b in range(n_batches)]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    args.gather_types = feat_types
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}
    # the timed region's launches carry events only on the sampler (the
    # dominant kernel) and the gather: events on every stage's launches cost
    # about 12% of a step here.  Every stage is timed in a profile pass after
    # the clock stops.

    if args.copy_calibration_mb > 0:
        # a copy of known size, untimed, for scaling the memory counters
        src = torch.ones(args.copy_calibration_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy of {args.copy_calibration_mb} MiB done")
        del src, dst

    def direct(u, ev=None):
        return g.sample_bundle([seeds[b] for b in u], fan, u, gather=feat_types,
                               stage_events=ev or stage_ev.get(u[0]))

    def submit(pipe, u):
        pipe.submit_bundle([seeds[b] for b in u], fan, u, stage_events=stage_ev.get(u[0]))

    # the stage with the most device time, found before the clock on the first
    # unit (direct calls with every stage timed, twice: the first call's setup
    # is left out); the timed region also carries events on that stage's
    # launches, for the roofline of the dominant kernel
    probe_u = (units or timed)[0]
    for _ in range(2):
        ev = hg.StageEvents(H)
        blist = direct(probe_u, ev)
        torch.cuda.synchronize()
        probe_ms = {name: sum(ev.stage_ms(h, st) for h in range(H))
                    for st, name in enumerate(hg.STAGE_NAMES)}
        probe_ms["gather"] = ev.gather_ms()
        del blist
    probe_dom = max(probe_ms, key=probe_ms.get)
    timed_stages = ("sample",) if probe_dom in ("sample", "gather") else ("sample", probe_dom)
    # events cost time on the launches that carry them (on every stage's
    # launches about 12% of a step), so on this stage only every ROOF_EVERY-th
    # timed unit carries them
    roof_units = [u for i, u in enumerate(timed) if i % ROOF_EVERY == 0]
    stage_ev = {u[0]: hg.StageEvents(H, stages=timed_stages if i % ROOF_EVERY == 0
                                     else ("sample",)) for i, u in enumerate(timed)}

    rec = []   # per timed unit: (unit, done_s, edges, rows_by_type, nd, ns, keys, ne)
    kept = []  # (batch, Blocks) checked against the oracle afterwards

    def account(u, blist, t_done):
        nd = np.zeros((H, g.T), np.int64)
        ns = np.zeros((H, g.T), np.int64)
        ne = np.zeros((H, g.R), np.int64)
        keys = None
        rows = {t: 0 for t in feat_types}
        for b, blocks in zip(u, blist):
            d, s, k = blocks.counts()
            nd += d
            ns += s
            keys = k  # a bundle's handles hold the bundle's totals
            ne += np.asarray(blocks.edge_counts(), np.int64).reshape(H, g.R)
            for t in feat_types:
                rows[t] += blocks.num_input_nodes(t)
            if len(kept) < 2:  # compared with the same units made again after the clock
                kept.append((b, blocks))
        rec.append((u, t_done, int(ne.sum()), rows, nd, ns, keys, ne))

    log(f"warm-up: {warm_n} mini-batches in units of {sorted(set(len(u) for u in units))}; "
        f"timed: {args.steps} in units of {B} ({pipeline_name(args)})")
    elapsed = run_units(args, g, units, timed, direct, submit, account)
    steps = args.steps
    edges = sum(r[2] for r in rec)
    gbytes = sum(n * row_bytes[t] for r in rec for t, n in r[3].items())
    ms_per_step = elapsed / steps * 1e3
    # per-step spread: the interval between successive units' returns
    per_step, prev = [], 0.0
    for u, t_done, *_ in rec:
        per_step.append((t_done - prev) / len(u) * 1e3)
        prev = t_done
    p10, p50, p90 = percentiles(per_step)

    # device time of the sampler's and the gather's launches over the timed
    # region, from the events those launches carried
    sample_ms = sum(stage_ev[u[0]].stage_ms(h, hg.HG_STAGE_SAMPLE) for u in timed
                    for h in range(H))
    sample_launches = len(timed) * H
    gather_ms = sum(stage_ev[u[0]].gather_ms() for u in timed)
    keys = sum(int(r[6].sum()) for r in rec)
    g_alg = sum(n * (2 * row_bytes[t] + 8) for r in rec for t, n in r[3].items())
    if args.host_features:
        g_alg = gbytes  # the rows cross the host link once; that link is the roof

    # profile pass (untimed): the first timed units again, direct calls on one
    # stream, every stage's launches carrying events
    prof_units = timed[:max(1, min(len(timed), args.profile_units))]
    stage_ms = {name: 0.0 for name in hg.STAGE_NAMES}
    prof_alg = prof_steps = prof_keys = 0
    prof_stage_alg = {name: 0 for name in hg.STAGE_NAMES}
    hop_ms = [{name: 0.0 for name in hg.STAGE_NAMES} for _ in range(H)]
    hop_keys = np.zeros(H, np.int64)
    hop_kept = np.zeros(H, np.int64)
    prof_gather_ms = 0.0
    for u in prof_units:
        ev = hg.StageEvents(H)
        blist = direct(u, ev)
        torch.cuda.synchronize()
        for h in range(H):
            for st, name in enumerate(hg.STAGE_NAMES):
                stage_ms[name] += ev.stage_ms(h, st)
                hop_ms[h][name] += ev.stage_ms(h, st)
        hop_keys += np.asarray(blist[0].counts()[2], np.int64)  # the bundle's keys per hop
        prof_gather_ms += ev.gather_ms()
        nd = sum(b.counts()[0] for b in blist)
        ns = sum(b.counts()[1] for b in blist)
        ne = sum(np.asarray(b.edge_counts(), np.int64).reshape(H, g.R) for b in blist)
        hop_kept += ne.sum(axis=1)
        for name, v in stage_bytes_model(g, nd, ns, ne, len(u)).items():
            prof_stage_alg[name] += v
            prof_alg += v
        prof_keys += int(np.asarray(blist[0].counts()[2]).sum())  # the bundle's keys
        prof_steps += len(u)
        del blist
    sc_ms = sum(stage_ms.values())

    # the sampler's key loop alone, over as many keys as a timed step
    hip_ev = hg.HipEvents(2)
    n_groups = 64 * (1 << 22)
    hg.bench_philox(1, 0, 0, 64 * 1024, 1000)  # first launch, untimed
    cnt = hg.bench_philox(7, 1, 2, n_groups, 1 << 20, events=tuple(hip_ev.events))
    torch.cuda.synchronize()
    loop_ms = hip_ev.elapsed_ms(*hip_ev.events)
    loop_keys_s = 4 * n_groups / (loop_ms / 1e3)
    del cnt

    # context for the peak: a plain 4 GiB device-to-device copy, best of 6
    copy_gbps = None
    if not args.host_features:
        src = torch.ones(1 << 32, dtype=torch.uint8, device=dev)
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

    traffic = counter_traffic(args.workload, B)
    peak = HOST_LINK_PEAK_GBS if args.host_features else HBM_PEAK_GBS
    g_gbps = g_alg / (gather_ms / 1e3) / 1e9 if gather_ms > 0 else 0.0
    gather = {"kernel": "k_gather_multi (all featured types, one launch per bundle)",
              "achieved": g_gbps, "peak": peak, "unit": "GB/s", "frac": g_gbps / peak,
              "bound": "host link" if args.host_features else "hbm",
              "ms_per_step": gather_ms / steps,
              "algorithmic_bytes_per_step": g_alg / steps,
              "traffic_per_step": traffic["gather"] if traffic else None,
              "l2_hit_rate": traffic.get("gather_l2_hit_rate") if traffic else None}
    sample_s = sample_ms / 1e3
    philox = {"keys_per_step": keys / steps,
              "keys_per_s": keys / sample_s if sample_s > 0 else None,
              "peak_keys_per_s": PHILOX_PEAK_KEYS,
              "frac": (keys / sample_s) / PHILOX_PEAK_KEYS if sample_s > 0 else None,
              "loop_alone_keys_per_s": loop_keys_s,
              "loop_alone_frac": loop_keys_s / PHILOX_PEAK_KEYS,
              "hub_loop_issue_bound_keys_per_s": VALU_LANE_OPS * 4 / PHILOX_HUB_VALU_PER_CALL,
              "peak_derivation": f"{VALU_LANE_OPS:.4g} lane-ops/s x 4 keys / "
                                 f"{PHILOX_VALU_PER_CALL} vector instructions per call"}
    sc = {"kernels": "counting pass, sampler, hub selection, compaction, relabel",
          "measured": f"profile pass: {prof_steps} of the timed mini-batches again, direct "
                      f"calls on one stream, every stage's launches carrying HIP events",
          "ms_per_step": sc_ms / prof_steps,
          "stage_ms_per_step": {k: v / prof_steps for k, v in stage_ms.items()},
          "per_hop": [{"stage_ms_per_step": {k: v / prof_steps for k, v in hop_ms[h].items()},
                       "kept_edges_per_step": int(hop_kept[h]) / prof_steps,
                       "keys_per_step": int(hop_keys[h]) / prof_steps,
                       "sampler_keys_per_s": (int(hop_keys[h]) / (hop_ms[h]["sample"] / 1e3)
                                              if hop_ms[h]["sample"] > 0 else None)}
                      for h in range(H)],
          "gather_ms_per_step": prof_gather_ms / prof_steps,
          "algorithmic_bytes_per_step": prof_alg / prof_steps,
          "algorithmic_GBps": prof_alg / (sc_ms / 1e3) / 1e9 if sc_ms > 0 else None,
          "algorithmic_frac": prof_alg / (sc_ms / 1e3) / 1e9 / HBM_PEAK_GBS if sc_ms > 0 else None,
          "counter_bytes_per_step": traffic["sample_compact"] if traffic else None}
    if traffic:
        rate = traffic["sample_compact"] / (sc_ms / prof_steps / 1e3) / 1e9
        sc["counter_GBps"] = rate
        sc["counter_frac"] = rate / HBM_PEAK_GBS
        sc["counter_over_algorithmic"] = traffic["sample_compact"] / (prof_alg / prof_steps)
        sc["l2_hit_rate"] = traffic.get("sample_compact_l2_hit_rate")
    # the roofline of the kernel with the most device time (from the profile
    # pass), its rate measured over the timed region; a stage whose launches
    # carried no events there (the probe before the clock chose another) is
    # passed over for the largest one that did
    per_kernel = dict(stage_ms, gather=prof_gather_ms)
    dominant = max(per_kernel, key=per_kernel.get)
    timed_kinds = ("gather",) + timed_stages
    reported = dominant if dominant in timed_kinds else max(timed_kinds, key=per_kernel.get)
    if reported == "gather":
        n_l = len(timed)
        roofline = {"bound": gather["bound"], "kernel": gather["kernel"],
                    "achieved": g_gbps, "peak": peak, "unit": "GB/s", "frac": g_gbps / peak,
                    "traffic": traffic["gather_per_launch"] if traffic else None,
                    "algorithmic_per_launch": g_alg / n_l,
                    "avg_launch_us": gather_ms / n_l * 1e3}
    elif reported != "sample":
        # a memory-bound stage: its share of the byte model over its launches
        st = hg.STAGE_NAMES.index(reported)
        d_ms = sum(stage_ev[u[0]].stage_ms(h, st) for u in roof_units for h in range(H))
        n_l = len(roof_units) * H
        first = {u[0] for u in roof_units}
        alg = sum(stage_bytes_model(g, r[4], r[5], r[7], len(r[0]))[reported]
                  for r in rec if r[0][0] in first)
        a_gbps = alg / (d_ms / 1e3) / 1e9 if d_ms > 0 else 0.0
        roofline = {"bound": "hbm", "kernel": STAGE_KERNELS[reported],
                    "achieved": a_gbps, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": a_gbps / HBM_PEAK_GBS, "traffic": None,
                    "algorithmic_per_launch": alg / n_l, "avg_launch_us": d_ms / n_l * 1e3,
                    "per_launch": "one hop of one call (a bundle's mini-batches together)",
                    "measured_on": f"{len(roof_units)} of the {len(timed)} timed units "
                                   f"(every {ROOF_EVERY}th carries events on this stage)"}
        if stage_ms[reported] > 0:
            alone = prof_stage_alg[reported] / (stage_ms[reported] / 1e3) / 1e9
            roofline["alone"] = {
                "achieved": alone, "frac": alone / HBM_PEAK_GBS,
                "measured": f"profile pass (the first timed units again, direct calls on one "
                            f"stream): the {reported} stage's launches with nothing beside them"}
    else:
        achieved = keys / sample_s / 1e9 if sample_s > 0 else 0.0
        roofline = {"bound": "alu", "kernel": "k_sample (the sampler: random keys of every "
                    "in-edge of a selecting pair, then the kept edges)",
                    "achieved": achieved, "peak": PHILOX_PEAK_KEYS / 1e9, "unit": "Gkeys/s",
                    "frac": achieved / (PHILOX_PEAK_KEYS / 1e9),
                    "traffic": traffic["k_sample_per_launch"] if traffic else None,
                    "algorithmic_per_launch": keys / sample_launches,
                    "avg_launch_us": sample_ms / sample_launches * 1e3,
                    "peak_source": philox["peak_derivation"]}
        # the same launches alone on the GPU: the profile pass (one stream)
        if stage_ms["sample"] > 0:
            alone = prof_keys / (stage_ms["sample"] / 1e3) / 1e9
            roofline["alone"] = {
                "achieved": alone, "frac": alone / (PHILOX_PEAK_KEYS / 1e9),
                "measured": "profile pass (the first timed units again, direct calls on one "
                            "stream): k_sample launches with nothing beside them"}
    if reported != dominant:
        roofline["note"] = (f"the {dominant} stage had the most device time in the profile "
                            f"pass, but the probe before the clock found {probe_dom}: the "
                            f"roofline of {reported}, whose launches carried events, is "
                            f"reported")
    roofline["device_copy_GBps"] = copy_gbps
    result = {
        "metric": "sampled edges/s + gathered feature GB/s per mini-batch (1 GPU), % of HBM peak",
        "value": edges / elapsed,
        "unit": "sampled edges/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "warmup_run": warm_n,
        "ms_per_step": ms_per_step,
        "ms_per_step_p10": p10, "ms_per_step_p50": p50, "ms_per_step_p90": p90,
        "probe": {"dominant": probe_dom, "calls": 2, "mini_batches": 2 * len(probe_u),
                  "measured": "before warm-up: the first unit twice, direct calls, every "
                              "stage timed"},
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
                   "bundle": B, "pipeline": pipeline_name(args)},
        "gathered_GBps": gbytes / elapsed / 1e9,
        "sampled_edges_per_step": edges / steps,
        "roofline": roofline,
        "gather": gather,
        "sample_compact": sc,
        "philox": philox,
    }
    if not args.no_cpu_baseline or args.check_batches != 0:
        def remake(u):  # the timed unit again: direct call, no events
            blist = g.sample_bundle([seeds[b] for b in u], fan, u, gather=feat_types)
            torch.cuda.synchronize()
            return blist
        parity, base = oracle_check(args, wl, gen, fan, kept, not args.no_cpu_baseline, timed,
                                    remake)
        result["parity"] = parity
        if not args.no_cpu_baseline:
            result["cpu_baseline"] = base
    print(json.dumps(result), flush=True)


# ---------------------------------------------------------------------------
# Link prediction and layer-wise tasks

def drive_units(args, g, direct, submit, account):
    units, timed, warm_n = make_units(args, max(1, args.bundle))

    def acc(u, blist, _t):
        for b in blist:
            account(b)

    elapsed = run_units(args, g, units, timed, lambda u: direct(u[0], u[-1] + 1),
                        lambda pipe, u: submit(pipe, u[0], u[-1] + 1), acc)
    return elapsed, warm_n


def link_main(args, wl, gen, g):
    """Edge-seeded (link-prediction) mini-batches: targets of one forward
    relation, their endpoints as seeds, one negative per target, targets and
    their reverse edges excluded, the paper's link-prediction fanouts [25, 15]
    per hop, every featured type gathered."""
    import torch

    import paper_2112_15345_amd as hg
    import workloads as W

    dev = g.device
    rev_et, rev_eid = W.reverse_maps(gen)
    exclude = hg.HG_EXCLUDE_REVERSE if rev_et is not None else hg.HG_EXCLUDE_SELF
    link_et = gen.etype_names.index("cites") if "cites" in gen.etype_names else 0
    fan = [[k] * g.R for k in W.LINK_FANOUTS]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    args.gather_types = feat_types
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}
    n_max = make_units(args, max(1, args.bundle))[2] + args.steps
    targets = [[None if x is None else torch.as_tensor(x, device=dev)
                for x in W.link_targets(gen, b, link_et)] for b in range(n_max)]
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

    elapsed, warm_n = drive_units(args, g, direct, submit, account)
    edges, rows, gbytes = totals
    print(json.dumps({
        "metric": "sampled edges/s + gathered feature GB/s per mini-batch (1 GPU), % of HBM peak",
        "value": edges / elapsed, "unit": "sampled edges/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "warmup_run": warm_n,
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
    }), flush=True)


def layers_main(args, wl, gen, g):
    """Layer-wise (LADIES) mini-batches: the workload's seeds, 512 draws per
    node type in each of two hops, every featured type gathered."""
    import torch

    import workloads as W

    dev = g.device
    sizes = [[k] * g.T for k in W.LAYER_SIZES]
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    args.gather_types = feat_types
    row_bytes = {t: gen.feats[t].shape[1] * gen.feats[t].element_size() for t in feat_types}
    n_max = make_units(args, max(1, args.bundle))[2] + args.steps
    seeds = [[None if s is None else torch.as_tensor(s, device=dev)
              for s in W.seeds_per_type(wl, b)] for b in range(n_max)]

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

    elapsed, warm_n = drive_units(args, g, direct, submit, account)
    edges, rows, gbytes = totals
    result = {
        "metric": "kept edges/s + gathered feature GB/s per layer-wise mini-batch (1 GPU)",
        "value": edges / elapsed, "unit": "kept edges/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "warmup_run": warm_n,
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
        host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False,
                                lib=oracle.load_omp())
        spent = 0.0
        cedges = nb = 0
        first = n_max - args.steps
        for b in range(first, n_max):
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
            "value": cedges / spent, "unit": "kept edges/s", "cores": oracle.threads(host.lib),
            "kind": "oracle",
            "sample": f"{nb} whole layer-wise mini-batches (batches {first}..{first + nb - 1}: "
                      f"sampling, compaction, gather) in {spent:.2f} s, OpenMP build",
            **host_info()}
    print(json.dumps(result), flush=True)


# ---------------------------------------------------------------------------
# The sampler's key loop alone

def philox_main(args):
    """The sampler's key loop (hg_bench_philox) over 2^30 key groups, timed by
    HIP events carried by its launch: the measured rate of the random keys
    beside the vector-ALU roof derived from the chip's unit counts."""
    import torch

    import paper_2112_15345_amd as hg

    ev = hg.HipEvents(2)
    n_groups = 1 << 30
    hg.bench_philox(1, 0, 0, 64 * 1024, 1000)
    rates = []
    for rep in range(max(1, args.steps)):
        hg.bench_philox(rep, 1, 2, n_groups, 1 << 20, events=tuple(ev.events))
        torch.cuda.synchronize()
        rates.append(4 * n_groups / (ev.elapsed_ms(*ev.events) / 1e3))
    best = max(rates)
    med = sorted(rates)[len(rates) // 2]
    print(json.dumps({
        "metric": "random keys/s of the sampler's key loop alone (1 GPU)",
        "value": best, "unit": "keys/s", "n_gpus": 1, "steps": len(rates), "warmup": 1,
        "ms_per_step": 4 * n_groups / med * 1e3,
        "higher_is_better": True, "dtype": "u32", "data": "synthetic",
        "config": {"workload": "Philox4x32-10 edge keys of 2^32 edge IDs, one (seed, hop, edge "
                               "type) line, candidate threshold 2^20"},
        "roofline": {"bound": "alu", "achieved": best / 1e9, "peak": PHILOX_PEAK_KEYS / 1e9,
                     "unit": "Gkeys/s", "frac": best / PHILOX_PEAK_KEYS, "traffic": None,
                     "peak_source": f"{VALU_LANE_OPS:.4g} lane-ops/s x 4 keys / "
                                    f"{PHILOX_VALU_PER_CALL} vector instructions per call",
                     "loop_peak_Gkeys": VALU_LANE_OPS * 4 / PHILOX_LOOP_VALU_PER_CALL / 1e9},
        "median_keys_per_s": med,
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed mini-batches (default per workload: 40 for workload 3)")
    ap.add_argument("--warmup", type=int, default=5,
                    help="untimed mini-batches first, at least; every unit size the timed "
                         "region uses is also warmed up twice per worker stream")
    ap.add_argument("--workload", type=int, default=3,
                    help="1 tiny, 2 academic, 3 billion-edge share (default), 4 knowledge "
                         "graph, 5 gather-heavy academic")
    ap.add_argument("--workers", type=int, default=None,
                    help="pipeline worker threads (own streams); 0 = direct calls on one "
                         "stream (default per workload)")
    ap.add_argument("--bundle", type=int, default=None,
                    help="mini-batches per launch sequence (1..32; default per workload)")
    ap.add_argument("--depth", type=int, default=0,
                    help="mini-batches outstanding in the pipeline (default 2 x workers x "
                         "bundle)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--check-batches", type=int, default=None,
                    help="timed mini-batches compared with the oracle, from the first (default "
                         "-1: every one); 0 skips the check")
    ap.add_argument("--profile-units", type=int, default=4,
                    help="timed units re-run after the timed region with every stage timed")
    ap.add_argument("--cpu-budget", type=float, default=20.0,
                    help="seconds of oracle time after which the check stops")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after warm-up (untimed), copy this many MiB device to device "
                         "once: a copy of known size for scaling memory counters")
    ap.add_argument("--host-features", action="store_true",
                    help="feature tables in pinned host memory, gathered over the host link "
                         "(zero-copy); the gather rate then includes that link")
    ap.add_argument("--task", choices=("vertex", "link", "layers"), default="vertex")
    ap.add_argument("--mode", choices=("step", "philox"), default="step",
                    help="step: mini-batches (default); philox: the sampler's key loop alone")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        sys.exit(2)
    if args.mode == "philox":
        if args.steps is None:
            args.steps = 5
        return philox_main(args)
    dw, db, ds = DEFAULTS.get(args.workload, (2, 32, 320))
    if args.workers is None:
        args.workers = dw
    if args.bundle is None:
        args.bundle = db
    if args.steps is None:
        args.steps = ds
    if args.check_batches is None:
        args.check_batches = -1  # every timed mini-batch

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
    return vertex_main(args, wl, gen, g)


if __name__ == "__main__":
    main()
