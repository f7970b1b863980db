"""HIP path against the oracle on the two largest workloads, at full size: the
billion-edge single-GPU share (3 node types, 1.2B edges, 3 hops) and the
200-relation knowledge graph (20M nodes, 300M edges).  Every block array and
the gathered feature bytes are compared element by element for three
mini-batches each (different seeds, sampling seeds and hub mixes); the
definition checks of the pins run on the first GPU result as well.  On the
billion-edge share the first two mini-batches go through the launch bench.py
times by default (a pipeline of 3 worker streams, bundles of 2), the third
through a single call.  The oracle is its OpenMP build (the same source,
every host core)."""
import sys
import time

import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import compare, gpu_seeds, result_dict

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("idx,batches", [(4, (0, 1, 7)), (3, (0, 1, 7))])
def test_large_workload_parity(idx, batches):
    torch.cuda.empty_cache()
    wl = W.WORKLOADS[idx]
    t0 = time.time()
    gen = W.make_graph(wl, device="cuda")
    torch.cuda.synchronize()
    say(f"workload {idx}: generated in {time.time() - t0:.1f}s")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    fan = wl.fanout_matrix()
    got, outs = {}, {}

    def keep(b, blocks):
        outs[b] = {t: blocks.features(t).contiguous().view(torch.uint8).cpu().numpy()
                   for t, f in enumerate(gen.feats) if f is not None}
        got[b] = result_dict(g, blocks)

    single = list(batches)
    if idx == 3:
        # bench.py's default launch: 3 worker streams, bundles of 2
        t0 = time.time()
        pair = list(batches[:2])
        pipe = hg.Pipeline(g, workers=3, capacity=12, gather="all")
        try:
            pipe.submit_bundle([gpu_seeds(W.seeds_per_type(wl, b)) for b in pair], fan, pair)
            for b in pair:
                blocks = pipe.next()
                keep(b, blocks)
                del blocks
        finally:
            pipe.close()
        single = list(batches[2:])
        say(f"workload {idx} batches {pair}: pipeline bundle and copy-out in "
            f"{time.time() - t0:.1f}s")
    for b in single:
        t0 = time.time()
        blocks = g.sample_blocks(gpu_seeds(W.seeds_per_type(wl, b)), fan, b, gather="all")
        keep(b, blocks)
        del blocks
        say(f"workload {idx} batch {b}: GPU mini-batch and copy-out in {time.time() - t0:.1f}s")
    del g

    t0 = time.time()
    host_et = gen.host_etypes()
    host_nt = gen.host_ntypes()
    del gen
    torch.cuda.empty_cache()
    say(f"workload {idx}: host copies in {time.time() - t0:.1f}s")
    host = oracle.HostGraph(host_nt, host_et, check=False, lib=oracle.load_omp())
    for b in batches:
        t0 = time.time()
        seeds = W.seeds_per_type(wl, b)
        ref = host.sample_blocks(seeds, fan, b)
        say(f"workload {idx} batch {b}: oracle mini-batch in {time.time() - t0:.1f}s "
            f"({sum(v[3].size for v in ref['edges'].values())} edges, "
            f"{oracle.threads(host.lib)} threads)")
        diffs = compare(ref, got[b], len(host_nt), len(host_et), len(fan))
        assert not diffs, f"batch {b}: " + "\n".join(diffs[:10])
        if b == batches[0]:
            fails = pins.check_blocks([n for n, _ in host_nt], host_et, seeds, fan, b, 32,
                                      got[b], brute=False)
            assert not fails, "\n".join(fails[:5])
        for t, x in outs[b].items():
            want = host.gather(t, ref["input"][t])
            assert x.tobytes() == want.tobytes(), f"batch {b} type {t}: gathered bytes differ"
        say(f"workload {idx} batch {b}: equal")
