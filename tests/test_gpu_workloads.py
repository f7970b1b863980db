"""HIP path against the oracle on full-size workloads, with the same calls and
launch configuration that bench.py times: every block array of every hop and
the gathered feature bytes, element by element."""
import sys

import numpy as np
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


_cache = {}


def workload_graph(idx):
    """(generated graph on the GPU, library graph, oracle host graph), cached."""
    if idx not in _cache:
        _cache.clear()
        torch.cuda.empty_cache()
        wl = W.WORKLOADS[idx]
        say(f"generating workload {idx}: {wl.name}")
        gen = W.make_graph(wl, device="cuda")
        g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
        # the OpenMP build of the oracle: the same results on every host core
        host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False,
                                lib=oracle.load_omp())
        _cache[idx] = (wl, gen, g, host)
    return _cache[idx]


# at least 20 mini-batches each (different seeds, sampling seeds and hub mixes)
@pytest.mark.parametrize("idx,batches", [(2, tuple(range(20))), (5, tuple(range(20)))])
def test_workload_parity(idx, batches):
    wl, gen, g, host = workload_graph(idx)
    fan = wl.fanout_matrix()
    for b in batches:
        seeds = W.seeds_per_type(wl, b)
        say(f"workload {idx} batch {b}: GPU")
        # the call bench.py times: blocks and input features together
        blocks = g.sample_blocks(gpu_seeds(seeds), fan, b, gather="all")
        got = result_dict(g, blocks)
        say(f"workload {idx} batch {b}: oracle")
        ref = host.sample_blocks(seeds, fan, b)
        diffs = compare(ref, got, g.T, g.R, len(fan))
        assert not diffs, f"batch {b}: " + "\n".join(diffs[:10])
        allx = g.gather_features_all(blocks)
        for t, f in enumerate(gen.feats):
            if f is None:
                assert blocks.features(t) is None
                continue
            ids = ref["input"][t]
            want = host.gather(t, ids).tobytes()
            for x in (blocks.features(t), allx[t]):
                assert x.contiguous().view(torch.uint8).cpu().numpy().tobytes() == want, \
                    f"batch {b} type {t}: gathered bytes differ"
        say(f"workload {idx} batch {b}: equal "
            f"({sum(v[3].size for v in ref['edges'].values())} edges)")


@pytest.mark.parametrize("idx,B,first", [(2, 32, 192), (5, 8, 48)])
def test_workload_pipeline_launch(idx, B, first):
    """A workload as bench.py runs it by default: bundles of B mini-batches
    (32 on the academic graph, 8 on the gather-heavy one) submitted to a
    pipeline of 3 worker streams (at most 6 B outstanding), here the first
    three timed bundles.  Every mini-batch comes back in order and equals its
    own single call (blocks and gathered bytes); every mini-batch of the first
    bundle, and the first and last of the others, also equal the oracle."""
    wl, gen, g, host = workload_graph(idx)
    fan = wl.fanout_matrix()
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    batches = list(range(first, first + 3 * B))
    bundles = [batches[i:i + B] for i in range(0, len(batches), B)]
    seeds = {b: gpu_seeds(W.seeds_per_type(wl, b)) for b in batches}
    pipe = hg.Pipeline(g, workers=3, capacity=6 * B, gather=feat_types)
    try:
        for u in bundles:
            pipe.submit_bundle([seeds[b] for b in u], fan, u)
        got = {b: pipe.next() for b in batches}
    finally:
        pipe.close()
    for u in bundles:
        say(f"pipeline bundle {u[0]}..{u[-1]}")
        for b in u:
            direct = g.sample_blocks(seeds[b], fan, b, gather="all")
            mine = result_dict(g, got[b])
            diffs = compare(result_dict(g, direct), mine, g.T, g.R, len(fan))
            assert not diffs, f"batch {b}: " + "\n".join(diffs[:10])
            for t in feat_types:
                assert torch.equal(got[b].features(t).view(torch.uint8),
                                   direct.features(t).view(torch.uint8)), f"batch {b} type {t}"
            if u is bundles[0] or b in (u[0], u[-1]):
                ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
                diffs = compare(ref, mine, g.T, g.R, len(fan))
                assert not diffs, f"batch {b} vs oracle: " + "\n".join(diffs[:10])
                for t in feat_types:
                    want = host.gather(t, ref["input"][t]).tobytes()
                    assert got[b].features(t).contiguous().view(torch.uint8).cpu().numpy() \
                        .tobytes() == want, f"batch {b} type {t}: gathered bytes differ"
                say(f"batch {b}: equal to the oracle")
            del direct


def test_workload_invariants_with_forced_ties():
    """Academic workload with 4-bit keys (ties everywhere, hub fallbacks), one
    batch: GPU == oracle, and the definition checks hold on the GPU result."""
    wl, gen, g, host = workload_graph(2)
    fan = [[10] * g.R]
    seeds = W.seeds_per_type(wl, 3)
    blocks = g.sample_blocks(gpu_seeds(seeds), fan, 3, key_bits=4)
    got = result_dict(g, blocks)
    ref = host.sample_blocks(seeds, fan, 3, key_bits=4)
    assert not compare(ref, got, g.T, g.R, 1)
    ets = gen.host_etypes()
    fails = pins.check_blocks(gen.num_nodes, ets, seeds, fan, 3, 4, got, brute=False)
    assert not fails, "\n".join(fails[:5])
