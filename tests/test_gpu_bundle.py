"""Bundled mini-batches (hg_sample_blocks_bundle) against single calls and the
oracle: every batch of a bundle is the mini-batch its own call would make
(blocks and gathered features), for bundles of several sizes, on random
heterographs (hubs, ties, take-all) and the tiny and academic workloads."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import compare, gpu_graph, gpu_seeds, result_dict

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def feats_of(g, b):
    return {t: b.features(t).cpu().numpy().tobytes() for t, (_, f) in enumerate(g.ntypes)
            if f is not None}


def check_bundle(g, seeds_list, fan, sigmas, H):
    bundle = g.sample_bundle(seeds_list, fan, sigmas, gather="all")
    assert len(bundle) == len(seeds_list)
    for k, (seeds, sg) in enumerate(zip(seeds_list, sigmas)):
        single = g.sample_blocks(seeds, fan, sg, gather="all")
        diffs = compare(result_dict(g, single), result_dict(g, bundle[k]), g.T, g.R, H)
        assert not diffs, f"batch {k}: " + "\n".join(diffs[:10])
        assert feats_of(g, bundle[k]) == feats_of(g, single)
    return bundle


@pytest.mark.parametrize("B", [2, 3, 5])
def test_bundle_tiny_workload(B):
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    fan = wl.fanout_matrix()
    seeds_list = [gpu_seeds(W.seeds_per_type(wl, b)) for b in range(B)]
    bundle = check_bundle(g, seeds_list, fan, list(range(B)), len(fan))
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes())
    ref = host.sample_blocks(W.seeds_per_type(wl, B - 1), fan, B - 1)
    assert not compare(ref, result_dict(g, bundle[B - 1]), g.T, g.R, len(fan))
    # freeing the handles in any order keeps the others valid
    first = result_dict(g, bundle[0])
    del bundle[1:]
    torch.cuda.synchronize()
    assert not compare(first, result_dict(g, bundle[0]), g.T, g.R, len(fan))


@pytest.mark.parametrize("B", [8, 13, 32])
def test_bundle_tiny_workload_per_xcd(B):
    """Bundles of 8 or more mini-batches order the sampler's and the relabel's
    blocks per XCD (each XCD takes a contiguous eighth of every role); 8 gives
    one block per XCD and role, 13 splits mini-batches between XCDs, 32 is the
    largest bundle.  Every mini-batch equals its own single call and the
    oracle."""
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    fan = wl.fanout_matrix()
    batches = list(range(3, 3 + B))
    bundle = check_bundle(g, [gpu_seeds(W.seeds_per_type(wl, b)) for b in batches], fan,
                          batches, len(fan))
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes())
    for b, blocks in zip(batches, bundle):
        ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
        diffs = compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
        assert not diffs, f"batch {b}: " + "\n".join(diffs[:10])


def test_bundle_random_heterographs_per_xcd():
    """Random heterographs (selections, take-all, empty seed lists) in bundles
    of 8 to 12, then a graph with hubs of 2900 in-edges (chunked hub
    sampling) in a bundle of 9: the per-XCD block order against single
    calls."""
    rng = np.random.default_rng(2024)
    for c in range(6):
        nn, ets, feats, seeds, fanouts, sigma, bits = pins.random_case(rng, max_nodes=300,
                                                                       max_deg=300)
        g = gpu_graph(nn, ets, feats)
        B = int(rng.integers(8, 13))
        seeds_list = []
        for k in range(B):
            s = [np.sort(rng.choice(n, size=min(n, int(rng.integers(0, 12))), replace=False))
                 if n else np.zeros(0, np.int64) for n in nn]
            seeds_list.append(gpu_seeds(s))
        say(f"case {c}: T={len(nn)} R={len(ets)} H={len(fanouts)} B={B}")
        check_bundle(g, seeds_list, fanouts, [sigma + 7 * k for k in range(B)], len(fanouts))
    n = 3000
    deg = np.where(np.arange(n) % 97 == 0, 2900, rng.integers(0, 40, n))
    indptr = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    indices = np.concatenate([np.sort(rng.choice(n, size=int(d), replace=False))
                              for d in deg]).astype(np.int64)
    g = gpu_graph([n], [(0, 0, indptr, indices)], [None])
    # every seed list holds a hub; hop 1 reaches more of them
    seeds_list = [gpu_seeds([np.unique(np.append(rng.choice(n, size=39, replace=False),
                                                 97 * k))]) for k in range(9)]
    say("hub case: B=9")
    check_bundle(g, seeds_list, [[10], [5]], [3 + k for k in range(9)], 2)


def test_bundle_random_heterographs():
    rng = np.random.default_rng(77)
    for c in range(12):
        nn, ets, feats, seeds, fanouts, sigma, bits = pins.random_case(rng, max_nodes=60,
                                                                       max_deg=40)
        g = gpu_graph(nn, ets, feats)
        B = int(rng.integers(2, 5))
        seeds_list = []
        for k in range(B):
            s = [np.sort(rng.choice(n, size=min(n, int(rng.integers(0, 6))), replace=False))
                 if n else np.zeros(0, np.int64) for n in nn]
            seeds_list.append(gpu_seeds(s))
        say(f"case {c}: T={len(nn)} R={len(ets)} H={len(fanouts)} B={B}")
        check_bundle(g, seeds_list, fanouts, [sigma + 11 * k for k in range(B)], len(fanouts))


def test_bundle_academic_workload():
    """Bundles of 4 and of 32 academic mini-batches: each equals its own
    single call, and every mini-batch of both bundles equals the oracle
    (blocks and gathered bytes)."""
    wl = W.WORKLOADS[2]
    gen = W.make_graph(wl, device="cuda")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False,
                            lib=oracle.load_omp())
    fan = wl.fanout_matrix()
    seeds_list = [gpu_seeds(W.seeds_per_type(wl, b)) for b in (4, 5, 6, 7)]
    check_bundle(g, seeds_list, fan, [4, 5, 6, 7], len(fan))
    feat_types = [t for t, f in enumerate(gen.feats) if f is not None]
    for first, B in ((4, 4), (40, 32)):
        batches = list(range(first, first + B))
        say(f"academic bundle of {B}: batches {batches[0]}..{batches[-1]} against the oracle")
        got = g.sample_bundle([gpu_seeds(W.seeds_per_type(wl, b)) for b in batches], fan,
                              batches, gather="all")
        for b, blocks in zip(batches, got):
            seeds = W.seeds_per_type(wl, b)
            ref = host.sample_blocks(seeds, fan, b)
            diffs = compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
            assert not diffs, f"batch {b}: " + "\n".join(diffs[:10])
            for t in feat_types:
                want = host.gather(t, ref["input"][t]).tobytes()
                assert blocks.features(t).contiguous().view(torch.uint8).cpu().numpy() \
                    .tobytes() == want, f"batch {b} type {t}: gathered bytes differ"
        del got


def test_bundle_errors():
    indptr = np.array([0, 1, 3, 3], np.int64)
    indices = np.array([2, 0, 1], np.int64)
    g = gpu_graph([3], [(0, 0, indptr, indices)], [None])
    good = gpu_seeds([np.array([0, 1])])
    bad = gpu_seeds([np.array([2, 2])])
    with pytest.raises(hg.HGError) as e:
        g.sample_bundle([good, bad], [[1]], [0, 1], gather=[])
    assert e.value.status == hg.HG_EINVAL
    with pytest.raises(hg.HGError):
        g.sample_bundle([good] * 33, [[1]], list(range(33)), gather=[])
    # the graph (and its bundle workspaces) still work
    out = g.sample_bundle([good, good], [[1]], [0, 0], gather=[])
    assert not compare(result_dict(g, out[0]), result_dict(g, out[1]), 1, 1, 1)
