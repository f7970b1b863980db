"""The mini-batch pipeline (worker threads with their own streams) against the
direct call and the oracle: every mini-batch, returned in submission order,
equals the one hg_sample_blocks_gather makes on its own (and, for layer-wise
and edge-seeded submissions, the one hg_sample_layers_bundle or
hg_sample_edge_blocks_bundle makes), and a bad mini-batch fails alone."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import workloads as W
import pins
from gpu_harness import (compare, compare_edges, edge_result_dict, gpu_graph, gpu_seeds,
                         result_dict)

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def tiny():
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes())
    return wl, gen, g, host


def features(g, b):
    return {t: b.features(t).cpu().numpy().tobytes() for t, (_, f) in enumerate(g.ntypes)
            if f is not None}


@pytest.mark.parametrize("workers,capacity", [(1, 1), (2, 3), (4, 8)])
def test_pipeline_matches_direct_calls(tiny, workers, capacity):
    wl, gen, g, host = tiny
    fan = wl.fanout_matrix()
    batches = list(range(10))
    seeds = {b: gpu_seeds(W.seeds_per_type(wl, b)) for b in batches}
    pipe = hg.Pipeline(g, workers=workers, capacity=capacity, gather="all")
    got = []
    pending = list(batches)
    for _ in range(min(capacity, len(pending))):
        b = pending.pop(0)
        pipe.submit(seeds[b], fan, b)
    for _ in batches:
        got.append(pipe.next())
        if pending:
            b = pending.pop(0)
            pipe.submit(seeds[b], fan, b)
    pipe.close()
    for b, blocks in zip(batches, got):
        say(f"workers {workers}: batch {b}")
        direct = g.sample_blocks(seeds[b], fan, b, gather="all")
        assert not compare(result_dict(g, direct), result_dict(g, blocks), g.T, g.R, len(fan))
        assert features(g, blocks) == features(g, direct)
    # and two of them against the oracle
    for b in (0, 7):
        ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
        assert not compare(ref, result_dict(g, got[b]), g.T, g.R, len(fan))
        for t, x in features(g, got[b]).items():
            assert x == host.gather(t, ref["input"][t]).tobytes()


def test_pipeline_bad_minibatch_fails_alone(tiny):
    wl, gen, g, host = tiny
    fan = wl.fanout_matrix()
    good = gpu_seeds(W.seeds_per_type(wl, 1))
    bad = [torch.tensor([5, 5], dtype=torch.int64, device="cuda"), None]  # repeated seed
    pipe = hg.Pipeline(g, workers=2, capacity=4)
    pipe.submit(good, fan, 1)
    pipe.submit(bad, fan, 2)
    pipe.submit(good, fan, 3)
    first = pipe.next()
    with pytest.raises(hg.HGError) as e:
        pipe.next()
    assert e.value.status == hg.HG_EINVAL
    third = pipe.next()
    with pytest.raises(hg.HGError):
        pipe.next()  # nothing outstanding
    direct = g.sample_blocks(good, fan, 3, gather="all")
    assert not compare(result_dict(g, direct), result_dict(g, third), g.T, g.R, len(fan))
    assert not compare(result_dict(g, g.sample_blocks(good, fan, 1)), result_dict(g, first),
                       g.T, g.R, len(fan))
    pipe.close()


def test_pipeline_close_with_outstanding_minibatches(tiny):
    wl, gen, g, host = tiny
    fan = wl.fanout_matrix()
    pipe = hg.Pipeline(g, workers=3, capacity=6)
    for b in range(6):
        pipe.submit(gpu_seeds(W.seeds_per_type(wl, b)), fan, b)
    blocks = pipe.next()
    pipe.close()  # five never returned: finished and freed
    # the returned one outlives the pipeline
    ref = host.sample_blocks(W.seeds_per_type(wl, 0), fan, 0)
    assert not compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
    # and the graph keeps working
    b = g.sample_blocks(gpu_seeds(W.seeds_per_type(wl, 9)), fan, 9)
    assert not compare(host.sample_blocks(W.seeds_per_type(wl, 9), fan, 9), result_dict(g, b),
                       g.T, g.R, len(fan))


def test_pipeline_bundles(tiny):
    """Bundled submits: each mini-batch of a bundle comes back on its own, in
    order, equal to its single call; a bad mini-batch fails its whole bundle
    only; a bundle larger than the capacity is refused."""
    wl, gen, g, host = tiny
    fan = wl.fanout_matrix()
    seeds = {b: gpu_seeds(W.seeds_per_type(wl, b)) for b in range(8)}
    pipe = hg.Pipeline(g, workers=2, capacity=6)
    pipe.submit_bundle([seeds[0], seeds[1], seeds[2]], fan, [0, 1, 2])
    pipe.submit(seeds[3], fan, 3)
    bad = [torch.tensor([7, 7], dtype=torch.int64, device="cuda"), None]
    pipe.submit_bundle([seeds[4], bad], fan, [4, 5])
    got = [pipe.next() for _ in range(4)]
    for b, blocks in zip(range(4), got):
        direct = g.sample_blocks(seeds[b], fan, b, gather="all")
        assert not compare(result_dict(g, direct), result_dict(g, blocks), g.T, g.R, len(fan))
        assert features(g, blocks) == features(g, direct)
    for _ in range(2):
        with pytest.raises(hg.HGError) as e:
            pipe.next()
        assert e.value.status == hg.HG_EINVAL
    with pytest.raises(hg.HGError):
        pipe.submit_bundle([seeds[b] for b in range(7)], fan, list(range(7)))
    pipe.submit_bundle([seeds[6], seeds[7]], fan, [6, 7])
    last = [pipe.next(), pipe.next()]
    pipe.close()
    for b, blocks in zip((6, 7), last):
        ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
        assert not compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))


def dev(xs):
    return None if xs is None else [None if x is None else torch.as_tensor(x, device="cuda")
                                    for x in xs]


def all_features(g, b):
    return {t: b.features(t).cpu().numpy().tobytes() for t, (_, f) in enumerate(g.ntypes)
            if f is not None}


@pytest.mark.parametrize("chunk", range(2))
def test_pipeline_layer_and_edge_bundles(chunk):
    """One pipeline (3 workers) takes layer-wise, edge-seeded and vertex
    bundles in turn, with a bad layer-wise bundle and a bad edge-seeded bundle
    among them: every mini-batch comes back in submission order, equal to the
    same bundle made by a direct call (blocks and gathered bytes), and the bad
    bundles fail alone; the last batches of each kind also equal the oracle."""
    rng = np.random.default_rng(9700 + chunk)
    for c in range(6):
        nn, ets, feats, seeds, sizes, sigma = pins.random_layer_case(rng, max_nodes=60,
                                                                     max_deg=40)
        ecase = pins.random_edge_case(rng, max_nodes=60, max_deg=40)
        enn, eets, efeats, tg, q, x, rev_et, rev_eid, efan, esig, _bits = ecase
        g = gpu_graph(nn, ets, feats)
        eg = gpu_graph(enn, eets, efeats)
        B = [2, 3, 5][c % 3]
        seeds_list = [seeds] + [[None if s is None else
                                 rng.choice(nn[t], size=s.size, replace=False).astype(np.int64)
                                 for t, s in enumerate(seeds)] for _ in range(B - 1)]
        lsig = [sigma + 7 * b for b in range(B)]
        tgs = [tg] + [[None if t is None else
                       rng.integers(0, max(int(e[3].size), 1), size=t.size).astype(np.int64)
                       if e[3].size else t for t, e in zip(tg, eets)] for _ in range(B - 1)]
        esigs = [esig + 13 * b for b in range(B)]
        say(f"pipeline kinds chunk {chunk} case {c}: B={B}")
        # layer-wise batches on g's pipeline; a repeated seed fails its bundle
        bad_t = next((t for t, s in enumerate(seeds) if s is not None and s.size), None)
        lp = hg.Pipeline(g, workers=3, capacity=4 * B, gather="all")
        lp.submit_layers_bundle([gpu_seeds(s) for s in seeds_list], sizes, lsig)
        if bad_t is not None:
            bad = [None] * len(nn)
            bad[bad_t] = np.array([seeds[bad_t][0]] * 2, np.int64)
            lp.submit_layers_bundle([gpu_seeds(seeds), gpu_seeds(bad)], sizes, [1, 2])
        lp.submit_layers_bundle([gpu_seeds(s) for s in seeds_list], sizes, lsig[::-1])
        first = [lp.next() for _ in range(B)]
        if bad_t is not None:
            for _ in range(2):
                with pytest.raises(hg.HGError) as e:
                    lp.next()
                assert e.value.status == hg.HG_EINVAL
        second = [lp.next() for _ in range(B)]
        lp.close()
        direct = g.sample_layers_bundle([gpu_seeds(s) for s in seeds_list], sizes, lsig,
                                        gather="all")
        direct2 = g.sample_layers_bundle([gpu_seeds(s) for s in seeds_list], sizes, lsig[::-1],
                                         gather="all")
        H = len(sizes)
        for got, want in zip(first + second, direct + direct2):
            diffs = compare(result_dict(g, want), result_dict(g, got), len(nn), len(ets), H)
            assert not diffs, f"case {c} layers: " + "\n".join(diffs[:10])
            assert all_features(g, got) == all_features(g, want)
        ref = oracle.HostGraph(list(zip(nn, feats)), ets).sample_layers(seeds_list[-1], sizes,
                                                                        lsig[-1])
        assert not compare(ref, result_dict(g, first[-1]), len(nn), len(ets), H)
        # edge-seeded batches, then a vertex bundle, on eg's pipeline; a target
        # out of range fails its bundle
        ep = hg.Pipeline(eg, workers=3, capacity=4 * B, gather="all")
        ep.submit_edge_bundle([dev(t) for t in tgs], efan, esigs, n_neg=q, exclude=x,
                              rev_etype=rev_et, rev_eid=dev(rev_eid))
        badt = [None] * len(eets)
        badt[0] = np.array([int(eets[0][3].size) + 5], np.int64)
        ep.submit_edge_bundle([dev(tgs[0]), dev(badt)], efan, [3, 4], n_neg=q, exclude=x,
                              rev_etype=rev_et, rev_eid=dev(rev_eid))
        vseeds = [[None if n == 0 else rng.choice(n, size=min(n, 5), replace=False)
                   .astype(np.int64) for n in enn] for _ in range(2)]
        vfan = [[3] * len(eets)]
        ep.submit_bundle([gpu_seeds(s) for s in vseeds], vfan, [8, 9])
        egot = [ep.next() for _ in range(B)]
        for _ in range(2):
            with pytest.raises(hg.HGError) as e:
                ep.next()
            assert e.value.status == hg.HG_EINVAL
        vgot = [ep.next() for _ in range(2)]
        ep.close()
        edirect = eg.sample_edge_bundle([dev(t) for t in tgs], efan, esigs, n_neg=q, exclude=x,
                                        rev_etype=rev_et, rev_eid=dev(rev_eid), gather="all")
        for got, want in zip(egot, edirect):
            diffs = compare_edges(edge_result_dict(eg, want), edge_result_dict(eg, got),
                                  len(enn), len(eets), len(efan))
            assert not diffs, f"case {c} edges: " + "\n".join(diffs[:10])
            assert all_features(eg, got) == all_features(eg, want)
        eref = oracle.HostGraph(list(zip(enn, efeats)), eets).sample_edge_blocks(
            tgs[-1], efan, esigs[-1], n_neg=q, exclude=x, rev_etype=rev_et, rev_eid=rev_eid)
        assert not compare_edges(eref, edge_result_dict(eg, egot[-1]), len(enn), len(eets),
                                 len(efan))
        for s, sg, got in zip(vseeds, (8, 9), vgot):
            want = eg.sample_blocks(gpu_seeds(s), vfan, sg, gather="all")
            assert not compare(result_dict(eg, want), result_dict(eg, got), len(enn), len(eets),
                               1)
            assert all_features(eg, got) == all_features(eg, want)
