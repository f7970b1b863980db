"""The mini-batch pipeline (worker threads with their own streams) against the
direct call and the oracle: every mini-batch, returned in submission order,
equals the one hg_sample_blocks_gather makes on its own, and a bad
mini-batch fails alone."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import workloads as W
from gpu_harness import compare, gpu_seeds, result_dict

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
