"""Edge-seeded (link-prediction) mini-batches: the HIP path through the C ABI
against the CPU oracle, element by element (seeds, pair graphs, every block
array, gathered bytes), on random heterographs with reverse edge types, on
hub pairs whose in-edges are excluded (every sampler role), and on the academic
workload's graph with the paper's link-prediction fanouts."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import compare_edges, edge_result_dict, gpu_graph

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def olib():
    return oracle.load()


def dev(xs):
    return None if xs is None else [None if x is None else torch.as_tensor(x, device="cuda")
                                    for x in xs]


def run_edge_both(olib, nn, ets, feats, targets, n_neg, exclude, rev_et, rev_eid, fanouts,
                  sigma):
    g = gpu_graph(nn, ets, feats)
    featured = [t for t, f in enumerate(feats) if f is not None]
    b = g.sample_edge_blocks(dev(targets), fanouts, sigma, n_neg=n_neg, exclude=exclude,
                             rev_etype=rev_et, rev_eid=dev(rev_eid), gather=featured)
    got = edge_result_dict(g, b)
    ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_edge_blocks(
        targets, fanouts, sigma, n_neg=n_neg, exclude=exclude, rev_etype=rev_et,
        rev_eid=rev_eid)
    return g, b, ref, got


@pytest.mark.parametrize("chunk", range(3))
def test_edge_random_heterographs(olib, chunk):
    rng = np.random.default_rng(5000 + chunk)
    for c in range(40):
        case = pins.random_edge_case(rng, max_nodes=60, max_deg=40)
        nn, ets, feats, tg, q, x, rev_et, rev_eid, fanouts, sigma, bits = case
        say(f"edge chunk {chunk} case {c}: T={len(nn)} R={len(ets)} H={len(fanouts)} "
            f"neg={q} exclude={x}")
        g, b, ref, got = run_edge_both(olib, nn, ets, feats, tg, q, x, rev_et, rev_eid, fanouts,
                                       sigma)
        diffs = compare_edges(ref, got, len(nn), len(ets), len(fanouts))
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])
        fails = pins.check_edge_blocks(nn, ets, tg, q, x, rev_et, rev_eid, fanouts, sigma, 32,
                                       got, brute=False)
        assert not fails, "\n".join(fails[:5])
        for t, f in enumerate(feats):
            if f is not None:
                assert b.features(t).cpu().numpy().tobytes() == f[got["input"][t]].tobytes()


def hub_with_reverse(deg, extra=(3, 0, 7, 40)):
    """One node type: destination 0 has `deg` in-edges, a few others follow;
    plus the transpose as edge type 1 and the reverse maps."""
    degs = [deg, *extra]
    n_src = max(degs) + 10
    rng = np.random.default_rng(deg)
    idx = np.concatenate([np.sort(rng.choice(n_src, size=d, replace=False)) for d in degs])
    indptr = np.concatenate([[0], np.cumsum(degs), np.full(n_src - len(degs), sum(degs))])
    nn = [n_src]
    ets, rev_et, rev_eid = pins.with_reverses(nn, [(0, 0, indptr.astype(np.int64),
                                                   idx.astype(np.int64))])
    return nn, ets, [None], rev_et, rev_eid


# (deg, K): the hub candidate path, its bisection fallback (more candidates
# than fit), one wavefront selecting, the take-all of the remaining edges,
# and every in-edge (K = -1)
@pytest.mark.parametrize("deg,k", [(5000, 25), (70000, 15), (3000, 600), (1500, 5),
                                   (1500, 1490), (40, 38), (40, -1), (20, 25)])
@pytest.mark.parametrize("exclude", [1, 2])
def test_edge_exclusion_on_hubs(olib, deg, k, exclude):
    nn, ets, feats, rev_et, rev_eid = hub_with_reverse(deg)
    rng = np.random.default_rng(deg + k)
    # targets into the hub (repeats included) and into a small destination
    tg0 = np.concatenate([rng.choice(deg, size=min(12, deg), replace=False), [3, 3],
                          [deg + 1]]).astype(np.int64)
    targets = [tg0, None]
    for sigma in (0, 7, 2**40 + 3):
        say(f"hub exclusion deg={deg} K={k} exclude={exclude} sigma={sigma}")
        g, b, ref, got = run_edge_both(olib, nn, ets, feats, targets, 2, exclude, rev_et,
                                       rev_eid, [[k, k], [k, k]], sigma)
        diffs = compare_edges(ref, got, 1, 2, 2)
        assert not diffs, "\n".join(diffs[:10])


def test_edge_errors_and_recovery(olib):
    nn, ets, feats, rev_et, rev_eid = hub_with_reverse(100)
    g = gpu_graph(nn, ets, feats)
    good = [torch.tensor([1, 2], device="cuda"), None]
    fan = [[3, 3]]
    for bad in ([torch.tensor([10_000], device="cuda"), None],
                [torch.tensor([-1], device="cuda"), None]):
        with pytest.raises(hg.HGError) as ex:
            g.sample_edge_blocks(bad, fan, 0)
        assert ex.value.status == hg.HG_EINVAL
    wrong = [x.copy() for x in rev_eid]
    wrong[0][1], wrong[0][2] = wrong[0][2], wrong[0][1]
    with pytest.raises(hg.HGError) as ex:
        g.sample_edge_blocks(good, fan, 0, exclude=2, rev_etype=rev_et, rev_eid=dev(wrong))
    assert ex.value.status == hg.HG_EINVAL
    for kw in ({"n_neg": hg.HG_MAX_NEG + 1}, {"exclude": 3}, {"exclude": 2}):
        with pytest.raises(hg.HGError):
            g.sample_edge_blocks(good, fan, 0, **kw)
    with pytest.raises(hg.HGError):
        g.sample_edge_blocks(good, fan, 0, exclude=2, rev_etype=[0, 0], rev_eid=dev(rev_eid))
    # a vertex-seeded batch has no pair graph
    vb = g.sample_blocks([torch.tensor([0], device="cuda")], fan, 0)
    with pytest.raises(hg.HGError):
        vb.edge_pairs(0)
    # the failures left the workspaces clean: a good call still matches
    tg = [np.array([1, 2], np.int64), None]
    ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_edge_blocks(
        tg, fan, 0, n_neg=3, exclude=2, rev_etype=rev_et, rev_eid=rev_eid)
    b = g.sample_edge_blocks(dev(tg), fan, 0, n_neg=3, exclude=2, rev_etype=rev_et,
                             rev_eid=dev(rev_eid))
    diffs = compare_edges(ref, edge_result_dict(g, b), 1, 2, 1)
    assert not diffs, "\n".join(diffs[:10])
    # no hops: the input frontier is the seeds
    b0 = g.sample_edge_blocks(dev(tg), [], 0, n_neg=1)
    ref0 = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_edge_blocks(
        tg, [], 0, n_neg=1)
    assert np.array_equal(b0.input_nodes(0).cpu().numpy(), ref0["input"][0])
    assert np.array_equal(b0.seeds(0).cpu().numpy(), ref0["seeds"][0])


@pytest.mark.slow
def test_edge_workload_academic(olib):
    """Link-prediction batches on the academic graph: 1000 target edges of
    paper-cites-paper, one negative each, targets and their reverses excluded,
    fanouts [25, 15] per hop, every featured type gathered."""
    wl = W.WORKLOADS[2]
    gen = W.make_graph(wl, device="cuda")
    rev_et, rev_eid = W.reverse_maps(gen)
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=olib, check=False)
    rev_host = [x.cpu().numpy() for x in rev_eid]
    R = g.R
    fan = [[k] * R for k in W.LINK_FANOUTS]
    cites = gen.etype_names.index("cites")
    for bno in range(2):
        tg = W.link_targets(gen, bno, cites)
        say(f"academic link batch {bno}")
        b = g.sample_edge_blocks(dev(tg), fan, bno, n_neg=W.LINK_NEG, exclude=2,
                                 rev_etype=rev_et, rev_eid=rev_eid, gather="all")
        got = edge_result_dict(g, b)
        ref = host.sample_edge_blocks(tg, fan, bno, n_neg=W.LINK_NEG, exclude=2,
                                      rev_etype=rev_et, rev_eid=rev_host)
        diffs = compare_edges(ref, got, g.T, R, len(fan))
        assert not diffs, "\n".join(diffs[:10])
        for t in range(g.T):
            want = host.gather(t, ref["input"][t])
            assert b.features(t).cpu().numpy().tobytes() == want.tobytes(), f"type {t}"
        say(f"academic link batch {bno}: equal "
            f"({sum(v[3].size for v in ref['edges'].values())} sampled edges)")


def edge_feats(g, b):
    return {t: b.features(t).cpu().numpy().tobytes() for t, (_, f) in enumerate(g.ntypes)
            if f is not None}


@pytest.mark.parametrize("chunk", range(2))
def test_edge_bundles_equal_single_calls(olib, chunk):
    """Every batch of an edge-seeded bundle is the batch its own call makes
    (seeds, pair graphs, blocks, gathered bytes), and the oracle's."""
    rng = np.random.default_rng(9100 + chunk)
    for c in range(12):
        case = pins.random_edge_case(rng, max_nodes=60, max_deg=40)
        nn, ets, feats, tg, q, x, rev_et, rev_eid, fanouts, sigma, bits = case
        g = gpu_graph(nn, ets, feats)
        B = [2, 3, 7][c % 3]
        # other target lists for the other batches: the same edge types, new picks
        tgs = [tg]
        for b in range(1, B):
            tgs.append([None if t is None else
                        rng.integers(0, max(int(e[3].size), 1), size=t.size).astype(np.int64)
                        if e[3].size else t for t, e in zip(tg, ets)])
        sigmas = [sigma + 17 * b for b in range(B)]
        say(f"edge bundle chunk {chunk} case {c}: B={B} R={len(ets)} neg={q} exclude={x}")
        bl = g.sample_edge_bundle([dev(t) for t in tgs], fanouts, sigmas, n_neg=q, exclude=x,
                                  rev_etype=rev_et, rev_eid=dev(rev_eid), gather="all")
        assert len(bl) == B
        host = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib)
        for b in range(B):
            single = g.sample_edge_blocks(dev(tgs[b]), fanouts, sigmas[b], n_neg=q, exclude=x,
                                          rev_etype=rev_et, rev_eid=dev(rev_eid), gather="all")
            got = edge_result_dict(g, bl[b])
            diffs = compare_edges(edge_result_dict(g, single), got, len(nn), len(ets),
                                  len(fanouts))
            assert not diffs, f"case {c} batch {b}: " + "\n".join(diffs[:10])
            assert edge_feats(g, bl[b]) == edge_feats(g, single)
            if b == B - 1:
                ref = host.sample_edge_blocks(tgs[b], fanouts, sigmas[b], n_neg=q, exclude=x,
                                              rev_etype=rev_et, rev_eid=rev_eid)
                diffs = compare_edges(ref, got, len(nn), len(ets), len(fanouts))
                assert not diffs, f"case {c} batch {b} vs oracle: " + "\n".join(diffs[:10])


def test_edge_bundle_errors(olib):
    nn, ets, feats, rev_et, rev_eid = hub_with_reverse(100)
    g = gpu_graph(nn, ets, feats)
    good = [torch.tensor([1, 2], device="cuda"), None]
    bad = [torch.tensor([10_000], device="cuda"), None]
    with pytest.raises(hg.HGError):
        g.sample_edge_bundle([good, bad], [[3, 3]], [0, 1])
    with pytest.raises(hg.HGError):
        g.sample_edge_bundle([good] * 33, [[3, 3]], list(range(33)))
    out = g.sample_edge_bundle([good, good], [[3, 3]], [5, 5], n_neg=2)
    a, b = edge_result_dict(g, out[0]), edge_result_dict(g, out[1])
    assert not compare_edges(a, b, 1, 2, 1)
