"""Layer-wise (LADIES) mini-batches: the HIP path through the C ABI against
the CPU oracle, element by element (every hop's source lists, every block
array, gathered bytes), on random heterographs with every kind of layer size,
on draws that land on interval boundaries, on hubs whose importance rounds to
zero, and on the academic workload's graph."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import compare, gpu_graph, gpu_seeds, many_relations, result_dict

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def olib():
    return oracle.load()


def run_layer_both(olib, nn, ets, feats, seeds, sizes, sigma, g=None):
    g = g or gpu_graph(nn, ets, feats)
    featured = [t for t, f in enumerate(feats) if f is not None]
    b = g.sample_layers(gpu_seeds(seeds), sizes, sigma, gather=featured)
    got = result_dict(g, b)
    ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_layers(seeds, sizes, sigma)
    return g, b, ref, got


@pytest.mark.parametrize("chunk", range(3))
def test_layer_random_heterographs(olib, chunk):
    rng = np.random.default_rng(7000 + chunk)
    for c in range(40):
        nn, ets, feats, seeds, sizes, sigma = pins.random_layer_case(rng, max_nodes=60,
                                                                     max_deg=40)
        say(f"layer chunk {chunk} case {c}: T={len(nn)} R={len(ets)} sizes={sizes}")
        g, b, ref, got = run_layer_both(olib, nn, ets, feats, seeds, sizes, sigma)
        diffs = compare(ref, got, len(nn), len(ets), len(sizes))
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])
        fails = pins.check_layer_blocks(nn, ets, seeds, sizes, sigma, got)
        assert not fails, "\n".join(fails[:5])
        for t, f in enumerate(feats):
            if f is not None:
                assert b.features(t).cpu().numpy().tobytes() == f[got["input"][t]].tobytes()
        # the same graph again with other draws: the importance array and the
        # flags were left clean
        sigma2 = (sigma * 3 + 1) & (2**64 - 1)
        g, b, ref, got = run_layer_both(olib, nn, ets, feats, seeds, sizes, sigma2, g=g)
        diffs = compare(ref, got, len(nn), len(ets), len(sizes))
        assert not diffs, f"case {c} again: " + "\n".join(diffs[:10])


def test_layer_boundary_draws(olib):
    """One destination of in-degree 65536: every source has importance 1, so
    each draw r lands on the first point of candidate r's interval; the second
    hop draws among their ring neighbours."""
    n, d = 65536 + 70000, 65536
    indptr = np.concatenate([[0], d + np.arange(0, n, dtype=np.int64)])
    indices = np.concatenate([np.arange(1, d + 1), 65537 + (np.arange(1, n) % 69999)])
    ets = [(0, 0, indptr.astype(np.int64), indices.astype(np.int64))]
    g = gpu_graph([n], ets, [None])
    for sizes in ([[40], [40]], [[3000], [-1]], [[-1], [700]]):
        for sigma in (3, 77, 2**63 + 5):
            say(f"boundary sizes={sizes} sigma={sigma}")
            _, _, ref, got = run_layer_both(olib, [n], ets, [None], [np.array([0])], sizes, sigma,
                                            g=g)
            diffs = compare(ref, got, 1, 1, 2)
            assert not diffs, "\n".join(diffs[:10])


def hubs():
    """Destinations 0 .. 3 with in-degrees 70000 (importance 0 per edge),
    5000, 300 and 0, sources spread over 100000 vertices; two node types so
    that candidates of both types arise."""
    rng = np.random.default_rng(11)
    n0, n1 = 100_000, 3_000
    degs = [70000, 5000, 300, 0]
    idx0 = [np.sort(rng.choice(n0, size=k, replace=False)) for k in degs]
    ip0 = np.concatenate([[0], np.cumsum(degs), np.full(n1 - len(degs), sum(degs))])
    # type-1 destinations from type-0 sources, and type-0 destinations from type 1
    degs1 = [40, 2000] + [0] * (n0 - 2)
    idx1 = [np.sort(rng.choice(n1, size=k, replace=False)) for k in degs1[:2]]
    ip1 = np.concatenate([[0], np.cumsum(degs1)])
    ets = [(0, 1, ip0.astype(np.int64), np.concatenate(idx0).astype(np.int64)),
           (1, 0, ip1.astype(np.int64), np.concatenate(idx1).astype(np.int64))]
    return [n0, n1], ets


@pytest.mark.parametrize("sizes", [[[-1, -1]], [[300, 10], [64, 64]], [[0, 5000], [1, -1]],
                                   [[100000, 0], [2, 2]]])
def test_layer_hubs(olib, sizes):
    nn, ets = hubs()
    g = gpu_graph(nn, ets, [None, None])
    seeds = [np.array([1, 0]), np.array([0, 1, 3, 2])]
    for sigma in (0, 9):
        say(f"hubs sizes={sizes} sigma={sigma}")
        _, _, ref, got = run_layer_both(olib, nn, ets, [None, None], seeds, sizes, sigma, g=g)
        diffs = compare(ref, got, 2, 2, len(sizes))
        assert not diffs, "\n".join(diffs[:10])


def test_layer_errors_and_recovery(olib):
    rng = np.random.default_rng(3)
    nn, ets, feats = W.random_hetero(rng, max_nodes=30, max_deg=10)
    g = gpu_graph(nn, ets, feats)
    T = len(nn)
    seeds = [np.array([0], np.int64) if n > 0 else None for n in nn]
    for bad in ([[-2] * T], [[1] * (T + 1)]):
        with pytest.raises((hg.HGError, ValueError)):
            g.sample_layers(gpu_seeds(seeds), bad, 0)
    t0 = next(t for t in range(T) if nn[t] > 0)
    rep = list(seeds)
    rep[t0] = np.array([0, 0], np.int64)
    with pytest.raises(hg.HGError) as ex:
        g.sample_layers(gpu_seeds(rep), [[1] * T], 0)
    assert ex.value.status == hg.HG_EINVAL
    far = list(seeds)
    far[t0] = np.array([nn[t0]], np.int64)
    with pytest.raises(hg.HGError) as ex:
        g.sample_layers(gpu_seeds(far), [[1] * T], 0)
    assert ex.value.status == hg.HG_EINVAL
    # nine node types (the per-type tables live on the device, not in the launch)
    many_nn = [2] * 9
    many_ets = [(0, 1, np.array([0, 1, 1]), np.array([1])),
                (1, 0, np.array([0, 1, 1]), np.array([0]))]
    many = gpu_graph(many_nn, many_ets, [None] * 9)
    mseeds = [np.array([0])] + [None] * 8
    _, _, mref, mgot = run_layer_both(olib, many_nn, many_ets, [None] * 9, mseeds,
                                      [[1] * 9, [-1] * 9], 3, g=many)
    assert not compare(mref, mgot, 9, 2, 2)
    # the failures left the workspaces clean
    sizes = [[-1] * T, [2] * T]
    _, _, ref, got = run_layer_both(olib, nn, ets, feats, seeds, sizes, 5, g=g)
    diffs = compare(ref, got, T, len(ets), 2)
    assert not diffs, "\n".join(diffs[:10])
    # no hops: the input frontier is the seeds
    b0 = g.sample_layers(gpu_seeds(seeds), [], 0)
    for t in range(T):
        want = np.zeros(0, np.int64) if seeds[t] is None else seeds[t]
        assert np.array_equal(b0.input_nodes(t).cpu().numpy(), want)


@pytest.mark.slow
def test_layer_workload_academic(olib):
    """Layer-wise batches on the academic graph: the workload's 1024 paper
    seeds, 512 draws per node type in each of two hops, every featured type
    gathered."""
    wl = W.WORKLOADS[2]
    gen = W.make_graph(wl, device="cuda")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=olib, check=False)
    sizes = [[k] * g.T for k in W.LAYER_SIZES]
    for bno in range(2):
        seeds = W.seeds_per_type(wl, bno)
        say(f"academic layer batch {bno}")
        b = g.sample_layers(gpu_seeds(seeds), sizes, bno, gather="all")
        got = result_dict(g, b)
        ref = host.sample_layers(seeds, sizes, bno)
        diffs = compare(ref, got, g.T, g.R, len(sizes))
        assert not diffs, "\n".join(diffs[:10])
        for t in range(g.T):
            want = host.gather(t, ref["input"][t])
            assert b.features(t).cpu().numpy().tobytes() == want.tobytes(), f"type {t}"
        say(f"academic layer batch {bno}: equal "
            f"({sum(v[3].size for v in ref['edges'].values())} kept edges)")


@pytest.mark.parametrize("chunk", range(2))
def test_layer_bundles_equal_single_calls(olib, chunk):
    """Every batch of a layer-wise bundle is the batch its own call makes
    (blocks and gathered bytes), and the oracle's."""
    rng = np.random.default_rng(9300 + chunk)
    for c in range(10):
        nn, ets, feats, seeds, sizes, sigma = pins.random_layer_case(rng, max_nodes=60,
                                                                     max_deg=40)
        g = gpu_graph(nn, ets, feats)
        B = [2, 4, 9][c % 3]
        seeds_list = [seeds]
        for b in range(1, B):
            seeds_list.append([None if s is None else
                               rng.choice(nn[t], size=s.size, replace=False).astype(np.int64)
                               for t, s in enumerate(seeds)])
        sigmas = [sigma + 29 * b for b in range(B)]
        say(f"layer bundle chunk {chunk} case {c}: B={B} T={len(nn)} sizes={sizes}")
        bl = g.sample_layers_bundle([gpu_seeds(s) for s in seeds_list], sizes, sigmas,
                                    gather="all")
        assert len(bl) == B
        for b in range(B):
            single = g.sample_layers(gpu_seeds(seeds_list[b]), sizes, sigmas[b], gather="all")
            got = result_dict(g, bl[b])
            diffs = compare(result_dict(g, single), got, len(nn), len(ets), len(sizes))
            assert not diffs, f"case {c} batch {b}: " + "\n".join(diffs[:10])
            for t, f in enumerate(feats):
                if f is not None:
                    assert bl[b].features(t).cpu().numpy().tobytes() == \
                        single.features(t).cpu().numpy().tobytes()
            if b == B - 1:
                ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_layers(
                    seeds_list[b], sizes, sigmas[b])
                diffs = compare(ref, got, len(nn), len(ets), len(sizes))
                assert not diffs, f"case {c} batch {b} vs oracle: " + "\n".join(diffs[:10])


def sparse_relations(rng, R, n0=300, n1=80):
    """Two node types and R edge types with a handful of edges each: about 3%
    of the destinations of an edge type have 1 to 3 in-edges."""
    nn = [n0, n1]
    ets = []
    for _e in range(R):
        s, d = int(rng.integers(0, 2)), int(rng.integers(0, 2))
        indptr, indices = [0], []
        for _v in range(nn[d]):
            k = int(rng.integers(1, 4)) if rng.random() < 0.03 else 0
            indices.extend(int(x) for x in np.sort(rng.choice(nn[s], size=k, replace=False)))
            indptr.append(len(indices))
        ets.append((s, d, np.array(indptr, np.int64), np.array(indices, np.int64)))
    feats = [rng.standard_normal((n0, 4)).astype(np.float32), None]
    return nn, ets, feats


@pytest.mark.parametrize("R", [6, 40, 70])
def test_layer_many_relations(olib, R):
    """Many sparse edge types: a tile of in-edges (2048 in the importance
    kernel, 512 in the kept-edge scan) then spans more etypes than the
    kernels' per-tile tables hold (32), and the etype of each edge is searched
    for instead; with 6 a tile spans few.  Single calls and a bundle of 4
    against the oracle."""
    rng = np.random.default_rng(8800 + R)
    nn, ets, feats = many_relations(rng, R) if R <= 6 else sparse_relations(rng, R)
    g = gpu_graph(nn, ets, feats)
    host = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib)
    for c in range(4):
        seeds = [rng.choice(nn[0], size=int(rng.integers(20, 200)), replace=False).astype(np.int64),
                 rng.choice(nn[1], size=int(rng.integers(0, 30)), replace=False).astype(np.int64)]
        H = int(rng.integers(1, 4))
        sizes = [[[-1, 0, 1, 5, 40][int(rng.integers(0, 5))] for _ in range(2)] for _ in range(H)]
        sigma = int(rng.integers(0, 1 << 63))
        say(f"layer many relations R={R} case {c}: H={H} sizes={sizes}")
        b = g.sample_layers(gpu_seeds(seeds), sizes, sigma, gather="all")
        got = result_dict(g, b)
        ref = host.sample_layers(seeds, sizes, sigma)
        diffs = compare(ref, got, 2, R, H)
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])
        assert b.features(0).cpu().numpy().tobytes() == feats[0][got["input"][0]].tobytes()
        # four copies of 70 etypes: the next-hop plan scans its 280 etypes in two chunks
        sigmas = [sigma, sigma + 1, sigma + 2, sigma + 3]
        bl = g.sample_layers_bundle([gpu_seeds(seeds)] * 4, sizes, sigmas, gather=[])
        for k in range(4):
            refk = ref if k == 0 else host.sample_layers(seeds, sizes, sigmas[k])
            diffs = compare(refk, result_dict(g, bl[k]), 2, R, H)
            assert not diffs, f"case {c} bundle copy {k}: " + "\n".join(diffs[:10])
