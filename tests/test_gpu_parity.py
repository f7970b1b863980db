"""HIP path (through the C ABI) against the CPU oracle, element by element, on
random tiny heterographs and the tiny workload.  All outputs are integers or
copied bits, so the bar is exact equality."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import many_relations, compare, gpu_graph, gpu_seeds, result_dict

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def olib():
    return oracle.load()


def test_philox_device_matches_oracle(olib):
    rng = np.random.default_rng(1)
    n = 4096
    ctr = rng.integers(0, 1 << 32, size=(n, 4), dtype=np.uint64).astype(np.uint32)
    ctr[0] = 0
    ctr[1] = 0xFFFFFFFF
    key = int(rng.integers(0, 1 << 63)) * 2 + 1
    got = hg.debug_philox(torch.as_tensor(ctr.view(np.int32), device="cuda"), key)
    got = got.cpu().numpy().view(np.uint32)
    for i in range(0, n, 97):
        ref = oracle.philox4x32_10(ctr[i], [key & 0xFFFFFFFF, key >> 32], olib)
        assert np.array_equal(got[i], ref), f"counter {ctr[i]}"
    # and all of them against rocRAND's key definition for the zero-key case
    z = hg.debug_philox(torch.zeros((1, 4), dtype=torch.int32, device="cuda"), 0)
    assert np.array_equal(z.cpu().numpy().view(np.uint32)[0], pins.rr_block(0, 0, 0))


@pytest.mark.parametrize("sigma,hop,etype,lim", [(0, 0, 0, 1 << 31), (2**64 - 1, 2, 5, 123457),
                                                  (987654321, 1, 1199, 0xFFFFFFFF),
                                                  (5, 7, 3, 0)])
def test_key_loop_counts_match_oracle(olib, sigma, hop, etype, lim):
    """The sampler's key loop run alone (hg_bench_philox, the key-rate
    microbenchmark): its count of keys <= lim over edge IDs 0 .. 4n-1 equals
    the oracle's keys of the same edges."""
    n_groups = 64 * 160
    got = int(hg.bench_philox(sigma, hop, etype, n_groups, lim).item())
    keys = np.array([oracle.edge_key(sigma, hop, etype, eid, 32, olib)
                     for eid in range(4 * n_groups)], dtype=np.uint64)
    assert got == int((keys <= lim).sum())
    with pytest.raises(hg.HGError):
        hg.bench_philox(sigma, hop, etype, 100, lim)  # not a multiple of 64


def run_both(olib, nn, ets, feats, seeds, fanouts, sigma, bits):
    g = gpu_graph(nn, ets, feats)
    b = g.sample_blocks(gpu_seeds(seeds), fanouts, sigma, key_bits=bits)
    got = result_dict(g, b)
    ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_blocks(seeds, fanouts,
                                                                              sigma, bits)
    return g, b, ref, got


@pytest.mark.parametrize("chunk", range(4))
def test_random_heterographs(olib, chunk):
    rng = np.random.default_rng(1000 + chunk)
    for c in range(40):
        case = pins.random_case(rng, max_nodes=60, max_deg=40)
        nn, ets, feats, seeds, fanouts, sigma, bits = case
        say(f"chunk {chunk} case {c}: T={len(nn)} R={len(ets)} H={len(fanouts)} bits={bits}")
        g, b, ref, got = run_both(olib, *case)
        diffs = compare(ref, got, len(nn), len(ets), len(fanouts))
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])
        fails = pins.check_blocks(nn, ets, seeds, fanouts, sigma, bits, got, brute=False)
        assert not fails, "\n".join(fails[:5])
        # every block's edge count in one call
        assert b.edge_counts() == [[ref["edges"][(h, e)][3].size for e in range(len(ets))]
                                   for h in range(len(fanouts))]
        # gather of the input frontier, every type with features (one call)
        featured = [t for t, f in enumerate(feats) if f is not None]
        allx = g.gather_features_all(b, featured)
        for t in featured:
            assert allx[t].cpu().numpy().tobytes() == feats[t][got["input"][t]].tobytes()
        # and per type
        for t, f in enumerate(feats):
            if f is None:
                with pytest.raises(hg.HGError):
                    g.gather_features(b, t)
                continue
            x = g.gather_features(b, t).cpu().numpy()
            assert x.tobytes() == f[got["input"][t]].tobytes()
        # the fused call: same blocks, and the features it gathered itself
        if bits == 32:
            bf = g.sample_blocks(gpu_seeds(seeds), fanouts, sigma, gather=featured)
            diffs = compare(ref, result_dict(g, bf), len(nn), len(ets), len(fanouts))
            assert not diffs, f"case {c} (fused): " + "\n".join(diffs[:10])
            for t, f in enumerate(feats):
                x = bf.features(t)
                if f is None:
                    assert x is None
                    continue
                assert x.shape == (got["input"][t].size, f.shape[1])
                assert x.cpu().numpy().tobytes() == f[got["input"][t]].tobytes()


def hub_graph(deg, n_src=None, extra=(3, 0, 7)):
    """One node type; destination 0 has `deg` in-edges, a few small ones follow."""
    n_src = n_src or deg + 10
    degs = [deg, *extra]
    indptr = np.concatenate([[0], np.cumsum(degs)]).astype(np.int64)
    rng = np.random.default_rng(deg)
    idx = np.concatenate([np.sort(rng.choice(n_src, size=d, replace=False)) for d in degs])
    n = max(n_src, len(degs))
    indptr = np.concatenate([indptr, np.full(n - len(degs), indptr[-1])]).astype(np.int64)
    return [n], [(0, 0, indptr, idx.astype(np.int64))], [None]


@pytest.mark.parametrize("deg,k,bits", [
    (700, 5, 32), (5000, 25, 32), (70000, 15, 32),      # candidate path
    (3000, 5, 2), (3000, 5, 1), (1200, 600, 32),        # bisection fallback
    (2000, 400, 4), (640, 639, 32), (64, 63, 32), (65, 64, 32),
    # every in-edge kept from more than one chunk's worth: chunked copies
    (70000, -1, 32), (5000, 5000, 32), (2049, 3000, 32), (4097, -1, 32),
])
def test_hub_selection(olib, deg, k, bits):
    nn, ets, feats = hub_graph(deg)
    seeds = [np.array([0, 1, 2, 3], np.int64)]
    for sigma in (0, 1, 2**40 + 3):
        say(f"hub deg={deg} K={k} bits={bits} sigma={sigma}")
        g, b, ref, got = run_both(olib, nn, ets, feats, seeds, [[k], [k]], sigma, bits)
        diffs = compare(ref, got, 1, 1, 2)
        assert not diffs, "\n".join(diffs)


# 16 etypes into a type: the smallest with a mask; 33 and 70: rows of 2 and
# 3 words
@pytest.mark.parametrize("R", [16, 33, 70])
def test_many_relations(olib, R):
    rng = np.random.default_rng(70 + R)
    nn, ets, feats = many_relations(rng, R)
    g = gpu_graph(nn, ets, feats)
    host = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib)
    for c in range(6):
        seeds = [rng.choice(nn[0], size=int(rng.integers(1, 60)), replace=False).astype(np.int64),
                 rng.choice(nn[1], size=int(rng.integers(0, 10)), replace=False).astype(np.int64)]
        H = int(rng.integers(1, 4))
        fan = [[[-1, 0, 1, 3, 10][int(rng.integers(0, 5))] for _ in range(R)] for _ in range(H)]
        sigma = int(rng.integers(0, 1 << 63))
        say(f"many relations R={R} case {c}: H={H}")
        b = g.sample_blocks(gpu_seeds(seeds), fan, sigma, gather="all")
        got = result_dict(g, b)
        ref = host.sample_blocks(seeds, fan, sigma)
        diffs = compare(ref, got, 2, R, H)
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])
        assert b.features(0).cpu().numpy().tobytes() == feats[0][got["input"][0]].tobytes()
        # the same batches bundled (the copies share the masks); four copies of
        # 70 etypes: the next-hop plan scans its 280 etypes in two chunks
        bl = g.sample_bundle([gpu_seeds(seeds)] * 4, fan, [sigma + k for k in range(4)],
                             gather=[])
        for k in range(4):
            refk = ref if k == 0 else host.sample_blocks(seeds, fan, sigma + k)
            diffs = compare(refk, result_dict(g, bl[k]), 2, R, H)
            assert not diffs, f"case {c} bundle copy {k}: " + "\n".join(diffs[:10])


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_forced_ties(olib, bits):
    rng = np.random.default_rng(77 + bits)
    for c in range(15):
        nn, ets, feats, seeds, fanouts, sigma, _ = pins.random_case(rng, max_nodes=80, max_deg=70)
        say(f"ties bits={bits} case {c}")
        g, b, ref, got = run_both(olib, nn, ets, feats, seeds, fanouts, sigma, bits)
        diffs = compare(ref, got, len(nn), len(ets), len(fanouts))
        assert not diffs, f"case {c}: " + "\n".join(diffs[:10])


def test_tiny_workload_batches(olib):
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    hgraph = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=olib)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    for bno in range(20):
        seeds = W.seeds_per_type(wl, bno)
        say(f"tiny workload batch {bno}")
        b = g.sample_blocks(gpu_seeds(seeds), wl.fanout_matrix(), bno)
        got = result_dict(g, b)
        ref = hgraph.sample_blocks(seeds, wl.fanout_matrix(), bno)
        diffs = compare(ref, got, g.T, g.R, len(wl.fanouts))
        assert not diffs, f"batch {bno}: " + "\n".join(diffs[:10])
        for t in range(g.T):
            x = g.gather_features(b, t).cpu().numpy()
            assert x.tobytes() == hgraph.gather(t, ref["input"][t]).tobytes()


def test_error_codes_match_oracle(olib):
    indptr = np.array([0, 1, 3, 3], np.int64)
    indices = np.array([2, 0, 1], np.int64)
    g = gpu_graph([3], [(0, 0, indptr, indices)], [None])
    ho = oracle.HostGraph([(3, None)], [(0, 0, indptr, indices)], lib=olib)
    for seeds, fo, kb in [([[1, 1]], [[2]], 32), ([[3]], [[2]], 32), ([[-1]], [[2]], 32),
                          ([[0]], [[-2]], 32), ([[0]], [[1]], 0), ([[0]], [[1]], 33),
                          ([[0, 0]], [], 32)]:
        with pytest.raises(oracle.OracleError) as eo:
            ho.sample_blocks([np.array(seeds[0])], fo, 0, kb)
        with pytest.raises(hg.HGError) as eg:
            g.sample_blocks(gpu_seeds([np.array(seeds[0])]), fo, 0, key_bits=kb)
        assert eo.value.status == eg.value.status == hg.HG_EINVAL
    # a featureless type cannot be gathered, by either call
    b = g.sample_blocks(gpu_seeds([np.array([0])]), [[1]], 0)
    with pytest.raises(hg.HGError):
        g.gather_features(b, 0)
    for gl in ([0], [1], [-1]):
        with pytest.raises(hg.HGError) as e:
            g.sample_blocks(gpu_seeds([np.array([0])]), [[1]], 0, gather=gl)
        assert e.value.status == hg.HG_EINVAL
    with pytest.raises(ValueError):
        g.sample_blocks(gpu_seeds([np.array([0])]), [[1]], 0, key_bits=8, gather=[])
    # invalid CSC arrays are refused at creation
    for ip, ix in [(np.array([0, 1, 3, 2]), indices), (indptr, np.array([2, 0, 3])),
                   (np.array([1, 1, 3, 3]), indices)]:
        with pytest.raises(hg.HGError) as e:
            gpu_graph([3], [(0, 0, ip, ix)], [None])
        assert e.value.status == hg.HG_EINVAL
    # the graph still works after failed calls (map and bitmap left clean)
    b = g.sample_blocks(gpu_seeds([np.array([1, 0])]), [[-1], [-1]], 3)
    got = result_dict(g, b)
    ref = ho.sample_blocks([np.array([1, 0])], [[-1], [-1]], 3)
    assert not compare(ref, got, 1, 1, 2)


def test_zero_hops_and_empty_seeds(olib):
    rng = np.random.default_rng(5)
    nn, ets, feats = W.random_hetero(rng, max_types=2, max_nodes=30)[:3]
    seeds = [np.arange(min(3, n), dtype=np.int64) for n in nn]
    for fanouts in ([], [[2] * len(ets)]):
        g, b, ref, got = run_both(olib, nn, ets, feats, seeds, fanouts, 9, 32)
        assert not compare(ref, got, len(nn), len(ets), len(fanouts))
    empty = [np.zeros(0, np.int64) for _ in nn]
    g, b, ref, got = run_both(olib, nn, ets, feats, empty, [[3] * len(ets)] * 2, 1, 32)
    assert not compare(ref, got, len(nn), len(ets), 2)


def test_determinism_and_two_streams(olib):
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    seeds = gpu_seeds(W.seeds_per_type(wl, 3))
    first = result_dict(g, g.sample_blocks(seeds, wl.fanout_matrix(), 3))
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(s1):
        b1 = g.sample_blocks(seeds, wl.fanout_matrix(), 3, stream=s1)
    with torch.cuda.stream(s2):
        b2 = g.sample_blocks(seeds, wl.fanout_matrix(), 3, stream=s2)
    torch.cuda.synchronize()
    for b in (b1, b2):
        assert not compare(first, result_dict(g, b), g.T, g.R, 2)


def test_allocator_failure_releases_everything(olib):
    """An allocator that fails after a few allocations: HG_ENOMEM, every block
    it handed out is returned, and the graph keeps working."""
    state = {"live": {}, "budget": 0, "allocs": 0}

    def alloc(ctx, nbytes, stream):
        if state["allocs"] >= state["budget"]:
            return None
        state["allocs"] += 1
        t = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        state["live"][t.data_ptr()] = t
        return t.data_ptr()

    def free(ctx, ptr, stream):
        state["live"].pop(ptr)

    a = hg.Allocator(None, hg.ALLOC_FN(alloc), hg.FREE_FN(free))
    rng = np.random.default_rng(3)
    nn, ets, feats = W.random_hetero(rng, max_types=2, max_nodes=40)[:3]
    nts = [(n, None if f is None else torch.as_tensor(f).cuda()) for n, f in zip(nn, feats)]
    g = hg.Graph(nts, [(s, d, torch.as_tensor(ip).cuda(), torch.as_tensor(ix).cuda())
                       for s, d, ip, ix in ets], allocator=a)
    seeds = [np.arange(min(4, n), dtype=np.int64) for n in nn]
    fo = [[3] * len(ets)] * 3
    ref = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib).sample_blocks(seeds, fo, 11)
    for budget in range(0, 12):
        state.update(budget=budget, allocs=0)
        try:
            b = g.sample_blocks(gpu_seeds(seeds), fo, 11)
        except hg.HGError as e:
            assert e.status == hg.HG_ENOMEM
            torch.cuda.synchronize()
            assert not state["live"], f"budget {budget}: {len(state['live'])} blocks leaked"
            continue
        got = result_dict(g, b)
        assert not compare(ref, got, len(nn), len(ets), 3)
        del b
        torch.cuda.synchronize()
        assert not state["live"]
        break
    else:
        pytest.fail("sampling never succeeded")


def expected_keys(ets, ref, fanouts):
    """Keys the sampler must evaluate per hop: the in-degree of every
    (frontier vertex, edge type) pair that keeps K of more than K in-edges."""
    out = []
    for h, row in enumerate(fanouts):
        k = 0
        for e, (s, d, ip, ix) in enumerate(ets):
            nd, sg = ref["nodes"][(h, d)]
            deg = ip[sg[:nd] + 1] - ip[sg[:nd]]
            if row[e] >= 0:
                k += int(deg[deg > row[e]].sum())
        out.append(k)
    return out


def test_block_counts_and_keys(olib):
    """hg_blocks_counts: per-hop frontier and source sizes equal the oracle's,
    and the sampler's key count equals the in-degrees of the pairs that
    select (a bundle reports the sum over its batches)."""
    rng = np.random.default_rng(31)
    for c in range(6):
        nn, ets, feats, seeds, fanouts, sigma, bits = pins.random_case(rng, max_nodes=300,
                                                                       max_deg=3000)
        g, b, ref, got = run_both(olib, nn, ets, feats, seeds, fanouts, sigma, 32)
        nd, ns, keys = b.counts()
        for h in range(len(fanouts)):
            for t in range(len(nn)):
                assert nd[h, t] == ref["nodes"][(h, t)][0]
                assert ns[h, t] == ref["nodes"][(h, t)][1].size
        assert list(keys) == expected_keys(ets, ref, fanouts), f"case {c}"
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=olib)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    fan = wl.fanout_matrix()
    batches = [3, 4, 5]
    got = g.sample_bundle([gpu_seeds(W.seeds_per_type(wl, x)) for x in batches], fan, batches)
    want = np.zeros(len(fan), np.int64)
    for x in batches:
        ref = host.sample_blocks(W.seeds_per_type(wl, x), fan, x)
        want += expected_keys(gen.host_etypes(), ref, fan)
    for blocks in got:
        assert list(blocks.counts()[2]) == list(want)


@pytest.mark.parametrize("pad", [0, 3_000_000])
def test_reached_bit_mode(olib, pad):
    """Hops whose kept edges are few next to the graph's vertices mark reached
    sources with bits (atomicOr) instead of bytes; the tiny workload with and
    without 3M isolated extra vertices of each type (every hop in bit mode,
    or a mix) equals the oracle, blocks and gathered bytes."""
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    nn = [n + pad for n in gen.num_nodes]
    ets = []
    for s, d, ip, ix in gen.host_etypes():
        ets.append((s, d, np.concatenate([ip, np.full(pad, ip[-1], np.int64)]), ix))
    feats = [np.concatenate([f, np.zeros((pad,) + f.shape[1:], f.dtype)])
             for _, f in gen.host_ntypes()]
    g = gpu_graph(nn, ets, feats)
    host = oracle.HostGraph(list(zip(nn, feats)), ets, lib=olib)
    fan = wl.fanout_matrix()
    for b in range(3):
        seeds = W.seeds_per_type(wl, b)
        blocks = g.sample_blocks(gpu_seeds(seeds), fan, b, gather="all")
        ref = host.sample_blocks(seeds, fan, b)
        diffs = compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
        assert not diffs, f"pad {pad} batch {b}: " + "\n".join(diffs[:5])
        for t in range(g.T):
            assert blocks.features(t).cpu().numpy().tobytes() == \
                host.gather(t, ref["input"][t]).tobytes()
    # a bundle of 4 on the same graph (the virtual graph has 4x the vertices)
    got = g.sample_bundle([gpu_seeds(W.seeds_per_type(wl, b)) for b in range(4)], fan,
                          list(range(4)))
    for b, blocks in enumerate(got):
        ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
        assert not compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
