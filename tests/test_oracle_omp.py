"""The OpenMP build of the oracle (the same oracle.c compiled with -fopenmp,
whose pair, relabel and gather loops run on every host core; the benchmark's
all-core CPU baseline) gives the same mini-batches as the plain build:
random heterographs with hubs, forced ties, edge-seeded batches with
exclusion, and the tiny workload.  CPU only."""
import numpy as np
import pytest

import oracle
import workloads as W


def same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        if isinstance(a[k], dict):
            same(a[k], b[k])
        elif isinstance(a[k], tuple):
            assert len(a[k]) == len(b[k])
            for x, y in zip(a[k], b[k]):
                if isinstance(x, np.ndarray):
                    assert x.dtype == y.dtype and np.array_equal(x, y), k
                else:
                    assert x == y, k
        elif isinstance(a[k], np.ndarray):
            assert a[k].dtype == b[k].dtype and np.array_equal(a[k], b[k]), k
        else:
            assert a[k] == b[k], k


def test_omp_build_uses_threads():
    assert oracle.threads(oracle.load()) == 1
    assert oracle.threads(oracle.load_omp()) >= 1


@pytest.mark.parametrize("seed", range(12))
def test_random_heterographs_same_as_plain(seed):
    rng = np.random.default_rng(500 + seed)
    nn, ets, feats = W.random_hetero(rng, max_types=3, max_etypes=4, max_nodes=400, max_deg=60)
    # a hub on the first edge type: every source of its type into vertex 0
    s, d, ip, ix = ets[0]
    if nn[s] > 0 and nn[d] > 0:
        deg = np.diff(ip)
        deg[0] = nn[s]
        srcs = [np.arange(nn[s])] + [ix[ip[v]:ip[v + 1]] for v in range(1, nn[d])]
        ets[0] = (s, d, np.concatenate([[0], np.cumsum(deg)]).astype(np.int64),
                  np.concatenate(srcs).astype(np.int64))
    ntypes = list(zip(nn, feats))
    plain = oracle.HostGraph(ntypes, ets, lib=oracle.load())
    omp = oracle.HostGraph(ntypes, ets, lib=oracle.load_omp())
    seeds = [np.sort(rng.choice(n, size=min(n, 30), replace=False)).astype(np.int64)
             if n > 0 and t == 0 else None for t, n in enumerate(nn)]
    fan = [[int(rng.integers(-1, 12)) for _ in ets] for _ in range(3)]
    for kb in (32, 3):
        same(plain.sample_blocks(seeds, fan, seed, key_bits=kb),
             omp.sample_blocks(seeds, fan, seed, key_bits=kb))
    # edge-seeded, targets excluded
    R = len(ets)
    targets = [None] * R
    for e, (_, _, _, ix) in enumerate(ets):
        if ix.size:
            targets[e] = rng.choice(ix.size, size=min(ix.size, 8), replace=True).astype(np.int64)
    same(plain.sample_edge_blocks(targets, fan[:2], seed, n_neg=1, exclude=1),
         omp.sample_edge_blocks(targets, fan[:2], seed, n_neg=1, exclude=1))
    for t, (n, f) in enumerate(ntypes):
        if f is not None and n > 0:
            ids = rng.integers(0, n, size=50)
            assert plain.gather(t, ids).tobytes() == omp.gather(t, ids).tobytes()


def test_tiny_workload_same_as_plain():
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    plain = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=oracle.load())
    omp = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), lib=oracle.load_omp())
    for b in range(4):
        seeds = W.seeds_per_type(wl, b)
        same(plain.sample_blocks(seeds, wl.fanout_matrix(), b),
             omp.sample_blocks(seeds, wl.fanout_matrix(), b))
