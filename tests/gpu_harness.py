"""Runs the HIP path and the oracle on the same inputs and compares them."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2112_15345_amd as hg


def gpu_graph(nn, etypes, feats, device="cuda"):
    nts = []
    for n, f in zip(nn, feats):
        nts.append((n, None if f is None else torch.as_tensor(f).to(device).contiguous()))
    ets = [(s, d, torch.as_tensor(ip, device=device), torch.as_tensor(ix, device=device))
           for s, d, ip, ix in etypes]
    return hg.Graph(nts, ets, device=device)


def result_dict(graph: hg.Graph, blocks: hg.Blocks):
    """Copies every output of a Blocks handle to numpy (oracle result layout)."""
    torch.cuda.synchronize()
    res = {"n_hops": blocks.n_hops, "nodes": {}, "edges": {}, "input": {}}
    for h in range(blocks.n_hops):
        for t in range(graph.T):
            nd, sg = blocks.nodes(h, t)
            res["nodes"][(h, t)] = (nd, sg.cpu().numpy())
        for e in range(graph.R):
            res["edges"][(h, e)] = tuple(a.cpu().numpy() for a in blocks.edges(h, e))
    for t in range(graph.T):
        res["input"][t] = blocks.input_nodes(t).cpu().numpy()
    return res


def edge_result_dict(graph: hg.Graph, blocks: hg.Blocks):
    """result_dict plus the seeds and pair graphs of an edge-seeded batch."""
    res = result_dict(graph, blocks)
    res["seeds"] = {t: blocks.seeds(t).cpu().numpy() for t in range(graph.T)}
    res["pairs"] = {e: tuple(a.cpu().numpy() for a in blocks.edge_pairs(e))
                    for e in range(graph.R)}
    return res


def compare_edges(ref, got, T, R, H):
    """compare() plus the seeds and the pair graphs."""
    diffs = compare(ref, got, T, R, H)
    for t in range(T):
        if not np.array_equal(ref["seeds"][t], got["seeds"][t]):
            diffs.append(f"seeds of type {t} differ: {ref['seeds'][t][:6]} / {got['seeds'][t][:6]}")
    for e in range(R):
        for name, x, y in zip(("pos_src", "pos_dst", "neg_dst"), ref["pairs"][e], got["pairs"][e]):
            if x.dtype != y.dtype or not np.array_equal(x, y):
                diffs.append(f"etype {e} {name} differs: {x[:6]} / {y[:6]}")
    return diffs


def gpu_seeds(seeds, device="cuda"):
    return [None if s is None else torch.as_tensor(np.asarray(s, np.int64), device=device)
            for s in seeds]


def compare(ref, got, T, R, H):
    """Element-by-element comparison; returns a list of differences."""
    diffs = []
    for h in range(H):
        for t in range(T):
            a, b = ref["nodes"][(h, t)], got["nodes"][(h, t)]
            if a[0] != b[0] or not np.array_equal(a[1], b[1]):
                diffs.append(f"hop {h} type {t}: n_dst {a[0]}/{b[0]}, n_src {a[1].size}/{b[1].size}")
        for e in range(R):
            for name, x, y in zip(("indptr", "src_local", "dst_local", "eid"),
                                  ref["edges"][(h, e)], got["edges"][(h, e)]):
                if x.dtype != y.dtype or not np.array_equal(x, y):
                    first = None
                    if x.shape == y.shape:
                        bad = np.nonzero(x != y)[0]
                        first = int(bad[0]) if bad.size else None
                    diffs.append(f"hop {h} etype {e} {name}: sizes {x.size}/{y.size}, "
                                 f"dtypes {x.dtype}/{y.dtype}, first mismatch at {first}")
    for t in range(T):
        if not np.array_equal(ref["input"][t], got["input"][t]):
            diffs.append(f"input frontier of type {t} differs")
    return diffs


def many_relations(rng, R, n0=300, n1=80):
    """Two node types and R edge types, the first 40 and most others into type
    0 (so that type 0 gets the per-vertex non-empty mask): per edge type a share of the
    destinations (none, few, some, all) has in-edges, some edge types empty."""
    nn = [n0, n1]
    ets = []
    for e in range(R):
        d = 0 if e < 40 or rng.random() < 0.85 else 1
        s = int(rng.integers(0, 2))
        share = [0.0, 0.02, 0.2, 1.0][int(rng.integers(0, 4))]
        indptr, indices = [0], []
        for _v in range(nn[d]):
            k = int(rng.integers(1, 12)) if rng.random() < share else 0
            indices.extend(int(x) for x in np.sort(rng.choice(nn[s], size=k, replace=False)))
            indptr.append(len(indices))
        ets.append((s, d, np.array(indptr, np.int64), np.array(indices, np.int64)))
    feats = [rng.standard_normal((n0, 4)).astype(np.float32), None]
    return nn, ets, feats
