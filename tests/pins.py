"""Checks that pin the CPU oracle to things other than itself.

- Philox4x32-10 and the edge key are compared with rocRAND's engine (an
  independent implementation, reached through tests/rocrand_ref.cpp).
- The selection of one (destination, etype) pair is compared with brute force:
  numpy's lexsort over the rocRAND keys of every in-edge.
- Whole mini-batches are checked against the definitions of the method
  (DistDGLv2, arXiv 2112.15345, Sec. 3.2 and Sec. 4.2.2): sampled degree =
  min(deg, K); every kept edge exists and is one of the K smallest; the next
  frontier is the unique set of this hop's vertices (numpy set operations); the
  relabel maps each edge back to its endpoints.
- Gather against numpy fancy indexing; error codes; uniformity statistics.

Each pin returns a list of failure messages (empty = pass), so the same checks
can run against deliberately broken builds of the oracle.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
_RR_SRC = os.path.join(HERE, "rocrand_ref.cpp")
_RR_LIB = os.path.join(ROOT, "_build", "tests", "librocrand_ref.so")
M32 = (1 << 32) - 1

_rr = None


def rocrand_ref():
    """rocRAND's Philox4x32-10 engine on the host (built on first use)."""
    global _rr
    if _rr is None:
        if not os.path.exists(_RR_LIB) or os.path.getmtime(_RR_LIB) < os.path.getmtime(_RR_SRC):
            os.makedirs(os.path.dirname(_RR_LIB), exist_ok=True)
            tmp = f"{_RR_LIB}.{os.getpid()}.tmp"  # concurrent builders never share a file
            subprocess.run(["/opt/rocm/bin/hipcc", "-x", "hip", "-O1", "-fPIC", "-shared",
                            "--offload-arch=gfx950", "-I/opt/rocm/include", _RR_SRC, "-o",
                            tmp], check=True, capture_output=True)
            os.replace(tmp, _RR_LIB)
        lib = ctypes.CDLL(_RR_LIB)
        lib.rr_word.argtypes = [ctypes.c_uint64] * 3
        lib.rr_word.restype = ctypes.c_uint32
        lib.rr_block.argtypes = [ctypes.c_uint64] * 3 + [ctypes.c_void_p]
        lib.rr_block.restype = None
        _rr = lib
    return _rr


def rr_key(sigma: int, hop: int, etype: int, eid: int, key_bits: int = 32) -> int:
    """The edge key by its definition, computed by rocRAND: word (eid % 4) at
    counter (eid / 4, hop, etype), key sigma, truncated to key_bits bits."""
    w = rocrand_ref().rr_word(sigma & ((1 << 64) - 1), (hop & M32) | ((etype & M32) << 32), eid)
    return int(w) >> (32 - key_bits)


def rr_block(seed: int, subsequence: int, counter_lo64: int) -> np.ndarray:
    out = np.zeros(4, dtype=np.uint32)
    rocrand_ref().rr_block(seed, subsequence, counter_lo64, out.ctypes.data)
    return out


def brute_select(sigma, hop, etype, lo, hi, fanout, key_bits=32, excluded=None):
    """The kept edge IDs of one pair: all when deg <= K or K == -1, else the K
    smallest by (key, eid), in ascending eid.  Edge IDs in `excluded` take no
    part (they are removed before counting deg)."""
    eids = np.arange(lo, hi, dtype=np.int64)
    if excluded is not None and len(excluded):
        eids = eids[~np.isin(eids, excluded)]
    if fanout < 0 or eids.size <= fanout:
        return eids
    keys = np.array([rr_key(sigma, hop, etype, int(x), key_bits) for x in eids], dtype=np.int64)
    order = np.lexsort((eids, keys))
    return np.sort(eids[order[:fanout]])


# ---------------------------------------------------------------------------
# pins

def pin_philox(lib, rng, n=200):
    fails = []
    cases = [(0, 0, 0), ((1 << 64) - 1, (1 << 64) - 1, (1 << 62) - 1)]
    for _ in range(n):
        cases.append((int(rng.integers(0, 1 << 63)) * 2 + int(rng.integers(0, 2)),
                      int(rng.integers(0, 1 << 63)), int(rng.integers(0, 1 << 62))))
    for seed, sub, c in cases:
        ref = rr_block(seed, sub, c)
        got = oracle.philox4x32_10([c & M32, c >> 32, sub & M32, sub >> 32],
                                   [seed & M32, seed >> 32], lib)
        if not np.array_equal(ref, got):
            fails.append(f"philox seed={seed} sub={sub} ctr={c}: {got} != {ref}")
    return fails


def pin_edge_key(lib, rng, n=300):
    fails = []
    for i in range(n):
        sigma = int(rng.integers(0, 1 << 63)) * 2 + int(rng.integers(0, 2))
        hop, et = int(rng.integers(0, 8)), int(rng.integers(0, 400))
        eid = int(rng.integers(0, 1 << 40)) if i % 2 else int(rng.integers(0, 64))
        bits = [32, 16, 4, 1][i % 4]
        ref = rr_key(sigma, hop, et, eid, bits)
        got = oracle.edge_key(sigma, hop, et, eid, bits, lib)
        if ref != got:
            fails.append(f"edge_key({sigma},{hop},{et},{eid},{bits}) = {got} != {ref}")
    return fails


def pin_select(lib, rng, n=300):
    fails = []
    for i in range(n):
        lo = int(rng.integers(0, 1000))
        deg = int(rng.integers(0, 120))
        choices = [-1, 0, 1, 2, 3, 5, 10, 25, deg, deg + 1, max(deg - 1, 0)]
        k = choices[int(rng.integers(0, len(choices)))]
        sigma = int(rng.integers(0, 1 << 62))
        hop, et = int(rng.integers(0, 4)), int(rng.integers(0, 6))
        bits = [32, 32, 8, 3, 1][i % 5]
        ref = brute_select(sigma, hop, et, lo, lo + deg, k, bits)
        got = oracle.select(sigma, hop, et, lo, lo + deg, k, bits, lib)
        if not np.array_equal(ref, got):
            fails.append(f"select lo={lo} deg={deg} K={k} bits={bits}: {got} != {ref}")
    return fails


def check_blocks(ntypes, etypes, seeds, fanouts, sigma, key_bits, res, brute=True,
                 excluded=None):
    """Checks one mini-batch result against the definitions.

    ntypes: [num_nodes]; etypes: [(s, d, indptr, indices)] numpy; seeds: per
    type array or None; res: dict as returned by oracle.HostGraph.sample_blocks
    (or the same layout from the GPU path); excluded: {etype: edge IDs} that
    no hop may sample (edge-seeded mini-batches)."""
    fails = []
    T, R, H = len(ntypes), len(etypes), len(fanouts)
    F = [np.zeros(0, np.int64) if s is None else np.asarray(s, np.int64) for s in seeds]
    for h in range(H):
        src_lists = []
        for t in range(T):
            n_dst, sg = res["nodes"][(h, t)]
            if n_dst != F[t].size or not np.array_equal(sg[:n_dst], F[t]):
                fails.append(f"hop {h} type {t}: destination prefix is not the frontier")
            src_lists.append(sg)
        sampled_by_type = [[] for _ in range(T)]
        for e, (s, d, indptr, indices) in enumerate(etypes):
            ip, sl, dl, eid = res["edges"][(h, e)]
            k = fanouts[h][e]
            if ip.size != F[d].size + 1 or (ip.size and (ip[0] != 0 or ip[-1] != eid.size)):
                fails.append(f"hop {h} etype {e}: bad block indptr")
                continue
            if np.any(np.diff(ip) < 0):
                fails.append(f"hop {h} etype {e}: decreasing block indptr")
                continue
            xs = None if not excluded else excluded.get(e)
            if xs is not None and eid.size and np.any(np.isin(eid, xs)):
                fails.append(f"hop {h} etype {e}: an excluded edge was sampled")
            for i, v in enumerate(F[d]):
                a, b = int(ip[i]), int(ip[i + 1])
                lo, hi = int(indptr[v]), int(indptr[v + 1])
                deg = hi - lo
                if xs is not None:
                    deg -= int(np.count_nonzero((xs >= lo) & (xs < hi)))
                want_n = deg if (k < 0 or deg <= k) else k
                if b - a != want_n:
                    fails.append(f"hop {h} etype {e} dst {i}: {b - a} edges, want min(deg,K)={want_n}")
                    continue
                got = eid[a:b]
                if np.any(dl[a:b] != i):
                    fails.append(f"hop {h} etype {e} dst {i}: wrong dst_local")
                if np.any(got < lo) or np.any(got >= hi):
                    fails.append(f"hop {h} etype {e} dst {i}: edge not an in-edge of the vertex")
                    continue
                if np.any(np.diff(got) <= 0):
                    fails.append(f"hop {h} etype {e} dst {i}: edge IDs not strictly ascending")
                if brute and deg > 0:
                    ref = brute_select(sigma, h, e, lo, hi, k, key_bits, xs)
                    if not np.array_equal(ref, got):
                        fails.append(f"hop {h} etype {e} dst {i}: kept {got}, brute force {ref}")
            if eid.size:
                srcg = indices[eid]
                sampled_by_type[s].append(srcg)
                sl_ok = (sl >= 0) & (sl < src_lists[s].size)
                if not np.all(sl_ok) or not np.array_equal(src_lists[s][sl], srcg):
                    fails.append(f"hop {h} etype {e}: relabelled sources do not map back")
        for t in range(T):
            allsrc = np.concatenate(sampled_by_type[t]) if sampled_by_type[t] else np.zeros(0, np.int64)
            want_new = np.setdiff1d(np.unique(allsrc), F[t])
            got_new = src_lists[t][F[t].size:]
            if not np.array_equal(want_new, got_new):
                fails.append(f"hop {h} type {t}: new vertices {got_new[:8]}... != unique set "
                             f"minus frontier {want_new[:8]}...")
            F[t] = src_lists[t]
    for t in range(T):
        if not np.array_equal(res["input"][t], F[t]):
            fails.append(f"type {t}: input frontier differs from the last source list")
    return fails


def random_case(rng, max_nodes=40, max_deg=25):
    nn, ets, feats = workloads.random_hetero(rng, max_nodes=max_nodes, max_deg=max_deg)
    T, R = len(nn), len(ets)
    seeds = []
    for t in range(T):
        if nn[t] == 0 or rng.random() < 0.25:
            seeds.append(None if rng.random() < 0.5 else np.zeros(0, np.int64))
        else:
            seeds.append(rng.choice(nn[t], size=int(rng.integers(1, nn[t] + 1)), replace=False)
                         .astype(np.int64))
    H = int(rng.integers(0, 4))
    fchoices = [-1, 0, 1, 2, 3, 5, 8, 100]
    fanouts = [[fchoices[int(rng.integers(0, len(fchoices)))] for _ in range(R)] for _ in range(H)]
    sigma = int(rng.integers(0, 1 << 63))
    bits = 32 if rng.random() < 0.7 else int(rng.integers(1, 5))
    return nn, ets, feats, seeds, fanouts, sigma, bits


def pin_blocks(lib, rng, n=60):
    fails = []
    for c in range(n):
        nn, ets, feats, seeds, fanouts, sigma, bits = random_case(rng)
        hg = oracle.HostGraph(list(zip(nn, feats)), ets, lib=lib)
        res = hg.sample_blocks(seeds, fanouts, sigma, bits)
        f = check_blocks(nn, ets, seeds, fanouts, sigma, bits, res)
        fails += [f"case {c}: {m}" for m in f[:3]]
    return fails


def pin_gather(lib, rng, n=20):
    fails = []
    for c in range(n):
        rows = int(rng.integers(1, 50))
        dim = int(rng.integers(1, 9))
        dt = [np.float32, np.float16, np.uint16, np.int8][c % 4]
        feat = (rng.standard_normal((rows, dim)) * 100).astype(dt)
        ids = rng.integers(0, rows, size=int(rng.integers(0, 80))).astype(np.int64)
        hg = oracle.HostGraph([(rows, feat)], [], lib=lib)
        got = hg.gather(0, ids)
        if got.tobytes() != feat[ids].tobytes():
            fails.append(f"gather case {c}: bytes differ from feat[ids]")
    return fails


def pin_errors(lib):
    fails = []
    indptr = np.array([0, 1, 3, 3], np.int64)
    indices = np.array([2, 0, 1], np.int64)
    hg = oracle.HostGraph([(3, None)], [(0, 0, indptr, indices)], lib=lib)

    def expect(status, fn):
        try:
            fn()
        except oracle.OracleError as ex:
            if ex.status != status:
                fails.append(f"expected status {status}, got {ex.status}")
            return
        fails.append(f"expected status {status}, call succeeded")

    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([1, 1])], [[2]], 0))
    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([3])], [[2]], 0))
    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([-1])], [[2]], 0))
    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([0])], [[-2]], 0))
    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([0])], [[1]], 0, key_bits=0))
    expect(oracle.EINVAL, lambda: hg.sample_blocks([np.array([0])], [[1]], 0, key_bits=33))
    expect(oracle.EINVAL, lambda: hg.gather(0, np.array([0])))
    expect(oracle.EINVAL, lambda: oracle.HostGraph([(3, None)], [(0, 0, np.array([0, 1, 3, 2]),
                                                                     indices)], lib=lib))
    expect(oracle.EINVAL, lambda: oracle.HostGraph([(3, None)], [(0, 0, indptr,
                                                                 np.array([2, 0, 3]))], lib=lib))
    expect(oracle.EINVAL, lambda: oracle.HostGraph([(3, None)], [(0, 1, indptr, indices)], lib=lib))
    f3 = np.arange(6, dtype=np.float32).reshape(3, 2)
    hgf = oracle.HostGraph([(3, f3)], [], lib=lib)
    expect(oracle.EINVAL, lambda: hgf.gather(0, np.array([3])))
    # H = 0: the input frontier is the seeds
    r = hg.sample_blocks([np.array([2, 0])], [], 5)
    if not np.array_equal(r["input"][0], [2, 0]):
        fails.append("n_hops = 0: input frontier is not the seeds")
    return fails


def pin_special_fanouts(lib, rng):
    """-1 keeps all, 0 keeps none, K >= deg keeps all (closed forms)."""
    fails = []
    for _ in range(20):
        lo, deg = int(rng.integers(0, 100)), int(rng.integers(0, 40))
        sigma = int(rng.integers(0, 1 << 60))
        all_e = np.arange(lo, lo + deg)
        if not np.array_equal(oracle.select(sigma, 0, 0, lo, lo + deg, -1, 32, lib), all_e):
            fails.append("K=-1 does not keep every edge")
        if oracle.select(sigma, 0, 0, lo, lo + deg, 0, 32, lib).size != 0:
            fails.append("K=0 keeps an edge")
        if not np.array_equal(oracle.select(sigma, 1, 2, lo, lo + deg, deg, 32, lib), all_e):
            fails.append("K=deg does not keep every edge")
    return fails


def chi2_sf(x, k):
    """Survival function of the chi-squared distribution (scipy when present)."""
    try:
        from scipy.stats import chi2
        return float(chi2.sf(x, k))
    except Exception:  # pragma: no cover
        # Wilson-Hilferty approximation
        z = ((x / k) ** (1 / 3) - (1 - 2 / (9 * k))) / math.sqrt(2 / (9 * k))
        return 0.5 * math.erfc(z / math.sqrt(2))


def pin_statistics(lib, n_sigma=6000):
    """"Randomly pick at most K" (Sec. 3.2): every K-subset of the in-edges is
    equally likely over seeds, each edge is kept with probability K/deg, and the
    draws of different hops are independent."""
    fails = []
    deg, k = 6, 2
    counts = {}
    incl = np.zeros(deg)
    same = 0
    for sigma in range(n_sigma):
        a = tuple(oracle.select(sigma, 0, 3, 100, 100 + deg, k, 32, lib) - 100)
        b = tuple(oracle.select(sigma, 1, 3, 100, 100 + deg, k, 32, lib) - 100)
        counts[a] = counts.get(a, 0) + 1
        incl[list(a)] += 1
        same += a == b
    n_sub = math.comb(deg, k)
    if len(counts) != n_sub:
        fails.append(f"only {len(counts)} of {n_sub} subsets ever drawn")
    exp = n_sigma / n_sub
    x2 = sum((c - exp) ** 2 / exp for c in counts.values()) + (n_sub - len(counts)) * exp
    p = chi2_sf(x2, n_sub - 1)
    if p < 1e-3:
        fails.append(f"subset frequencies not uniform: chi2={x2:.1f}, p={p:.2g}")
    frac = incl / n_sigma
    if np.max(np.abs(frac - k / deg)) > 0.03:
        fails.append(f"per-edge inclusion {frac} far from K/deg={k / deg:.3f}")
    if abs(same / n_sigma - 1 / n_sub) > 0.02:
        fails.append(f"hop 0 and hop 1 agree {same / n_sigma:.3f}, independent draws agree "
                     f"{1 / n_sub:.3f}")
    return fails


# ---------------------------------------------------------------------------
# edge-seeded (link-prediction) mini-batches

def np_edge_dst(indptr, eids):
    """Destination of CSC slots: numpy's searchsorted (the last v with
    indptr[v] <= eid)."""
    return np.searchsorted(np.asarray(indptr), np.asarray(eids, np.int64), side="right") - 1


def rr_negative(sigma, etype, eid, k, n):
    """Negative k of edge eid by its definition, the two Philox words from
    rocRAND: counter (eid, 2^31 | k, etype), words 0 and 1, then
    floor(u * n / 2^64)."""
    rr = rocrand_ref()
    sub = ((0x80000000 | k) & M32) | ((etype & M32) << 32)
    w0 = int(rr.rr_word(sigma & ((1 << 64) - 1), sub, 4 * eid))
    w1 = int(rr.rr_word(sigma & ((1 << 64) - 1), sub, 4 * eid + 1))
    return ((w0 | (w1 << 32)) * n) >> 64


def with_reverses(nn, etypes):
    """The edge types followed by their transposes, and the reverse maps:
    rev_etype[e] and rev_eid[e][j] = slot of edge j's reverse (numpy)."""
    R = len(etypes)
    out = list(etypes)
    rev_etype = [R + e for e in range(R)] + list(range(R))
    fwd_maps, rev_maps = [], []
    for (s, d, ip, ix) in etypes:
        dst = np.repeat(np.arange(nn[d], dtype=np.int64), np.diff(ip))
        order = np.lexsort((dst, ix))  # by source, then destination
        rip = np.zeros(nn[s] + 1, np.int64)
        np.cumsum(np.bincount(ix, minlength=nn[s]), out=rip[1:])
        out.append((d, s, rip, dst[order]))
        fmap = np.empty(ix.size, np.int64)
        fmap[order] = np.arange(ix.size, dtype=np.int64)
        fwd_maps.append(fmap)
        rev_maps.append(order.astype(np.int64))
    return out, rev_etype, fwd_maps + rev_maps


def edge_batch_expect(nn, etypes, targets, n_neg, exclude, rev_etype, rev_eid, sigma):
    """Seeds, pair graphs (as global IDs) and excluded edges of an
    edge-seeded mini-batch, from numpy and rocRAND."""
    T, R = len(nn), len(etypes)
    ends = [[] for _ in range(T)]
    pairs = {}
    for e, (s, d, ip, ix) in enumerate(etypes):
        tg = np.zeros(0, np.int64) if targets[e] is None else np.asarray(targets[e], np.int64)
        src = ix[tg]
        dst = np_edge_dst(ip, tg)
        neg = np.array([rr_negative(sigma, e, int(j), k, nn[d]) for j in tg for k in range(n_neg)],
                       np.int64)
        ends[s].append(src)
        ends[d] += [dst, neg]
        pairs[e] = (src, dst, neg)
    seeds = [np.unique(np.concatenate(x)) if x else np.zeros(0, np.int64) for x in ends]
    excluded = {}
    if exclude >= 1:
        for e in range(R):
            x = [np.zeros(0, np.int64) if targets[e] is None else np.asarray(targets[e], np.int64)]
            if exclude == 2:
                for f in range(R):
                    if rev_etype[f] == e and targets[f] is not None:
                        x.append(rev_eid[f][np.asarray(targets[f], np.int64)])
            excluded[e] = np.unique(np.concatenate(x))
    return seeds, pairs, excluded


def check_edge_blocks(nn, etypes, targets, n_neg, exclude, rev_etype, rev_eid, fanouts, sigma,
                      key_bits, res, brute=True):
    """An edge-seeded result against the definitions: seeds = unique endpoints
    per type (numpy), the pair graphs map back to the targets' endpoints and
    negatives, and the blocks satisfy every vertex-seeded check from those
    seeds with the excluded edges removed."""
    fails = []
    seeds, pairs, excluded = edge_batch_expect(nn, etypes, targets, n_neg, exclude, rev_etype,
                                               rev_eid, sigma)
    for t in range(len(nn)):
        if not np.array_equal(res["seeds"][t], seeds[t]):
            fails.append(f"type {t}: seeds {res['seeds'][t][:8]} != unique endpoints {seeds[t][:8]}")
            return fails
    for e, (s, d, ip, ix) in enumerate(etypes):
        src, dst, neg = pairs[e]
        ps, pd, pn = res["pairs"][e]
        for name, loc, want, t in (("pos_src", ps, src, s), ("pos_dst", pd, dst, d),
                                   ("neg_dst", pn, neg, d)):
            if loc.size != want.size or np.any(loc < 0) or np.any(loc >= seeds[t].size) or \
                    not np.array_equal(seeds[t][loc], want):
                fails.append(f"etype {e}: {name} does not map back to the targets")
    fails += check_blocks(nn, etypes, seeds, fanouts, sigma, key_bits, res, brute=brute,
                          excluded=excluded)
    return fails


def random_edge_case(rng, max_nodes=30, max_deg=15):
    nn, ets, feats = workloads.random_hetero(rng, max_nodes=max_nodes, max_deg=max_deg,
                                             max_etypes=3)
    ets, rev_etype, rev_eid = with_reverses(nn, ets)
    R = len(ets)
    targets = []
    for e in range(R):
        nnz = ets[e][3].size
        if nnz == 0 or rng.random() < 0.3:
            targets.append(None)
        else:
            targets.append(rng.integers(0, nnz, size=int(rng.integers(1, 6))).astype(np.int64))
    H = int(rng.integers(0, 3))
    fchoices = [-1, 0, 1, 2, 3, 5]
    fanouts = [[fchoices[int(rng.integers(0, len(fchoices)))] for _ in range(R)] for _ in range(H)]
    sigma = int(rng.integers(0, 1 << 63))
    bits = 32 if rng.random() < 0.7 else int(rng.integers(1, 5))
    n_neg = int(rng.choice([0, 1, 3]))
    exclude = int(rng.integers(0, 3))
    return nn, ets, feats, targets, n_neg, exclude, rev_etype, rev_eid, fanouts, sigma, bits


def pin_edge_dst(lib, rng, n=40):
    fails = []
    for c in range(n):
        deg = rng.integers(0, 5, size=int(rng.integers(1, 30)))
        deg[rng.random(deg.size) < 0.3] = 0
        ip = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
        for j in range(int(ip[-1])):
            got = oracle.edge_dst(ip, j, lib)
            if got != int(np_edge_dst(ip, [j])[0]):
                fails.append(f"edge_dst case {c} eid {j}: {got}")
    return fails


def pin_negatives(lib, rng, n=200):
    fails = []
    for i in range(n):
        sigma = int(rng.integers(0, 1 << 63)) * 2 + int(rng.integers(0, 2))
        e, k = int(rng.integers(0, 300)), int(rng.integers(0, oracle.MAX_NEG))
        eid = int(rng.integers(0, 1 << 40)) if i % 2 else int(rng.integers(0, 64))
        nd = [1, 2, 7, 1000, 60_000_000, (1 << 40) + 3][i % 6]
        want = rr_negative(sigma, e, eid, k, nd)
        got = oracle.negative_dst(sigma, e, eid, k, nd, lib)
        if got != want:
            fails.append(f"negative({sigma},{e},{eid},{k},{nd}) = {got} != {want}")
    return fails


def pin_edge_blocks(lib, rng, n=40):
    fails = []
    for c in range(n):
        nn, ets, feats, tg, q, x, rev_et, rev_eid, fanouts, sigma, bits = random_edge_case(rng)
        hg = oracle.HostGraph(list(zip(nn, feats)), ets, lib=lib)
        res = hg.sample_edge_blocks(tg, fanouts, sigma, n_neg=q, exclude=x, rev_etype=rev_et,
                                    rev_eid=rev_eid, key_bits=bits)
        f = check_edge_blocks(nn, ets, tg, q, x, rev_et, rev_eid, fanouts, sigma, bits, res)
        fails += [f"edge case {c} (exclude {x}, neg {q}): {m}" for m in f[:3]]
    return fails


def pin_edge_errors(lib):
    fails = []
    nn = [3]
    ets = [(0, 0, np.array([0, 1, 3, 3], np.int64), np.array([2, 0, 1], np.int64))]
    ets, rev_et, rev_eid = with_reverses(nn, ets)
    hg = oracle.HostGraph([(3, None)], ets, lib=lib)

    def expect(fn):
        try:
            fn()
        except oracle.OracleError as ex:
            if ex.status != oracle.EINVAL:
                fails.append(f"expected EINVAL, got {ex.status}")
            return
        fails.append("expected EINVAL, call succeeded")

    ok = [np.array([1]), None]
    expect(lambda: hg.sample_edge_blocks([np.array([3]), None], [[1, 1]], 0))
    expect(lambda: hg.sample_edge_blocks([np.array([-1]), None], [[1, 1]], 0))
    expect(lambda: hg.sample_edge_blocks(ok, [[1, 1]], 0, n_neg=oracle.MAX_NEG + 1))
    expect(lambda: hg.sample_edge_blocks(ok, [[1, 1]], 0, exclude=3))
    expect(lambda: hg.sample_edge_blocks(ok, [[1, 1]], 0, exclude=2))
    bad = [rev_eid[0].copy(), rev_eid[1]]
    bad[0][1] = (bad[0][1] + 1) % 3  # the reverse of edge 1 named wrongly
    expect(lambda: hg.sample_edge_blocks(ok, [[1, 1]], 0, exclude=2, rev_etype=rev_et,
                                         rev_eid=bad))
    r = hg.sample_edge_blocks(ok, [[1, 1]], 0, exclude=2, rev_etype=rev_et, rev_eid=rev_eid)
    if not np.array_equal(r["seeds"][0], [0, 1]):
        fails.append(f"seeds of target edge 1 (0 -> 1): {r['seeds'][0]}")
    # a reverse edge type must run between the same node types the other way
    ets2 = [(0, 1, np.array([0, 1, 2], np.int64), np.array([0, 1], np.int64)),
            (0, 1, np.array([0, 1, 2], np.int64), np.array([1, 0], np.int64))]
    hg2 = oracle.HostGraph([(2, None), (2, None)], ets2, lib=lib)
    ident = [np.array([0, 1], np.int64), np.array([0, 1], np.int64)]
    expect(lambda: hg2.sample_edge_blocks([np.array([0]), None], [[1, 1]], 0, exclude=2,
                                          rev_etype=[1, 0], rev_eid=ident))
    # no hops: the input frontier is the seeds
    r = hg.sample_edge_blocks(ok, [], 0)
    if not np.array_equal(r["input"][0], [0, 1]):
        fails.append("n_hops = 0: input frontier is not the seeds")
    return fails


def pin_negative_uniformity(lib, n=6000):
    """Negatives are uniform on the destination type (chi-squared) and the
    draws for different k are independent."""
    fails = []
    nd = 7
    counts = np.zeros(nd)
    same = 0
    for eid in range(n):
        a = oracle.negative_dst(11, 2, eid, 0, nd, lib)
        b = oracle.negative_dst(11, 2, eid, 1, nd, lib)
        counts[a] += 1
        same += a == b
    exp = n / nd
    x2 = float(((counts - exp) ** 2 / exp).sum())
    p = chi2_sf(x2, nd - 1)
    if p < 1e-3:
        fails.append(f"negative destinations not uniform: chi2={x2:.1f}, p={p:.2g}")
    if abs(same / n - 1 / nd) > 0.02:
        fails.append(f"negatives 0 and 1 agree {same / n:.3f}, independent draws {1 / nd:.3f}")
    return fails


# ---------------------------------------------------------------------------
# layer-wise (LADIES) mini-batches

def rr_layer_draw(sigma, hop, ntype, k, total):
    """Draw k by its definition, the two Philox words from rocRAND: counter
    (k, 2^30 | hop, ntype), words 0 and 1, then floor(x * total / 2^64)."""
    rr = rocrand_ref()
    sub = ((0x40000000 | hop) & M32) | ((ntype & M32) << 32)
    w0 = int(rr.rr_word(sigma & ((1 << 64) - 1), sub, 4 * k))
    w1 = int(rr.rr_word(sigma & ((1 << 64) - 1), sub, 4 * k + 1))
    return ((w0 | (w1 << 32)) * total) >> 64


def layer_expect(nn, etypes, F, sizes_h, sigma, h):
    """One layer by numpy: per node type the candidates (ascending), their
    importance (sum of floor(2^32 / deg^2) over their edges into the
    frontier) and the drawn set (inverse CDF by searchsorted)."""
    T = len(nn)
    cands, weights = [], []
    for t in range(T):
        us, ws = [np.zeros(0, np.int64)], [np.zeros(0, np.int64)]
        for e, (s, d, ip, ix) in enumerate(etypes):
            if s != t or F[d].size == 0:
                continue
            deg = (ip[F[d] + 1] - ip[F[d]]).astype(np.int64)
            rows = np.repeat(np.arange(F[d].size), deg)
            slots = np.concatenate([np.arange(ip[v], ip[v + 1]) for v in F[d]]) \
                if deg.sum() else np.zeros(0, np.int64)
            w = np.where(deg > 0, (1 << 32) // np.maximum(deg, 1) ** 2, 0)[rows]
            us.append(ix[slots])
            ws.append(w)
        u = np.concatenate(us)
        w = np.concatenate(ws)
        keep = ~np.isin(u, F[t])
        u, w = u[keep], w[keep]
        c = np.unique(u)
        wt = np.zeros(c.size, np.int64)
        np.add.at(wt, np.searchsorted(c, u), w)
        cands.append(c)
        weights.append(wt)
    drawn = []
    for t in range(T):
        c, wt = cands[t], weights[t]
        k = sizes_h[t]
        if k < 0:
            drawn.append(c)
            continue
        total = int(wt.sum())
        if total == 0 or k == 0:
            drawn.append(np.zeros(0, np.int64))
            continue
        cum = np.cumsum(wt)  # inclusive: candidate i holds [cum[i] - wt[i], cum[i])
        r = np.array([rr_layer_draw(sigma, h, t, q, total) for q in range(k)], np.int64)
        drawn.append(np.unique(c[np.searchsorted(cum, r, side="right")]))
    return cands, weights, drawn


def check_layer_blocks(nn, etypes, seeds, layer_sizes, sigma, res):
    """A layer-wise result against the definitions: each hop's new vertices
    are the distinct draws (numpy, rocRAND), ascending after the frontier; the
    block holds exactly the in-edges of the frontier whose source is in the
    next frontier, grouped by destination and ascending edge ID."""
    fails = []
    T = len(nn)
    F = [np.zeros(0, np.int64) if s is None else np.asarray(s, np.int64) for s in seeds]
    for h, sizes in enumerate(layer_sizes):
        _, _, drawn = layer_expect(nn, etypes, F, sizes, sigma, h)
        NF = []
        for t in range(T):
            n_dst, sg = res["nodes"][(h, t)]
            want = np.concatenate([F[t], drawn[t]])
            if n_dst != F[t].size or not np.array_equal(sg, want):
                fails.append(f"hop {h} type {t}: source list {sg[:8]} != frontier + draws {want[:8]}")
            NF.append(want)
        for e, (s, d, ip, ix) in enumerate(etypes):
            bip, sl, dl, eid = res["edges"][(h, e)]
            want_eid, want_dl = [], []
            for i, v in enumerate(F[d]):
                slots = np.arange(ip[v], ip[v + 1])
                keep = slots[np.isin(ix[slots], NF[s])]
                want_eid.append(keep)
                want_dl.append(np.full(keep.size, i, np.int32))
            we = np.concatenate(want_eid) if want_eid else np.zeros(0, np.int64)
            wd = np.concatenate(want_dl) if want_dl else np.zeros(0, np.int32)
            if not np.array_equal(eid, we) or not np.array_equal(dl, wd):
                fails.append(f"hop {h} etype {e}: block edges differ from the filtered in-edges")
                continue
            counts = np.bincount(wd, minlength=F[d].size) if F[d].size else np.zeros(0, np.int64)
            if not np.array_equal(bip, np.concatenate([[0], np.cumsum(counts)])):
                fails.append(f"hop {h} etype {e}: block indptr is not the scan of the counts")
            if eid.size and not np.array_equal(NF[s][sl], ix[eid]):
                fails.append(f"hop {h} etype {e}: relabelled sources do not map back")
        F = NF
    for t in range(T):
        if not np.array_equal(res["input"][t], F[t]):
            fails.append(f"type {t}: input frontier differs from the last source list")
    return fails


def random_layer_case(rng, max_nodes=40, max_deg=20):
    nn, ets, feats = workloads.random_hetero(rng, max_nodes=max_nodes, max_deg=max_deg)
    T = len(nn)
    seeds = []
    for t in range(T):
        if nn[t] == 0 or rng.random() < 0.3:
            seeds.append(None)
        else:
            seeds.append(rng.choice(nn[t], size=int(rng.integers(1, nn[t] + 1)), replace=False)
                         .astype(np.int64))
    H = int(rng.integers(1, 4))  # weights must be cleared between hops
    choices = [-1, 0, 1, 2, 5, 12, 40]
    sizes = [[choices[int(rng.integers(0, len(choices)))] for _ in range(T)] for _ in range(H)]
    return nn, ets, feats, seeds, sizes, int(rng.integers(0, 1 << 63))


def pin_layer_draw(lib, rng, n=200):
    fails = []
    for i in range(n):
        sigma = int(rng.integers(0, 1 << 63)) * 2 + int(rng.integers(0, 2))
        h, t, k = int(rng.integers(0, 6)), int(rng.integers(0, 50)), int(rng.integers(0, 1 << 20))
        total = [1, 7, 1 << 32, (1 << 62) + 11, int(rng.integers(1, 1 << 62))][i % 5]
        want = rr_layer_draw(sigma, h, t, k, total)
        got = oracle.layer_draw(sigma, h, t, k, total, lib)
        if got != want:
            fails.append(f"layer_draw({sigma},{h},{t},{k},{total}) = {got} != {want}")
    return fails


def pin_layer_weight(lib, rng, n=300):
    """floor(2^32 / d^2): w <= 2^32 / d^2 < w + 1, in exact rationals."""
    from fractions import Fraction
    fails = []
    degs = [1, 2, 3, 255, 256, 65535, 65536, 65537, 1 << 20, 5_000_000] + \
        [int(x) for x in rng.integers(1, 10_000_000, size=n)]
    for d in degs:
        w = oracle.layer_weight(d, lib)
        q = Fraction(1 << 32, d * d)
        if not (w <= q < w + 1):
            fails.append(f"layer_weight({d}) = {w}, 2^32/d^2 = {float(q)}")
    if oracle.layer_weight(0, lib) != 0:
        fails.append("layer_weight(0) != 0")
    return fails


def pin_layer_blocks(lib, rng, n=40):
    fails = []
    for c in range(n):
        nn, ets, feats, seeds, sizes, sigma = random_layer_case(rng)
        hg = oracle.HostGraph(list(zip(nn, feats)), ets, lib=lib)
        res = hg.sample_layers(seeds, sizes, sigma)
        f = check_layer_blocks(nn, ets, seeds, sizes, sigma, res)
        fails += [f"layer case {c}: {m}" for m in f[:3]]
    return fails


def pin_layer_boundaries(lib, n_draw=40):
    """Draws that land exactly on interval boundaries: one destination of
    in-degree 65536 gives each of its 65536 distinct sources weight
    floor(2^32 / 65536^2) = 1, so every draw r is the first point of the
    interval of candidate r; a second hop draws among those sources' own
    in-neighbours (a ring), with the first hop's weights cleared."""
    fails = []
    n = 65536 + 70000
    d = 65536
    # vertex 0 has sources 1 .. 65536; vertex v >= 1 has one in-edge from
    # 65537 + (v % 69999)
    indptr = np.concatenate([[0], d + np.arange(0, n, dtype=np.int64)])
    indices = np.concatenate([np.arange(1, d + 1), 65537 + (np.arange(1, n) % 69999)])
    indices = indices.astype(np.int64)
    ets = [(0, 0, indptr.astype(np.int64), indices)]
    hg = oracle.HostGraph([(n, None)], ets, lib=lib)
    for sigma in (3, 77):
        res = hg.sample_layers([np.array([0])], [[n_draw], [n_draw]], sigma)
        f = check_layer_blocks([n], ets, [np.array([0])], [[n_draw], [n_draw]], sigma, res)
        fails += [f"boundary sigma {sigma}: {m}" for m in f[:3]]
    return fails


def pin_layer_errors(lib):
    fails = []
    indptr = np.array([0, 1, 3, 3], np.int64)
    indices = np.array([2, 0, 1], np.int64)
    hg = oracle.HostGraph([(3, None)], [(0, 0, indptr, indices)], lib=lib)
    for seeds, sizes in (([np.array([1, 1])], [[2]]), ([np.array([3])], [[2]]),
                         ([np.array([0])], [[-2]])):
        try:
            hg.sample_layers(seeds, sizes, 0)
            fails.append(f"layer batch {seeds} {sizes} accepted")
        except oracle.OracleError as ex:
            if ex.status != oracle.EINVAL:
                fails.append(f"expected EINVAL, got {ex.status}")
    return fails


def pin_layer_statistics(lib, n_sigma=4000):
    """LADIES' importance sampling: over many sigma, single draws land on each
    candidate with probability weight / total."""
    fails = []
    # one destination of degree 2 and one of degree 4 in the frontier; five
    # candidate sources with different multiplicities into them
    indptr = np.array([0, 2, 6, 6, 6, 6, 6, 6], np.int64)
    indices = np.array([2, 3, 2, 4, 5, 6], np.int64)
    hg = oracle.HostGraph([(7, None)], [(0, 0, indptr, indices)], lib=lib)
    w2, w4 = (1 << 32) // 4, (1 << 32) // 16
    weights = {2: w2 + w4, 3: w2, 4: w4, 5: w4, 6: w4}
    total = sum(weights.values())
    counts = {u: 0 for u in weights}
    for sigma in range(n_sigma):
        res = hg.sample_layers([np.array([0, 1])], [[1]], sigma)
        drawn = res["nodes"][(0, 0)][1][2:]
        for u in drawn:
            counts[int(u)] += 1
    x2 = sum((counts[u] - n_sigma * w / total) ** 2 / (n_sigma * w / total)
             for u, w in weights.items())
    p = chi2_sf(x2, len(weights) - 1)
    if p < 1e-3:
        fails.append(f"draw frequencies {counts} not proportional to importance: p={p:.2g}")
    return fails


ALL_PINS = {
    "philox": pin_philox,
    "edge_key": pin_edge_key,
    "select": pin_select,
    "special_fanouts": pin_special_fanouts,
    "blocks": pin_blocks,
    "gather": lambda lib, rng: pin_gather(lib, rng),
    "errors": lambda lib, rng: pin_errors(lib),
    "edge_dst": pin_edge_dst,
    "negatives": pin_negatives,
    "edge_blocks": pin_edge_blocks,
    "edge_errors": lambda lib, rng: pin_edge_errors(lib),
    "layer_draw": pin_layer_draw,
    "layer_weight": pin_layer_weight,
    "layer_blocks": pin_layer_blocks,
    "layer_errors": lambda lib, rng: pin_layer_errors(lib),
    "layer_boundaries": lambda lib, rng: pin_layer_boundaries(lib),
}
