"""Seeded synthetic heterographs, feature tables and seed batches.

This module only makes inputs.  It holds none of the method's arithmetic, and both
the GPU library's tests and the CPU oracle read its outputs.  The shapes follow the
paper's workloads (arXiv 2112.15345, Table 1 datasets and Appendix A.1 fanouts and
batch sizes); the graphs themselves are synthetic stand-ins, since the public
datasets are not available here.

Generator for one edge type G(n_src, n_dst, E, alpha, seed):
  1. raw_v = floor(U^(-1/(alpha-1))), U ~ Uniform(0, 1], per destination v: a
     discrete power law with P(raw >= k) = k^-(alpha-1), i.e. pmf ~ k^-alpha; clipped
     to n_src.
  2. d_v = floor(c*raw_v) + Bernoulli(frac(c*raw_v)), c = E / sum(raw), clipped to
     n_src; then +-1 on random eligible vertices until sum(d) == E exactly.
  3. d_v distinct uniform sources per destination (draw, drop duplicates after a
     sort by (dst, src), redraw), ascending within a destination: CSC by dst.
  Reverse edge types are exact transposes of their forward type.
Features: standard normal float32, cast to fp16 / bf16 where asked.
Seeds of batch b: numpy Generator(PCG64(10000*cfg + b)).choice(n, B, replace=False);
sampling seed sigma = b.  Graph seed of edge type e: 1000*cfg + e; feature seed of
node type t: 2000*cfg + t.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class NodeType:
    name: str
    num_nodes: int
    dtype: str | None  # "f32" | "f16" | "bf16" | None (no features)
    dim: int


@dataclasses.dataclass(frozen=True)
class EdgeType:
    src: str
    name: str
    dst: str
    nnz: int


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg: int            # 1-based workload number used in the seed recipe
    name: str
    ntypes: tuple
    etypes: tuple       # forward edge types
    reverse: bool       # append the transpose of every forward type
    alpha: float
    fanouts: tuple      # per hop; applied to every edge type
    seed_type: str
    batch: int

    def all_etypes(self):
        ets = list(self.etypes)
        if self.reverse:
            ets += [EdgeType(e.dst, "rev_" + e.name, e.src, e.nnz) for e in self.etypes]
        return ets

    def fanout_matrix(self):
        R = len(self.all_etypes())
        return [[int(k)] * R for k in self.fanouts]


def _kg_sizes(total=300_000_000, R=200, s=1.2):
    w = np.array([(r + 1) ** -s for r in range(R)])
    sizes = np.floor(w / w.sum() * total).astype(np.int64)
    sizes[0] += total - int(sizes.sum())
    return sizes


_ACADEMIC_NT = (NodeType("paper", 736_000, "f32", 128), NodeType("author", 1_130_000, "f32", 128),
                NodeType("institution", 8_700, "f32", 128), NodeType("field", 60_000, "f32", 128))
_ACADEMIC_ET = (EdgeType("author", "writes", "paper", 7_100_000),
                EdgeType("paper", "cites", "paper", 5_400_000),
                EdgeType("paper", "has_field", "field", 7_500_000),
                EdgeType("author", "affiliated", "institution", 1_000_000))

WORKLOADS = {
    1: Workload(1, "tiny-hetero: A 6k, B 4k nodes; A->A 40k, A->B 30k, B->A 30k edges; "
                   "f32x16; fanout [5,5]; 64 A seeds",
                (NodeType("A", 6_000, "f32", 16), NodeType("B", 4_000, "f32", 16)),
                (EdgeType("A", "aa", "A", 40_000), EdgeType("A", "ab", "B", 30_000),
                 EdgeType("B", "ba", "A", 30_000)),
                False, 1.5, (5, 5), "A", 64),
    2: Workload(2, "academic: paper 736k, author 1.13M, institution 8.7k, field 60k; "
                   "4 relations + reverses (42M edges); f32x128; fanout [25,20]; 1024 paper seeds",
                _ACADEMIC_NT, _ACADEMIC_ET, True, 2.1, (25, 20), "paper", 1024),
    3: Workload(3, "billion-share: user 60M, item 30M, seller 2M; 3 relations + reverses "
                   "(1.2B edges); f16x128 on user, item; fanout [15,10,5]; 4096 user seeds",
                (NodeType("user", 60_000_000, "f16", 128), NodeType("item", 30_000_000, "f16", 128),
                 NodeType("seller", 2_000_000, None, 0)),
                (EdgeType("user", "clicks", "item", 450_000_000),
                 EdgeType("user", "follows", "user", 120_000_000),
                 EdgeType("item", "sold_by", "seller", 30_000_000)),
                True, 1.8, (15, 10, 5), "user", 4096),
    4: Workload(4, "knowledge-graph: 1 type 20M nodes; 200 relations, Zipf(1.2) sizes, 300M "
                   "edges; f32x64; fanout [10,10]; 2048 seeds",
                (NodeType("entity", 20_000_000, "f32", 64),),
                tuple(EdgeType("entity", f"r{r}", "entity", int(n))
                      for r, n in enumerate(_kg_sizes())),
                False, 2.1, (10, 10), "entity", 2048),
    5: Workload(5, "gather-heavy academic: config-2 graph, bf16x512 features on all types; "
                   "fanout [10,10]; 8192 paper seeds",
                tuple(NodeType(n.name, n.num_nodes, "bf16", 512) for n in _ACADEMIC_NT),
                _ACADEMIC_ET, True, 2.1, (10, 10), "paper", 8192),
}

TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def powerlaw_degrees(n_dst: int, n_src: int, E: int, alpha: float, gen, device) -> torch.Tensor:
    """Steps 1-2 of the recipe: int64 in-degrees summing exactly to E, each <= n_src."""
    if E > n_dst * n_src:
        raise ValueError("more edges than distinct (src, dst) pairs")
    if n_dst == 0:
        return torch.zeros(0, dtype=torch.int64, device=device)
    u = 1.0 - torch.rand(n_dst, generator=gen, device=device, dtype=torch.float64)
    raw = torch.floor(u.pow(-1.0 / (alpha - 1.0))).clamp_(max=float(n_src))
    x = raw * (E / float(raw.sum()))
    d = torch.floor(x)
    bump = torch.rand(n_dst, generator=gen, device=device, dtype=torch.float64) < (x - d)
    d = (d + bump.to(torch.float64)).clamp_(max=float(n_src)).to(torch.int64)
    for _ in range(10_000):
        diff = int(E - int(d.sum()))
        if diff == 0:
            return d
        elig = torch.nonzero(d < n_src if diff > 0 else d > 0).flatten()
        pick = elig[torch.randperm(elig.numel(), generator=gen, device=device)[: abs(diff)]]
        d[pick] += 1 if diff > 0 else -1
    raise RuntimeError("degree fix-up did not converge")


def distinct_sources(deg: torch.Tensor, n_src: int, gen, device):
    """Step 3: CSC (indptr, indices) with deg[v] distinct uniform sources per v."""
    n_dst = deg.numel()
    E = int(deg.sum())
    indptr = torch.zeros(n_dst + 1, dtype=torch.int64, device=device)
    torch.cumsum(deg, 0, out=indptr[1:])
    if E == 0:
        return indptr, torch.zeros(0, dtype=torch.int64, device=device)
    dst = torch.repeat_interleave(torch.arange(n_dst, device=device, dtype=torch.int64), deg)
    key = dst * n_src + torch.randint(n_src, (E,), generator=gen, device=device, dtype=torch.int64)
    del dst
    for _ in range(10_000):
        key = torch.sort(key).values
        dup = torch.zeros(E, dtype=torch.bool, device=device)
        dup[1:] = key[1:] == key[:-1]
        nd = int(dup.sum())
        if nd == 0:
            return indptr, key % n_src
        redo = key[dup] // n_src
        key[dup] = redo * n_src + torch.randint(n_src, (nd,), generator=gen, device=device,
                                                dtype=torch.int64)
    raise RuntimeError("duplicate-edge redraw did not converge")


def transpose_csc(indptr: torch.Tensor, indices: torch.Tensor, n_src: int):
    """CSC of the reverse edge type: destinations become sources."""
    n_dst = indptr.numel() - 1
    device = indptr.device
    deg = indptr[1:] - indptr[:-1]
    dst = torch.repeat_interleave(torch.arange(n_dst, device=device, dtype=torch.int64), deg)
    key = torch.sort(indices * n_dst + dst).values
    del dst
    rdeg = torch.bincount(indices, minlength=n_src)
    rindptr = torch.zeros(n_src + 1, dtype=torch.int64, device=device)
    torch.cumsum(rdeg, 0, out=rindptr[1:])
    return rindptr, key % n_dst


def edge_type_graph(n_src, n_dst, E, alpha, seed, device):
    gen = _gen(seed, device)
    deg = powerlaw_degrees(n_dst, n_src, E, alpha, gen, device)
    return distinct_sources(deg, n_src, gen, device)


@dataclasses.dataclass
class Graph:
    """A generated heterograph: torch tensors on `device`."""
    workload: Workload
    ntype_names: list
    num_nodes: list
    etypes: list          # (src_type, dst_type, indptr, indices)
    feats: list           # tensor [n, dim] or None per node type
    etype_names: list

    def host_ntypes(self):
        """(num_nodes, numpy feature array or None) per type, for the oracle."""
        out = []
        for n, f in zip(self.num_nodes, self.feats):
            if f is None:
                out.append((n, None))
            elif f.dtype == torch.bfloat16:
                out.append((n, f.view(torch.int16).cpu().numpy().view(np.uint16)))
            else:
                out.append((n, f.cpu().numpy()))
        return out

    def host_etypes(self):
        return [(s, d, ip.cpu().numpy(), ix.cpu().numpy()) for s, d, ip, ix in self.etypes]


def make_graph(workload: Workload, device="cpu", features=True, feat_device=None) -> Graph:
    names = [n.name for n in workload.ntypes]
    idx = {n: i for i, n in enumerate(names)}
    nn = [n.num_nodes for n in workload.ntypes]
    fwd = []
    for e, et in enumerate(workload.etypes):
        s, d = idx[et.src], idx[et.dst]
        ip, ix = edge_type_graph(nn[s], nn[d], et.nnz, workload.alpha,
                                 1000 * workload.cfg + e, device)
        fwd.append((s, d, ip, ix))
    ets = list(fwd)
    if workload.reverse:
        for (s, d, ip, ix) in fwd:
            rip, rix = transpose_csc(ip, ix, nn[s])
            ets.append((d, s, rip, rix))
    feats = []
    fdev = feat_device or device
    for t, nt in enumerate(workload.ntypes):
        if not features or nt.dtype is None:
            feats.append(None)
            continue
        feats.append(random_features(nt.num_nodes, nt.dim, nt.dtype, 2000 * workload.cfg + t, fdev))
    return Graph(workload, names, nn, ets, feats, [e.name for e in workload.all_etypes()])


def random_features(n, dim, dtype, seed, device, chunk_rows=1 << 22):
    gen = _gen(seed, device)
    out = torch.empty((n, dim), dtype=TORCH_DTYPES[dtype], device=device)
    for r0 in range(0, n, chunk_rows):
        r1 = min(n, r0 + chunk_rows)
        out[r0:r1] = torch.randn((r1 - r0, dim), generator=gen, device=device,
                                 dtype=torch.float32).to(out.dtype)
    return out


def batch_seeds(workload: Workload, b: int) -> np.ndarray:
    t = [n.name for n in workload.ntypes].index(workload.seed_type)
    n = workload.ntypes[t].num_nodes
    rng = np.random.Generator(np.random.PCG64(10000 * workload.cfg + b))
    return rng.choice(n, size=min(workload.batch, n), replace=False).astype(np.int64)


def seeds_per_type(workload: Workload, b: int):
    """Seed arrays indexed by node type (None for types without seeds)."""
    t = [n.name for n in workload.ntypes].index(workload.seed_type)
    out = [None] * len(workload.ntypes)
    out[t] = batch_seeds(workload, b)
    return out


# Edge-seeded (link-prediction) batches on a workload's graph: the paper's
# link-prediction runs use two sampling hops of fanout 25 and 15 and the batch
# size of its other runs (Appendix A.1); the targets are edges of one forward
# relation, drawn without replacement.
# Layer-wise (LADIES) batches on a workload's graph: the workload's seeds,
# 512 draws per node type in each of two hops (LADIES samples 512 vertices
# per layer in its main experiments).
LAYER_SIZES = (512, 512)

LINK_FANOUTS = (25, 15)
LINK_BATCH = 1000
LINK_NEG = 1


def reverse_maps(graph: Graph):
    """rev_etype[e] and rev_eid[e] (int64 tensor [nnz_e] on the graph's device)
    for a workload whose reverse edge types are transposes: the slot of every
    edge's reverse in its reverse type.  None, None when there are no reverses."""
    wl = graph.workload
    if not wl.reverse:
        return None, None
    R0 = len(wl.etypes)
    rev_etype = [R0 + e for e in range(R0)] + list(range(R0))
    fmaps, rmaps = [], []
    for (s, d, ip, ix) in graph.etypes[:R0]:
        n_dst = ip.numel() - 1
        deg = ip[1:] - ip[:-1]
        dst = torch.repeat_interleave(torch.arange(n_dst, device=ip.device, dtype=torch.int64), deg)
        # the transpose orders its slots by (source, destination), all distinct
        order = torch.argsort(ix * n_dst + dst)
        del dst
        fmap = torch.empty_like(order)
        fmap[order] = torch.arange(order.numel(), device=order.device, dtype=torch.int64)
        fmaps.append(fmap)
        rmaps.append(order)
    return rev_etype, fmaps + rmaps


def link_targets(graph: Graph, b: int, etype: int, size: int = LINK_BATCH):
    """Target edge IDs of link-prediction batch b: `size` distinct edges of
    edge type `etype`, numpy Generator(PCG64(30000*cfg + b)); a list per edge
    type (None for the others)."""
    nnz = int(graph.etypes[etype][3].numel())
    rng = np.random.Generator(np.random.PCG64(30000 * graph.workload.cfg + b))
    out = [None] * len(graph.etypes)
    out[etype] = rng.choice(nnz, size=min(size, nnz), replace=False).astype(np.int64)
    return out


def random_hetero(rng: np.random.Generator, max_types=3, max_etypes=4, max_nodes=50,
                  max_deg=30, feat_dim=4):
    """A tiny random heterograph for brute-force and invariant checks (numpy CSC).

    Degrees 0..max_deg (capped by the source count), distinct sources, self-loops
    allowed when source and destination types coincide."""
    T = int(rng.integers(1, max_types + 1))
    nn = [int(rng.integers(0, max_nodes + 1)) for _ in range(T)]
    R = int(rng.integers(1, max_etypes + 1))
    etypes = []
    for _ in range(R):
        s, d = int(rng.integers(0, T)), int(rng.integers(0, T))
        indptr = [0]
        indices = []
        for _v in range(nn[d]):
            k = int(rng.integers(0, min(max_deg, nn[s]) + 1)) if nn[s] > 0 else 0
            if rng.random() < 0.3:
                k = min(k, 2)
            srcs = np.sort(rng.choice(nn[s], size=k, replace=False)) if k else np.zeros(0, np.int64)
            indices.extend(int(x) for x in srcs)
            indptr.append(len(indices))
        etypes.append((s, d, np.array(indptr, np.int64), np.array(indices, np.int64)))
    feats = []
    for t in range(T):
        if rng.random() < 0.8:
            feats.append(rng.standard_normal((nn[t], feat_dim)).astype(np.float32))
        else:
            feats.append(None)
    return nn, etypes, feats


def graph_stats(graph: Graph, fanout: int | None = None) -> dict:
    """Shape statistics of a generated graph (max degree, share of zero in-degree,
    share of destinations above a fanout, edge-biased mean degree)."""
    st = {}
    for name, (s, d, ip, ix) in zip(graph.etype_names, graph.etypes):
        deg = (ip[1:] - ip[:-1]).to(torch.float64)
        nz = deg.sum().item()
        st[name] = {
            "nnz": int(ix.numel()),
            "max_deg": int(deg.max().item()) if deg.numel() else 0,
            "zero_in_deg": float((deg == 0).to(torch.float64).mean().item()) if deg.numel() else 1.0,
            "edge_biased_mean_deg": float((deg * deg).sum().item() / nz) if nz else 0.0,
        }
        if fanout is not None and deg.numel():
            st[name]["above_fanout"] = float((deg > fanout).to(torch.float64).mean().item())
    return st


def human_bytes(n: int) -> str:
    for unit in ("B", "KB", "MB", "GB", "TB"):
        if n < 1024 or unit == "TB":
            return f"{n:.1f} {unit}" if unit != "B" else f"{n} B"
        n /= 1024.0
    return str(n)


__all__ = ["NodeType", "EdgeType", "Workload", "WORKLOADS", "Graph", "make_graph",
           "reverse_maps", "link_targets", "LAYER_SIZES", "LINK_FANOUTS", "LINK_BATCH", "LINK_NEG",
           "batch_seeds", "seeds_per_type", "random_hetero", "graph_stats", "powerlaw_degrees",
           "distinct_sources", "transpose_csc", "random_features"]
