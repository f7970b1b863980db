"""Python binding of libhg.so (include/hg.h): heterogeneous mini-batch
generation on MI355X (DistDGLv2, arXiv 2112.15345, Sec. 3.2 and Sec. 4.2).

Argument marshalling only: every step of the path runs in the library's gfx950
kernels.  PyTorch supplies device memory (the graph, feature tables, outputs)
and the stream (the current torch stream).  Import fails loudly if the library
is not built; there is no CPU path.

    g = Graph(ntypes=[(num_nodes, feat_or_None), ...],
              etypes=[(src_type, dst_type, indptr, indices), ...])
    b = g.sample_blocks(seeds=[ids_or_None per node type], fanouts=[[K]*R]*H,
                        rng_seed=0)
    n_dst, src_gid = b.nodes(hop, ntype)
    indptr, src_local, dst_local, eid = b.edges(hop, etype)
    x = g.gather_features(b, ntype)
"""
from __future__ import annotations

import collections
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhg.so")

HG_OK, HG_EINVAL, HG_ENOMEM, HG_EDEVICE, HG_EUNSUPPORTED = 0, -1, -2, -3, -4
HG_DT_NONE, HG_DT_F32, HG_DT_F16, HG_DT_BF16 = 0, 1, 2, 3
_DTYPE_CODE = {torch.float32: HG_DT_F32, torch.float16: HG_DT_F16,
               torch.bfloat16: HG_DT_BF16}

# Every entry point declared in include/hg.h.
ABI_SYMBOLS = ("hg_create", "hg_destroy", "hg_retire_stream", "hg_sample_blocks", "hg_sample_blocks_ex",
               "hg_blocks_num_hops", "hg_blocks_nodes", "hg_blocks_edges",
               "hg_blocks_input_nodes", "hg_gather_features", "hg_gather_features_multi",
               "hg_gather_features_multi_timed", "hg_gather_rows",
               "hg_sample_blocks_gather", "hg_sample_blocks_bundle", "hg_blocks_features",
               "hg_graph_types",
               "hg_pipeline_create", "hg_pipeline_submit", "hg_pipeline_next",
               "hg_pipeline_destroy", "hg_sample_edge_blocks", "hg_blocks_seeds",
               "hg_blocks_edge_pairs", "hg_sample_layers", "hg_blocks_edge_counts",
               "hg_sample_edge_blocks_bundle", "hg_sample_layers_bundle",
               "hg_pipeline_submit_layers", "hg_pipeline_submit_edges",
               "hg_blocks_free", "hg_last_error", "hg_debug_philox", "hg_bench_philox",
               "hg_sample_blocks_bundle_timed", "hg_pipeline_submit_timed", "hg_blocks_counts",
               "hg_gather_rows_noalloc")

HG_MAX_NEG = 64
HG_MAX_TIMED_HOPS = 8
HG_STAGE_COUNT, HG_STAGE_SAMPLE, HG_STAGE_SELECT, HG_STAGE_COMPACT, HG_STAGE_RELABEL = range(5)
HG_NUM_STAGES = 5
STAGE_NAMES = ("count", "sample", "select", "compact", "relabel")
HG_EXCLUDE_NONE, HG_EXCLUDE_SELF, HG_EXCLUDE_REVERSE = 0, 1, 2


class HGError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"hg status {status}: {message}")
        self.status = status


class NTypeDesc(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("feat", ctypes.c_void_p),
                ("dtype", ctypes.c_int32), ("dim", ctypes.c_int32)]


class ETypeDesc(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("nnz", ctypes.c_int64), ("indptr", ctypes.c_void_p),
                ("indices", ctypes.c_void_p)]


class StageEventsStruct(ctypes.Structure):
    _fields_ = [("start", (ctypes.c_void_p * HG_NUM_STAGES) * HG_MAX_TIMED_HOPS),
                ("stop", (ctypes.c_void_p * HG_NUM_STAGES) * HG_MAX_TIMED_HOPS),
                ("gather_start", ctypes.c_void_p), ("gather_stop", ctypes.c_void_p)]


class EdgeBatch(ctypes.Structure):
    _fields_ = [("eids", ctypes.c_void_p), ("n_eids", ctypes.c_void_p),
                ("n_neg", ctypes.c_int32), ("exclude", ctypes.c_int32),
                ("rev_etype", ctypes.c_void_p), ("rev_eid", ctypes.c_void_p)]


ALLOC_FN = ctypes.CFUNCTYPE(ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p)
FREE_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p)


class Allocator(ctypes.Structure):
    _fields_ = [("ctx", ctypes.c_void_p), ("alloc", ALLOC_FN), ("free", FREE_FN)]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_I32 = ctypes.c_int32
_PP = ctypes.POINTER(ctypes.c_void_p)
_PI64 = ctypes.POINTER(ctypes.c_int64)


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    sig = {
        "hg_create": ([_P, _I32, _P, _I32, _P, _P, _PP], _I32),
        "hg_destroy": ([_P], None),
        "hg_retire_stream": ([_P, _P], _I32),
        "hg_sample_blocks": ([_P, _P, _P, _I32, _P, ctypes.c_uint64, _P, _PP], _I32),
        "hg_sample_blocks_ex": ([_P, _P, _P, _I32, _P, ctypes.c_uint64, _I32, _P, _PP], _I32),
        "hg_blocks_num_hops": ([_P], _I32),
        "hg_blocks_nodes": ([_P, _I32, _I32, _PI64, _PI64, _PP], _I32),
        "hg_blocks_edges": ([_P, _I32, _I32, _PI64, _PP, _PP, _PP, _PP], _I32),
        "hg_blocks_input_nodes": ([_P, _I32, _PI64, _PP], _I32),
        "hg_gather_features": ([_P, _P, _I32, _P, _P], _I32),
        "hg_gather_features_multi": ([_P, _P, _P, _P, _I32, _P], _I32),
        "hg_gather_features_multi_timed": ([_P, _P, _P, _P, _I32, _P, _P, _P], _I32),
        "hg_gather_rows": ([_P, _I32, _P, _I64, _P, _P], _I32),
        "hg_gather_rows_noalloc": ([_P, _I32, _P, _I64, _P, _P], _I32),
        "hg_sample_blocks_gather": ([_P, _P, _P, _I32, _P, ctypes.c_uint64, _P, _I32, _P, _P, _P,
                                     _PP], _I32),
        "hg_blocks_features": ([_P, _I32, _PI64, _PP], _I32),
        "hg_sample_blocks_bundle": ([_P, _I32, _P, _P, _I32, _P, _P, _P, _I32, _P, _P, _P, _P],
                                    _I32),
        "hg_graph_types": ([_P, ctypes.POINTER(_I32), ctypes.POINTER(_I32)], _I32),
        "hg_pipeline_create": ([_P, _I32, _I32, _P, _I32, _PP], _I32),
        "hg_pipeline_submit": ([_P, _I32, _P, _P, _I32, _P, _P, _P, _P], _I32),
        "hg_pipeline_next": ([_P, _PP], _I32),
        "hg_pipeline_destroy": ([_P], None),
        "hg_blocks_free": ([_P], None),
        "hg_last_error": ([], ctypes.c_char_p),
        "hg_debug_philox": ([_P, ctypes.c_uint64, _I64, _P, _P], _I32),
        "hg_sample_blocks_bundle_timed": ([_P, _I32, _P, _P, _I32, _P, _P, _P, _I32, _P, _P,
                                           _P], _I32),
        "hg_blocks_counts": ([_P, _P, _P, _P], _I32),
        "hg_pipeline_submit_timed": ([_P, _I32, _P, _P, _I32, _P, _P, _P], _I32),
        "hg_bench_philox": ([ctypes.c_uint64, _I32, _I32, _I64, ctypes.c_uint32, _P, _P, _P, _P],
                            _I32),
        "hg_sample_edge_blocks": ([_P, _P, _I32, _P, ctypes.c_uint64, _P, _I32, _P, _PP], _I32),
        "hg_blocks_seeds": ([_P, _I32, _PI64, _PP], _I32),
        "hg_blocks_edge_pairs": ([_P, _I32, _PI64, _PP, _PP, _PI64, _PP], _I32),
        "hg_sample_layers": ([_P, _P, _P, _I32, _P, ctypes.c_uint64, _P, _I32, _P, _PP], _I32),
        "hg_blocks_edge_counts": ([_P, _P], _I32),
        "hg_sample_edge_blocks_bundle": ([_P, _I32, _P, _I32, _P, _P, _P, _I32, _P, _P], _I32),
        "hg_sample_layers_bundle": ([_P, _I32, _P, _P, _I32, _P, _P, _P, _I32, _P, _P], _I32),
        "hg_pipeline_submit_layers": ([_P, _I32, _P, _P, _I32, _P, _P], _I32),
        "hg_pipeline_submit_edges": ([_P, _I32, _P, _I32, _P, _P], _I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads libhg.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with "
                              "`python -m paper_2112_15345_amd.build`")
        _lib = _bind(ctypes.CDLL(path))
    return _lib


def _check(st: int):
    if st != HG_OK:
        raise HGError(st, load_library().hg_last_error().decode(errors="replace"))


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _dev_i64(x, device) -> torch.Tensor:
    t = torch.as_tensor(x, dtype=torch.int64, device=device)
    return t.contiguous()


class _DeviceArray:
    """Presents library-owned device memory through __cuda_array_interface__;
    holds a reference to the owning handle so that it outlives the view."""

    def __init__(self, ptr: int, n: int, typestr: str, owner):
        self.__cuda_array_interface__ = {"shape": (n,), "typestr": typestr,
                                         "data": (ptr, False), "version": 3,
                                         "strides": None, "stream": None}
        self._owner = owner


_TYPESTR = {torch.int64: "<i8", torch.int32: "<i4", torch.uint8: "|u1"}


def _view(ptr: int, n: int, dtype, owner, device) -> torch.Tensor:
    if n == 0 or not ptr:
        return torch.empty(0, dtype=dtype, device=device)
    return torch.as_tensor(_DeviceArray(ptr, n, _TYPESTR[dtype], owner), device=device)


class Blocks:
    """The blocks of one mini-batch; owns the library's output arrays."""

    def __init__(self, graph: "Graph", handle: ctypes.c_void_p, n_hops: int):
        self.graph = graph
        self._h = handle
        self.n_hops = n_hops
        self.device = graph.device

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.hg_blocks_free(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    def nodes(self, hop: int, ntype: int):
        """(n_dst, src_gid): src_gid[:n_dst] is the frontier of this hop."""
        nd, ns, p = _I64(), _I64(), ctypes.c_void_p()
        _check(load_library().hg_blocks_nodes(self._h, hop, ntype, ctypes.byref(nd),
                                              ctypes.byref(ns), ctypes.byref(p)))
        return nd.value, _view(p.value, ns.value, torch.int64, self, self.device)

    def edges(self, hop: int, etype: int):
        """(indptr, src_local, dst_local, eid) of one edge type in block `hop`."""
        ne = _I64()
        pi, ps, pd, pe = (ctypes.c_void_p() for _ in range(4))
        _check(load_library().hg_blocks_edges(self._h, hop, etype, ctypes.byref(ne),
                                              ctypes.byref(pi), ctypes.byref(ps),
                                              ctypes.byref(pd), ctypes.byref(pe)))
        d = self.graph.etypes[etype][1]
        n_dst = self.nodes(hop, d)[0]
        return (_view(pi.value, n_dst + 1, torch.int64, self, self.device),
                _view(ps.value, ne.value, torch.int32, self, self.device),
                _view(pd.value, ne.value, torch.int32, self, self.device),
                _view(pe.value, ne.value, torch.int64, self, self.device))

    def num_edges(self, hop: int, etype: int) -> int:
        ne = _I64()
        _check(load_library().hg_blocks_edges(self._h, hop, etype, ctypes.byref(ne),
                                              None, None, None, None))
        return ne.value

    def edge_counts(self):
        """Kept edges of every block: a list [n_hops][n_etypes] (one call)."""
        R = self.graph.R
        buf = (ctypes.c_int64 * max(self.n_hops * R, 1))()
        _check(load_library().hg_blocks_edge_counts(self._h, buf))
        return [[buf[h * R + e] for e in range(R)] for h in range(self.n_hops)]

    def counts(self):
        """(n_dst, n_src, keys): numpy int64 [n_hops, T], [n_hops, T] and
        [n_hops] (keys: the random keys the sampler evaluated per hop; a
        bundle's handles hold the bundle's totals)."""
        import numpy as np
        H, T = self.n_hops, self.graph.T
        nd = np.zeros(max(H * T, 1), np.int64)
        ns = np.zeros(max(H * T, 1), np.int64)
        ky = np.zeros(max(H, 1), np.int64)
        _check(load_library().hg_blocks_counts(self._h, nd.ctypes.data, ns.ctypes.data,
                                               ky.ctypes.data))
        return nd[:H * T].reshape(H, T), ns[:H * T].reshape(H, T), ky[:H]

    def total_edges(self) -> int:
        """Kept edges over every hop and edge type."""
        return sum(sum(row) for row in self.edge_counts())

    def input_nodes(self, ntype: int) -> torch.Tensor:
        n, p = _I64(), ctypes.c_void_p()
        _check(load_library().hg_blocks_input_nodes(self._h, ntype, ctypes.byref(n),
                                                    ctypes.byref(p)))
        return _view(p.value, n.value, torch.int64, self, self.device)

    def features(self, ntype: int):
        """Rows gathered for `ntype` by sample_blocks(..., gather=...): a
        [rows, dim] tensor of the type's dtype (a view of library memory), or
        None when the type was not gathered."""
        rows, p = _I64(), ctypes.c_void_p()
        _check(load_library().hg_blocks_features(self._h, ntype, ctypes.byref(rows),
                                                 ctypes.byref(p)))
        if not p.value:
            return None
        feat = self.graph.ntypes[ntype][1]
        dim = feat.shape[1]
        nbytes = rows.value * dim * feat.element_size()
        return _view(p.value, nbytes, torch.uint8, self, self.device).view(feat.dtype).view(
            rows.value, dim)

    def num_input_nodes(self, ntype: int) -> int:
        n = _I64()
        _check(load_library().hg_blocks_input_nodes(self._h, ntype, ctypes.byref(n), None))
        return n.value

    def seeds(self, ntype: int) -> torch.Tensor:
        """The seeds of `ntype`: an edge-seeded batch's endpoints in ascending
        ID, or the given seeds of a vertex-seeded one."""
        n, p = _I64(), ctypes.c_void_p()
        _check(load_library().hg_blocks_seeds(self._h, ntype, ctypes.byref(n), ctypes.byref(p)))
        return _view(p.value, n.value, torch.int64, self, self.device)

    def edge_pairs(self, etype: int):
        """(pos_src, pos_dst, neg_dst) of an edge-seeded batch: local IDs among
        the seeds; negative i * n_neg + k has source pos_src[i]."""
        npos, nneg = _I64(), _I64()
        ps, pd, pn = (ctypes.c_void_p() for _ in range(3))
        _check(load_library().hg_blocks_edge_pairs(self._h, etype, ctypes.byref(npos),
                                                   ctypes.byref(ps), ctypes.byref(pd),
                                                   ctypes.byref(nneg), ctypes.byref(pn)))
        return (_view(ps.value, npos.value, torch.int32, self, self.device),
                _view(pd.value, npos.value, torch.int32, self, self.device),
                _view(pn.value, nneg.value, torch.int32, self, self.device))


class Graph:
    """An immutable heterograph over borrowed device tensors.

    ntypes: [(num_nodes, feat)] with feat a contiguous [num_nodes, dim] float32 /
    float16 / bfloat16 device tensor or None.  etypes: [(src_type, dst_type,
    indptr, indices)] with int64 device tensors (CSC keyed by destination)."""

    def __init__(self, ntypes, etypes, device=None, allocator: Allocator | None = None,
                 stream=None):
        lib = load_library()
        self.device = torch.device(device or "cuda")
        self.ntypes = []
        self.etypes = []
        nt = (NTypeDesc * max(len(ntypes), 1))()
        et = (ETypeDesc * max(len(etypes), 1))()
        for t, (n, feat) in enumerate(ntypes):
            if feat is not None:
                if not feat.is_contiguous() or feat.dim() != 2 or feat.shape[0] != n:
                    raise ValueError(f"node type {t}: features must be contiguous [n, dim]")
                if feat.dtype not in _DTYPE_CODE:
                    raise ValueError(f"node type {t}: unsupported dtype {feat.dtype}")
                nt[t] = NTypeDesc(int(n), feat.data_ptr() if feat.numel() else None,
                                  _DTYPE_CODE[feat.dtype], int(feat.shape[1]))
            else:
                nt[t] = NTypeDesc(int(n), None, HG_DT_NONE, 0)
            self.ntypes.append((int(n), feat))
        for e, (s, d, indptr, indices) in enumerate(etypes):
            indptr = _dev_i64(indptr, self.device)
            indices = _dev_i64(indices, self.device)
            et[e] = ETypeDesc(int(s), int(d), int(indices.numel()), indptr.data_ptr(),
                              indices.data_ptr() if indices.numel() else None)
            self.etypes.append((int(s), int(d), indptr, indices))
        self._allocator = allocator
        h = ctypes.c_void_p()
        _check(lib.hg_create(ctypes.addressof(nt), len(ntypes), ctypes.addressof(et),
                             len(etypes),
                             ctypes.addressof(allocator) if allocator is not None else None,
                             _stream(stream), ctypes.byref(h)))
        self._h = h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.hg_destroy(h)
            self._h = None

    @property
    def T(self) -> int:
        return len(self.ntypes)

    @property
    def R(self) -> int:
        return len(self.etypes)

    def sample_blocks(self, seeds, fanouts, rng_seed: int = 0, key_bits: int = 32,
                      stream=None, gather=None, events=None) -> Blocks:
        """seeds: per node type an int64 device tensor or None; fanouts:
        [n_hops][n_etypes] (hop 0 starts from the seeds; -1 = all).
        gather: None, "all" (every featured type) or a list of node types whose
        input-frontier rows the same call gathers (Blocks.features); events:
        optional (start, stop) raw hipEvent_t handles carried by that gather."""
        lib = load_library()
        T, R = self.T, self.R
        if len(seeds) != T:
            raise ValueError("one seed entry per node type")
        keep = []
        ptrs = (ctypes.c_void_p * T)()
        counts = (ctypes.c_int64 * T)()
        for t, s in enumerate(seeds):
            if s is None:
                counts[t] = 0
                continue
            s = _dev_i64(s, self.device)
            keep.append(s)
            counts[t] = s.numel()
            ptrs[t] = s.data_ptr() if s.numel() else None
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        h = ctypes.c_void_p()
        if gather is None:
            _check(lib.hg_sample_blocks_ex(self._h, ptrs, counts, H, fo,
                                           int(rng_seed) & (2**64 - 1), int(key_bits),
                                           _stream(stream), ctypes.byref(h)))
            return Blocks(self, h, H)
        if key_bits != 32:
            raise ValueError("gather=... samples with full 32-bit keys")
        if isinstance(gather, str):
            if gather != "all":
                raise ValueError('gather must be None, "all" or a list of node types')
            gather = [t for t, (_, f) in enumerate(self.ntypes) if f is not None]
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        start, stop = events if events is not None else (None, None)
        _check(lib.hg_sample_blocks_gather(self._h, ptrs, counts, H, fo,
                                           int(rng_seed) & (2**64 - 1), gt, len(gather),
                                           start, stop, _stream(stream), ctypes.byref(h)))
        return Blocks(self, h, H)

    def sample_bundle(self, seeds_list, fanouts, rng_seeds, gather="all", events=None,
                      stream=None, stage_events=None):
        """Several mini-batches in one launch sequence (hg_sample_blocks_bundle):
        seeds_list[b] per node type as in sample_blocks, rng_seeds[b]; returns
        one Blocks per batch (with gathered features for `gather`)."""
        lib = load_library()
        T, R = self.T, self.R
        B = len(seeds_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per batch")
        keep = []
        ptrs = (ctypes.c_void_p * max(B * T, 1))()
        counts = (ctypes.c_int64 * max(B * T, 1))()
        for b, seeds in enumerate(seeds_list):
            if len(seeds) != T:
                raise ValueError("one seed entry per node type")
            for t, sd in enumerate(seeds):
                if sd is None:
                    continue
                sd = _dev_i64(sd, self.device)
                keep.append(sd)
                counts[b * T + t] = sd.numel()
                ptrs[b * T + t] = sd.data_ptr() if sd.numel() else None
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(x) & (2**64 - 1) for x in rng_seeds])
        if isinstance(gather, str):
            if gather != "all":
                raise ValueError('gather must be "all" or a list of node types')
            gather = [t for t, (_, f) in enumerate(self.ntypes) if f is not None]
        gather = list(gather or [])
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        start, stop = events if events is not None else (None, None)
        hs = (ctypes.c_void_p * max(B, 1))()
        if stage_events is not None:
            _check(lib.hg_sample_blocks_bundle_timed(self._h, B, ptrs, counts, H, fo, sg, gt,
                                                     len(gather),
                                                     ctypes.addressof(stage_events.struct),
                                                     _stream(stream), hs))
        else:
            _check(lib.hg_sample_blocks_bundle(self._h, B, ptrs, counts, H, fo, sg, gt,
                                               len(gather), start, stop, _stream(stream), hs))
        return [Blocks(self, ctypes.c_void_p(hs[b]), H) for b in range(B)]

    def sample_layers(self, seeds, layer_sizes, rng_seed: int = 0, gather=None,
                      stream=None) -> Blocks:
        """A layer-wise (LADIES) mini-batch (hg_sample_layers): seeds per node
        type as in sample_blocks; layer_sizes [n_hops][n_ntypes], the draws of
        each node type per hop (-1 = every candidate).  gather as in
        sample_blocks."""
        lib = load_library()
        T = self.T
        if len(seeds) != T:
            raise ValueError("one seed entry per node type")
        keep = []
        ptrs = (ctypes.c_void_p * T)()
        counts = (ctypes.c_int64 * T)()
        for t, s in enumerate(seeds):
            if s is None:
                continue
            s = _dev_i64(s, self.device)
            keep.append(s)
            counts[t] = s.numel()
            ptrs[t] = s.data_ptr() if s.numel() else None
        H = len(layer_sizes)
        flat = [int(k) for row in layer_sizes for k in row]
        if len(flat) != H * T:
            raise ValueError("layer_sizes must be [n_hops][n_ntypes]")
        ls = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        if isinstance(gather, str):
            if gather != "all":
                raise ValueError('gather must be None, "all" or a list of node types')
            gather = [t for t, (_, f) in enumerate(self.ntypes) if f is not None]
        gather = list(gather or [])
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        h = ctypes.c_void_p()
        st = lib.hg_sample_layers(self._h, ptrs, counts, H, ls, int(rng_seed) & (2**64 - 1), gt,
                                  len(gather), _stream(stream), ctypes.byref(h))
        del keep
        _check(st)
        return Blocks(self, h, H)

    def _edge_batch(self, targets, n_neg, exclude, rev_etype, rev_eid, keep):
        """An EdgeBatch over ctypes arrays that `keep` holds alive."""
        R = self.R
        if len(targets) != R:
            raise ValueError("one target entry per edge type")
        tptr = (ctypes.c_void_p * max(R, 1))()
        tcnt = (ctypes.c_int64 * max(R, 1))()
        for e, x in enumerate(targets):
            if x is None:
                continue
            x = _dev_i64(x, self.device)
            keep.append(x)
            tcnt[e] = x.numel()
            tptr[e] = x.data_ptr() if x.numel() else None
        rv = None
        rptr = None
        if rev_etype is not None:
            rv = (ctypes.c_int32 * max(R, 1))(*[int(r) for r in rev_etype])
        if rev_eid is not None:
            rptr = (ctypes.c_void_p * max(R, 1))()
            for e, x in enumerate(rev_eid):
                if x is None:
                    continue
                x = _dev_i64(x, self.device)
                keep.append(x)
                rptr[e] = x.data_ptr() if x.numel() else None
        keep.extend([tptr, tcnt, rv, rptr])
        return EdgeBatch(ctypes.addressof(tptr), ctypes.addressof(tcnt), int(n_neg),
                         int(exclude), ctypes.addressof(rv) if rv is not None else None,
                         ctypes.addressof(rptr) if rptr is not None else None)

    def _gather_list(self, gather):
        if isinstance(gather, str):
            if gather != "all":
                raise ValueError('gather must be None, "all" or a list of node types')
            gather = [t for t, (_, f) in enumerate(self.ntypes) if f is not None]
        return list(gather or [])

    def sample_layers_bundle(self, seeds_list, layer_sizes, rng_seeds, gather=None,
                             stream=None):
        """Several layer-wise mini-batches in one launch sequence
        (hg_sample_layers_bundle): seeds_list[b] per node type as in
        sample_layers, rng_seeds[b]; the same layer_sizes for all.  Returns one
        Blocks per batch."""
        lib = load_library()
        T = self.T
        B = len(seeds_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per batch")
        keep = []
        ptrs = (ctypes.c_void_p * max(B * T, 1))()
        counts = (ctypes.c_int64 * max(B * T, 1))()
        for b, seeds in enumerate(seeds_list):
            if len(seeds) != T:
                raise ValueError("one seed entry per node type")
            for t, s in enumerate(seeds):
                if s is None:
                    continue
                s = _dev_i64(s, self.device)
                keep.append(s)
                counts[b * T + t] = s.numel()
                ptrs[b * T + t] = s.data_ptr() if s.numel() else None
        H = len(layer_sizes)
        flat = [int(k) for row in layer_sizes for k in row]
        if len(flat) != H * T:
            raise ValueError("layer_sizes must be [n_hops][n_ntypes]")
        ls = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(s) & (2**64 - 1) for s in rng_seeds])
        gather = self._gather_list(gather)
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        hs = (ctypes.c_void_p * max(B, 1))()
        st = lib.hg_sample_layers_bundle(self._h, B, ptrs, counts, H, ls, sg, gt, len(gather),
                                         _stream(stream), hs)
        del keep
        _check(st)
        return [Blocks(self, ctypes.c_void_p(hs[b]), H) for b in range(B)]

    def sample_edge_blocks(self, targets, fanouts, rng_seed: int = 0, n_neg: int = 0,
                           exclude: int = HG_EXCLUDE_NONE, rev_etype=None, rev_eid=None,
                           gather=None, stream=None) -> Blocks:
        """An edge-seeded mini-batch (link prediction): targets per edge type an
        int64 device tensor of edge IDs or None; n_neg negatives per target;
        exclude HG_EXCLUDE_NONE / _SELF / _REVERSE, the last with rev_etype
        (per edge type its reverse type or -1) and rev_eid (per edge type an
        int64 device tensor [nnz] or None).  gather as in sample_blocks."""
        lib = load_library()
        R = self.R
        keep = []
        batch = self._edge_batch(targets, n_neg, exclude, rev_etype, rev_eid, keep)
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        gather = self._gather_list(gather)
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        h = ctypes.c_void_p()
        st = lib.hg_sample_edge_blocks(self._h, ctypes.addressof(batch), H, fo,
                                       int(rng_seed) & (2**64 - 1), gt, len(gather),
                                       _stream(stream), ctypes.byref(h))
        # the call waits on the stream before it returns, so the target
        # tensors are read by then
        del keep
        _check(st)
        return Blocks(self, h, H)

    def sample_edge_bundle(self, targets_list, fanouts, rng_seeds, n_neg: int = 0,
                           exclude: int = HG_EXCLUDE_NONE, rev_etype=None, rev_eid=None,
                           gather=None, stream=None):
        """Several edge-seeded mini-batches in one launch sequence
        (hg_sample_edge_blocks_bundle): targets_list[b] per edge type as in
        sample_edge_blocks, rng_seeds[b]; the same n_neg, exclusion and reverse
        maps for all.  Returns one Blocks per batch."""
        lib = load_library()
        R = self.R
        B = len(targets_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per batch")
        keep = []
        batches = (EdgeBatch * max(B, 1))()
        for b, targets in enumerate(targets_list):
            batches[b] = self._edge_batch(targets, n_neg, exclude, rev_etype, rev_eid, keep)
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(s) & (2**64 - 1) for s in rng_seeds])
        gather = self._gather_list(gather)
        gt = (ctypes.c_int32 * max(len(gather), 1))(*[int(t) for t in gather])
        hs = (ctypes.c_void_p * max(B, 1))()
        st = lib.hg_sample_edge_blocks_bundle(self._h, B, batches, H, fo, sg, gt, len(gather),
                                              _stream(stream), hs)
        del keep
        _check(st)
        return [Blocks(self, ctypes.c_void_p(hs[b]), H) for b in range(B)]

    def gather_features(self, blocks: Blocks, ntype: int, out: torch.Tensor | None = None,
                        stream=None) -> torch.Tensor:
        n, feat = self.ntypes[ntype]
        if feat is None:
            raise HGError(HG_EINVAL, f"node type {ntype} has no features")
        rows = blocks.num_input_nodes(ntype)
        if out is None:
            out = torch.empty((rows, feat.shape[1]), dtype=feat.dtype, device=self.device)
        _check(load_library().hg_gather_features(self._h, blocks.handle, ntype,
                                                 out.data_ptr() if out.numel() else None,
                                                 _stream(stream)))
        return out

    def gather_outputs(self, blocks: Blocks, ntypes=None):
        """Empty output tensors for gather_features_all: {ntype: [rows, dim]}."""
        if ntypes is None:
            ntypes = [t for t, (_, f) in enumerate(self.ntypes) if f is not None]
        outs = {}
        for t in ntypes:
            feat = self.ntypes[t][1]
            if feat is None:
                raise HGError(HG_EINVAL, f"node type {t} has no features")
            outs[t] = torch.empty((blocks.num_input_nodes(t), feat.shape[1]), dtype=feat.dtype,
                                  device=self.device)
        return outs

    def gather_features_all(self, blocks: Blocks, ntypes=None, outs=None, stream=None,
                            events=None):
        """Input-frontier rows of every featured node type (or of `ntypes`), in
        as few launches as possible, into `outs` (made by gather_outputs when
        not given).  `events`: optional (start, stop) raw hipEvent_t handles
        that the gather kernels record themselves.  Returns {ntype: tensor}."""
        if outs is None:
            outs = self.gather_outputs(blocks, ntypes)
        ts_list = list(outs.keys())
        n = len(ts_list)
        ts = (ctypes.c_int32 * max(n, 1))(*ts_list)
        ps = (ctypes.c_void_p * max(n, 1))(
            *[outs[t].data_ptr() if outs[t].numel() else None for t in ts_list])
        start, stop = events if events is not None else (None, None)
        _check(load_library().hg_gather_features_multi_timed(self._h, blocks.handle, ts, ps, n,
                                                             _stream(stream), start, stop))
        return outs

    def gather_rows_noalloc(self, ntype: int, ids: torch.Tensor, out: torch.Tensor,
                            stream=None) -> torch.Tensor:
        """hg_gather_rows_noalloc: the same pull with no device allocation (its
        counter lives in the library's static scratch); `out` is required."""
        ids = _dev_i64(ids, self.device)
        _check(load_library().hg_gather_rows_noalloc(self._h, ntype,
                                                     ids.data_ptr() if ids.numel() else None,
                                                     ids.numel(),
                                                     out.data_ptr() if out.numel() else None,
                                                     _stream(stream)))
        return out

    def gather_rows(self, ntype: int, ids: torch.Tensor, out: torch.Tensor | None = None,
                    stream=None) -> torch.Tensor:
        n, feat = self.ntypes[ntype]
        ids = _dev_i64(ids, self.device)
        if out is None:
            if feat is None:
                raise HGError(HG_EINVAL, f"node type {ntype} has no features")
            out = torch.empty((ids.numel(), feat.shape[1]), dtype=feat.dtype, device=self.device)
        _check(load_library().hg_gather_rows(self._h, ntype,
                                             ids.data_ptr() if ids.numel() else None,
                                             ids.numel(),
                                             out.data_ptr() if out.numel() else None,
                                             _stream(stream)))
        return out


class Pipeline:
    """Mini-batches generated ahead of use (hg_pipeline_*): `workers` host
    threads with their own streams run submitted mini-batches concurrently;
    next() returns them in submission order, complete on the device.  At most
    `capacity` are outstanding (submit waits).  gather: node types whose input
    features every mini-batch gathers ("all": every featured type)."""

    def __init__(self, graph: Graph, workers: int = 2, capacity: int = 4, gather="all"):
        self.graph = graph
        if isinstance(gather, str):
            if gather != "all":
                raise ValueError('gather must be "all" or a list of node types')
            gather = [t for t, (_, f) in enumerate(graph.ntypes) if f is not None]
        gather = [int(t) for t in (gather or [])]
        gt = (ctypes.c_int32 * max(len(gather), 1))(*gather)
        h = ctypes.c_void_p()
        _check(load_library().hg_pipeline_create(graph._h, int(workers), int(capacity), gt,
                                                 len(gather), ctypes.byref(h)))
        self._h = h
        self._held = collections.deque()  # seed tensors of outstanding mini-batches

    def submit(self, seeds, fanouts, rng_seed: int = 0, events=None):
        """Queues one mini-batch (seeds per node type, as in Graph.sample_blocks)."""
        self.submit_bundle([seeds], fanouts, [rng_seed], events)

    def submit_bundle(self, seeds_list, fanouts, rng_seeds, events=None, stage_events=None):
        """Queues len(seeds_list) mini-batches sampled together as one bundle
        (Graph.sample_bundle); next() returns them one by one, in order."""
        g = self.graph
        T, R = g.T, g.R
        B = len(seeds_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per mini-batch")
        keep = []
        ptrs = (ctypes.c_void_p * max(B * T, 1))()
        counts = (ctypes.c_int64 * max(B * T, 1))()
        for b, seeds in enumerate(seeds_list):
            if len(seeds) != T:
                raise ValueError("one seed entry per node type")
            for t, sd in enumerate(seeds):
                if sd is None:
                    continue
                sd = _dev_i64(sd, g.device)
                keep.append(sd)
                counts[b * T + t] = sd.numel()
                ptrs[b * T + t] = sd.data_ptr() if sd.numel() else None
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(x) & (2**64 - 1) for x in rng_seeds])
        start, stop = events if events is not None else (None, None)
        if stage_events is not None:
            _check(load_library().hg_pipeline_submit_timed(
                self._h, B, ptrs, counts, H, fo, sg, ctypes.addressof(stage_events.struct)))
        else:
            _check(load_library().hg_pipeline_submit(self._h, B, ptrs, counts, H, fo, sg, start,
                                                     stop))
        for _ in range(B):
            self._held.append(keep)

    def submit_layers_bundle(self, seeds_list, layer_sizes, rng_seeds):
        """Queues len(seeds_list) layer-wise mini-batches made as one bundle
        (Graph.sample_layers_bundle, hg_pipeline_submit_layers); next()
        returns them one by one, in order."""
        g = self.graph
        T = g.T
        B = len(seeds_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per mini-batch")
        keep = []
        ptrs = (ctypes.c_void_p * max(B * T, 1))()
        counts = (ctypes.c_int64 * max(B * T, 1))()
        for b, seeds in enumerate(seeds_list):
            if len(seeds) != T:
                raise ValueError("one seed entry per node type")
            for t, sd in enumerate(seeds):
                if sd is None:
                    continue
                sd = _dev_i64(sd, g.device)
                keep.append(sd)
                counts[b * T + t] = sd.numel()
                ptrs[b * T + t] = sd.data_ptr() if sd.numel() else None
        H = len(layer_sizes)
        flat = [int(k) for row in layer_sizes for k in row]
        if len(flat) != H * T:
            raise ValueError("layer_sizes must be [n_hops][n_ntypes]")
        ls = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(x) & (2**64 - 1) for x in rng_seeds])
        _check(load_library().hg_pipeline_submit_layers(self._h, B, ptrs, counts, H, ls, sg))
        for _ in range(B):
            self._held.append(keep)

    def submit_edge_bundle(self, targets_list, fanouts, rng_seeds, n_neg: int = 0,
                           exclude: int = HG_EXCLUDE_NONE, rev_etype=None, rev_eid=None):
        """Queues len(targets_list) edge-seeded mini-batches made as one bundle
        (Graph.sample_edge_bundle, hg_pipeline_submit_edges); next() returns
        them one by one, in order."""
        g = self.graph
        R = g.R
        B = len(targets_list)
        if len(rng_seeds) != B:
            raise ValueError("one rng seed per mini-batch")
        keep = []
        batches = (EdgeBatch * max(B, 1))()
        for b, targets in enumerate(targets_list):
            batches[b] = g._edge_batch(targets, n_neg, exclude, rev_etype, rev_eid, keep)
        H = len(fanouts)
        flat = [int(k) for row in fanouts for k in row]
        if len(flat) != H * R:
            raise ValueError("fanouts must be [n_hops][n_etypes]")
        fo = (ctypes.c_int32 * max(len(flat), 1))(*flat)
        sg = (ctypes.c_uint64 * max(B, 1))(*[int(x) & (2**64 - 1) for x in rng_seeds])
        _check(load_library().hg_pipeline_submit_edges(self._h, B, batches, H, fo, sg))
        for _ in range(B):
            self._held.append(keep)

    def next(self) -> Blocks:
        if not self._held:
            raise HGError(HG_EINVAL, "no mini-batch outstanding")
        h = ctypes.c_void_p()
        st = load_library().hg_pipeline_next(self._h, ctypes.byref(h))
        self._held.popleft()  # the oldest mini-batch is returned, or its error
        _check(st)
        return Blocks(self.graph, h, load_library().hg_blocks_num_hops(h))

    def close(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.hg_pipeline_destroy(h)
            self._h = None
            self._held.clear()

    def __del__(self):
        self.close()


class HipEvents:
    """Raw HIP timing events (hipEvent_t) from the HIP runtime, for
    gather_features_all(events=...)."""

    def __init__(self, n: int):
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self._hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float),
                                                  ctypes.c_void_p, ctypes.c_void_p]
        self._hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self._hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.events = []
        for _ in range(n):
            e = ctypes.c_void_p()
            if self._hip.hipEventCreate(ctypes.byref(e)) != 0:
                raise HGError(HG_EDEVICE, "hipEventCreate failed")
            self.events.append(e.value)

    def elapsed_ms(self, start: int, stop: int) -> float:
        ms = ctypes.c_float()
        self._hip.hipEventSynchronize(stop)
        if self._hip.hipEventElapsedTime(ctypes.byref(ms), start, stop) != 0:
            raise HGError(HG_EDEVICE, "hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        for e in getattr(self, "events", []):
            self._hip.hipEventDestroy(e)


class StageEvents:
    """Timing events for the stages of up to n_hops hops and the gather of one
    call (hg_stage_events), created through the HIP runtime; durations in ms.
    stages: the names (STAGE_NAMES) that get events, default all; gather:
    whether the gather gets them.  A stage without events is not timed (its
    launches stay plain) and reports None."""

    def __init__(self, n_hops: int, stages=STAGE_NAMES, gather: bool = True):
        if n_hops > HG_MAX_TIMED_HOPS:
            raise ValueError(f"at most {HG_MAX_TIMED_HOPS} timed hops")
        self.n_hops = n_hops
        self.stages = tuple(stages)
        self.gather = gather
        n = 2 * n_hops * len(self.stages) + (2 if gather else 0)
        self._ev = HipEvents(n)
        self.struct = StageEventsStruct()
        k = 0
        for h in range(n_hops):
            for st, name in enumerate(STAGE_NAMES):
                if name in self.stages:
                    self.struct.start[h][st] = self._ev.events[k]
                    self.struct.stop[h][st] = self._ev.events[k + 1]
                    k += 2
        if gather:
            self.struct.gather_start = self._ev.events[k]
            self.struct.gather_stop = self._ev.events[k + 1]

    def stage_ms(self, hop: int, stage: int):
        if STAGE_NAMES[stage] not in self.stages:
            return None
        return self._ev.elapsed_ms(self.struct.start[hop][stage], self.struct.stop[hop][stage])

    def gather_ms(self):
        if not self.gather:
            return None
        return self._ev.elapsed_ms(self.struct.gather_start, self.struct.gather_stop)


def debug_philox(ctr: torch.Tensor, key: int, stream=None) -> torch.Tensor:
    """Philox4x32-10 of each row of a [n, 4] counter tensor (int32 bits)."""
    ctr = ctr.contiguous()
    out = torch.empty_like(ctr)
    _check(load_library().hg_debug_philox(ctr.data_ptr() if ctr.numel() else None,
                                          int(key) & (2**64 - 1), ctr.shape[0],
                                          out.data_ptr() if out.numel() else None,
                                          _stream(stream)))
    return out


def bench_philox(rng_seed: int, hop: int, etype: int, n_groups: int, lim: int,
                 events=None, stream=None) -> torch.Tensor:
    """The sampler's key loop alone (hg_bench_philox): the number of keys <=
    lim among the keys of edge IDs 0 .. 4 * n_groups - 1 of (rng_seed, hop,
    etype), as a one-element int64 device tensor.  events: optional (start,
    stop) raw hipEvent_t handles carried by the launch."""
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    start, stop = events if events is not None else (None, None)
    _check(load_library().hg_bench_philox(int(rng_seed) & (2**64 - 1), int(hop), int(etype),
                                          int(n_groups), int(lim) & 0xFFFFFFFF,
                                          count.data_ptr(), start, stop, _stream(stream)))
    return count
