"""Test infrastructure only: ctypes access to the plain C oracle (oracle.c).

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  It shares no code with the GPU library
(``paper_2112_15345_amd``); both follow the written definition of DistDGLv2's
mini-batch generation (arXiv 2112.15345, Sec. 3.2 and Sec. 4.2.2).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# The same source built with OpenMP: independent loops (the pairs of a hop,
# the relabelled edges, the gathered rows) run on every host core.
_LIB_OMP = os.path.join(_HERE, "liboracle_omp.so")

OK, EINVAL, ENOMEM, EUNSUPPORTED = 0, -1, -2, -4


def build(out: str = _LIB, extra_flags=(), src: str = _SRC) -> str:
    """Compile oracle.c with gcc into a shared library (plain C11, -O2); with
    the default output also its OpenMP build (liboracle_omp.so)."""
    tmp = f"{out}.{os.getpid()}.tmp"  # concurrent builders never share a file
    cmd = ["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-Wall", "-Wextra",
           "-Wno-unknown-pragmas", "-I", _HERE, *extra_flags, src, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    if out == _LIB and not extra_flags and src == _SRC:
        build(_LIB_OMP, extra_flags=("-fopenmp",))
    return out


class _NType(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int64), ("feat", ctypes.c_void_p),
                ("row_bytes", ctypes.c_int64)]


class _EType(ctypes.Structure):
    _fields_ = [("src_type", ctypes.c_int32), ("dst_type", ctypes.c_int32),
                ("nnz", ctypes.c_int64), ("indptr", ctypes.c_void_p),
                ("indices", ctypes.c_void_p)]


_P = ctypes.c_void_p
_I64P = ctypes.POINTER(ctypes.c_int64)


def _bind(lib):
    lib.oracle_philox4x32_10.argtypes = [_P, _P, _P]
    lib.oracle_philox4x32_10.restype = None
    lib.oracle_edge_key.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int64, ctypes.c_int32]
    lib.oracle_edge_key.restype = ctypes.c_uint32
    lib.oracle_select.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_int32, _P, _I64P]
    lib.oracle_select.restype = ctypes.c_int
    lib.oracle_check_graph.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_int32]
    lib.oracle_check_graph.restype = ctypes.c_int
    lib.oracle_sample_blocks.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_int32, _P, _P,
                                         ctypes.c_int32, _P, ctypes.c_uint64,
                                         ctypes.c_int32, ctypes.POINTER(_P)]
    lib.oracle_sample_blocks.restype = ctypes.c_int
    lib.oracle_blocks_free.argtypes = [_P]
    lib.oracle_blocks_free.restype = None
    lib.oracle_blocks_nodes.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, _I64P, _I64P,
                                        ctypes.POINTER(_P)]
    lib.oracle_blocks_nodes.restype = ctypes.c_int
    lib.oracle_blocks_edges.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, _I64P,
                                        ctypes.POINTER(_P), ctypes.POINTER(_P),
                                        ctypes.POINTER(_P), ctypes.POINTER(_P)]
    lib.oracle_blocks_edges.restype = ctypes.c_int
    lib.oracle_blocks_input_nodes.argtypes = [_P, ctypes.c_int32, _I64P, ctypes.POINTER(_P)]
    lib.oracle_blocks_input_nodes.restype = ctypes.c_int
    lib.oracle_gather_rows.argtypes = [_P, ctypes.c_int64, ctypes.c_int64, _P,
                                       ctypes.c_int64, _P]
    lib.oracle_gather_rows.restype = ctypes.c_int
    lib.oracle_edge_dst.argtypes = [_P, ctypes.c_int64, ctypes.c_int64, _I64P]
    lib.oracle_edge_dst.restype = ctypes.c_int
    lib.oracle_negative_dst.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64,
                                        ctypes.c_int32, ctypes.c_int64, _I64P]
    lib.oracle_negative_dst.restype = ctypes.c_int
    lib.oracle_sample_edge_blocks.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_int32, _P,
                                              ctypes.c_int32, _P, ctypes.c_uint64,
                                              ctypes.c_int32, ctypes.POINTER(_P)]
    lib.oracle_sample_edge_blocks.restype = ctypes.c_int
    lib.oracle_blocks_seeds.argtypes = [_P, ctypes.c_int32, _I64P, ctypes.POINTER(_P)]
    lib.oracle_blocks_seeds.restype = ctypes.c_int
    lib.oracle_blocks_pairs.argtypes = [_P, ctypes.c_int32, _I64P, ctypes.POINTER(_P),
                                        ctypes.POINTER(_P), _I64P, ctypes.POINTER(_P)]
    lib.oracle_blocks_pairs.restype = ctypes.c_int
    lib.oracle_layer_weight.argtypes = [ctypes.c_int64]
    lib.oracle_layer_weight.restype = ctypes.c_uint64
    lib.oracle_layer_draw.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_uint64]
    lib.oracle_layer_draw.restype = ctypes.c_uint64
    lib.oracle_sample_layers.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_int32, _P, _P,
                                         ctypes.c_int32, _P, ctypes.c_uint64, ctypes.POINTER(_P)]
    lib.oracle_sample_layers.restype = ctypes.c_int
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = ctypes.c_int
    return lib


_lib_cache: dict[str, ctypes.CDLL] = {}


def load(path: str = _LIB) -> ctypes.CDLL:
    """Load (building first if absent) the oracle library at ``path``."""
    if path not in _lib_cache:
        if not os.path.exists(path):
            build(path, extra_flags=("-fopenmp",) if path == _LIB_OMP else ())
        _lib_cache[path] = _bind(ctypes.CDLL(path))
    return _lib_cache[path]


def load_omp() -> ctypes.CDLL:
    """The OpenMP build of the same source (every host core; same results)."""
    return load(_LIB_OMP)


def threads(lib=None) -> int:
    """Threads the library's parallel loops use (1 for the plain build)."""
    return int((lib or load()).oracle_threads())


def _ptr(a: np.ndarray | None) -> int | None:
    return None if a is None else a.ctypes.data


def _arr_i64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int64))


def philox4x32_10(ctr, key, lib=None) -> np.ndarray:
    lib = lib or load()
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib.oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def edge_key(sigma: int, hop: int, etype: int, eid: int, key_bits: int = 32, lib=None) -> int:
    lib = lib or load()
    return int(lib.oracle_edge_key(sigma, hop, etype, eid, key_bits))


def select(sigma, hop, etype, lo, hi, fanout, key_bits=32, lib=None):
    """Chosen edge IDs of one (destination, etype) pair with slots lo..hi-1."""
    lib = lib or load()
    out = np.zeros(max(hi - lo, 1), dtype=np.int64)
    n = ctypes.c_int64(0)
    st = lib.oracle_select(sigma, hop, etype, lo, hi, fanout, key_bits, _ptr(out),
                           ctypes.byref(n))
    if st != OK:
        raise OracleError(st)
    return out[: n.value].copy()


def edge_dst(indptr, eid, lib=None) -> int:
    """The destination vertex of CSC slot `eid`."""
    lib = lib or load()
    ip = _arr_i64(indptr)
    v = ctypes.c_int64(0)
    st = lib.oracle_edge_dst(_ptr(ip), ip.size - 1, eid, ctypes.byref(v))
    if st != OK:
        raise OracleError(st)
    return v.value


def negative_dst(sigma, etype, eid, k, n_dst, lib=None) -> int:
    """Negative destination k of target edge `eid` of `etype`."""
    lib = lib or load()
    v = ctypes.c_int64(0)
    st = lib.oracle_negative_dst(sigma, etype, eid, k, n_dst, ctypes.byref(v))
    if st != OK:
        raise OracleError(st)
    return v.value


def layer_weight(deg, lib=None) -> int:
    """One edge's share of its source's importance: floor(2^32 / deg^2)."""
    lib = lib or load()
    return int(lib.oracle_layer_weight(deg))


def layer_draw(sigma, hop, ntype, k, total, lib=None) -> int:
    """Draw k of a hop and node type: a point in [0, total)."""
    lib = lib or load()
    return int(lib.oracle_layer_draw(sigma, hop, ntype, k, total))


MAX_NEG = 64
EXCLUDE_NONE, EXCLUDE_SELF, EXCLUDE_REVERSE = 0, 1, 2


class _EdgeBatch(ctypes.Structure):
    _fields_ = [("eids", ctypes.c_void_p), ("n_eids", ctypes.c_void_p),
                ("n_neg", ctypes.c_int32), ("exclude", ctypes.c_int32),
                ("rev_etype", ctypes.c_void_p), ("rev_eid", ctypes.c_void_p)]


class OracleError(RuntimeError):
    def __init__(self, status: int):
        super().__init__(f"oracle status {status}")
        self.status = status


class HostGraph:
    """A heterograph in host memory, as numpy arrays, for the oracle.

    ntypes: list of (num_nodes, feat ndarray [num_nodes, ...] or None)
    etypes: list of (src_type, dst_type, indptr int64, indices int64)
    """

    def __init__(self, ntypes, etypes, lib=None, check=True):
        self.lib = lib or load()
        self.ntypes = []
        self.etypes = []
        self._nt = (_NType * max(len(ntypes), 1))()
        self._et = (_EType * max(len(etypes), 1))()
        for t, (n, feat) in enumerate(ntypes):
            if feat is not None:
                feat = np.ascontiguousarray(feat)
                row_bytes = feat.nbytes // max(int(n), 1) if n > 0 else feat.strides[0]
            else:
                row_bytes = 0
            self.ntypes.append((int(n), feat, int(row_bytes)))
            self._nt[t] = _NType(int(n), _ptr(feat) if feat is not None else None, int(row_bytes))
        for e, (s, d, indptr, indices) in enumerate(etypes):
            indptr = _arr_i64(indptr)
            indices = _arr_i64(indices)
            self.etypes.append((int(s), int(d), indptr, indices))
            self._et[e] = _EType(int(s), int(d), int(indices.shape[0]), _ptr(indptr),
                                 _ptr(indices) if indices.shape[0] > 0 else None)
        if check:
            st = self.lib.oracle_check_graph(ctypes.addressof(self._nt), len(self.ntypes),
                                             ctypes.addressof(self._et), len(self.etypes))
            if st != OK:
                raise OracleError(st)

    @property
    def T(self):
        return len(self.ntypes)

    @property
    def R(self):
        return len(self.etypes)

    def sample_blocks(self, seeds, fanouts, sigma, key_bits=32):
        """seeds: list (per node type) of int64 arrays (or None); fanouts:
        [n_hops][n_etypes].  Returns a dict of numpy arrays (see result_dict)."""
        T, R = self.T, self.R
        seed_arrs = []
        for t in range(T):
            s = None if (seeds[t] is None) else _arr_i64(seeds[t])
            seed_arrs.append(s)
        ptrs = (ctypes.c_void_p * T)(*[(_ptr(s) if s is not None and s.size else None)
                                       for s in seed_arrs])
        ns = np.array([0 if s is None else s.size for s in seed_arrs], dtype=np.int64)
        H = len(fanouts)
        fo = np.ascontiguousarray(np.asarray(fanouts, dtype=np.int32).reshape(H * R)) \
            if H * R > 0 else np.zeros(1, dtype=np.int32)
        handle = ctypes.c_void_p()
        st = self.lib.oracle_sample_blocks(ctypes.addressof(self._nt), T,
                                           ctypes.addressof(self._et), R, ptrs, _ptr(ns), H,
                                           _ptr(fo), sigma, key_bits, ctypes.byref(handle))
        if st != OK:
            raise OracleError(st)
        try:
            return _result_dict(self.lib, handle, H, T, R, [e[1] for e in self.etypes])
        finally:
            self.lib.oracle_blocks_free(handle)

    def sample_edge_blocks(self, targets, fanouts, sigma, n_neg=0, exclude=0, rev_etype=None,
                           rev_eid=None, key_bits=32):
        """An edge-seeded mini-batch.  targets: per edge type an int64 array of
        target edge IDs (or None); rev_etype: per edge type its reverse type or
        -1; rev_eid: per edge type an int64 array [nnz] (or None).  Returns the
        result dict of sample_blocks plus "seeds" {t: gids} and "pairs"
        {e: (pos_src, pos_dst, neg_dst)}."""
        T, R = self.T, self.R
        tg = [None if (targets[e] is None) else _arr_i64(targets[e]) for e in range(R)]
        tptr = (ctypes.c_void_p * max(R, 1))(*[(_ptr(x) if x is not None and x.size else None)
                                               for x in tg])
        tn = np.array([0 if x is None else x.size for x in tg] + [0], dtype=np.int64)
        rv = None
        rptr = None
        if rev_etype is not None:
            rv = np.ascontiguousarray(np.asarray(rev_etype, dtype=np.int32))
        keep = []
        if rev_eid is not None:
            arrs = [None if x is None else _arr_i64(x) for x in rev_eid]
            keep = arrs
            rptr = (ctypes.c_void_p * max(R, 1))(*[(_ptr(x) if x is not None and x.size else None)
                                                   for x in arrs])
        batch = _EdgeBatch(ctypes.addressof(tptr), _ptr(tn), int(n_neg), int(exclude),
                           _ptr(rv), None if rptr is None else ctypes.addressof(rptr))
        H = len(fanouts)
        fo = np.ascontiguousarray(np.asarray(fanouts, dtype=np.int32).reshape(H * R)) \
            if H * R > 0 else np.zeros(1, dtype=np.int32)
        handle = ctypes.c_void_p()
        st = self.lib.oracle_sample_edge_blocks(ctypes.addressof(self._nt), T,
                                                ctypes.addressof(self._et), R,
                                                ctypes.addressof(batch), H, _ptr(fo), sigma,
                                                key_bits, ctypes.byref(handle))
        del keep
        if st != OK:
            raise OracleError(st)
        try:
            res = _result_dict(self.lib, handle, H, T, R, [e[1] for e in self.etypes])
            res["seeds"] = {}
            res["pairs"] = {}
            for t in range(T):
                n = ctypes.c_int64()
                p = ctypes.c_void_p()
                self.lib.oracle_blocks_seeds(handle, t, ctypes.byref(n), ctypes.byref(p))
                res["seeds"][t] = _copy(p.value, n.value, ctypes.c_int64, np.int64)
            for e in range(R):
                npos, nneg = ctypes.c_int64(), ctypes.c_int64()
                ps, pd, pn = (ctypes.c_void_p() for _ in range(3))
                self.lib.oracle_blocks_pairs(handle, e, ctypes.byref(npos), ctypes.byref(ps),
                                             ctypes.byref(pd), ctypes.byref(nneg),
                                             ctypes.byref(pn))
                res["pairs"][e] = (_copy(ps.value, npos.value, ctypes.c_int32, np.int32),
                                   _copy(pd.value, npos.value, ctypes.c_int32, np.int32),
                                   _copy(pn.value, nneg.value, ctypes.c_int32, np.int32))
            return res
        finally:
            self.lib.oracle_blocks_free(handle)

    def sample_layers(self, seeds, layer_sizes, sigma):
        """A layer-wise (LADIES) mini-batch: seeds per node type; layer_sizes
        [n_hops][n_ntypes] draws per hop and node type (-1: every candidate).
        Returns the result dict of sample_blocks."""
        T, R = self.T, self.R
        seed_arrs = [None if (seeds[t] is None) else _arr_i64(seeds[t]) for t in range(T)]
        ptrs = (ctypes.c_void_p * T)(*[(_ptr(x) if x is not None and x.size else None)
                                       for x in seed_arrs])
        ns = np.array([0 if x is None else x.size for x in seed_arrs], dtype=np.int64)
        H = len(layer_sizes)
        ls = np.ascontiguousarray(np.asarray(layer_sizes, dtype=np.int32).reshape(H * T)) \
            if H > 0 else np.zeros(1, dtype=np.int32)
        handle = ctypes.c_void_p()
        st = self.lib.oracle_sample_layers(ctypes.addressof(self._nt), T,
                                           ctypes.addressof(self._et), R, ptrs, _ptr(ns), H,
                                           _ptr(ls), sigma, ctypes.byref(handle))
        if st != OK:
            raise OracleError(st)
        try:
            return _result_dict(self.lib, handle, H, T, R, [e[1] for e in self.etypes])
        finally:
            self.lib.oracle_blocks_free(handle)

    def gather(self, ntype, ids):
        n, feat, row_bytes = self.ntypes[ntype]
        if feat is None or row_bytes == 0:
            raise OracleError(EINVAL)
        ids = _arr_i64(ids)
        out = np.empty((ids.size,) + feat.shape[1:], dtype=feat.dtype)
        st = self.lib.oracle_gather_rows(_ptr(feat), n, row_bytes,
                                         _ptr(ids) if ids.size else None, ids.size,
                                         _ptr(out) if ids.size else None)
        if st != OK:
            raise OracleError(st)
        return out


def _copy(ptr, n, ctype, dtype):
    if n == 0:
        return np.zeros(0, dtype=dtype)
    buf = (ctype * n).from_address(ptr)
    return np.frombuffer(buf, dtype=dtype, count=n).copy()


def _result_dict(lib, handle, H, T, R, dst_types):
    """Copy every output array of an oracle result into numpy.

    nodes[(h, t)] = (n_dst, src_gid); edges[(h, e)] = (indptr, src_local, dst_local,
    eid); input[t] = input-frontier vertex IDs."""
    res = {"n_hops": H, "nodes": {}, "edges": {}, "input": {}}
    for h in range(H):
        for t in range(T):
            nd, ns = ctypes.c_int64(), ctypes.c_int64()
            p = ctypes.c_void_p()
            lib.oracle_blocks_nodes(handle, h, t, ctypes.byref(nd), ctypes.byref(ns),
                                    ctypes.byref(p))
            res["nodes"][(h, t)] = (nd.value, _copy(p.value, ns.value, ctypes.c_int64, np.int64))
        for e in range(R):
            ne = ctypes.c_int64()
            pi, ps, pd, pe = (ctypes.c_void_p() for _ in range(4))
            lib.oracle_blocks_edges(handle, h, e, ctypes.byref(ne), ctypes.byref(pi),
                                    ctypes.byref(ps), ctypes.byref(pd), ctypes.byref(pe))
            n_dst = res["nodes"][(h, dst_types[e])][0]
            res["edges"][(h, e)] = (
                _copy(pi.value, n_dst + 1, ctypes.c_int64, np.int64),
                _copy(ps.value, ne.value, ctypes.c_int32, np.int32),
                _copy(pd.value, ne.value, ctypes.c_int32, np.int32),
                _copy(pe.value, ne.value, ctypes.c_int64, np.int64),
            )
    for t in range(T):
        n = ctypes.c_int64()
        p = ctypes.c_void_p()
        lib.oracle_blocks_input_nodes(handle, t, ctypes.byref(n), ctypes.byref(p))
        res["input"][t] = _copy(p.value, n.value, ctypes.c_int64, np.int64)
    return res
