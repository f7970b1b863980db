"""The C-ABI library loads and exports every entry point include/hg.h declares
(no device calls; runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hg.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*[A-Za-z_][\w\s\*]*?\b(hg_\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    from paper_2112_15345_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    return ctypes.CDLL(build.LIB)


def test_header_declares_the_binding_symbols():
    import paper_2112_15345_amd as hg
    assert declared_functions() == sorted(hg.ABI_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    missing = [f for f in declared_functions() if not hasattr(lib, f)]
    assert not missing, f"missing exports: {missing}"


def test_library_argument_checks_without_device(lib):
    """Host-side checks return HG_EINVAL before any device work."""
    import paper_2112_15345_amd as hg
    hg.load_library()
    out = ctypes.c_void_p()
    assert hg._lib.hg_create(None, 0, None, 0, None, None, ctypes.byref(out)) == hg.HG_EINVAL
    assert b"node type" in hg._lib.hg_last_error()
    assert hg._lib.hg_sample_blocks(None, None, None, 1, None, 0, None,
                                    ctypes.byref(out)) == hg.HG_EINVAL
    assert hg._lib.hg_blocks_num_hops(None) == -1
    assert hg._lib.hg_blocks_nodes(None, 0, 0, None, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_gather_rows(None, 0, None, 0, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_debug_philox(None, 0, -1, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_graph_types(None, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_blocks_features(None, 0, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_sample_blocks_gather(None, None, None, 1, None, 0, None, 0, None, None,
                                           None, ctypes.byref(out)) == hg.HG_EINVAL
    assert hg._lib.hg_pipeline_create(None, 2, 4, None, 0, ctypes.byref(out)) == hg.HG_EINVAL
    assert hg._lib.hg_pipeline_submit(None, 1, None, None, 1, None, None, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_pipeline_next(None, ctypes.byref(out)) == hg.HG_EINVAL
    assert hg._lib.hg_pipeline_submit_layers(None, 1, None, None, 1, None, None) == hg.HG_EINVAL
    assert hg._lib.hg_pipeline_submit_edges(None, 1, None, 1, None, None) == hg.HG_EINVAL
    hg._lib.hg_pipeline_destroy(None)


def test_create_descriptor_checks_without_device(lib):
    """hg_create validates every descriptor before it makes any HIP call, so
    these run on the CPU; the pointers are never dereferenced (fake, non-NULL).
    An edge type of 2^32 edges or more is refused with HG_EUNSUPPORTED: edge
    IDs enter the key counter as (eid >> 2) below 2^30, and the sampler's
    per-hub edge offsets are 32-bit."""
    import paper_2112_15345_amd as hg
    hg.load_library()
    fake = ctypes.c_void_p(0x1000)
    out = ctypes.c_void_p()

    def create(nt, et):
        nts = (hg.NTypeDesc * len(nt))(*nt)
        ets = (hg.ETypeDesc * max(len(et), 1))(*et)
        return hg._lib.hg_create(nts, len(nt), ets, len(et), None, None, ctypes.byref(out))

    def nt(n=10, feat=None, dtype=0, dim=0):
        return hg.NTypeDesc(n, feat, dtype, dim)

    def et(src=0, dst=0, nnz=5, indptr=fake, indices=fake):
        return hg.ETypeDesc(src, dst, nnz, indptr, indices)

    assert create([nt(-1)], []) == hg.HG_EINVAL
    assert b"negative num_nodes" in hg._lib.hg_last_error()
    assert create([nt(dtype=7, dim=4, feat=fake)], []) == hg.HG_EINVAL
    assert create([nt(dtype=hg.HG_DT_F32, dim=0, feat=fake)], []) == hg.HG_EINVAL
    assert create([nt(dtype=hg.HG_DT_F32, dim=4, feat=None)], []) == hg.HG_EINVAL
    assert create([nt()], [et(src=1)]) == hg.HG_EINVAL
    assert b"node type out of range" in hg._lib.hg_last_error()
    assert create([nt()], [et(indptr=None)]) == hg.HG_EINVAL
    assert create([nt()], [et(indices=None)]) == hg.HG_EINVAL
    assert create([nt()], [et(nnz=-1)]) == hg.HG_EINVAL
    assert create([nt()], [et(nnz=1 << 32)]) == hg.HG_EUNSUPPORTED
    assert b"below 2^32" in hg._lib.hg_last_error()
    assert out.value is None
