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
