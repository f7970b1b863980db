"""The allocation-free row pull (hg_gather_rows_noalloc) against the existing
pull (hg_gather_rows) through the C ABI: two calls in a row on the academic
graph's paper features, the second with fewer rows, each byte-equal to
hg_gather_rows and to the rows of the table; IDs out of range give HG_EINVAL
with the valid rows gathered, and the next call starts from a clean count."""
import ctypes
import sys

import numpy as np
import pytest
import torch

import paper_2112_15345_amd as hg
import workloads as W

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def pull(g, fn, t, ids, dim, dtype):
    out = torch.full((ids.numel(), dim), -1, dtype=dtype, device="cuda")
    st = getattr(hg.load_library(), fn)(g._h, t, ids.data_ptr() if ids.numel() else None,
                                        ids.numel(), out.data_ptr() if out.numel() else None,
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return st, out


def test_noalloc_pull_equals_gather_rows():
    wl = W.WORKLOADS[2]
    gen = W.make_graph(wl, device="cuda")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    t = 0
    f = gen.feats[t]
    n, dim = f.shape
    rng = np.random.default_rng(3)
    for rows in (300_000, 1_001):
        say(f"pull of {rows} rows")
        ids = torch.as_tensor(rng.integers(0, n, size=rows), device="cuda")
        st0, want = pull(g, "hg_gather_rows", t, ids, dim, f.dtype)
        st1, got = pull(g, "hg_gather_rows_noalloc", t, ids, dim, f.dtype)
        assert st0 == hg.HG_OK and st1 == hg.HG_OK
        assert torch.equal(got.view(torch.uint8), want.view(torch.uint8))
        assert torch.equal(got.view(torch.uint8), f.index_select(0, ids).view(torch.uint8))
    say("IDs out of range")
    ids = torch.as_tensor([0, n - 1, n, -5, 7], device="cuda")
    st, got = pull(g, "hg_gather_rows_noalloc", t, ids, dim, f.dtype)
    assert st == hg.HG_EINVAL
    assert b"2 IDs are outside" in hg.load_library().hg_last_error()
    ok = torch.tensor([0, 1, 4])
    assert torch.equal(got[ok].view(torch.uint8),
                       f.index_select(0, ids[ok.cuda()]).view(torch.uint8))
    assert not got[2:4].view(torch.uint8).any()
    st, got = pull(g, "hg_gather_rows_noalloc", t, ids[:2], dim, f.dtype)
    assert st == hg.HG_OK
    assert hg.load_library().hg_gather_rows_noalloc(g._h, 3 + 1, None, 0, None, None) == \
        hg.HG_EINVAL
