"""Feature tables in pinned host memory (the paper keeps features in CPU
memory, Sec. 4.1): the gathers read them through their device mapping over
the host link.  The gathered bytes must equal the oracle's, as for tables in
HBM; pageable host memory is refused."""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import workloads as W
from gpu_harness import compare, gpu_seeds, result_dict

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def pinned(t):
    return None if t is None else torch.empty(t.shape, dtype=t.dtype, pin_memory=True).copy_(t)


@pytest.mark.parametrize("idx,batches", [(1, range(3)), (2, range(2))])
def test_host_resident_features(idx, batches):
    wl = W.WORKLOADS[idx]
    gen = W.make_graph(wl, device="cuda", feat_device="cpu")
    feats = [pinned(f) for f in gen.feats]
    g = hg.Graph(list(zip(gen.num_nodes, feats)), gen.etypes)
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes(), check=False)
    fan = wl.fanout_matrix()
    featured = [t for t, f in enumerate(feats) if f is not None]
    for b in batches:
        say(f"workload {idx} batch {b}: pinned host features")
        seeds = W.seeds_per_type(wl, b)
        blocks = g.sample_blocks(gpu_seeds(seeds), fan, b, gather="all")
        got = result_dict(g, blocks)
        ref = host.sample_blocks(seeds, fan, b)
        diffs = compare(ref, got, g.T, g.R, len(fan))
        assert not diffs, "\n".join(diffs[:10])
        for t in featured:
            want = host.gather(t, ref["input"][t]).tobytes()
            assert blocks.features(t).cpu().numpy().tobytes() == want, f"type {t} (fused)"
            assert g.gather_features(blocks, t).cpu().numpy().tobytes() == want, f"type {t}"
        outs = g.gather_features_all(blocks, featured)
        for t in featured:
            assert outs[t].cpu().numpy().tobytes() == host.gather(t, ref["input"][t]).tobytes()
    # arbitrary rows by ID; an ID out of range is reported (HG_EINVAL), with
    # the valid rows gathered and zero rows for the bad ones
    t = featured[0]
    f = gen.host_ntypes()[t][1]
    ok_ids = torch.tensor([0, gen.num_nodes[t] - 1, 5], device="cuda")
    x = g.gather_rows(t, ok_ids).cpu().numpy()
    assert x.tobytes() == f[[0, gen.num_nodes[t] - 1, 5]].tobytes()
    ids = torch.tensor([0, gen.num_nodes[t] - 1, 5, gen.num_nodes[t], -3], device="cuda")
    out = torch.empty((5, f.shape[1]), dtype=feats[t].dtype, device="cuda")
    with pytest.raises(hg.HGError) as ex:
        g.gather_rows(t, ids, out=out)
    assert ex.value.status == hg.HG_EINVAL
    x = out.cpu().numpy()
    assert x[:3].tobytes() == f[[0, gen.num_nodes[t] - 1, 5]].tobytes()
    assert not x[3:].view(np.uint8).any()
    # the error does not stick: the next pull succeeds
    assert g.gather_rows(t, ok_ids).cpu().numpy().tobytes() == f[[0, gen.num_nodes[t] - 1, 5]].tobytes()


def test_pageable_host_features_refused():
    f = torch.randn(10, 4)  # ordinary (pageable) host memory
    with pytest.raises(hg.HGError) as ex:
        hg.Graph([(10, f)], [(0, 0, torch.zeros(11, dtype=torch.int64),
                              torch.zeros(0, dtype=torch.int64))])
    assert ex.value.status == hg.HG_EINVAL
