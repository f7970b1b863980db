"""HIP path against the oracle on the two largest workloads, at full size and
with the calls bench.py makes: the billion-edge single-GPU share (3 node types,
1.2B edges, 3 hops) and the 200-relation knowledge graph (20M nodes, 300M
edges).  Every block array and the gathered feature bytes are compared element
by element for one mini-batch each; the definition checks of the pins run on
the GPU result as well."""
import sys
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2112_15345_amd as hg
import pins
import workloads as W
from gpu_harness import compare, gpu_seeds, result_dict

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("idx,batch", [(4, 0), (3, 0)])
def test_large_workload_parity(idx, batch):
    torch.cuda.empty_cache()
    wl = W.WORKLOADS[idx]
    t0 = time.time()
    gen = W.make_graph(wl, device="cuda")
    torch.cuda.synchronize()
    say(f"workload {idx}: generated in {time.time() - t0:.1f}s")
    g = hg.Graph(list(zip(gen.num_nodes, gen.feats)), gen.etypes)
    fan = wl.fanout_matrix()
    seeds = W.seeds_per_type(wl, batch)
    t0 = time.time()
    blocks = g.sample_blocks(gpu_seeds(seeds), fan, batch, gather="all")
    outs = {t: blocks.features(t) for t, f in enumerate(gen.feats) if f is not None}
    got = result_dict(g, blocks)
    say(f"workload {idx}: GPU mini-batch and copy-out in {time.time() - t0:.1f}s")

    t0 = time.time()
    host_et = gen.host_etypes()
    host_nt = gen.host_ntypes()
    del gen
    say(f"workload {idx}: host copies in {time.time() - t0:.1f}s")
    t0 = time.time()
    host = oracle.HostGraph(host_nt, host_et, check=False)
    ref = host.sample_blocks(seeds, fan, batch)
    say(f"workload {idx}: oracle mini-batch in {time.time() - t0:.1f}s "
        f"({sum(v[3].size for v in ref['edges'].values())} edges)")
    diffs = compare(ref, got, g.T, g.R, len(fan))
    assert not diffs, "\n".join(diffs[:10])
    fails = pins.check_blocks([n for n, _ in host_nt], host_et, seeds, fan, batch, 32, got,
                              brute=False)
    assert not fails, "\n".join(fails[:5])
    for t, x in outs.items():
        want = host.gather(t, ref["input"][t])
        assert x.contiguous().view(torch.uint8).cpu().numpy().tobytes() == want.tobytes(), \
            f"type {t}: gathered bytes differ"
    say(f"workload {idx}: equal")
