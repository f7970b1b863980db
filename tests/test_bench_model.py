"""The bench's byte model (no GPU): the per-stage split of the algorithmic
bytes of sampling and compaction adds up to the model's total per hop,
8 D + 16 P + 8 S + 8 (P + R) + 16 S + 8 (D + U), with R counted once per
mini-batch of a call."""
import os
import sys
from types import SimpleNamespace

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def test_stage_bytes_model_adds_up():
    rng = np.random.default_rng(5)
    # 2 node types, 3 edge types (dst types 0, 1, 0)
    g = SimpleNamespace(R=3, etypes=[(0, 0, None, None), (0, 1, None, None), (1, 0, None, None)])
    for n_batches in (1, 4):
        H = 3
        nd = rng.integers(0, 1000, size=(H, 2))
        ns = nd + rng.integers(0, 500, size=(H, 2))
        ne = rng.integers(0, 5000, size=(H, 3))
        got = bench.stage_bytes_model(g, nd, ns, ne, n_batches)
        want = 0
        for h in range(H):
            D, U, S = nd[h].sum(), (ns[h] - nd[h]).sum(), ne[h].sum()
            P = nd[h, 0] * 2 + nd[h, 1]  # two edge types end in type 0
            R = 3 * n_batches
            want += 8 * D + 16 * P + 8 * S + 8 * (P + R) + 16 * S + 8 * (D + U)
        assert sum(got.values()) == want
        assert got["select"] == 0
        assert got["relabel"] == 4 * ne.sum()
        assert got["compact"] == 8 * ns.sum()
        assert got["count"] == sum(8 * nd[h].sum() + 16 * (2 * nd[h, 0] + nd[h, 1])
                                   for h in range(H))
