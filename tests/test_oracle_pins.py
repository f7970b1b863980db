"""The CPU oracle against its pins (no GPU)."""
import numpy as np
import pytest

import oracle
import pins


@pytest.fixture(scope="module")
def lib():
    oracle.build()
    return oracle.load()


@pytest.mark.parametrize("name", sorted(pins.ALL_PINS))
def test_pin(lib, name):
    fails = pins.ALL_PINS[name](lib, np.random.default_rng(12345))
    assert not fails, "\n".join(fails[:10])


def test_statistics(lib):
    fails = pins.pin_statistics(lib)
    assert not fails, "\n".join(fails)


def test_negative_statistics(lib):
    fails = pins.pin_negative_uniformity(lib)
    assert not fails, "\n".join(fails)


def test_layer_statistics(lib):
    fails = pins.pin_layer_statistics(lib)
    assert not fails, "\n".join(fails)


def test_philox_zero_counter_known_answer(lib):
    # Philox4x32-10 with zero counter and zero key, from rocRAND's engine.
    ref = pins.rr_block(0, 0, 0)
    assert np.array_equal(oracle.philox4x32_10([0, 0, 0, 0], [0, 0], lib), ref)


def test_blocks_larger_graph(lib):
    """A few larger random graphs: more hops and wider frontiers than the pins."""
    rng = np.random.default_rng(7)
    for _ in range(3):
        nn, ets, feats, seeds, fanouts, sigma, bits = pins.random_case(rng, max_nodes=300,
                                                                       max_deg=60)
        hg = oracle.HostGraph(list(zip(nn, feats)), ets, lib=lib)
        res = hg.sample_blocks(seeds, fanouts, sigma, bits)
        fails = pins.check_blocks(nn, ets, seeds, fanouts, sigma, bits, res)
        assert not fails, "\n".join(fails[:10])


def test_tiny_workload(lib):
    """The tiny workload (6k/4k nodes, 100k edges), batch 0: every invariant and
    the brute-force selection of every pair."""
    import workloads as W
    wl = W.WORKLOADS[1]
    g = W.make_graph(wl)
    hg = oracle.HostGraph(g.host_ntypes(), g.host_etypes(), lib=lib)
    seeds = W.seeds_per_type(wl, 0)
    res = hg.sample_blocks(seeds, wl.fanout_matrix(), 0)
    fails = pins.check_blocks(g.num_nodes, g.host_etypes(), seeds, wl.fanout_matrix(), 0, 32,
                              res)
    assert not fails, "\n".join(fails[:10])
