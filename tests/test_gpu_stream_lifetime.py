"""Streams that go away: a pipeline creates worker streams, runs bundles on
them and destroys them when it closes; a caller may do the same with its own
stream (hg_retire_stream before destroying it).  Afterwards a direct call
with the same bundle size (which takes over the workspaces those streams
used), hg_destroy and the next torch launch must all work, equal the oracle,
and leave no HIP error pending on the thread."""
import ctypes
import sys

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


def hip():
    lib = ctypes.CDLL("libamdhip64.so")
    lib.hipPeekAtLastError.restype = ctypes.c_int
    lib.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    lib.hipStreamSynchronize.argtypes = [ctypes.c_void_p]
    return lib


def tiny_graph():
    wl = W.WORKLOADS[1]
    gen = W.make_graph(wl)
    g = hg.Graph([(n, f.cuda()) for n, f in zip(gen.num_nodes, gen.feats)],
                 [(s, d, ip.cuda(), ix.cuda()) for s, d, ip, ix in gen.etypes])
    host = oracle.HostGraph(gen.host_ntypes(), gen.host_etypes())
    return wl, gen, g, host


def check_batches(wl, g, host, batches, got):
    fan = wl.fanout_matrix()
    for b, blocks in zip(batches, got):
        ref = host.sample_blocks(W.seeds_per_type(wl, b), fan, b)
        diffs = compare(ref, result_dict(g, blocks), g.T, g.R, len(fan))
        assert not diffs, f"batch {b}: " + "\n".join(diffs[:5])
        for t in range(g.T):
            want = host.gather(t, ref["input"][t]).tobytes()
            assert blocks.features(t).cpu().numpy().tobytes() == want, f"batch {b} type {t}"


def test_pipeline_close_then_direct_call_and_destroy():
    lib = hip()
    wl, gen, g, host = tiny_graph()
    fan = wl.fanout_matrix()
    sizes = W.LAYER_SIZES
    say("pipeline: vertex bundles of 4 and 1, a layer-wise bundle of 3, on 2 worker streams")
    pipe = hg.Pipeline(g, workers=2, capacity=8, gather="all")
    seeds = {b: gpu_seeds(W.seeds_per_type(wl, b)) for b in range(12)}
    pipe.submit_bundle([seeds[b] for b in range(4)], fan, list(range(4)))
    pipe.submit_bundle([seeds[b] for b in range(4, 8)], fan, list(range(4, 8)))
    first = [pipe.next() for _ in range(8)]
    pipe.submit(seeds[8], fan, 8)
    pipe.submit_layers_bundle([seeds[b] for b in range(9, 12)], [[k] * g.T for k in sizes],
                              list(range(9, 12)))
    more = [pipe.next() for _ in range(4)]
    pipe.close()
    assert lib.hipPeekAtLastError() == 0, "the pipeline's teardown left a HIP error pending"
    check_batches(wl, g, host, list(range(9)), first + more[:1])
    del first, more

    say("direct bundle of 4 on the current stream after the pipeline closed")
    got = g.sample_bundle([seeds[b] for b in range(4)], fan, list(range(4)))
    check_batches(wl, g, host, list(range(4)), got)
    got1 = g.sample_blocks(seeds[5], fan, 5, gather="all")
    check_batches(wl, g, host, [5], [got1])
    del got, got1
    assert lib.hipPeekAtLastError() == 0

    say("hg_destroy, then a torch launch")
    del g
    assert lib.hipPeekAtLastError() == 0, "hg_destroy left a HIP error pending"
    x = torch.rand(1 << 16, device="cuda")
    torch.cuda.synchronize()
    assert float(x.sum()) > 0


def test_caller_stream_retired_before_destroy():
    lib = hip()
    wl, gen, g, host = tiny_graph()
    fan = wl.fanout_matrix()
    seeds = {b: gpu_seeds(W.seeds_per_type(wl, b)) for b in range(6)}
    s = ctypes.c_void_p()
    assert lib.hipStreamCreate(ctypes.byref(s)) == 0
    say("bundle of 3 and a single call on a caller-made stream")
    torch.cuda.synchronize()  # the seeds were copied on the current stream
    ext = torch.cuda.ExternalStream(s.value)
    got = g.sample_bundle([seeds[b] for b in range(3)], fan, list(range(3)), stream=ext)
    one = g.sample_blocks(seeds[3], fan, 3, gather="all", stream=ext)
    assert lib.hipStreamSynchronize(s) == 0
    # the handles are freed on their own stream: free them before it goes
    check_batches(wl, g, host, list(range(3)), got)
    check_batches(wl, g, host, [3], [one])
    del got, one
    assert lib.hipStreamSynchronize(s) == 0
    assert hg.load_library().hg_retire_stream(g._h, s) == hg.HG_OK
    assert lib.hipStreamDestroy(s) == 0
    assert lib.hipPeekAtLastError() == 0

    say("the same calls on the current stream after the caller's stream is gone")
    got = g.sample_bundle([seeds[b] for b in range(3)], fan, list(range(3)))
    one = g.sample_blocks(seeds[4], fan, 4, gather="all")
    check_batches(wl, g, host, list(range(3)), got)
    check_batches(wl, g, host, [4], [one])
    del got, one
    del g
    assert lib.hipPeekAtLastError() == 0
    x = torch.rand(1 << 16, device="cuda")
    torch.cuda.synchronize()
    assert float(x.sum()) > 0
    assert hg.load_library().hg_retire_stream(None, None) == hg.HG_EINVAL
