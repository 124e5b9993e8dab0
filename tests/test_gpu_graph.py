"""The whole pass captured in a HIP graph (through torch.cuda.graph) and
replayed: every replay must equal the eager pass bit for bit. The pass
records no memset and allocates nothing, so it can be captured; the cache is
restored between replays by eager copies outside the graph."""
import numpy as np
import pytest
import torch

from paper_2506_15745_amd import ipv
from tests import parity as P
from tests.test_gpu_parity import cache_of
from synth import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", [0, ipv.TAR_ADJACENT | ipv.HEAD_SHARED])
def test_compress_graph_replays_equal_eager(mode):
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    L = 8  # a few layers keep the test short
    K, V, fr, pa = (np.ascontiguousarray(a[:, :L]) for a in (K, V, fr, pa))
    pristine = (P.to_device(K, "bf16"), P.to_device(V, "bf16"), P.to_device(fr), P.to_device(pa))
    work = tuple(t.clone() for t in pristine)
    comp = ipv.Compressor(work[0], w.grid_h, w.grid_w, w.budget)

    def run():
        comp.compress(*work, w.n_tokens, 0.5, w.recent_frames, mode=mode)

    def restore():
        for dst, src in zip(work, pristine):
            dst.copy_(src)

    def snapshot():
        return [t.clone() for t in work] + [comp.tar.clone(), comp.van.clone(), comp.keep_idx.clone()]

    # eager reference
    run()
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    ref = snapshot()

    # capture on a side stream (torch.cuda.graph does), after a warm-up there
    restore()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    restore()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()

    for rep in range(4):
        restore()
        for t in (comp.tar, comp.van):
            t.fill_(-1.0)
        comp.keep_idx.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = snapshot()
        for a, b in zip(got, ref):
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.uint8) if b.dtype == torch.bfloat16 else b), "replay %d differs" % rep
        # an eager pass between the replays, as a real caller would have
        restore()
        run()
        torch.cuda.synchronize()
        assert all(torch.equal(x, y) for x, y in zip(snapshot()[2:], ref[2:]))
    assert comp.device_errors() == 0


def test_noalloc_pass_graph_replays_equal_eager():
    """The allocation-free entry point is the one meant for capture: captured
    after one eager call (which looks up the per-GPU workspace), every replay
    equals the eager ipv_compress pass bit for bit, error word included."""
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    L = 8
    K, V, fr, pa = (np.ascontiguousarray(a[:, :L]) for a in (K, V, fr, pa))
    pristine = (P.to_device(K, "bf16"), P.to_device(V, "bf16"), P.to_device(fr), P.to_device(pa))
    work = tuple(t.clone() for t in pristine)
    comp = ipv.Compressor(work[0], w.grid_h, w.grid_w, w.budget)
    tar, van, keep = torch.empty_like(comp.tar), torch.empty_like(comp.van), torch.empty_like(comp.keep_idx)
    err = torch.zeros((1,), dtype=torch.int32, device="cuda:0")

    def run():
        ipv.ipv_compress_noalloc(*work, w.n_tokens, w.budget, 0.5, w.recent_frames, None, tar, van, keep,
                                 w.grid_h, w.grid_w, device_errors=err)

    def restore():
        for dst, src in zip(work, pristine):
            dst.copy_(src)

    # reference: the ordinary entry point with its own workspace
    comp.compress(*work, w.n_tokens, 0.5, w.recent_frames)
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    ref = [t.clone() for t in work] + [comp.tar.clone(), comp.van.clone(), comp.keep_idx.clone()]

    restore()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()  # eager warm-up: also resolves the per-GPU workspace outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    restore()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()

    for rep in range(4):
        restore()
        tar.fill_(-1.0)
        van.fill_(-1.0)
        keep.fill_(-1)
        err.fill_(0x5A5A5A5A)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [t.clone() for t in work] + [tar.clone(), van.clone(), keep.clone()]
        for a, b in zip(got, ref):
            assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.uint8) if b.dtype == torch.bfloat16 else b), "replay %d differs" % rep
        assert int(err.item()) == 0, "replay %d error word %#x" % (rep, int(err.item()))
        # eager work between the replays, as a real caller would have
        restore()
        comp.compress(*work, w.n_tokens, 0.5, w.recent_frames)
        torch.cuda.synchronize()
