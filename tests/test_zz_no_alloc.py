"""ipv_compress_noalloc: the pass with the library's own per-GPU workspace.

Its results must equal ipv_compress's on the same inputs (same kernels), and
match the oracle by the usual rule. Two calls in a row with different shapes,
the second smaller, check that what the first call left in the shared
workspace does not leak into the second; a third repeats the first, and
Uniform Select calls (whose selection zeroes the compaction flags) follow.
"""
import numpy as np
import pytest
import torch

from paper_2506_15745_amd import ipv
from synth import workloads as W
from tests import parity as P
from tests.test_gpu_parity import cache_of

pytestmark = pytest.mark.gpu


def noalloc_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau=None, mode=0):
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd, fd, pd = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    B, L, H, S, D = K.shape
    # recognisable contents: every value the pass must write is overwritten
    tar = torch.full((B, L, H, S), float("nan"), dtype=torch.float32, device="cuda:0")
    van = torch.full_like(tar, float("nan"))
    keep = torch.full((B, L, H, budget), -7, dtype=torch.int32, device="cuda:0")
    err = torch.full((1,), 0x5A5A5A5A, dtype=torch.int32, device="cuda:0")
    ipv.ipv_compress_noalloc(Kd, Vd, fd, pd, n, budget, alpha, r, tau, tar, van, keep, gh, gw, device_errors=err,
                             mode=mode)
    torch.cuda.synchronize()
    return P.GpuPass(P.to_host(tar), P.to_host(van), P.to_host(keep), P.to_host(Kd), P.to_host(Vd), P.to_host(fd),
                     P.to_host(pd), int(err.item()))


def compress_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau=None, mode=0):
    """The same pass through ipv_compress with a workspace of its own."""
    if mode == 0:
        return P.gpu_compress(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau)
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd, fd, pd = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, gh, gw, budget)
    comp.compress(Kd, Vd, fd, pd, n, alpha, r, tau, mode=mode)
    torch.cuda.synchronize()
    return P.GpuPass(P.to_host(comp.tar), P.to_host(comp.van), P.to_host(comp.keep_idx), P.to_host(Kd),
                     P.to_host(Vd), P.to_host(fd), P.to_host(pd), comp.device_errors())


def check_against_compress(name, K, V, fr, pa, n, budget, alpha, r, gh, gw, tau=None, mode=0):
    print("case", name, K.shape, n, budget, alpha, mode, flush=True)
    got = noalloc_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau, mode)
    ref = compress_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau, mode)
    assert got.errors == 0 and ref.errors == 0
    # the same kernels on the same inputs: identical scores, keep sets and cache
    if not mode & ipv.UNIFORM_SELECT:  # Uniform Select writes no scores
        assert np.array_equal(got.tar[..., :n].view(np.uint32), ref.tar[..., :n].view(np.uint32))
        assert np.array_equal(got.van[..., :n].view(np.uint32), ref.van[..., :n].view(np.uint32))
    assert np.array_equal(got.keep, ref.keep)
    C = budget
    for a, b in ((got.K, ref.K), (got.V, ref.V), (got.frame_idx, ref.frame_idx), (got.patch_idx, ref.patch_idx)):
        assert np.array_equal(a[:, :, :, :C].view(np.uint8), b[:, :, :, :C].view(np.uint8))
    # and the oracle's rule, as for every pass
    P.check_pass(name, K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, got, tau)


def test_noalloc_equals_compress_on_consecutive_calls():
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    check_against_compress("7b-class", K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w)
    # second call: fewer layers and rows, another budget and a pooled VaN
    n = 3000
    k2, v2, f2, p2 = (np.ascontiguousarray(a[:, :5, :, :n]) for a in (K, V, fr, pa))
    check_against_compress("7b-class, 5 layers, 3000 rows", k2, v2, f2, p2, n, 1700, 0.6, w.recent_frames,
                           w.grid_h, w.grid_w, tau=(0.3, 0.5, 0.7))
    # third: the tiny fp32 cache, then the first case again
    t = W.TINY
    check_against_compress("tiny", *cache_of(t), t.n_tokens, t.budget, 0.5, t.recent_frames, t.grid_h, t.grid_w)
    check_against_compress("7b-class again", K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h,
                           w.grid_w)
    # Uniform Select runs no score kernel, so its selection zeroes the compaction's
    # flags and tickets, which the calls before left set in the shared workspace
    check_against_compress("7b-class, Uniform Select", K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames,
                           w.grid_h, w.grid_w, mode=ipv.UNIFORM_SELECT)
    check_against_compress("7b-class, 5 layers, 3000 rows, Uniform Select, heads shared", k2, v2, f2, p2, n, 1700,
                           0.6, w.recent_frames, w.grid_h, w.grid_w, mode=ipv.UNIFORM_SELECT | ipv.HEAD_SHARED)
    check_against_compress("7b-class after Uniform Select", K, V, fr, pa, w.n_tokens, w.budget, 0.5,
                           w.recent_frames, w.grid_h, w.grid_w)


def test_noalloc_reports_device_errors():
    # a budget below the recent window is only visible on the device
    t = W.TINY
    K, V, fr, pa = cache_of(t)
    got = noalloc_pass(K, V, fr, pa, t.n_tokens, 15, 0.5, t.recent_frames, t.grid_h, t.grid_w)
    assert got.errors == ipv.DEV_RECENT_OVER
    # the next call clears the word first
    got = noalloc_pass(K, V, fr, pa, t.n_tokens, t.budget, 0.5, t.recent_frames, t.grid_h, t.grid_w)
    assert got.errors == 0
