"""GPU parity at the workloads' full sizes.

The 72B-class and batched caches are compressed whole, in the launch
configuration the benchmark uses; the oracle then checks a sample of slices
one by one, and properties that hold for every slice are checked for all of
them. The streaming workload runs all of its passes and compares each pass
in full, then hands the oracle's state to the GPU (teacher forcing) so that a
permitted near-threshold difference cannot grow over later passes.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads as W
from tests import parity as P
from paper_2506_15745_amd import ipv

pytestmark = pytest.mark.gpu


def stream_cache(w, s, n=None):
    n = w.n_tokens if n is None else n
    return synth.fresh_cache(w.seeds[s], w.layers, w.kv_heads, max(n, w.capacity), w.head_dim, w.grid_h, w.grid_w,
                             n, w.dtype, w.rho_specs[s], w.value_sigma)


def slice_arrays(K, V, fr, pa, idx):
    """One (b, l, h) slice as a [1, 1, 1, S, ...] cache."""
    one = lambda a: np.ascontiguousarray(a[idx][None, None, None])
    return one(K), one(V), one(fr), one(pa)


def check_sampled_slices(w, K, V, fr, pa, alpha, got, samples, n, budget):
    for idx in samples:
        print("  slice", idx, flush=True)
        k1, v1, f1, p1 = slice_arrays(K, V, fr, pa, idx)
        tar64 = oracle.tar_scores(k1, f1, p1, n, w.recent_frames, w.grid_h, w.grid_w)
        van64, _ = oracle.van_scores(v1, f1, p1, n, w.grid_h, w.grid_w)
        sel = oracle.select(tar64.astype(np.float32), van64.astype(np.float32), f1, n, budget, alpha,
                            w.recent_frames)
        g_tar = got["tar"][idx][None, None, None]
        g_van = got["van"][idx][None, None, None]
        g_keep = got["keep"][idx][None, None, None]
        P.check_scores(g_tar, g_van, tar64, van64, n, str(idx))
        P.check_keep(g_keep, sel, tar64, van64)
        sel_g = oracle.select(np.ascontiguousarray(g_tar), np.ascontiguousarray(g_van), f1, n, budget, alpha,
                              w.recent_frames)
        assert np.array_equal(sel_g.keep_idx, g_keep)
        Ko, Vo, fo, po = oracle.compact(k1, v1, f1, p1, n, np.ascontiguousarray(g_keep))
        C = budget
        assert np.array_equal(got["K"][idx][:C].view(np.uint8), Ko[0, 0, 0, :C].view(np.uint8))
        assert np.array_equal(got["V"][idx][:C].view(np.uint8), Vo[0, 0, 0, :C].view(np.uint8))
        assert np.array_equal(got["fr"][idx][:C], fo[0, 0, 0, :C])
        assert np.array_equal(got["pa"][idx][:C], po[0, 0, 0, :C])


def check_all_slices(w, fr0, keep, n, budget):
    """Properties of every slice's keep set: size, order, recent window kept."""
    assert keep.shape[-1] == budget
    assert np.all(np.diff(keep, axis=-1) > 0) and keep.min() >= 0 and keep.max() < n
    last = fr0[..., n - 1]
    thr = last - w.recent_frames + 1
    n_recent = (fr0[..., :n] >= thr[..., None]).sum(-1)
    # the window is a suffix of length n_recent, so the keep set ends with it
    tail_ok = keep[..., budget - n_recent.max():] == np.arange(n - n_recent.max(), n)
    assert np.all(n_recent == n_recent.flat[0]) and np.all(tail_ok)


def run_gpu(K, V, fr, pa, w, n, budget, alpha):
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd, fd, pd = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, w.grid_h, w.grid_w, budget)
    comp.compress(Kd, Vd, fd, pd, n, alpha, w.recent_frames)
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    return Kd, Vd, fd, pd, comp


def test_72b_class_full_size_sampled():
    w = W.SEVENTY_B
    print("generating %s" % w.name, flush=True)
    st = stream_cache(w, 0)
    K, V, fr, pa = (getattr(st, a)[None] for a in ("K", "V", "frame_idx", "patch_idx"))
    n, C, alpha = w.n_tokens, w.budget, w.alphas[0]
    assert n % w.p == 36  # 167 whole frames and a partial one
    Kd, Vd, fd, pd, comp = run_gpu(K, V, fr, pa, w, n, C, alpha)
    keep = comp.keep_idx.cpu().numpy()
    check_all_slices(w, fr, keep, n, C)
    samples = [(0, 0, 0), (0, 13, 5), (0, 40, 2), (0, 62, 7), (0, 79, 0), (0, 79, 7)]
    got = {"tar": {}, "van": {}, "keep": {}, "K": {}, "V": {}, "fr": {}, "pa": {}}
    for idx in samples:
        got["tar"][idx] = comp.tar[idx].cpu().numpy()
        got["van"][idx] = comp.van[idx].cpu().numpy()
        got["keep"][idx] = keep[idx]
        got["K"][idx] = P.to_host(Kd[idx][:C])
        got["V"][idx] = P.to_host(Vd[idx][:C])
        got["fr"][idx] = fd[idx][:C].cpu().numpy()
        got["pa"][idx] = pd[idx][:C].cpu().numpy()
    del Kd, Vd
    check_sampled_slices(w, K, V, fr, pa, alpha, got, samples, n, C)


@functools.lru_cache(maxsize=1)
def batched_cache():
    w = W.BATCHED
    print("generating %s" % w.name, flush=True)
    sts = [stream_cache(w, s) for s in range(w.streams)]
    return tuple(np.stack([getattr(s, a) for s in sts]) for a in ("K", "V", "frame_idx", "patch_idx"))


@pytest.mark.parametrize("alpha", [0.5, 1.0, 0.0])
def test_batched_streams_full_size_sampled(alpha):
    w = W.BATCHED
    K, V, fr, pa = batched_cache()
    n, C = w.n_tokens, w.budget
    Kd, Vd, fd, pd, comp = run_gpu(K, V, fr, pa, w, n, C, alpha)
    keep = comp.keep_idx.cpu().numpy()
    check_all_slices(w, fr, keep, n, C)
    rng = np.random.default_rng(int(alpha * 10))
    samples = [(int(b), int(rng.integers(w.layers)), int(rng.integers(w.kv_heads))) for b in (0, 1, 6, 9, 15)]
    got = {"tar": {}, "van": {}, "keep": {}, "K": {}, "V": {}, "fr": {}, "pa": {}}
    for idx in samples:
        got["tar"][idx] = comp.tar[idx].cpu().numpy()
        got["van"][idx] = comp.van[idx].cpu().numpy()
        got["keep"][idx] = keep[idx]
        got["K"][idx] = P.to_host(Kd[idx][:C])
        got["V"][idx] = P.to_host(Vd[idx][:C])
        got["fr"][idx] = fd[idx][:C].cpu().numpy()
        got["pa"][idx] = pd[idx][:C].cpu().numpy()
    check_sampled_slices(w, K, V, fr, pa, alpha, got, samples, n, C)


def test_streaming_all_passes():
    w = W.STREAMING
    cap, C, alpha, r = w.n_tokens, w.budget, w.alphas[0], w.recent_frames
    st = synth.Stream(w.seeds[0], w.layers, w.kv_heads, cap, w.head_dim, w.grid_h, w.grid_w, w.dtype,
                      w.rho_specs[0], tuple(w.value_sigma))
    Kd = P.to_device(st.K[None], "bf16")
    Vd = P.to_device(st.V[None], "bf16")
    fd, pd = P.to_device(st.frame_idx[None]), P.to_device(st.patch_idx[None])
    comp = ipv.Compressor(Kd, w.grid_h, w.grid_w, C)
    passes = near = 0
    for f in range(w.stream_frames):
        n0 = st.n
        st.append(1)
        rows = slice(n0, st.n)
        Kd[0, :, :, rows] = torch.from_numpy(st.K[:, :, rows]).view(torch.bfloat16).to("cuda:0")
        Vd[0, :, :, rows] = torch.from_numpy(st.V[:, :, rows]).view(torch.bfloat16).to("cuda:0")
        fd[0, :, :, rows] = torch.from_numpy(st.frame_idx[:, :, rows]).to("cuda:0")
        pd[0, :, :, rows] = torch.from_numpy(st.patch_idx[:, :, rows]).to("cuda:0")
        if st.n < cap:
            continue
        n = st.n
        print("pass %d at frame %d" % (passes, f), flush=True)
        K, V, fr, pa = st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None]
        tar64 = oracle.tar_scores(K, fr, pa, n, r, w.grid_h, w.grid_w)
        van64, _ = oracle.van_scores(V, fr, pa, n, w.grid_h, w.grid_w)
        sel = oracle.select(tar64.astype(np.float32), van64.astype(np.float32), fr, n, C, alpha, r)
        comp.compress(Kd, Vd, fd, pd, n, alpha, r)
        torch.cuda.synchronize()
        assert comp.device_errors() == 0
        g_tar, g_van, g_keep = comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy()
        P.check_scores(g_tar, g_van, tar64, van64, n, "pass %d" % passes)
        near += P.check_keep(g_keep, sel, tar64, van64)
        got = P.GpuPass(g_tar, g_van, g_keep, P.to_host(Kd), P.to_host(Vd), fd.cpu().numpy(), pd.cpu().numpy(), 0)
        P.oracle_gather_equal(K, V, fr, pa, n, g_keep, got)
        # the oracle's pass becomes the state of both sides (teacher forcing)
        Ko, Vo, fo, po = oracle.compact(K, V, fr, pa, n, sel.keep_idx)
        st.K[:, :, :C], st.V[:, :, :C] = Ko[0, :, :, :C], Vo[0, :, :, :C]
        st.frame_idx[:, :, :C], st.patch_idx[:, :, :C] = fo[0, :, :, :C], po[0, :, :, :C]
        st.n = C
        Kd[0, :, :, :C] = torch.from_numpy(st.K[:, :, :C]).view(torch.bfloat16).to("cuda:0")
        Vd[0, :, :, :C] = torch.from_numpy(st.V[:, :, :C]).view(torch.bfloat16).to("cuda:0")
        fd[0, :, :, :C] = torch.from_numpy(st.frame_idx[:, :, :C]).to("cuda:0")
        pd[0, :, :, :C] = torch.from_numpy(st.patch_idx[:, :, :C]).to("cuda:0")
        passes += 1
    print("passes %d, near-threshold rows %d" % (passes, near), flush=True)
    assert passes == 20 and st.n == 8192
