"""GPU parity: the HIP pass, called through the C ABI, against the CPU oracle
on the same seeded inputs."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from synth import workloads as W
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu


def cache_of(w: W.Workload, streams=None, n=None, capacity=None):
    """Stacked numpy cache [B, L, H, S, D] for the workload's streams."""
    idx = range(w.streams) if streams is None else streams
    n = w.n_tokens if n is None else n
    cap = capacity or max(n, w.capacity)
    sts = [synth.fresh_cache(w.seeds[s], w.layers, w.kv_heads, cap, w.head_dim, w.grid_h, w.grid_w, n, w.dtype,
                             w.rho_specs[s], w.value_sigma) for s in idx]
    st = lambda a: np.ascontiguousarray(np.stack([getattr(s, a) for s in sts]))
    return st("K"), st("V"), st("frame_idx"), st("patch_idx")


def oracle_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, tau=None):
    tar64 = oracle.tar_scores(K, fr, pa, n, r, gh, gw)
    van64, pool = oracle.van_scores(V, fr, pa, n, gh, gw, tau)
    sel = oracle.select(tar64.astype(np.float32), van64.astype(np.float32), fr, n, budget, alpha, r)
    return tar64, van64, pool, sel


def full_check(w, K, V, fr, pa, alpha, steps=False, tau=None, n=None, budget=None):
    n = w.n_tokens if n is None else n
    budget = w.budget if budget is None else budget
    print("case %s alpha=%s n=%d C=%d steps=%s" % (w.name, alpha, n, budget, steps), flush=True)
    tar64, van64, pool, sel = oracle_pass(K, V, fr, pa, n, budget, alpha, w.recent_frames, w.grid_h, w.grid_w, tau)
    got = P.gpu_compress(K, V, fr, pa, n, budget, alpha, w.recent_frames, w.grid_h, w.grid_w, tau, steps=steps)
    assert got.errors == 0
    et, ev = P.check_scores(got.tar, got.van, tar64, van64, n, w.name)
    P.check_ascending(got.keep, n)
    near = P.check_keep(got.keep, sel, tar64, van64)
    P.oracle_gather_equal(K, V, fr, pa, n, got.keep, got)
    # the oracle's selection on the GPU's own scores must give the GPU's keep set exactly
    sel_g = oracle.select(np.ascontiguousarray(got.tar), np.ascontiguousarray(got.van), fr, n, budget, alpha,
                          w.recent_frames)
    assert np.array_equal(sel_g.keep_idx, got.keep)
    if steps and tau is not None:
        assert np.array_equal(got.pool_size, pool)
    print("  max abs err tar %.2e van %.2e (tolerance used %.3f / %.3f), near-threshold rows %d"
          % (et["max_abs"], ev["max_abs"], et["max_tol_frac"], ev["max_tol_frac"], near), flush=True)
    return got


@pytest.mark.parametrize("steps", [False, True])
def test_tiny_fp32_end_to_end(steps):
    w = W.TINY
    full_check(w, *cache_of(w), 0.5, steps=steps)


@pytest.mark.parametrize("alpha", [0.5, 1.0, 0.0])
def test_7b_class_end_to_end(alpha):
    w = W.SEVEN_B
    full_check(w, *cache_of(w), alpha)


def test_7b_class_step_entry_points():
    w = W.SEVEN_B
    full_check(w, *cache_of(w), 0.5, steps=True)


def test_select_is_bit_exact_on_oracle_scores():
    # the same fp32 scores in, the same keep set out
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    n = w.n_tokens
    tar32 = oracle.tar_scores(K, fr, pa, n, w.recent_frames, w.grid_h, w.grid_w).astype(np.float32)
    van32 = oracle.van_scores(V, fr, pa, n, w.grid_h, w.grid_w)[0].astype(np.float32)
    # coarsen the scores so that many ties occur and the index tie-break matters
    tar32 = np.round(tar32 * 64) / 64
    van32 = np.round(van32 * 4) / 4
    tar32[..., ::5] = -0.0
    from paper_2506_15745_amd import ipv
    for alpha in (0.5, 1.0, 0.0, 0.3):
        sel = oracle.select(tar32, van32, fr, n, w.budget, alpha, w.recent_frames)
        td, vd, fd = P.to_device(tar32), P.to_device(van32), P.to_device(fr)
        keep = torch.zeros(sel.keep_idx.shape, dtype=torch.int32, device="cuda:0")
        ws = ipv.alloc_workspace(ipv.Shape(1, w.layers, w.kv_heads, w.head_dim, w.n_tokens, w.grid_h, w.grid_w, 0),
                                 "cuda:0")
        ipv.ipv_select(td, vd, fd, n, w.budget, alpha, w.recent_frames, keep, ws, w.grid_h, w.grid_w)
        torch.cuda.synchronize()
        assert ipv.ipv_read_device_errors(ws) == 0
        assert np.array_equal(keep.cpu().numpy(), sel.keep_idx), alpha


@pytest.mark.parametrize("dtype,D,gh,gw,frames,extra,r", [
    (synth.BF16, 64, 3, 5, 7, 4, 2),      # ragged: partial last frame, odd grid
    (synth.BF16, 32, 2, 2, 40, 3, 3),
    (synth.BF16, 256, 4, 4, 9, 0, 1),
    (synth.F32, 128, 5, 3, 11, 7, 2),
    (synth.F32, 32, 1, 7, 20, 1, 4),
    (synth.F32, 256, 2, 3, 12, 5, 3),
])
def test_ragged_shapes_and_head_dims(dtype, D, gh, gw, frames, extra, r):
    p = gh * gw
    n = frames * p + extra
    w = W.Workload(name="ragged-D%d" % D, streams=2, layers=3, kv_heads=2, head_dim=D, grid_h=gh, grid_w=gw,
                   n_tokens=n, budget=max(r * p + 1, n // 2), recent_frames=r, alphas=(0.5,), dtype=dtype,
                   seeds=(21, 22), rho_specs=(synth.RhoSpec(), synth.RhoSpec(0, 0.9, 0.3)))
    K, V, fr, pa = cache_of(w, capacity=n + 13)
    for alpha in (0.5, 0.9):
        full_check(w, K, V, fr, pa, alpha)


def test_degenerate_budgets():
    w = W.Workload(name="degenerate", streams=1, layers=2, kv_heads=2, head_dim=128, grid_h=4, grid_w=4,
                   n_tokens=16 * 10, budget=0, recent_frames=2, alphas=(0.5,), dtype=synth.BF16, seeds=(5,),
                   rho_specs=(synth.RhoSpec(),))
    K, V, fr, pa = cache_of(w)
    n, R = w.n_tokens, 2 * 16
    for budget in (R, R + 1, n - 1, n):  # only the window; window + 1; drop one row; keep everything
        got = full_check(w, K, V, fr, pa, 0.5, budget=budget)
        if budget == n:
            assert np.array_equal(got.keep[0, 0, 0], np.arange(n))
        if budget == R:
            assert np.array_equal(got.keep[0, 0, 0], np.arange(n - R, n))


@pytest.mark.parametrize("dtype,D,gh,gw,n,S,r,budget,alpha", [
    # the largest count a slice takes (1024 selection threads x 64 rows), 16-byte row runs
    (synth.BF16, 64, 16, 16, 65536, 65536, 4, 32768, 0.5),
    # one row fewer, a capacity that is not a multiple of 4 (4-byte row loads), a
    # ragged last frame and a 256-frame recent window
    (synth.F32, 32, 7, 9, 65535, 65535, 256, 40000, 0.3),
    # the longest recent window with the narrowest bf16 rows: the table's slot
    # array at its largest (64 position groups x 256 frames of LDS)
    (synth.BF16, 32, 2, 2, 4099, 4100, 256, 2048, 0.5),
])
def test_largest_sizes(dtype, D, gh, gw, n, S, r, budget, alpha):
    w = W.Workload(name="largest-D%d-r%d" % (D, r), streams=1, layers=1, kv_heads=2, head_dim=D, grid_h=gh, grid_w=gw,
                   n_tokens=n, budget=budget, recent_frames=r, alphas=(alpha,), dtype=dtype, seeds=(31,),
                   rho_specs=(synth.RhoSpec(0.0, 0.99, static_frac=0.2, static_rho=0.999),))
    K, V, fr, pa = cache_of(w, capacity=S)
    full_check(w, K, V, fr, pa, alpha)


def test_pool_workload():
    w = W.POOL
    got = full_check(w, *cache_of(w), 0.5, steps=True, tau=w.cv_tau)
    assert set(got.pool_size.ravel().tolist()) == {7, 5, 3, 1}


def test_deterministic_over_repeated_runs():
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    K, V, fr, pa = K[:, :6], V[:, :6], fr[:, :6], pa[:, :6]
    K, V, fr, pa = (np.ascontiguousarray(a) for a in (K, V, fr, pa))
    ref = P.gpu_compress(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w)
    for _ in range(19):
        got = P.gpu_compress(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w)
        for a in ("tar", "van", "keep", "K", "V", "frame_idx", "patch_idx"):
            assert np.array_equal(getattr(got, a).view(np.uint8), getattr(ref, a).view(np.uint8)), a


@pytest.mark.parametrize("dtype,D", [(synth.BF16, 128), (synth.F32, 64), (synth.BF16, 32)])
def test_compaction_adversarial_patterns(dtype, D):
    # in-place gather against numpy fancy indexing, on keep patterns that stress
    # the write-after-read hazard; rows [n, S) hold a poison pattern that must
    # never reach the output and must stay untouched
    from paper_2506_15745_amd import ipv
    rng = np.random.default_rng(77)
    B, L, H, n, S = 1, 2, 3, 5000, 5003
    edt = np.uint16 if dtype == synth.BF16 else np.float32
    K = rng.integers(0, 2**15, size=(B, L, H, S, D)).astype(np.uint16)
    V = rng.integers(0, 2**15, size=(B, L, H, S, D)).astype(np.uint16)
    if dtype == synth.F32:
        K = rng.standard_normal((B, L, H, S, D)).astype(np.float32)
        V = rng.standard_normal((B, L, H, S, D)).astype(np.float32)
    K[..., n:, :] = K.dtype.type(0x7fc0) if dtype == synth.BF16 else np.float32(np.nan)
    fr = np.tile(np.arange(S, dtype=np.int32), (B, L, H, 1))
    pa = fr + 1000000
    patterns = {
        "drop-row-0": np.arange(1, n),
        "prefix": np.arange(0, 3000),
        "alternate": np.arange(0, n, 2),
        "window-plus-one": np.concatenate([[0], np.arange(n - 700, n)]),
        "last-rows": np.arange(n - 2500, n),
        "random": np.sort(rng.choice(n, 2222, replace=False)),
    }
    for name, keep1 in patterns.items():
        print("pattern", name, flush=True)
        C = len(keep1)
        keep = np.ascontiguousarray(np.broadcast_to(keep1.astype(np.int32), (B, L, H, C)))
        kind = "bf16" if dtype == synth.BF16 else "raw"
        Kd, Vd, fd, pd = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
        kd = P.to_device(keep)
        shape = ipv.shape_of(Kd, 1, 1)
        ws = ipv.alloc_workspace(shape, "cuda:0")
        ipv.ipv_compact(Kd, Vd, fd, pd, n, kd, C, ws, 1, 1)
        torch.cuda.synchronize()
        assert ipv.ipv_read_device_errors(ws) == 0
        Kh, Vh, fh, ph = P.to_host(Kd), P.to_host(Vd), P.to_host(fd), P.to_host(pd)
        assert np.array_equal(Kh[..., :C, :].view(np.uint8), K[..., keep1, :].view(np.uint8)), name
        assert np.array_equal(Vh[..., :C, :].view(np.uint8), V[..., keep1, :].view(np.uint8)), name
        assert np.array_equal(fh[..., :C], fr[..., keep1]) and np.array_equal(ph[..., :C], pa[..., keep1]), name
        assert np.array_equal(Kh[..., n:, :].view(np.uint8), K[..., n:, :].view(np.uint8)), name


def test_workspace_reused_across_calls_of_different_sizes():
    # the pass zeroes the compaction flags it uses in its first kernel: one
    # workspace serves many calls, of any budget, with no clearing between them
    from paper_2506_15745_amd import ipv
    w = W.Workload(name="reuse", streams=1, layers=3, kv_heads=2, head_dim=128, grid_h=8, grid_w=8,
                   n_tokens=64 * 40, budget=0, recent_frames=3, alphas=(0.5,), dtype=synth.BF16, seeds=(9,),
                   rho_specs=(synth.RhoSpec(),))
    K, V, fr, pa = cache_of(w)
    shape = ipv.Shape(1, w.layers, w.kv_heads, w.head_dim, w.n_tokens, w.grid_h, w.grid_w, 0)
    ws = ipv.alloc_workspace(shape, "cuda:0")
    for i, budget in enumerate((1280, 200, 2559, 900, 1280, 640, 2000, 192)):
        print("call", i, "budget", budget, flush=True)
        Kd, Vd = P.to_device(K, "bf16"), P.to_device(V, "bf16")
        fd, pd = P.to_device(fr), P.to_device(pa)
        comp = ipv.Compressor(Kd, w.grid_h, w.grid_w, budget)
        comp.ws = ws
        comp.compress(Kd, Vd, fd, pd, w.n_tokens, 0.5, w.recent_frames)
        torch.cuda.synchronize()
        assert ipv.ipv_read_device_errors(ws) == 0
        keep = comp.keep_idx.cpu().numpy()
        got = P.GpuPass(comp.tar.cpu().numpy(), comp.van.cpu().numpy(), keep, P.to_host(Kd), P.to_host(Vd),
                        P.to_host(fd), P.to_host(pd), 0)
        P.check_ascending(keep, w.n_tokens)
        P.oracle_gather_equal(K, V, fr, pa, w.n_tokens, keep, got)


def test_nan_scores_are_reported_and_the_pass_stays_well_formed():
    # bf16 quiet NaNs in one past key and one past value: their NaN scores
    # are reported in the device error word, the two rows' ranks are
    # unspecified, and the pass still keeps exactly C ascending rows, the
    # whole recent window, and compacts the rows it names
    from paper_2506_15745_amd import ipv
    w = W.SEVEN_B
    L = 2
    K, V, fr, pa = (np.ascontiguousarray(a[:, :L]) for a in cache_of(w))
    K[0, 1, 2, 500, 7] = 0x7fc0
    V[0, 0, 3, 1200, 0] = 0x7fc0
    got = P.gpu_compress(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, None)
    print("device errors", got.errors, flush=True)
    assert got.errors & ipv.DEV_NAN
    assert got.errors & ~(ipv.DEV_NAN) == 0
    # both NaNs reach the scores, as in the oracle's exact arithmetic
    assert np.isnan(got.tar[0, 1, 2, 500]) and np.isnan(got.van[0, 0, 3, 1200])
    P.check_ascending(got.keep, w.n_tokens)
    n_recent = w.recent_frames * w.p
    assert np.all(got.keep[..., -n_recent:] == np.arange(w.n_tokens - n_recent, w.n_tokens, dtype=np.int32))
    P.oracle_gather_equal(K, V, fr, pa, w.n_tokens, got.keep, got)


@pytest.mark.parametrize("C", [1, 511, 512, 513, 1024, 1025, 1999])
def test_compaction_at_chunk_boundaries(C):
    # keep sets whose size falls on, just below and just above the compaction's
    # chunk boundaries (512 rows), with sources spread over the whole slice
    from paper_2506_15745_amd import ipv
    rng = np.random.default_rng(91 + C)
    B, L, H, n, S, D = 1, 2, 2, 2000, 2003, 128
    K = rng.integers(0, 2**15, size=(B, L, H, S, D)).astype(np.uint16)
    V = rng.integers(0, 2**15, size=(B, L, H, S, D)).astype(np.uint16)
    fr = np.tile(np.arange(S, dtype=np.int32), (B, L, H, 1))
    pa = fr + 5000
    keep1 = np.sort(rng.choice(n, C, replace=False)).astype(np.int32)
    keep = np.ascontiguousarray(np.broadcast_to(keep1, (B, L, H, C)))
    Kd, Vd, fd, pd = P.to_device(K, "bf16"), P.to_device(V, "bf16"), P.to_device(fr), P.to_device(pa)
    ws = ipv.alloc_workspace(ipv.shape_of(Kd, 1, 1), "cuda:0")
    ipv.ipv_compact(Kd, Vd, fd, pd, n, P.to_device(keep), C, ws, 1, 1)
    torch.cuda.synchronize()
    assert ipv.ipv_read_device_errors(ws) == 0
    Kh, Vh, fh, ph = P.to_host(Kd), P.to_host(Vd), P.to_host(fd), P.to_host(pd)
    assert np.array_equal(Kh[..., :C, :], K[..., keep1, :]) and np.array_equal(Vh[..., :C, :], V[..., keep1, :])
    assert np.array_equal(fh[..., :C], fr[..., keep1]) and np.array_equal(ph[..., :C], pa[..., keep1])
    assert np.array_equal(Kh[..., n:, :], K[..., n:, :])


@pytest.mark.parametrize("mode", [0, ipv.UNIFORM_SELECT, ipv.TAR_REVERSE | ipv.VAN_REVERSE])
def test_more_slices_than_compute_units(mode):
    # 320 slices of few rows: the selection takes 16 rows a thread so that
    # several of its blocks share a CU
    L, H, D, gh, gw, r = 80, 4, 32, 14, 14, 2
    n = 8 * gh * gw
    st = synth.fresh_cache(61, L, H, n, D, gh, gw, n, synth.BF16, synth.RhoSpec(0.0, 0.99), (0.5,))
    K, V, fr, pa = (np.ascontiguousarray(getattr(st, a)[None]) for a in ("K", "V", "frame_idx", "patch_idx"))
    budget = n // 2
    Kd, Vd, frd, pad = P.to_device(K, "bf16"), P.to_device(V, "bf16"), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, gh, gw, budget)
    comp.compress(Kd, Vd, frd, pad, n, 0.5, r, mode=mode)
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    got = P.GpuPass(P.to_host(comp.tar), P.to_host(comp.van), P.to_host(comp.keep_idx), P.to_host(Kd), P.to_host(Vd),
                    P.to_host(frd), P.to_host(pad), 0)
    near = P.check_pass("320 slices mode %d" % mode, K, V, fr, pa, n, budget, 0.5, r, gh, gw, mode, got)
    print("  near-threshold rows %d" % near, flush=True)
