"""GPU parity of Uniform Select (IPV_UNIFORM_SELECT): frames at regular
intervals, from frame ids alone. The keep sets are integer work and must equal
the oracle's bit for bit; the compaction must equal the oracle's gather; the
score buffers are neither read nor written."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2506_15745_amd import ipv
from synth import workloads as W
from tests import parity as P
from tests.test_gpu_parity import cache_of

pytestmark = pytest.mark.gpu
U = ipv.UNIFORM_SELECT


def uniform_pass(K, V, fr, pa, n, budget, r, gh, gw, mode=U, steps=False, scores=True):
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    B, L, H, S, D = K.shape
    # score buffers with a sentinel: the mode must leave them alone (or get None)
    tar = torch.full((B, L, H, S), 1.5, dtype=torch.float32, device="cuda:0") if scores else None
    van = torch.full((B, L, H, S), 2.5, dtype=torch.float32, device="cuda:0") if scores else None
    keep = torch.full((B, L, H, budget), -1, dtype=torch.int32, device="cuda:0")
    shape = ipv.shape_of(Kd, gh, gw)
    ws = ipv.alloc_workspace(shape, "cuda:0")
    if steps:
        ipv.ipv_select(tar, van, frd, n, budget, 0.5, r, keep, ws, gh, gw, head_dim=D, dtype=shape.dtype, mode=mode)
        ipv.ipv_compact(Kd, Vd, frd, pad, n, keep, budget, ws, gh, gw)
    else:
        ipv.ipv_compress(Kd, Vd, frd, pad, n, budget, 0.3, r, None, tar, van, keep, ws, gh, gw, mode=mode)
    torch.cuda.synchronize()
    if scores:
        assert bool((tar == 1.5).all()) and bool((van == 2.5).all()), "score buffers were written"
    z = np.zeros((B, L, H, S), np.float32)
    return P.GpuPass(z, z, P.to_host(keep), P.to_host(Kd), P.to_host(Vd), P.to_host(frd), P.to_host(pad),
                     ipv.ipv_read_device_errors(ws))


def check(name, K, V, fr, pa, n, budget, r, gh, gw, mode=U, **kw):
    print("case %s n=%d C=%d r=%d mode=%d %s" % (name, n, budget, r, mode, kw), flush=True)
    got = uniform_pass(K, V, fr, pa, n, budget, r, gh, gw, mode, **kw)
    assert got.errors == 0
    P.check_pass(name, K, V, fr, pa, n, budget, 0.5, r, gh, gw, mode, got)
    return got


@pytest.mark.parametrize("steps,scores", [(False, True), (True, True), (True, False), (False, False)])
def test_7b_class(steps, scores):
    w = W.SEVEN_B
    check(w.name, *cache_of(w), w.n_tokens, w.budget, w.recent_frames, w.grid_h, w.grid_w, steps=steps,
          scores=scores)


def test_7b_class_takes_every_other_frame():
    # 28 past frames and room for 14 of them: ranks 0, 2, 4, ...
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    got = uniform_pass(K, V, fr, pa, w.n_tokens, 4 * 196 + 14 * 196, w.recent_frames, w.grid_h, w.grid_w)
    frames = np.unique(got.keep[0, 0, 0] // 196)
    assert frames.tolist() == list(range(0, 28, 2)) + [28, 29, 30, 31]


@pytest.mark.parametrize("budget", [784, 785, 1000, 3136, 6271, 6272])
def test_budgets(budget):
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w)
    check("7b budget %d" % budget, K[:, :3], V[:, :3], fr[:, :3], pa[:, :3], w.n_tokens, budget, w.recent_frames,
          w.grid_h, w.grid_w)


def test_tiny_fp32_and_head_shared():
    w = W.TINY
    K, V, fr, pa = cache_of(w)
    check(w.name, K, V, fr, pa, w.n_tokens, w.budget, w.recent_frames, w.grid_h, w.grid_w)
    got = check(w.name + " head-shared", K, V, fr, pa, w.n_tokens, 40, w.recent_frames, w.grid_h, w.grid_w,
                mode=U | ipv.HEAD_SHARED)
    assert np.array_equal(got.keep[:, :, 0], got.keep[:, :, 1])


def test_fragmented_cache_after_a_pass():
    # a cache left by a published-method pass (frames lost rows), then new
    # frames, then Uniform Select: frames of every size, some ids missing
    w = W.SEVEN_B
    K, V, fr, pa = cache_of(w, n=w.n_tokens, capacity=w.n_tokens + 6 * 196)
    K, V, fr, pa = K[:, :4], V[:, :4], fr[:, :4], pa[:, :4]
    K, V, fr, pa = (np.ascontiguousarray(a) for a in (K, V, fr, pa))
    oracle.compress_inplace(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w)
    st = synth.fresh_cache(w.seeds[0] + 1, 4, w.kv_heads, 6 * 196, w.head_dim, w.grid_h, w.grid_w, 6 * 196, w.dtype,
                           w.rho_specs[0])
    n = w.budget + 6 * 196
    K[0, :, :, w.budget:n], V[0, :, :, w.budget:n] = st.K, st.V
    fr[0, :, :, w.budget:n] = st.frame_idx + 32
    pa[0, :, :, w.budget:n] = st.patch_idx
    for budget in (1500, 2500, 4000):
        check("fragmented C=%d" % budget, K, V, fr, pa, n, budget, w.recent_frames, w.grid_h, w.grid_w)


@pytest.mark.parametrize("S,n,p", [(50000, 50000, 196), (8192, 8190, 37), (4097, 4097, 64), (130, 129, 16)])
def test_row_counts_and_unaligned_slices(S, n, p):
    # 8 to 64 rows per thread; S not a multiple of 4 loads row runs 4 bytes at a time
    gh, gw = (14, 14) if p == 196 else ((1, 37) if p == 37 else ((8, 8) if p == 64 else (4, 4)))
    st = synth.fresh_cache(11, 1, 2, S, 32, gh, gw, n, synth.F32, synth.RhoSpec(0.0, 0.99))
    K, V, fr, pa = (np.ascontiguousarray(getattr(st, a)[None]) for a in ("K", "V", "frame_idx", "patch_idx"))
    r = 3
    rng = np.random.default_rng(n)
    window = int((fr[0, 0, 0, :n] >= fr[0, 0, 0, n - 1] - r + 1).sum())
    for budget in sorted({window, int(rng.integers(window, n + 1)), n}):
        check("S=%d n=%d C=%d" % (S, n, budget), K, V, fr, pa, n, budget, r, gh, gw)


def test_window_over_budget_is_flagged():
    w = W.TINY
    K, V, fr, pa = cache_of(w)
    got = uniform_pass(K, V, fr, pa, w.n_tokens, 15, w.recent_frames, w.grid_h, w.grid_w)
    assert got.errors == ipv.DEV_RECENT_OVER
    assert np.array_equal(got.keep, np.broadcast_to(np.arange(15), got.keep.shape))
