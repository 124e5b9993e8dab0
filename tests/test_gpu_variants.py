"""GPU parity of the variant modes (reversed TaR / VaN stages, consecutive-frame
TaR, head-shared selection), through the C ABI, against the oracle's modes."""
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


def gpu_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, steps=False, cv_tau=None):
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    B, L, H, S, D = K.shape
    tar = torch.zeros((B, L, H, S), dtype=torch.float32, device="cuda:0")
    van = torch.zeros_like(tar)
    keep = torch.zeros((B, L, H, budget), dtype=torch.int32, device="cuda:0")
    shape = ipv.shape_of(Kd, gh, gw)
    ws = ipv.alloc_workspace(shape, "cuda:0")
    if steps:
        ipv.ipv_tar_scores(Kd, frd, pad, n, r, tar, ws, gh, gw, mode=mode)
        ipv.ipv_van_scores(Vd, frd, pad, n, None, van, None, ws, gh, gw)
        ipv.ipv_select(tar, van, frd, n, budget, alpha, r, keep, ws, gh, gw, head_dim=D, dtype=shape.dtype, mode=mode)
        ipv.ipv_compact(Kd, Vd, frd, pad, n, keep, budget, ws, gh, gw)
    else:
        ipv.ipv_compress(Kd, Vd, frd, pad, n, budget, alpha, r, cv_tau, tar, van, keep, ws, gh, gw, mode=mode)
    torch.cuda.synchronize()
    return P.GpuPass(P.to_host(tar), P.to_host(van), P.to_host(keep), P.to_host(Kd), P.to_host(Vd), P.to_host(frd),
                     P.to_host(pad), ipv.ipv_read_device_errors(ws))


def mode_check(name, K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, steps=False, cv_tau=None):
    print("case %s mode=%d alpha=%s n=%d C=%d steps=%s" % (name, mode, alpha, n, budget, steps), flush=True)
    got = gpu_pass(K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, steps, cv_tau)
    assert got.errors == 0
    near = P.check_pass(name, K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, got, cv_tau)
    print("  near-threshold rows %d" % near, flush=True)
    return got


ALL_MODES = [ipv.TAR_REVERSE, ipv.VAN_REVERSE, ipv.TAR_REVERSE | ipv.VAN_REVERSE, ipv.TAR_ADJACENT,
             ipv.HEAD_SHARED, ipv.HEAD_SHARED | ipv.TAR_ADJACENT | ipv.VAN_REVERSE]


@pytest.mark.parametrize("mode", ALL_MODES)
def test_7b_class_modes(mode):
    w = W.SEVEN_B
    mode_check(w.name, *cache_of(w), w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, mode)


@pytest.mark.parametrize("mode", [ipv.TAR_ADJACENT | ipv.TAR_REVERSE, ipv.HEAD_SHARED])
def test_7b_class_modes_through_the_step_entry_points(mode):
    w = W.SEVEN_B
    mode_check(w.name, *cache_of(w), w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, mode,
               steps=True)


@pytest.mark.parametrize("mode", [ipv.TAR_ADJACENT, ipv.HEAD_SHARED | ipv.VAN_REVERSE])
def test_modes_with_layer_adaptive_pooling(mode):
    # VaN is pooled after the sweep (with consecutive-frame TaR: after the adjacent sweep that computes it)
    w = W.POOL
    mode_check(w.name, *cache_of(w), w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, mode,
               cv_tau=w.cv_tau)


@pytest.mark.parametrize("alpha", [1.0, 0.0])
def test_single_stage_reversed(alpha):
    w = W.TINY
    mode_check(w.name, *cache_of(w), w.n_tokens, w.budget, alpha, w.recent_frames, w.grid_h, w.grid_w,
               ipv.TAR_REVERSE | ipv.VAN_REVERSE)


@pytest.mark.parametrize("dtype,D,gh,gw,frames,extra,r", [
    (synth.BF16, 64, 3, 5, 7, 4, 2),      # partial last frame
    (synth.BF16, 32, 2, 2, 40, 3, 3),
    (synth.F32, 256, 2, 3, 12, 5, 1),
    (synth.F32, 128, 5, 3, 11, 0, 2),
    (synth.BF16, 256, 4, 4, 9, 7, 1),
])
def test_adjacent_ragged_shapes(dtype, D, gh, gw, frames, extra, r):
    p = gh * gw
    n = frames * p + extra
    st = synth.fresh_cache(17 + D, 2, 3, n + 5, D, gh, gw, n, dtype, synth.RhoSpec(0.0, 0.99, 0.3))
    K, V, fr, pa = st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None]
    budget = min(n, max(n // 2, r * p + (extra if extra else 0)))
    for mode in (ipv.TAR_ADJACENT, ipv.TAR_ADJACENT | ipv.HEAD_SHARED):
        mode_check("ragged", K, V, fr, pa, n, budget, 0.5, r, gh, gw, mode)


def fragmented_cache(seed, dtype, D, gh, gw, L=2, H=4, first=24, budget=150, later=9, r=2, mode=0):
    """A cache after one oracle pass (each slice keeps its own rows unless
    head-shared) with `later` whole frames appended since: old frames are
    gappy, so a row's previous frame often lacks its position."""
    p = gh * gw
    S = budget + later * p
    st = synth.Stream(seed, L, H, max(S, first * p), D, gh, gw, dtype, synth.RhoSpec(0.0, 0.95, 0.2))
    st.append(first)
    K, V, fr, pa = st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None]
    oracle.compress_inplace(K, V, fr, pa, first * p, budget, 0.5, r, gh, gw, mode=mode)
    st.n = budget
    st.append(later)
    return st


@pytest.mark.parametrize("mode", [ipv.TAR_ADJACENT, ipv.TAR_ADJACENT | ipv.HEAD_SHARED | ipv.TAR_REVERSE])
@pytest.mark.parametrize("dtype,D", [(synth.BF16, 128), (synth.F32, 64)])
def test_adjacent_on_a_fragmented_cache(mode, dtype, D):
    gh, gw, r = 4, 5, 2
    st = fragmented_cache(5, dtype, D, gh, gw, r=r, mode=P.oracle_mode(mode & ipv.HEAD_SHARED))
    n = st.n
    K, V, fr, pa = st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None]
    # gaps: some past row's previous frame lacks its position
    f0, p0 = fr[0, 0, 0, :n], pa[0, 0, 0, :n]
    have = set(zip(f0.tolist(), p0.tolist()))
    assert any((f - 1, q) not in have and f > f0[0] for f, q in zip(f0.tolist(), p0.tolist()))
    mode_check("fragmented", K, V, fr, pa, n, 200, 0.5, r, gh, gw, mode)


def test_adjacent_large_cache_spans_many_walk_chunks():
    # 72B-class row count (32768 rows: 32 chunks of the prev-row walk), few slices
    gh = gw = 14
    p = gh * gw
    n = 32768
    st = synth.fresh_cache(23, 1, 2, n, 128, gh, gw, n, synth.BF16, synth.RhoSpec(0.0, 0.99, 0.3))
    mode_check("long", st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None], n, n // 2, 0.5, 4, gh, gw,
               ipv.TAR_ADJACENT)


def test_adjacent_flags_a_repeated_frame_patch_pair():
    w = W.TINY
    K, V, fr, pa = cache_of(w)
    pa = pa.copy()
    pa[0, 0, 1, 20] = pa[0, 0, 1, 21]  # a pair repeats in slice (0, 0, 1), in a past frame
    with pytest.raises(oracle.OracleError):
        oracle.tar_scores(K, fr, pa, w.n_tokens, w.recent_frames, w.grid_h, w.grid_w, mode=oracle.TAR_ADJACENT)
    got = gpu_pass(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, ipv.TAR_ADJACENT)
    assert got.errors & ipv.DEV_BAD_FRAMES


def test_head_shared_flags_heads_with_different_frames():
    w = W.TINY
    K, V, fr, pa = cache_of(w)
    fr = fr.copy()
    fr[0, 0, 1, :16] = -1  # head 1's first frame carries another id (still non-decreasing)
    got = gpu_pass(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames, w.grid_h, w.grid_w, ipv.HEAD_SHARED)
    assert got.errors & ipv.DEV_BAD_FRAMES
    # the documented fallback: every head keeps rows 0..C-1
    assert np.array_equal(got.keep[0, 0], np.tile(np.arange(w.budget, dtype=np.int32), (2, 1)))


@pytest.mark.parametrize("mode", [0, ipv.TAR_ADJACENT | ipv.TAR_REVERSE])
def test_rows_up_to_the_selection_limit(mode):
    # 64 rows per thread in the selection (n > 32768) and 50 chunks of the prev-row walk
    gh = gw = 16
    n = 50000
    st = synth.fresh_cache(29, 1, 2, n + 3, 64, gh, gw, n, synth.BF16, synth.RhoSpec(0.0, 0.99, 0.3))
    mode_check("n50000", st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None], n, 20000, 0.5, 6, gh, gw,
               mode)


@pytest.mark.parametrize("gh,gw,frames,extra,r,mode,tau", [
    (64, 128, 3, 0, 1, 0, (0.3, 0.5, 0.7)),        # p = 8192, the largest grid: one pooled frame per round
    (64, 128, 3, 0, 1, ipv.TAR_ADJACENT, None),     # the prev-row walk's position table full
    (60, 60, 5, 100, 2, 0, None),                   # p = 3600 with a partial last frame
    (60, 60, 5, 100, 2, ipv.TAR_ADJACENT | ipv.HEAD_SHARED, None),
])
def test_large_patch_grids(gh, gw, frames, extra, r, mode, tau):
    # hundreds of table blocks and sweep column blocks per slice, more positions than rows per walk chunk
    p = gh * gw
    n = frames * p + extra
    st = synth.fresh_cache(31 + p, 1, 2, n + 4, 64, gh, gw, n, synth.BF16, synth.RhoSpec(0.0, 0.99, 0.3))
    budget = max(n // 2, min(n, r * p + extra))
    mode_check("grid%dx%d" % (gh, gw), st.K[None], st.V[None], st.frame_idx[None], st.patch_idx[None], n, budget,
               0.5, r, gh, gw, mode, cv_tau=tau)
