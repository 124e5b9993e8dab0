"""Pins of the oracle's continual-compression loop (Algorithm 1): append and
the memory-cap trigger. The loop state is checked against the generator
filling the same stream at once, against closed forms of the row counts, and
against the invariants a compressed cache must satisfy."""
import numpy as np
import pytest

import oracle
import synth

GH, GW, L, H, D = 3, 4, 2, 2, 32
P = GH * GW


def stream(S, seed=11):
    return synth.Stream(seed, L, H, S, D, GH, GW, synth.BF16, synth.RhoSpec(0.0, 0.9), (0.5,))


def frame_rows(src: synth.Stream, f):
    """The rows of frame f of a fully generated stream as [1, L, H, P, D]."""
    return src.K[None, :, :, f * P:(f + 1) * P].copy(), src.V[None, :, :, f * P:(f + 1) * P].copy()


def test_append_frame_by_frame_equals_filling_at_once():
    frames = 6
    full = synth.fresh_cache(11, L, H, frames * P, D, GH, GW, frames * P, synth.BF16, synth.RhoSpec(0.0, 0.9))
    S = frames * P + 5
    K = np.zeros((1, L, H, S, D), np.uint16)
    V = np.zeros_like(K)
    fr = np.full((1, L, H, S), -1, np.int32)
    pa = np.full((1, L, H, S), -1, np.int32)
    n = 0
    for f in range(frames):
        kn, vn = frame_rows(full, f)
        n = oracle.append(K, V, fr, pa, n, kn, vn, f)
        assert n == (f + 1) * P
    assert np.array_equal(K[0, :, :, :n], full.K[:, :, :n]) and np.array_equal(V[0, :, :, :n], full.V[:, :, :n])
    assert np.array_equal(fr[0, :, :, :n], full.frame_idx[:, :, :n])
    assert np.array_equal(pa[0, :, :, :n], full.patch_idx[:, :, :n])
    assert np.all(fr[..., n:] == -1) and np.all(K[..., n:, :] == 0)  # rows past n untouched


def test_append_partial_frame_and_overflow():
    full = synth.fresh_cache(11, L, H, 2 * P, D, GH, GW, 2 * P, synth.BF16, synth.RhoSpec(0.0, 0.9))
    K = np.zeros((1, L, H, P + 5, D), np.uint16)
    V, fr, pa = np.zeros_like(K), np.zeros((1, L, H, P + 5), np.int32), np.zeros((1, L, H, P + 5), np.int32)
    kn, vn = frame_rows(full, 0)
    n = oracle.append(K, V, fr, pa, 0, kn[:, :, :, 5:], vn[:, :, :, 5:], 0, first_patch=5)
    assert n == P - 5 and pa[0, 0, 0, 0] == 5 and pa[0, 1, 1, n - 1] == P - 1
    with pytest.raises(oracle.OracleError):
        oracle.append(K, V, fr, pa, n, *frame_rows(full, 1), 1)  # P rows do not fit in the 10 free rows


@pytest.mark.parametrize("cap,budget,r", [(6 * P, 3 * P, 1), (5 * P, 3 * P + 2, 2), (7 * P, 2 * P, 2)])
def test_ckv_loop_trigger_counts_and_invariants(cap, budget, r):
    frames = 20
    full = synth.fresh_cache(12, L, H, frames * P, D, GH, GW, frames * P, synth.BF16, synth.RhoSpec(0.0, 0.9))
    S = cap + P  # an append may overshoot the cap by less than a frame before the pass runs
    K = np.zeros((1, L, H, S, D), np.uint16)
    V = np.zeros_like(K)
    fr = np.full((1, L, H, S), -1, np.int32)
    pa = np.full((1, L, H, S), -1, np.int32)
    n, passes, expect_n = 0, 0, 0
    for f in range(frames):
        kn, vn = frame_rows(full, f)
        before = (K.copy(), V.copy(), fr.copy(), pa.copy())
        n, out = oracle.ckv_step(K, V, fr, pa, n, kn, vn, f, 0, cap, budget, 0.5, r, GH, GW)
        # closed form of the row count: grow by P, fall back to the budget at the cap
        expect_n += P
        fired = expect_n >= cap
        n_full = expect_n  # rows the pass runs on
        if fired:
            expect_n = budget
        assert n == expect_n and (out is not None) == fired
        if not fired:
            continue
        passes += 1
        tar, van, keep = out
        for idx in np.ndindex(keep.shape[:3]):
            k = keep[idx]
            assert len(k) == budget and np.all(np.diff(k) > 0) and k[-1] < n_full
            # the recent window (the last r frames: frames f-r+1 .. f) is kept
            recent = np.nonzero(np.arange(n_full) >= n_full - r * P)[0]
            assert set(recent.tolist()) <= set(k.tolist())
        # the compacted rows are the appended cache's rows at keep_idx
        Kb = before[0].copy()
        Kb[0, :, :, n_full - P:n_full] = kn[0]
        for idx in np.ndindex(keep.shape[:3]):
            assert np.array_equal(K[idx][:budget], Kb[idx][keep[idx]])
            assert np.all(fr[idx][:budget] <= f) and np.all(np.diff(fr[idx][:budget]) >= 0)
    # closed form of the number of passes
    expect_passes, m = 0, 0
    for _ in range(frames):
        m += P
        if m >= cap:
            expect_passes, m = expect_passes + 1, budget
    assert passes == expect_passes > 0
