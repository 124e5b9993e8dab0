"""Pins of the oracle's Uniform Select (the frame-sampling baseline of the
KV-compression comparison, appendix on KV cache compression details).

The oracle keeps the recent window and spends the rest of the budget on past
frames at regular intervals: k = ceil(b * q / |P|) frames at ranks
floor(j * q / k), all of their rows in row order, cut at b rows, and if the
taken frames hold fewer than b rows the lowest rows of the other past frames.
These tests hold it to hand-worked cases and to properties that fix the rule
independently of how the oracle computes it.
"""
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "uniform_select.json")


def uniform(frame_idx, budget, r=1, heads=1, mode=oracle.UNIFORM, scores=None):
    fr = np.ascontiguousarray(np.broadcast_to(np.asarray(frame_idx, np.int32), (1, 1, heads, len(frame_idx))))
    n = fr.shape[-1]
    t = v = None
    if scores is not None:
        t = np.ascontiguousarray(np.broadcast_to(scores[0], fr.shape).astype(np.float32))
        v = np.ascontiguousarray(np.broadcast_to(scores[1], fr.shape).astype(np.float32))
    return oracle.select(t, v, fr, n, budget, 0.5, r, mode=mode).keep_idx


def test_golden_cases():
    with open(GOLDEN) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        assert uniform(c["frame_idx"], c["budget"])[0, 0, 0].tolist() == c["keep"], c["derivation"]


def taken_by_condition(q, k):
    """Ranks with a sample point j*q/k in [i, i+1): ceil(i*k/q)*q < (i+1)*k."""
    return {i for i in range(q) if -(-i * k // q) * q < (i + 1) * k}


def frames_of(rows_per_frame, gaps):
    """Frame ids for frames of the given sizes, ids advancing by `gaps`."""
    ids, f = [], 0
    for size, g in zip(rows_per_frame, gaps):
        ids += [f] * size
        f += g
    return ids


@pytest.mark.parametrize("seed", range(40))
def test_whole_frames_at_regular_intervals(seed):
    # equal frames of s rows and a budget of m whole frames: exactly m whole
    # frames, the oldest first, consecutive taken ranks at most one apart in
    # their spacing (floor(q/m) or ceil(q/m) frames)
    rng = np.random.default_rng(seed)
    s, nf, r = int(rng.integers(1, 6)), int(rng.integers(3, 30)), int(rng.integers(1, 4))
    r = min(r, nf - 1)
    q = nf - r
    m = int(rng.integers(0, q + 1))
    fr = np.repeat(np.arange(nf), s)
    keep = uniform(fr, r * s + m * s, r)[0, 0, 0]
    past = keep[keep < q * s]
    assert np.array_equal(keep[len(past):], np.arange(q * s, nf * s))
    taken = sorted(set((past // s).tolist()))
    assert len(taken) == m and len(past) == m * s
    for f in taken:
        assert np.array_equal(past[past // s == f], np.arange(f * s, (f + 1) * s))
    if m:
        assert taken[0] == 0
        steps = np.diff(taken)
        assert steps.size == 0 or (steps.min() >= q // m and steps.max() <= -(-q // m))
        assert set(taken) == taken_by_condition(q, m)


@pytest.mark.parametrize("seed", range(40))
def test_any_budget_on_fragmented_frames(seed):
    # frames of different sizes and skipped ids (a cache after earlier passes)
    rng = np.random.default_rng(100 + seed)
    nf = int(rng.integers(2, 25))
    sizes = rng.integers(1, 7, nf).tolist()
    ids = frames_of(sizes, rng.integers(1, 4, nf).tolist())
    fr = np.asarray(ids)
    n, r = len(ids), int(rng.integers(1, 3))
    r = min(r, nf - 1)
    thr = fr[-1] - r + 1
    n_rec = int((fr >= thr).sum())
    n_past = n - n_rec
    b = int(rng.integers(0, n_past + 1))
    keep = uniform(fr, n_rec + b, r)[0, 0, 0]
    assert len(keep) == n_rec + b and np.all(np.diff(keep) > 0)
    assert np.array_equal(keep[b:], np.arange(n_past, n))
    past = keep[:b]
    if b == 0:
        return
    # ranks of the past frames, and the frames the rule takes
    ranks = np.cumsum(np.r_[1, np.diff(fr[:n_past]) != 0]) - 1
    q = int(ranks[-1]) + 1
    k = -(-b * q // n_past)
    taken = taken_by_condition(q, k)
    in_taken = np.array([ranks[x] in taken for x in range(n_past)])
    rows_taken = np.nonzero(in_taken)[0]
    if len(rows_taken) >= b:
        assert np.array_equal(past, rows_taken[:b])
    else:
        rest = np.nonzero(~in_taken)[0][:b - len(rows_taken)]
        assert np.array_equal(past, np.sort(np.r_[rows_taken, rest]))


def test_scores_are_ignored():
    fr = np.repeat(np.arange(10), 3)
    rng = np.random.default_rng(5)
    with_scores = uniform(fr, 12, 2, scores=(rng.normal(size=30), rng.normal(size=30)))
    assert np.array_equal(with_scores, uniform(fr, 12, 2))


def test_head_shared_gives_every_head_the_same_rows():
    fr = np.repeat(np.arange(9), 4)
    keep = uniform(fr, 14, 1, heads=3, mode=oracle.UNIFORM | oracle.HEAD_SHARED)
    assert np.array_equal(keep[0, 0, 0], keep[0, 0, 1]) and np.array_equal(keep[0, 0, 0], keep[0, 0, 2])
    bad = np.stack([fr, fr, np.r_[fr[:-1], 9]]).astype(np.int32)[None, None]
    with pytest.raises(oracle.OracleError):
        oracle.select(None, None, np.ascontiguousarray(bad), 36, 14, 0.5, 1, mode=oracle.UNIFORM | oracle.HEAD_SHARED)


def test_window_larger_than_budget_is_refused():
    with pytest.raises(oracle.OracleError):
        uniform(np.repeat(np.arange(4), 3), 2, 1)


def test_compress_moves_the_uniform_rows():
    # the whole pass in Uniform mode scores nothing and gathers the picked rows
    rng = np.random.default_rng(9)
    B, L, H, S, D = 1, 2, 2, 40, 8
    K = rng.normal(size=(B, L, H, S, D)).astype(np.float32)
    V = rng.normal(size=(B, L, H, S, D)).astype(np.float32)
    fr = np.ascontiguousarray(np.broadcast_to(np.repeat(np.arange(10, dtype=np.int32), 4), (B, L, H, S)))
    pa = np.ascontiguousarray(np.broadcast_to(np.tile(np.arange(4, dtype=np.int32), 10), (B, L, H, S)))
    keep_sel = oracle.select(None, None, fr, S, 18, 0.5, 2, mode=oracle.UNIFORM).keep_idx
    Kc, Vc, fc, pc = K.copy(), V.copy(), fr.copy(), pa.copy()
    tar, van, keep = oracle.compress_inplace(Kc, Vc, fc, pc, S, 18, 0.5, 2, 2, 2, None, oracle.UNIFORM)
    assert np.array_equal(keep, keep_sel)
    assert not tar.any() and not van.any()
    assert np.array_equal(Kc[..., :18, :], np.take_along_axis(K, keep[..., None].astype(np.int64), axis=3))
    assert np.array_equal(fc[..., :18], np.take_along_axis(fr, keep.astype(np.int64), axis=3))
