"""Pins of the oracle's variant modes (the Tab. 5 ablation rows TaR Reverse and
VaN Reverse, consecutive-frame TaR, and the head-shared reading of the
scores) to hand-worked fixtures, brute force and special cases."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from tests.tiny import slice_cache

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ----------------------------------------------------------------- consecutive-frame TaR

def test_golden_tar_adjacent_and_recent_differ():
    g = load("tar_adjacent_p2.json")
    K, V, fr, pa, n = slice_cache(g["K"], None, g["grid_h"], g["grid_w"], g["frames"], g["patches"])
    adj = oracle.tar_scores(K, fr, pa, n, g["recent_frames"], g["grid_h"], g["grid_w"], mode=oracle.TAR_ADJACENT)
    rec = oracle.tar_scores(K, fr, pa, n, g["recent_frames"], g["grid_h"], g["grid_w"])
    np.testing.assert_allclose(adj[0, 0, 0, :n], g["tar_adjacent"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(rec[0, 0, 0, :n], g["tar_recent"], rtol=0, atol=1e-12)


def test_adjacent_static_frames_score_minus_one_after_the_first():
    # every frame a positive multiple of the first: each past row is a copy of
    # its predecessor (cos 1, score -1), except the first frame, which has none
    rng = np.random.default_rng(3)
    p, f, D = 6, 5, 8
    base = rng.standard_normal((p, D))
    K = np.concatenate([base * (1.0 + t) for t in range(f)])
    Kc, V, fr, pa, n = slice_cache(K, None, 2, 3)
    s = oracle.tar_scores(Kc, fr, pa, n, 1, 2, 3, mode=oracle.TAR_ADJACENT)[0, 0, 0, :n]
    assert np.all(s[:p] == 0.0) and not np.any(np.signbit(s[:p]))
    np.testing.assert_allclose(s[p:(f - 1) * p], -1.0, atol=1e-12)
    assert np.all(s[(f - 1) * p:] == 0.0)


def brute_adjacent(K, frames, patches, n, r):
    """Dictionary walk over (frame, patch) -> row, frames searched downwards."""
    where = {(int(frames[x]), int(patches[x])): x for x in range(n)}
    last = int(frames[n - 1])
    out = np.zeros(n)
    for x in range(n):
        if frames[x] >= last - r + 1:
            continue
        for g in range(int(frames[x]) - 1, -1, -1):
            y = where.get((g, int(patches[x])))
            if y is not None:
                a, b = K[x].astype(np.float64), K[y].astype(np.float64)
                den = np.linalg.norm(a) * np.linalg.norm(b)
                out[x] = 0.0 if den == 0 else -float(a @ b) / den
                break
    return out


@pytest.mark.parametrize("seed", range(5))
def test_adjacent_matches_dictionary_walk_on_fragmented_caches(seed):
    rng = np.random.default_rng(seed)
    gh, gw, f, D, r = 2, 3, 9, 4, 2
    p = gh * gw
    full = rng.standard_normal((f * p, D)).astype(np.float32)
    full[rng.integers(0, f * p, 3)] = 0.0  # zero keys: cos 0
    # a compacted cache: a random subset of the old frames, recent frames whole
    keep = np.sort(np.concatenate([np.flatnonzero(rng.random((f - r) * p) < 0.4), np.arange((f - r) * p, f * p)]))
    frames, patches = keep // p, keep % p
    K, V, fr, pa, n = slice_cache(full[keep], None, gh, gw, frames, patches)
    got = oracle.tar_scores(K, fr, pa, n, r, gh, gw, mode=oracle.TAR_ADJACENT)[0, 0, 0, :n]
    np.testing.assert_allclose(got, brute_adjacent(full[keep], frames, patches, n, r), rtol=1e-12, atol=1e-12)


def test_adjacent_rejects_a_repeated_frame_patch_pair():
    K, V, fr, pa, n = slice_cache([[1, 0], [0, 1], [1, 1], [2, 0]], None, 1, 2, [0, 0, 1, 1], [0, 1, 1, 1])
    oracle.tar_scores(K, fr, pa, n, 1, 1, 2)  # the recent-window score does not look at it
    with pytest.raises(oracle.OracleError):
        oracle.tar_scores(K, fr, pa, n, 1, 1, 2, mode=oracle.TAR_ADJACENT)


# ----------------------------------------------------------------- reversed stages

def brute_bottom(scores, cands, b):
    """The b-subset of cands with the smallest score sum; among equal sums the
    lexicographically smallest sorted index tuple."""
    best, best_key = None, None
    for sub in itertools.combinations(sorted(cands), b):
        key = (sum(scores[i] for i in sub), sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return set(best)


def brute_top(scores, cands, b):
    best, best_key = None, None
    for sub in itertools.combinations(sorted(cands), b):
        key = (-sum(scores[i] for i in sub), sub)
        if best_key is None or key < best_key:
            best, best_key = sub, key
    return set(best)


def arrays(rows, S):
    """[H, S] per-head lists -> [1, 1, H, S] float32."""
    a = np.zeros((1, 1, len(rows), S), np.float32)
    for h, row in enumerate(rows):
        a[0, 0, h, :len(row)] = row
    return a


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("mode", [oracle.TAR_REVERSE, oracle.VAN_REVERSE, oracle.TAR_REVERSE | oracle.VAN_REVERSE])
def test_reversed_stages_equal_brute_force(seed, mode):
    rng = np.random.default_rng(50 + seed)
    p = int(rng.integers(1, 4))
    n = min(p * int(rng.integers(3, 6)), 13)
    frames = [x // p for x in range(n)]
    r = int(rng.integers(1, 3))
    recent = {x for x in range(n) if frames[x] >= frames[-1] - r + 1}
    past = [x for x in range(n) if x not in recent]
    budget = int(rng.integers(len(recent), n + 1))
    alpha = float(rng.choice([0.0, 0.5, 0.75, 1.0]))
    tar = rng.integers(-3, 4, size=n).astype(np.float32)
    van = rng.integers(0, 4, size=n).astype(np.float32)
    fr = np.asarray(frames, np.int32).reshape(1, 1, 1, n)
    s = oracle.select(arrays([tar], n), arrays([van], n), fr, n, budget, alpha, r, mode=mode)
    bt = max(0, math.floor(alpha * budget) - len(recent))
    bv = budget - len(recent) - bt
    pick_t = brute_bottom if mode & oracle.TAR_REVERSE else brute_top
    pick_v = brute_bottom if mode & oracle.VAN_REVERSE else brute_top
    T = pick_t(tar, past, bt) if bt else set()
    Vs = pick_v(van, [x for x in past if x not in T], bv) if bv else set()
    assert list(s.keep_idx[0, 0, 0]) == sorted(recent | T | Vs)


@pytest.mark.parametrize("alpha", [1.0, 0.0])
def test_reversed_single_criterion_is_stable_ascending_argsort(alpha):
    rng = np.random.default_rng(9)
    p, f, r, budget = 8, 10, 2, 40
    n = p * f
    tar = np.round(rng.standard_normal(n), 1).astype(np.float32)
    van = np.round(rng.uniform(0, 3, n), 1).astype(np.float32)
    fr = (np.arange(n) // p).astype(np.int32).reshape(1, 1, 1, n)
    s = oracle.select(arrays([tar], n), arrays([van], n), fr, n, budget, alpha, r,
                      mode=oracle.TAR_REVERSE | oracle.VAN_REVERSE)
    past = np.arange(n - r * p)
    sc = tar if alpha == 1.0 else van
    low = past[np.argsort(sc[past], kind="stable")[: budget - r * p]]
    assert list(s.keep_idx[0, 0, 0]) == sorted(set(low.tolist()) | set(range(n - r * p, n)))


# ----------------------------------------------------------------- head-shared selection

@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("mode", [0, oracle.TAR_REVERSE | oracle.VAN_REVERSE])
def test_head_shared_equals_brute_force_on_the_head_sum(seed, mode):
    # integer scores: the fp32 head sums are exact
    rng = np.random.default_rng(200 + seed)
    H, p = 3, 2
    n = 12
    frames = [x // p for x in range(n)]
    r = 1
    recent = {x for x in range(n) if frames[x] >= frames[-1] - r + 1}
    past = [x for x in range(n) if x not in recent]
    budget = int(rng.integers(len(recent) + 1, n))
    alpha = 0.5
    tar = rng.integers(-2, 3, size=(H, n)).astype(np.float32)
    van = rng.integers(0, 3, size=(H, n)).astype(np.float32)
    fr = np.tile(np.asarray(frames, np.int32), (1, 1, H, 1))
    s = oracle.select(arrays(tar, n), arrays(van, n), fr, n, budget, alpha, r, mode=mode | oracle.HEAD_SHARED)
    st, sv = tar.sum(0), van.sum(0)
    bt = max(0, math.floor(alpha * budget) - len(recent))
    bv = budget - len(recent) - bt
    pick_t = brute_bottom if mode & oracle.TAR_REVERSE else brute_top
    pick_v = brute_bottom if mode & oracle.VAN_REVERSE else brute_top
    T = pick_t(st, past, bt) if bt else set()
    Vs = pick_v(sv, [x for x in past if x not in T], bv) if bv else set()
    want = sorted(recent | T | Vs)
    for h in range(H):
        assert list(s.keep_idx[0, 0, h]) == want


def test_head_shared_with_one_head_is_per_head():
    rng = np.random.default_rng(5)
    B, L, n, p = 2, 3, 60, 6
    tar = rng.standard_normal((B, L, 1, n)).astype(np.float32)
    van = rng.uniform(0, 2, (B, L, 1, n)).astype(np.float32)
    fr = np.broadcast_to((np.arange(n) // p).astype(np.int32), (B, L, 1, n)).copy()
    a = oracle.select(tar, van, fr, n, 30, 0.5, 2)
    b = oracle.select(tar, van, fr, n, 30, 0.5, 2, mode=oracle.HEAD_SHARED)
    assert np.array_equal(a.keep_idx, b.keep_idx)


def test_head_shared_sums_heads_in_fp32_in_head_order():
    # row 0: 2^24 + 1 rounds (to even) to 2^24 in fp32, and + 1 again to 2^24;
    # row 1: 2^24 + 0 + 2 = 2^24 + 2. An exact, wider or reordered sum ties the
    # two rows at 2^24 + 2 and would keep row 0
    n, p = 4, 1
    big = np.float32(2 ** 24)
    tar = np.array([[big, big, 0, 0], [1, 0, 0, 0], [1, 2, 0, 0]], np.float32)
    van = np.zeros((3, n), np.float32)
    fr = np.tile(np.arange(n, dtype=np.int32), (1, 1, 3, 1))
    s = oracle.select(arrays(tar, n), arrays(van, n), fr, n, 2, 1.0, 1, mode=oracle.HEAD_SHARED)
    assert list(s.keep_idx[0, 0, 0]) == [1, 3]


def test_head_shared_rejects_heads_with_different_frames():
    n = 8
    fr = np.tile(np.arange(n, dtype=np.int32) // 2, (1, 1, 2, 1))
    fr[0, 0, 1, 3] = 2  # head 1 holds a different frame at row 3 (still non-decreasing)
    z = np.zeros((1, 1, 2, n), np.float32)
    oracle.select(z, z, fr, n, 4, 0.5, 1)  # per head: fine
    with pytest.raises(oracle.OracleError):
        oracle.select(z, z, fr, n, 4, 0.5, 1, mode=oracle.HEAD_SHARED)


def test_unknown_mode_bits_are_rejected():
    z = np.zeros((1, 1, 1, 8), np.float32)
    fr = (np.arange(8, dtype=np.int32) // 2).reshape(1, 1, 1, 8)
    with pytest.raises(oracle.OracleError):
        oracle.select(z, z, fr, 8, 4, 0.5, 1, mode=32)
