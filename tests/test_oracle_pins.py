"""Pins of the CPU oracle to facts that do not come from the oracle itself:
hand-worked fixtures (tests/golden), closed forms, brute force over all
subsets, library routines for the special cases, and invariants of the
method. Each pin is chosen so that a plausible slip in the oracle (a dropped
term, a sign, a wrong index or operand, an off-by-one window) fails it.
"""
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


def tar_of(K, fr, pa, n, r, gh, gw):
    return oracle.tar_scores(K, fr, pa, n, r, gh, gw)[0, 0, 0, :n]


# ----------------------------------------------------------------- TaR (Sec. 3.1)

def test_golden_tar_p2_r1():
    g = load("tar_select_p2_r1.json")
    K, V, fr, pa, n = slice_cache(g["K"], g["V"], g["grid_h"], g["grid_w"])
    np.testing.assert_allclose(tar_of(K, fr, pa, n, g["recent_frames"], 1, 2), g["tar"], rtol=0, atol=1e-15)


def test_golden_tar_r2_averages_all_recent_frames():
    g = load("tar_r2_p1.json")
    K, V, fr, pa, n = slice_cache(g["K"], None, g["grid_h"], g["grid_w"])
    np.testing.assert_allclose(tar_of(K, fr, pa, n, g["recent_frames"], 1, 1), g["tar"], rtol=0, atol=1e-15)


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_identical_frames_give_minus_one(dtype):
    # a static video: every frame repeats the same keys -> full redundancy
    rng = np.random.default_rng(3)
    p, f, D = 6, 5, 16
    frame = rng.integers(-4, 5, size=(p, D)).astype(np.float32)
    frame[frame.sum(1) == 0, 0] = 1.0  # no zero rows
    K, V, fr, pa, n = slice_cache(np.tile(frame, (f, 1)), grid_h=2, grid_w=3)
    if dtype == np.uint16:  # small integers are exact in bf16
        K = (K.view(np.uint32) >> 16).astype(np.uint16)
    t = tar_of(K, fr, pa, n, 2, 2, 3)
    np.testing.assert_allclose(t[: (f - 2) * p], -1.0, atol=1e-15)
    assert np.all(t[(f - 2) * p:] == 0.0)


def test_negated_past_gives_plus_one_and_orthogonal_gives_positive_zero():
    D = 8
    e = np.eye(D, dtype=np.float32)
    # p=2, frames: 0 = (-e0, e3), 1 = recent (e0, e1) ; patch 1's past key e3 is orthogonal to e1
    K, V, fr, pa, n = slice_cache([-2 * e[0], e[3], 5 * e[0], e[1]], grid_h=1, grid_w=2)
    t = tar_of(K, fr, pa, n, 1, 1, 2)
    assert t[0] == 1.0
    assert t[1] == 0.0 and not math.copysign(1.0, t[1]) < 0  # canonical +0.0


def test_positive_rescaling_leaves_tar_unchanged():
    rng = np.random.default_rng(5)
    p, f, D = 4, 6, 32
    k = rng.standard_normal((p * f, D)).astype(np.float32)
    K, V, fr, pa, n = slice_cache(k, grid_h=2, grid_w=2)
    base = tar_of(K, fr, pa, n, 3, 2, 2)
    K2 = K.copy()
    K2[0, 0, 0, :n] *= rng.uniform(0.25, 4.0, size=(n, 1)).astype(np.float32)
    np.testing.assert_allclose(tar_of(K2, fr, pa, n, 3, 2, 2), base, rtol=1e-6, atol=1e-6)
    # a negative factor on one recent key flips that key's contribution only
    K3 = K.copy()
    K3[0, 0, 0, n - 1] *= -1.0  # last frame, patch 3; r=1 -> row x at patch 3 flips sign
    t3 = tar_of(K3, fr, pa, n, 1, 2, 2)
    b1 = tar_of(K, fr, pa, n, 1, 2, 2)
    past3 = [x for x in range(n - p) if x % p == 3]
    np.testing.assert_allclose(t3[past3], -b1[past3], atol=1e-12)


def test_tar_matches_pairwise_cosines_brute_force():
    # independent per-pair evaluation on a tiny random cache, rows in frame order
    rng = np.random.default_rng(11)
    p, f, D, r = 3, 5, 8, 2
    k = rng.standard_normal((p * f, D))
    K, V, fr, pa, n = slice_cache(k, grid_h=1, grid_w=3)
    t = tar_of(K, fr, pa, n, r, 1, 3)
    k32 = K[0, 0, 0, :n].astype(np.float64)
    for x in range((f - r) * p):
        q = x % p
        ys = [(f - r + j) * p + q for j in range(r)]
        cs = [k32[x] @ k32[y] / (np.linalg.norm(k32[x]) * np.linalg.norm(k32[y])) for y in ys]
        assert abs(t[x] - (-sum(cs) / r)) < 1e-12


def test_partial_last_frame_patch_without_recent_key_scores_zero():
    # p=4, r=1, last frame holds only patches 0 and 1
    rng = np.random.default_rng(2)
    k = rng.standard_normal((4 * 3 + 2, 8))
    K, V, fr, pa, n = slice_cache(k, grid_h=2, grid_w=2)
    t = tar_of(K, fr, pa, n, 1, 2, 2)
    past = np.arange(12)
    assert np.all(t[past[past % 4 >= 2]] == 0.0)
    assert np.all(t[past[past % 4 < 2]] != 0.0)
    # with r=2 the window is frames 2 and 3: patches 2,3 average one key, 0,1 two
    t2 = tar_of(K, fr, pa, n, 2, 2, 2)
    k64 = K[0, 0, 0, :n].astype(np.float64)
    cosf = lambda a, b: a @ b / np.linalg.norm(a) / np.linalg.norm(b)
    assert abs(t2[2] - (-cosf(k64[2], k64[10]))) < 1e-12
    assert abs(t2[1] - (-(cosf(k64[1], k64[9]) + cosf(k64[1], k64[13])) / 2)) < 1e-12


def test_zero_key_has_zero_cosine():
    D = 4
    K, V, fr, pa, n = slice_cache([[0, 0, 0, 0], [1, 2, 3, 4], [0, 0, 0, 0], [1, 0, 0, 0]], grid_h=1, grid_w=2)
    # row0 is zero (cos 0); row1's recent partner row3 is (1,0,0,0): cos = 1/sqrt(30)
    t = tar_of(K, fr, pa, n, 1, 1, 2)
    assert t[0] == 0.0
    # patch 0's recent key (row 2) is zero as well; patch 1: row1 vs row3 -> different patches
    K2, _, fr2, pa2, n2 = slice_cache([[1, 2, 3, 4], [0, 0, 0, 0], [1, 0, 0, 0], [0, 0, 0, 0]], grid_h=1, grid_w=2)
    t2 = tar_of(K2, fr2, pa2, n2, 1, 1, 2)
    assert abs(t2[0] - (-1 / math.sqrt(30))) < 1e-15 and t2[1] == 0.0


# ----------------------------------------------------------------- VaN (Sec. 3.2)

def van_of(V, fr, pa, n, gh, gw, tau=None):
    v, pool = oracle.van_scores(V, fr, pa, n, gh, gw, tau)
    return v[0, 0, 0, :n], pool


def test_van_closed_forms():
    D = 64
    rows = np.zeros((4, D), np.float32)
    rows[0, 17] = -3.5            # |c e_k| = |c|
    rows[1, :] = 1.0              # all-ones: sqrt(64) = 8
    rows[2, :2] = (3.0, 4.0)      # 3-4-5
    K, V, fr, pa, n = slice_cache(np.ones((4, D)), rows, grid_h=2, grid_w=2)
    v, pool = van_of(V, fr, pa, n, 2, 2)
    assert list(v) == [3.5, 8.0, 5.0, 0.0] and pool[0, 0] == 1


def test_golden_van_p2_r1():
    g = load("tar_select_p2_r1.json")
    K, V, fr, pa, n = slice_cache(g["K"], g["V"], 1, 2)
    v, _ = van_of(V, fr, pa, n, 1, 2)
    assert list(v) == g["van"]


@pytest.mark.parametrize("case", range(3))
def test_golden_pool_3x3(case):
    g = load("pool_3x3.json")
    c = g["cases"][case]
    K, V, fr, pa, n = slice_cache(np.ones((9, 1)), g["V"], 3, 3, frames=[0] * 9)
    v, pool = van_of(V, fr, pa, n, 3, 3, c["tau"])
    assert pool[0, 0] == c["pool_size"]
    np.testing.assert_allclose(v, c["van"], rtol=0, atol=1e-14)


def test_constant_field_pools_to_itself_with_k7():
    D = 16
    rows = np.zeros((2 * 9, D), np.float32)
    rows[:, 3] = 2.5
    K, V, fr, pa, n = slice_cache(np.ones((18, D)), rows, 3, 3)
    v, pool = van_of(V, fr, pa, n, 3, 3, (0.3, 0.5, 0.7))
    assert pool[0, 0] == 7  # CV = 0
    assert np.all(v == 2.5)


def test_spike_pools_over_present_in_grid_cells():
    # a single spike of height h on a 4x4 grid: CV = sqrt(15); tau -> k = 3
    h = 16.0
    rows = np.zeros((16, 1), np.float32)
    spike = 1 * 4 + 1  # cell (1,1)
    rows[spike, 0] = h
    K, V, fr, pa, n = slice_cache(np.ones((16, 1)), rows, 4, 4, frames=[0] * 16)
    v, pool = van_of(V, fr, pa, n, 4, 4, (1.0, 2.0, 10.0))
    assert pool[0, 0] == 3
    for c in range(16):
        i, j = divmod(c, 4)
        cells = [(a, b) for a in range(i - 1, i + 2) for b in range(j - 1, j + 2) if 0 <= a < 4 and 0 <= b < 4]
        want = h / len(cells) if (1, 1) in cells else 0.0
        assert abs(v[c] - want) < 1e-14, c
    # corner (0,0) sees a 4-cell window, edge (0,1) 6 cells, interior (1,1) 9 cells
    assert v[0] == h / 4 and v[1] == h / 6 and v[5] == h / 9


def test_pool_stays_inside_frame_and_skips_missing_cells():
    # frame 0 constant 1 on a 2x2 grid, frame 1 has cells 0,1,2 only (values 1,2,3)
    rows = np.array([[1], [1], [1], [1], [1], [2], [3]], np.float32)
    K, V, fr, pa, n = slice_cache(np.ones((7, 1)), rows, 2, 2, frames=[0, 0, 0, 0, 1, 1, 1],
                                  patches=[0, 1, 2, 3, 0, 1, 2])
    v, pool = van_of(V, fr, pa, n, 2, 2, (10.0, 11.0, 12.0))  # CV < tau1 -> k=7
    assert pool[0, 0] == 7
    np.testing.assert_allclose(v, [1, 1, 1, 1, 2, 2, 2], atol=1e-15)


@pytest.mark.parametrize("tau,k", [((0.4, 0.5, 0.6), 3), ((0.4, 0.51, 0.6), 5), ((0.5, 0.6, 0.7), 5),
                                   ((0.51, 0.6, 0.7), 7), ((0.1, 0.2, 0.5), 1)])
def test_cv_of_one_and_three_is_half(tau, k):
    # norms 1 and 3: mean 2, population std 1 -> CV = 0.5; the bands are [tau_i, tau_i+1)
    rows = np.array([[1.0], [3.0]], np.float32)
    K, V, fr, pa, n = slice_cache(np.ones((2, 1)), rows, 1, 2, frames=[0, 0])
    _, pool = van_of(V, fr, pa, n, 1, 2, tau)
    assert pool[0, 0] == k


def test_cv_spans_all_heads_of_a_layer():
    # head 0 all 1, head 1 all 3 -> the layer's CV is 0.5 although each head alone has CV 0
    Vc = np.zeros((1, 1, 2, 2, 1), np.float32)
    Vc[0, 0, 0] = 1.0
    Vc[0, 0, 1] = 3.0
    fr = np.zeros((1, 1, 2, 2), np.int32)
    pa = np.tile(np.arange(2, dtype=np.int32), (1, 1, 2, 1))
    _, pool = oracle.van_scores(Vc, fr, pa, 2, 1, 2, (0.4, 0.45, 0.6))
    assert pool[0, 0] == 3


# ----------------------------------------------------------------- selection (Alg. 1 (3)-(5))

def brute_top(scores, cands, b):
    """The b-subset of cands with the largest score sum; among equal sums the
    lexicographically smallest sorted index tuple (lowest index wins ties)."""
    best, best_key = None, None
    for sub in itertools.combinations(sorted(cands), b):
        key = (sum(scores[i] for i in sub), tuple(-i for i in sub))
        if best_key is None or key > best_key:
            best, best_key = sub, key
    return set(best)


def sel_slice(tar, van, fr, n, budget, alpha, r):
    S = len(tar)
    t = np.zeros((1, 1, 1, S), np.float32)
    v = np.zeros((1, 1, 1, S), np.float32)
    t[0, 0, 0] = tar
    v[0, 0, 0] = van
    f = np.asarray(fr, np.int32).reshape(1, 1, 1, S)
    return oracle.select(t, v, f, n, budget, alpha, r)


def test_golden_select():
    g = load("tar_select_p2_r1.json")
    fr = [x // 2 for x in range(6)]
    for a, keep in g["keep"].items():
        s = sel_slice(np.float32(g["tar"]), np.float32(g["van"]), fr, 6, g["budget"], float(a), 1)
        assert list(s.keep_idx[0, 0, 0]) == keep, a


@pytest.mark.parametrize("seed", range(12))
def test_select_equals_brute_force_over_all_subsets(seed):
    rng = np.random.default_rng(seed)
    p = int(rng.integers(1, 4))
    f = int(rng.integers(3, 6))
    n = min(p * f, 14)
    fr = [x // p for x in range(n)]
    r = int(rng.integers(1, 3))
    recent = {x for x in range(n) if fr[x] >= fr[-1] - r + 1}
    past = [x for x in range(n) if x not in recent]
    budget = int(rng.integers(len(recent), n + 1))
    alpha = float(rng.choice([0.0, 0.25, 0.5, 0.75, 1.0]))
    # integer-valued scores with many ties; sums are exact
    tar = rng.integers(-3, 4, size=n).astype(np.float32)
    van = rng.integers(0, 4, size=n).astype(np.float32)
    s = sel_slice(tar, van, fr, n, budget, alpha, r)
    bt = max(0, math.floor(alpha * budget) - len(recent))
    bv = budget - len(recent) - bt
    T = brute_top(tar, past, bt) if bt else set()
    Vs = brute_top(van, [x for x in past if x not in T], bv) if bv else set()
    assert list(s.keep_idx[0, 0, 0]) == sorted(recent | T | Vs)
    assert (s.b_tar[0, 0, 0], s.b_van[0, 0, 0], s.n_recent[0, 0, 0]) == (bt, bv, len(recent))


@pytest.mark.parametrize("seed", range(6))
def test_select_pairwise_characterisation(seed):
    # O(N^2) check at a size brute force cannot reach: in each stage every kept
    # candidate beats every dropped one, ties broken by the lower index
    rng = np.random.default_rng(100 + seed)
    p, f, r = 16, 12, 2
    n = p * f
    fr = [x // p for x in range(n)]
    tar = rng.integers(-20, 20, size=n).astype(np.float32) / 8
    van = rng.integers(0, 30, size=n).astype(np.float32) / 4
    tar[::7] = -0.0  # -0.0 must tie with +0.0
    tar[1::7] = 0.0
    budget, alpha = 100, 0.5
    s = sel_slice(tar, van, fr, n, budget, alpha, r)
    keep = set(s.keep_idx[0, 0, 0].tolist())
    recent = set(range(n - r * p, n))
    past = [x for x in range(n) if x not in recent]
    bt = int(s.b_tar[0, 0, 0])
    assert recent <= keep and len(keep) == budget
    assert list(s.keep_idx[0, 0, 0]) == sorted(keep)
    # reconstruct stage T as the best bt by (score, -index) and check the order property
    beats = lambda sc, a, b: sc[a] > sc[b] or (sc[a] == sc[b] and a < b)
    T = set(sorted(past, key=lambda x: (-tar[x], x))[:bt])
    assert T <= keep
    for a in T:
        for b in past:
            if b not in T:
                assert beats(tar, a, b)
    rest = [x for x in past if x not in T]
    Vk = [x for x in rest if x in keep]
    for a in Vk:
        for b in rest:
            if b not in keep:
                assert beats(van, a, b)


@pytest.mark.parametrize("alpha", [1.0, 0.0])
def test_single_criterion_special_cases_reduce_to_stable_argsort(alpha):
    # alpha=1 is the TaR-only compression of Sec. 3.1, alpha=0 VaN top-k plus the
    # recent window (Sec. 3.2); numpy's stable argsort of -score is a top-k with
    # lowest-index ties
    rng = np.random.default_rng(7)
    p, f, r = 8, 10, 2
    n = p * f
    fr = [x // p for x in range(n)]
    tar = np.round(rng.standard_normal(n), 1).astype(np.float32)
    van = np.round(rng.uniform(0, 3, n), 1).astype(np.float32)
    budget = 40
    s = sel_slice(tar, van, fr, n, budget, alpha, r)
    past = np.arange(n - r * p)
    sc = tar if alpha == 1.0 else van
    top = past[np.argsort(-sc[past], kind="stable")[: budget - r * p]]
    want = sorted(set(top.tolist()) | set(range(n - r * p, n)))
    assert list(s.keep_idx[0, 0, 0]) == want


def test_budget_equal_to_recent_window_keeps_only_it():
    fr = [x // 4 for x in range(20)]
    s = sel_slice(np.arange(20, dtype=np.float32), np.arange(20, dtype=np.float32), fr, 20, 8, 0.5, 2)
    assert list(s.keep_idx[0, 0, 0]) == list(range(12, 20))


def test_select_rejects_bad_inputs():
    fr = [x // 4 for x in range(20)]
    ones = np.ones(20, np.float32)
    with pytest.raises(oracle.OracleError):  # budget smaller than the recent window
        sel_slice(ones, ones, fr, 20, 7, 0.5, 2)
    bad = ones.copy()
    bad[0] = np.nan
    with pytest.raises(oracle.OracleError):
        sel_slice(bad, ones, fr, 20, 10, 0.5, 2)
    with pytest.raises(oracle.OracleError):  # frame ids must not decrease
        sel_slice(ones, ones, fr[::-1], 20, 10, 0.5, 2)


# ----------------------------------------------------------------- compaction (Alg. 1 (5))

@pytest.mark.parametrize("dtype", [np.uint16, np.float32])
def test_compaction_is_numpy_fancy_index_gather(dtype):
    rng = np.random.default_rng(4)
    B, L, H, S, D, n, C = 2, 2, 3, 40, 8, 36, 17
    K = rng.integers(0, 2**16, size=(B, L, H, S, D)).astype(np.uint16)
    V = rng.integers(0, 2**16, size=(B, L, H, S, D)).astype(np.uint16)
    if dtype == np.float32:
        K = rng.standard_normal((B, L, H, S, D)).astype(np.float32)
        V = rng.standard_normal((B, L, H, S, D)).astype(np.float32)
    fr = rng.integers(0, 9, size=(B, L, H, S)).astype(np.int32)
    pa = rng.integers(0, 9, size=(B, L, H, S)).astype(np.int32)
    keep = np.sort(np.stack([rng.choice(n, C, replace=False) for _ in range(B * L * H)]), -1)
    keep = keep.reshape(B, L, H, C).astype(np.int32)
    K2, V2, f2, p2 = oracle.compact(K, V, fr, pa, n, keep)
    for idx in np.ndindex(B, L, H):
        k = keep[idx]
        assert np.array_equal(K2[idx][:C].view(np.uint8), K[idx][k].view(np.uint8))
        assert np.array_equal(V2[idx][:C].view(np.uint8), V[idx][k].view(np.uint8))
        assert np.array_equal(f2[idx][:C], fr[idx][k]) and np.array_equal(p2[idx][:C], pa[idx][k])
        assert np.array_equal(K2[idx][C:], K[idx][C:])  # rows past the budget untouched


# ----------------------------------------------------------------- whole pass invariants

def test_whole_pass_invariants_on_tiny_workload():
    from synth.workloads import TINY as w
    st = synth.fresh_cache(w.seeds[0], w.layers, w.kv_heads, w.capacity, w.head_dim, w.grid_h, w.grid_w,
                           w.n_tokens, w.dtype, w.rho_specs[0])
    K, V, fr, pa = st.K[None].copy(), st.V[None].copy(), st.frame_idx[None].copy(), st.patch_idx[None].copy()
    K0, V0, fr0 = K.copy(), V.copy(), fr.copy()
    tar, van, keep = oracle.compress_inplace(K, V, fr, pa, w.n_tokens, w.budget, 0.5, w.recent_frames,
                                             w.grid_h, w.grid_w)
    p = w.p
    for idx in np.ndindex(keep.shape[:3]):
        k = keep[idx]
        assert len(k) == w.budget and np.all(np.diff(k) > 0)
        assert set(range(w.n_tokens - w.recent_frames * p, w.n_tokens)) <= set(k.tolist())
        assert np.array_equal(K[idx][: w.budget], K0[idx][k]) and np.array_equal(V[idx][: w.budget], V0[idx][k])
        assert np.array_equal(fr[idx][: w.budget], fr0[idx][k])


def test_generator_ar1_lag_correlation():
    # statistical check of the input generator (not of the method): for a
    # patch with coefficient rho, the correlation of keys one frame apart is rho
    spec = synth.RhoSpec(0.0, 0.99)
    st = synth.fresh_cache(9, 1, 1, 64 * 200, 64, 8, 8, 64 * 200, synth.F32, spec)
    k = st.K[0, 0].reshape(200, 64, 64).astype(np.float64)
    for q in (0, 17, 40):
        a, b = k[1:, q, :].ravel(), k[:-1, q, :].ravel()
        assert abs(np.corrcoef(a, b)[0, 1] - st.rho[q]) < 0.05
    z = synth.normals(1, 99, 200000)
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1) < 0.01


def test_acceptance_rule_counts():
    # the comparison rule of oracle/compare.py on a hand-made slice: cut scores
    # 0.5 (TaR) and 2.0 (VaN); row 3 sits 4e-4 from the TaR cut, so swapping it
    # for row 4 is a near-threshold flip, and row 9 (VaN score far from its cut)
    # may move once per TaR flip
    from oracle import compare
    o_tar = np.zeros((1, 12))
    o_van = np.zeros((1, 12))
    o_tar[0, 3], o_tar[0, 4] = 0.5004, 0.5
    o_van[0, 9], o_van[0, 8] = 9.0, 2.0
    o_keep = np.array([[0, 3, 8, 11]])
    cut_t, cut_v = np.array([0.5]), np.array([2.0])
    same = compare.keep_stats(o_keep, o_keep, cut_t, cut_v, o_tar, o_van)
    assert same["slices_differing"] == 0 and same["unexplained_rows"] == 0
    flip = compare.keep_stats(np.array([[0, 4, 8, 11]]), o_keep, cut_t, cut_v, o_tar, o_van)
    assert flip["mismatched_rows"] == 2 and flip["near_threshold_rows"] == 2 and flip["unexplained_rows"] == 0
    # a flip that also displaced a VaN row: one extra row is allowed per TaR flip
    disp = compare.keep_stats(np.array([[0, 4, 9, 11]]), o_keep, cut_t, cut_v, o_tar, o_van)
    assert disp["unexplained_rows"] == 0 and disp["mismatched_rows"] == 4
    # a row far from both cuts with no flip to explain it
    wrong = compare.keep_stats(np.array([[0, 3, 9, 11]]), o_keep, cut_t, cut_v, o_tar, o_van)
    assert wrong["unexplained_rows"] == 1 and wrong["worst_slice"] == [0]
    e = compare.score_errors(np.array([[1.0005, 0.0]], np.float32), np.array([[1.0, 2e-7]]), 2)
    assert e["max_tol_frac"] <= 1.0 and e["max_abs"] > 4e-4
    assert compare.score_errors(np.array([[1.0, 3e-6]]), np.array([[1.0, 0.0]]), 2)["max_tol_frac"] > 1.0
