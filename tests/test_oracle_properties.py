"""Property tests of the oracle over random tiny caches (hypothesis, CPU).

Each property is re-derived here in numpy from the paper's definitions, on
its own: TaR as minus the mean cosine against the recent keys at the same
patch position (Sec. 3.1, TaR equation), VaN as the value norm (Sec. 3.2),
the keep set as the recent window, then the top TaR share among past rows,
then the top VaN rows among the rest, each stage by score then lowest row
(Alg. 1 steps (3)-(5)), and the compaction as a gather in ascending row
order. Keys and values come from a small integer alphabet so that ties,
zero rows and repeated directions occur often.
"""
import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle


@st.composite
def caches(draw):
    gh, gw = draw(st.integers(1, 3)), draw(st.integers(1, 3))
    p = gh * gw
    frames = draw(st.integers(1, 5))
    extra = draw(st.integers(0, p - 1))
    n = frames * p + extra
    H = draw(st.integers(1, 2))
    D = draw(st.sampled_from([4, 8]))
    r = draw(st.integers(1, 3))
    S = n + draw(st.integers(0, 2))
    alphabet = st.integers(-2, 2)
    K = np.array(draw(st.lists(alphabet, min_size=H * S * D, max_size=H * S * D)), np.float32).reshape(1, 1, H, S, D)
    V = np.array(draw(st.lists(alphabet, min_size=H * S * D, max_size=H * S * D)), np.float32).reshape(1, 1, H, S, D)
    rows = np.arange(S)
    fr = np.where(rows < n, rows // p, -1).astype(np.int32)
    pa = np.where(rows < n, rows % p, -1).astype(np.int32)
    fr = np.ascontiguousarray(np.broadcast_to(fr, (1, 1, H, S)))
    pa = np.ascontiguousarray(np.broadcast_to(pa, (1, 1, H, S)))
    last = fr[0, 0, 0, n - 1]
    recent = (fr[0, 0, 0, :n] >= last - r + 1)
    window = int(recent.sum())
    budget = draw(st.integers(max(1, window), n))
    alpha = draw(st.sampled_from([0.0, 0.25, 0.5, 1.0]))
    return dict(K=K, V=V, fr=fr, pa=pa, n=n, r=r, gh=gh, gw=gw, budget=budget, alpha=alpha, recent=recent)


def numpy_tar(K, pa, n, recent):
    """Minus the mean cosine of each past key with the recent keys at its patch."""
    H = K.shape[2]
    out = np.zeros((H, n))
    for h in range(H):
        k = K[0, 0, h, :n].astype(np.float64)
        norm = np.sqrt((k * k).sum(axis=1))
        for x in np.flatnonzero(~recent):
            ys = [y for y in np.flatnonzero(recent) if pa[0, 0, h, y] == pa[0, 0, h, x]]
            if not ys:
                continue
            cos = [0.0 if norm[x] * norm[y] == 0 else float(k[x] @ k[y]) / (norm[x] * norm[y]) for y in ys]
            out[h, x] = -sum(cos) / len(ys)
    return out


def numpy_keep(tar32, van32, recent, budget, alpha):
    """Window, then the TaR share, then VaN, each by (score desc, row asc)."""
    n = len(recent)
    past = [x for x in range(n) if not recent[x]]
    b_t = max(0, math.floor(alpha * budget) - int(recent.sum()))
    b_v = budget - int(recent.sum()) - b_t
    by_tar = sorted(past, key=lambda x: (-float(tar32[x]), x))[:b_t]
    rest = [x for x in past if x not in set(by_tar)]
    by_van = sorted(rest, key=lambda x: (-float(van32[x]), x))[:b_v]
    return sorted(set(np.flatnonzero(recent)) | set(by_tar) | set(by_van))


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(caches())
def test_oracle_scores_equal_their_definitions(c):
    tar = oracle.tar_scores(c["K"], c["fr"], c["pa"], c["n"], c["r"], c["gh"], c["gw"])
    van, _ = oracle.van_scores(c["V"], c["fr"], c["pa"], c["n"], c["gh"], c["gw"])
    want = numpy_tar(c["K"], c["pa"], c["n"], c["recent"])
    np.testing.assert_allclose(tar[0, 0, :, :c["n"]], want, rtol=1e-12, atol=1e-12)
    v = c["V"][0, 0, :, :c["n"]].astype(np.float64)
    np.testing.assert_allclose(van[0, 0, :, :c["n"]], np.sqrt((v * v).sum(axis=2)), rtol=1e-12, atol=0)


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(caches())
def test_oracle_pass_keeps_the_defined_rows_and_gathers_them(c):
    n, C = c["n"], c["budget"]
    K, V, fr, pa = (c[k].copy() for k in ("K", "V", "fr", "pa"))
    tar32, van32, keep = oracle.compress_inplace(K, V, fr, pa, n, C, c["alpha"], c["r"], c["gh"], c["gw"])
    for h in range(K.shape[2]):
        got = keep[0, 0, h]
        assert len(got) == C and np.all(np.diff(got) > 0)
        assert set(np.flatnonzero(c["recent"])) <= set(got.tolist())
        assert got.tolist() == numpy_keep(tar32[0, 0, h, :n], van32[0, 0, h, :n], c["recent"], C, c["alpha"])
        # the compaction is the gather of the kept rows, in order, bit for bit
        assert np.array_equal(K[0, 0, h, :C].view(np.uint32), c["K"][0, 0, h, got].view(np.uint32))
        assert np.array_equal(V[0, 0, h, :C].view(np.uint32), c["V"][0, 0, h, got].view(np.uint32))
        assert np.array_equal(fr[0, 0, h, :C], c["fr"][0, 0, h, got])
        assert np.array_equal(pa[0, 0, h, :C], c["pa"][0, 0, h, got])
