"""Acceptance rule of a GPU pass against the oracle -- TEST INFRASTRUCTURE.

Used by the test suite and the benchmark's CPU-baseline leg only; plain numpy
on results already copied to the host, no GPU and no library calls.

  * scores: |gpu - oracle| <= 1e-3 * |oracle| + 1e-6, TaR and VaN alike,
    against the oracle's fp64 values;
  * keep sets: identical per slice, except rows whose oracle score lies within
    1e-3 * max(1, |cut|) of the stage's cut (the score of the stage's last
    pick); each such row that flips at the TaR cut may displace one more row
    at the VaN boundary (the VaN stage ranks the rows TaR left);
  * compaction: bit-exact (checked by the callers).
"""
from __future__ import annotations

import math

import numpy as np

REL = 1e-3
ABS = 1e-6
NEAR = 1e-3


def score_errors(gpu: np.ndarray, ref: np.ndarray, n: int) -> dict:
    """Largest absolute error over rows [0, n) and the largest share of the
    tolerance used (<= 1 passes)."""
    g = gpu[..., :n].astype(np.float64)
    o = ref[..., :n]
    err = np.abs(g - o)
    frac = err / (REL * np.abs(o) + ABS)
    bad = ~np.isfinite(frac)
    return {"max_abs": float(err.max(initial=0.0)), "max_tol_frac": float(frac.max(initial=0.0)),
            "nonfinite": int(bad.sum())}


def keep_stats(g_keep: np.ndarray, o_keep: np.ndarray, cut_tar: np.ndarray, cut_van: np.ndarray,
               o_tar: np.ndarray, o_van: np.ndarray) -> dict:
    """Per-slice comparison of keep sets [..., C]. o_tar / o_van are the oracle
    scores the distances are measured on (per head, or the head sums for a
    head-shared selection). Returns totals: slices compared and differing,
    rows in the symmetric differences, near-threshold rows among them, and
    rows the rule does not explain (0 passes)."""
    lead = g_keep.shape[:-1]
    differ = np.any(g_keep != o_keep, axis=-1)
    out = {"slices": int(np.prod(lead)), "slices_differing": int(differ.sum()), "mismatched_rows": 0,
           "near_threshold_rows": 0, "unexplained_rows": 0, "worst_slice": None}
    for idx in zip(*np.nonzero(differ)):
        g, o = set(g_keep[idx].tolist()), set(o_keep[idx].tolist())
        diff = g ^ o
        ct, cv = float(cut_tar[idx]), float(cut_van[idx])
        near_t = {x for x in diff if not math.isnan(ct) and abs(o_tar[idx][x] - ct) <= NEAR * max(1.0, abs(ct))}
        near_v = {x for x in diff if not math.isnan(cv) and abs(o_van[idx][x] - cv) <= NEAR * max(1.0, abs(cv))}
        rest = diff - near_t - near_v
        unexplained = max(0, len(rest) - len(near_t))
        out["mismatched_rows"] += len(diff)
        out["near_threshold_rows"] += len(near_t | near_v)
        out["unexplained_rows"] += unexplained
        if unexplained and out["worst_slice"] is None:
            out["worst_slice"] = [int(i) for i in idx]
    return out


def merge(a: dict | None, b: dict) -> dict:
    """Sum two keep_stats / score_errors records (maxima for the error fields)."""
    if a is None:
        return dict(b)
    out = dict(a)
    for k, v in b.items():
        if k in ("max_abs", "max_tol_frac"):
            out[k] = max(a[k], v)
        elif k == "worst_slice":
            out[k] = a[k] if a[k] is not None else v
        else:
            out[k] = a[k] + v
    return out
