"""GPU-vs-oracle comparison helpers (test infrastructure).

The acceptance rule itself (score tolerance, near-threshold keep rows) lives
in ``oracle/compare.py``, shared with the benchmark's parity record:
  * scores: |gpu - oracle| <= 1e-3 * |oracle| + 1e-6 for TaR and VaN, against
    the oracle's fp64 values;
  * keep sets: identical per slice, except rows whose oracle score lies within
    1e-3 * max(1, |cut|) of the stage's cut score (reported, and each such flip
    may displace one more row at the VaN boundary);
  * compaction: bit-exact against the oracle's gather with the GPU's keep_idx.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

import oracle
from oracle import compare
from paper_2506_15745_amd import ipv



def to_device(a: np.ndarray, kind: str = "raw", device="cuda:0") -> torch.Tensor:
    """numpy -> device tensor; kind 'bf16' reinterprets uint16 bits as bfloat16."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if kind == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(device)


def to_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
        return t.cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@dataclass
class GpuPass:
    tar: np.ndarray
    van: np.ndarray
    keep: np.ndarray
    K: np.ndarray
    V: np.ndarray
    frame_idx: np.ndarray
    patch_idx: np.ndarray
    errors: int
    pool_size: np.ndarray | None = None


def gpu_compress(K, V, fr, pa, n, budget, alpha, r, gh, gw, cv_tau=None, steps=False) -> GpuPass:
    """Run the pass on cuda:0 through the C ABI. steps=True calls the four
    entry points one by one instead of ipv_compress."""
    kind = "bf16" if K.dtype == np.uint16 else "raw"
    Kd, Vd = to_device(K, kind), to_device(V, kind)
    frd, pad = to_device(fr), to_device(pa)
    B, L, H, S, D = K.shape
    tar = torch.zeros((B, L, H, S), dtype=torch.float32, device="cuda:0")
    van = torch.zeros_like(tar)
    keep = torch.zeros((B, L, H, budget), dtype=torch.int32, device="cuda:0")
    shape = ipv.shape_of(Kd, gh, gw)
    ws = ipv.alloc_workspace(shape, "cuda:0")
    pool = torch.zeros((B, L), dtype=torch.int32, device="cuda:0")
    if steps:
        ipv.ipv_tar_scores(Kd, frd, pad, n, r, tar, ws, gh, gw)
        ipv.ipv_van_scores(Vd, frd, pad, n, cv_tau, van, pool, ws, gh, gw)
        ipv.ipv_select(tar, van, frd, n, budget, alpha, r, keep, ws, gh, gw, head_dim=D, dtype=shape.dtype)
        ipv.ipv_compact(Kd, Vd, frd, pad, n, keep, budget, ws, gh, gw)
    else:
        ipv.ipv_compress(Kd, Vd, frd, pad, n, budget, alpha, r, cv_tau, tar, van, keep, ws, gh, gw)
    torch.cuda.synchronize()
    errors = ipv.ipv_read_device_errors(ws)
    return GpuPass(to_host(tar), to_host(van), to_host(keep), to_host(Kd), to_host(Vd), to_host(frd),
                   to_host(pad), errors, to_host(pool) if steps else None)


def check_scores(g_tar, g_van, o_tar, o_van, n, name=""):
    """Both score columns within the tolerance; returns (TaR, VaN) error records."""
    et = compare.score_errors(g_tar, o_tar, n)
    ev = compare.score_errors(g_van, o_van, n)
    assert et["nonfinite"] == 0 and et["max_tol_frac"] <= 1.0, "%s TaR error %s" % (name, et)
    assert ev["nonfinite"] == 0 and ev["max_tol_frac"] <= 1.0, "%s VaN error %s" % (name, ev)
    return et, ev


def keep_record(g_keep, sel: oracle.Selection, o_tar, o_van):
    """The keep-set rule's counts (compare.keep_stats) for the oracle's selection."""
    return compare.keep_stats(g_keep, sel.keep_idx, sel.cut_tar, sel.cut_van, o_tar, o_van)


def check_keep(g_keep, sel: oracle.Selection, o_tar, o_van):
    """Keep-set rule; returns the near-threshold row count."""
    rec = keep_record(g_keep, sel, o_tar, o_van)
    assert rec["unexplained_rows"] == 0, "rows differ beyond the near-threshold rule: %s" % rec
    return rec["near_threshold_rows"]


def check_ascending(keep, n):
    assert np.all(np.diff(keep, axis=-1) > 0), "keep_idx not strictly ascending"
    assert keep.min() >= 0 and keep.max() < n


def oracle_gather_equal(K0, V0, fr0, pa0, n, keep, got: GpuPass):
    """Compaction parity: the oracle's gather of the ORIGINAL cache with the
    GPU's keep_idx must equal the GPU's compacted rows [0, C) bit for bit."""
    C = keep.shape[-1]
    Ko, Vo, fo, po = oracle.compact(K0, V0, fr0, pa0, n, np.ascontiguousarray(keep))
    assert np.array_equal(got.K[..., :C, :].view(np.uint8), Ko[..., :C, :].view(np.uint8)), "K compaction differs"
    assert np.array_equal(got.V[..., :C, :].view(np.uint8), Vo[..., :C, :].view(np.uint8)), "V compaction differs"
    assert np.array_equal(got.frame_idx[..., :C], fo[..., :C]), "frame_idx compaction differs"
    assert np.array_equal(got.patch_idx[..., :C], po[..., :C]), "patch_idx compaction differs"


def oracle_mode(mode: int) -> int:
    """The library's mode bits as the oracle's (the two define them separately)."""
    pairs = ((ipv.TAR_REVERSE, oracle.TAR_REVERSE), (ipv.VAN_REVERSE, oracle.VAN_REVERSE),
             (ipv.TAR_ADJACENT, oracle.TAR_ADJACENT), (ipv.HEAD_SHARED, oracle.HEAD_SHARED),
             (ipv.UNIFORM_SELECT, oracle.UNIFORM))
    return sum(o for g, o in pairs if mode & g)


def check_uniform_pass(name, K, V, fr, pa, n, budget, r, mode, got: GpuPass):
    """Uniform Select decides from frame ids alone (integer work): the keep
    set must equal the oracle's bit for bit, and the compaction its gather."""
    sel = oracle.select(None, None, fr, n, budget, 0.5, r, mode=oracle_mode(mode))
    check_ascending(got.keep, n)
    assert np.array_equal(got.keep, sel.keep_idx), "%s: Uniform Select keep set differs" % name
    oracle_gather_equal(K, V, fr, pa, n, got.keep, got)
    return 0


def check_pass(name, K, V, fr, pa, n, budget, alpha, r, gh, gw, mode, got: GpuPass, cv_tau=None):
    """Every rule above for one pass in any mode; K, V, fr, pa are the cache
    before the pass. Returns the near-threshold row count."""
    if mode & ipv.UNIFORM_SELECT:
        return check_uniform_pass(name, K, V, fr, pa, n, budget, r, mode, got)
    om = oracle_mode(mode)
    tar64 = oracle.tar_scores(K, fr, pa, n, r, gh, gw, mode=om)
    van64, _ = oracle.van_scores(V, fr, pa, n, gh, gw, cv_tau)
    sel = oracle.select(tar64.astype(np.float32), van64.astype(np.float32), fr, n, budget, alpha, r, mode=om)
    check_scores(got.tar, got.van, tar64, van64, n, name)
    check_ascending(got.keep, n)
    if mode & ipv.HEAD_SHARED:
        # the decision is taken on the heads' summed scores: the rule's distances too
        H = K.shape[2]
        st = np.repeat(tar64.sum(axis=2, keepdims=True), H, axis=2)
        sv = np.repeat(van64.sum(axis=2, keepdims=True), H, axis=2)
        near = check_keep(got.keep, sel, st, sv)
        assert np.array_equal(got.keep, np.repeat(got.keep[:, :, :1], H, axis=2)), "heads kept different rows"
    else:
        near = check_keep(got.keep, sel, tar64, van64)
    oracle_gather_equal(K, V, fr, pa, n, got.keep, got)
    # the oracle's decision on the GPU's own fp32 scores is the GPU's keep set
    sel_g = oracle.select(np.ascontiguousarray(got.tar), np.ascontiguousarray(got.van), fr, n, budget, alpha, r,
                          mode=om)
    assert np.array_equal(sel_g.keep_idx, got.keep), "%s: keep set differs from the oracle's on the GPU scores" % name
    return near
