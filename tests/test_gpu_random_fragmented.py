"""Seeded random configurations on fragmented caches: each stream's cache is
the state the oracle's continual-compression loop (Algorithm 1) leaves after
a random number of frames, so most of its past rows were moved by earlier
passes and sit off their frame-plane positions, with whole recent frames
appended since (and sometimes a partial frame after them). One pass with its
own random budget, TaR share, variant mode and pooling then runs on the GPU
and in the oracle on that state; each case prints its draw."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu

MODES = [0, 0, ipv.TAR_REVERSE, ipv.VAN_REVERSE, ipv.TAR_ADJACENT, ipv.HEAD_SHARED,
         ipv.TAR_ADJACENT | ipv.HEAD_SHARED, ipv.UNIFORM_SELECT]


def loop_state(seed, L, H, D, gh, gw, dtype, frames, cap, budget, alpha, r, mode, tau, partial):
    """The oracle loop's cache after `frames` frames (cap and budget of the
    loop), then `partial` rows of one more frame appended without a pass."""
    p = gh * gw
    S = cap + p
    total = frames + 1
    full = synth.fresh_cache(seed, L, H, total * p, D, gh, gw, total * p, dtype, synth.RhoSpec(0.0, 0.99, 0.3),
                             (0.1, 0.55, 1.0))
    edt = np.uint16 if dtype == synth.BF16 else np.float32
    K = np.zeros((1, L, H, S, D), edt)
    V = np.zeros_like(K)
    fr = np.full((1, L, H, S), -1, np.int32)
    pa = np.full((1, L, H, S), -1, np.int32)
    n = passes = 0
    for f in range(frames):
        kn = np.ascontiguousarray(full.K[None, :, :, f * p:(f + 1) * p])
        vn = np.ascontiguousarray(full.V[None, :, :, f * p:(f + 1) * p])
        n, out = oracle.ckv_step(K, V, fr, pa, n, kn, vn, f, 0, cap, budget, alpha, r, gh, gw, tau,
                                 mode=P.oracle_mode(mode))
        passes += out is not None
    if partial and n + partial <= S:
        kn = np.ascontiguousarray(full.K[None, :, :, frames * p:frames * p + partial])
        vn = np.ascontiguousarray(full.V[None, :, :, frames * p:frames * p + partial])
        n = oracle.append(K, V, fr, pa, n, kn, vn, frames)
    return K[0], V[0], fr[0], pa[0], n, passes


def draw(seed):
    rng = np.random.default_rng(5000 + seed)
    dtype = synth.BF16 if rng.random() < 0.7 else synth.F32
    D = int(rng.choice([32, 64, 128, 256]))
    gh, gw = int(rng.integers(1, 8)), int(rng.integers(1, 8))
    p = gh * gw
    B, L, H = int(rng.integers(1, 4)), int(rng.integers(1, 3)), int(rng.integers(1, 4))
    r = int(rng.integers(1, 4))
    cap = int(rng.integers(r + 2, r + 9)) * p + int(rng.integers(0, p))
    loop_budget = int(rng.integers(r * p, cap - p + 1))
    if rng.random() < 0.5:  # whole frames kept: later frames land at their frame-plane positions again
        loop_budget = max(r * p, loop_budget // p * p)
    streams = []
    for b in range(B):
        if b > 0 and rng.random() < 0.1:
            streams.append(None)  # an empty stream beside the others
            continue
        streams.append(dict(frames=int(rng.integers(r, 4 * (cap // p) + 2)),
                            partial=int(rng.integers(1, p)) if p > 1 and rng.random() < 0.3 else 0,
                            alpha=float(rng.choice([0.0, 0.5, 1.0])), mode=int(rng.choice(MODES[:7])),
                            tau=(0.3, 0.5, 0.7) if rng.random() < 0.3 else None))
    pass_alpha = float(rng.choice([0.0, 0.3, 0.5, 0.8, 1.0]))
    pass_mode = int(rng.choice(MODES))
    pass_tau = (0.3, 0.5, 0.7) if rng.random() < 0.3 else None
    if pass_mode & ipv.HEAD_SHARED:  # a head-shared pass needs every head to hold the same frame ids
        for st in streams:
            if st is not None:
                st["mode"] |= ipv.HEAD_SHARED
    return dict(dtype=dtype, D=D, gh=gh, gw=gw, B=B, L=L, H=H, r=r, cap=cap, loop_budget=loop_budget,
                streams=streams, alpha=pass_alpha, mode=pass_mode, tau=pass_tau, u=float(rng.random()))


@pytest.mark.parametrize("seed", range(1024))
def test_random_fragmented_cache(seed):
    c = draw(seed)
    print("draw", seed, c, flush=True)
    p, S = c["gh"] * c["gw"], c["cap"] + c["gh"] * c["gw"]
    edt = np.uint16 if c["dtype"] == synth.BF16 else np.float32
    K = np.zeros((c["B"], c["L"], c["H"], S, c["D"]), edt)
    V = np.zeros_like(K)
    fr = np.full((c["B"], c["L"], c["H"], S), -1, np.int32)
    pa = np.full_like(fr, -1)
    counts, passes = [], []
    for b, st in enumerate(c["streams"]):
        if st is None:
            counts.append(0)
            continue
        Kb, Vb, fb, pb, n, ps = loop_state(9000 + 17 * seed + b, c["L"], c["H"], c["D"], c["gh"], c["gw"],
                                           c["dtype"], st["frames"], c["cap"], c["loop_budget"], st["alpha"],
                                           c["r"], st["mode"], st["tau"], st["partial"])
        K[b], V[b], fr[b], pa[b] = Kb, Vb, fb, pb
        counts.append(n)
        passes.append(ps)
    live = [n for n in counts if n]
    # the pass's budget holds every stream's largest possible window and fits every stream
    lo, hi = max(min(n, c["r"] * p) for n in live), min(live)
    assert lo <= hi  # every stream saw at least r frames
    budget = lo + int(c["u"] * (hi - lo + 1)) if hi > lo else lo
    budget = min(budget, hi)
    print("  rows per stream %s, earlier passes %s, budget %d" % (counts, passes, budget), flush=True)

    kind = "bf16" if c["dtype"] == synth.BF16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, c["gh"], c["gw"], budget)
    ipv.ipv_compress(Kd, Vd, frd, pad, counts, budget, c["alpha"], c["r"], c["tau"], comp.tar, comp.van,
                     comp.keep_idx, comp.ws, c["gh"], c["gw"], mode=c["mode"])
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    tar, van, keep = comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy()
    Kg, Vg, fg, pg = P.to_host(Kd), P.to_host(Vd), frd.cpu().numpy(), pad.cpu().numpy()
    for b, n in enumerate(counts):
        sl = slice(b, b + 1)
        if n == 0:
            assert np.array_equal(Kg[sl].view(np.uint8), K[sl].view(np.uint8))
            continue
        got = P.GpuPass(tar[sl], van[sl], keep[sl], Kg[sl], Vg[sl], fg[sl], pg[sl], 0)
        near = P.check_pass("seed %d stream %d" % (seed, b), K[sl], V[sl], fr[sl], pa[sl], n, budget,
                            c["alpha"], c["r"], c["gh"], c["gw"], c["mode"], got, c["tau"])
        print("  stream %d: n=%d near-threshold rows %d" % (b, n, near), flush=True)
