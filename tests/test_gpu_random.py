"""Seeded random configurations through the whole pass against the oracle:
shapes, dtypes, grids, recent windows, budgets, TaR shares, variant modes,
pooling and per-stream row counts drawn at random (each case prints its
draw), so that corners no hand-picked case names still meet the same rules."""
import numpy as np
import pytest
import torch

import synth
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu

MODES = [0, ipv.TAR_REVERSE, ipv.VAN_REVERSE, ipv.TAR_ADJACENT, ipv.HEAD_SHARED,
         ipv.TAR_ADJACENT | ipv.HEAD_SHARED | ipv.VAN_REVERSE, ipv.UNIFORM_SELECT,
         ipv.UNIFORM_SELECT | ipv.HEAD_SHARED]


def draw(seed):
    rng = np.random.default_rng(1000 + seed)
    dtype = synth.BF16 if rng.random() < 0.7 else synth.F32
    D = int(rng.choice([32, 64, 128, 256]))
    gh, gw = int(rng.integers(1, 9)), int(rng.integers(1, 9))
    p = gh * gw
    B, L, H = int(rng.integers(1, 4)), int(rng.integers(1, 4)), int(rng.integers(1, 4))
    r = int(rng.integers(1, 5))
    frames = int(rng.integers(1, r + 20))  # also caches shorter than the recent window
    counts = []
    for _ in range(B):
        n = frames * p + (int(rng.integers(0, p)) if rng.random() < 0.5 else 0)
        counts.append(0 if rng.random() < 0.15 else n)
    if not any(counts):
        counts[0] = frames * p
    S = max(counts) + int(rng.integers(0, 5))
    window = max(min(n, r * p) for n in counts if n)
    lo = window
    hi = min(n for n in counts if n)
    if hi < lo:  # no budget fits every stream: every non-empty stream gets the largest count
        top = max(counts)
        counts = [top if n else 0 for n in counts]
        lo, hi = min(top, r * p), top
    budget = int(rng.integers(lo, hi + 1))
    alpha = float(rng.choice([0.0, 0.3, 0.5, 0.8, 1.0]))
    mode = int(rng.choice(MODES))
    tau = (0.3, 0.5, 0.7) if rng.random() < 0.3 else None
    return dict(dtype=dtype, D=D, gh=gh, gw=gw, B=B, L=L, H=H, r=r, counts=counts, S=S, budget=budget,
                alpha=alpha, mode=mode, tau=tau)


@pytest.mark.parametrize("seed", range(1024))
def test_random_configuration(seed):
    c = draw(seed)
    print("draw", seed, c, flush=True)
    sts = [synth.fresh_cache(7000 + 31 * seed + b, c["L"], c["H"], c["S"], c["D"], c["gh"], c["gw"], n, c["dtype"],
                             synth.RhoSpec(0.0, 0.99, 0.3), (0.1, 0.55, 1.0)) for b, n in enumerate(c["counts"])]
    st = lambda a: np.ascontiguousarray(np.stack([getattr(x, a) for x in sts]))
    K, V, fr, pa = st("K"), st("V"), st("frame_idx"), st("patch_idx")
    kind = "bf16" if c["dtype"] == synth.BF16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, c["gh"], c["gw"], c["budget"])
    ipv.ipv_compress(Kd, Vd, frd, pad, c["counts"], c["budget"], c["alpha"], c["r"], c["tau"], comp.tar, comp.van,
                     comp.keep_idx, comp.ws, c["gh"], c["gw"], mode=c["mode"])
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    tar, van, keep = comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy()
    Kg, Vg, fg, pg = P.to_host(Kd), P.to_host(Vd), frd.cpu().numpy(), pad.cpu().numpy()
    for b, n in enumerate(c["counts"]):
        sl = slice(b, b + 1)
        if n == 0:
            assert np.array_equal(Kg[sl].view(np.uint8), K[sl].view(np.uint8))
            continue
        got = P.GpuPass(tar[sl], van[sl], keep[sl], Kg[sl], Vg[sl], fg[sl], pg[sl], 0)
        near = P.check_pass("seed %d stream %d" % (seed, b), K[sl], V[sl], fr[sl], pa[sl], n, c["budget"],
                            c["alpha"], c["r"], c["gh"], c["gw"], c["mode"], got, c["tau"])
        print("  stream %d: n=%d near-threshold rows %d" % (b, n, near), flush=True)
