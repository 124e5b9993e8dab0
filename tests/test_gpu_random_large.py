"""Seeded random configurations with long slices (4097 to 65536 rows): every
rows-a-thread step of the selection (8, 12, 16, 32, 64), budgets above the
8192 positions its LDS stage holds at once (keep sets written in rounds),
capacities that are not a multiple of 4, partial last frames, every mode;
one or two slices so that the oracle stays quick. Each case prints its draw."""
import numpy as np
import pytest
import torch

import synth
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu

MODES = [0, 0, ipv.TAR_REVERSE, ipv.VAN_REVERSE, ipv.TAR_ADJACENT, ipv.UNIFORM_SELECT,
         ipv.HEAD_SHARED, ipv.TAR_ADJACENT | ipv.VAN_REVERSE]


def draw(seed):
    rng = np.random.default_rng(9000 + seed)
    dtype = synth.BF16 if rng.random() < 0.8 else synth.F32
    D = int(rng.choice([32, 64]))
    gh, gw = int(rng.integers(4, 17)), int(rng.integers(4, 17))
    p = gh * gw
    n = int(rng.integers(4097, 65537))
    r = int(rng.integers(1, 5))
    while r * p > n // 2:  # the window leaves room for past rows and a budget
        r -= 1
    r = max(r, 1)
    S = n + int(rng.integers(0, 4))
    window = min(n, r * p)
    budget = int(rng.integers(window, n + 1))
    if rng.random() < 0.4:  # a keep set larger than the LDS stage
        budget = int(rng.integers(max(window, 8193), n + 1)) if n > 8193 else budget
    H = int(rng.integers(1, 3))
    return dict(dtype=dtype, D=D, gh=gh, gw=gw, n=n, S=S, r=r, budget=budget, H=H,
                alpha=float(rng.choice([0.0, 0.3, 0.5, 1.0])), mode=int(rng.choice(MODES)),
                tau=(0.3, 0.5, 0.7) if rng.random() < 0.3 else None)


@pytest.mark.parametrize("seed", range(192))
def test_random_long_slices(seed):
    c = draw(seed)
    print("draw", seed, c, flush=True)
    st = synth.fresh_cache(20000 + seed, 1, c["H"], c["S"], c["D"], c["gh"], c["gw"], c["n"], c["dtype"],
                           synth.RhoSpec(0.0, 0.99, 0.3), (0.1, 0.55, 1.0))
    K, V, fr, pa = (np.ascontiguousarray(getattr(st, a)[None]) for a in ("K", "V", "frame_idx", "patch_idx"))
    kind = "bf16" if c["dtype"] == synth.BF16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, c["gh"], c["gw"], c["budget"])
    comp.compress(Kd, Vd, frd, pad, c["n"], c["alpha"], c["r"], c["tau"], mode=c["mode"])
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    got = P.GpuPass(P.to_host(comp.tar), P.to_host(comp.van), P.to_host(comp.keep_idx), P.to_host(Kd), P.to_host(Vd),
                    P.to_host(frd), P.to_host(pad), 0)
    near = P.check_pass("seed %d" % seed, K, V, fr, pa, c["n"], c["budget"], c["alpha"], c["r"], c["gh"], c["gw"],
                        c["mode"], got, c["tau"])
    print("  near-threshold rows %d" % near, flush=True)
