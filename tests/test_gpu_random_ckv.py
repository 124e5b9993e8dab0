"""Seeded random configurations of the continual-compression loop
(Algorithm 1) through ipv_ckv_step, frame by frame against the oracle's
loop and teacher-forced at every pass (the loop of tests/test_gpu_ckv.py):
shape, grid, cap, budget (down to the largest recent window), TaR share,
variant mode and pooling drawn at random; each case prints its draw."""
import numpy as np
import pytest

import synth
from paper_2506_15745_amd import ipv
from tests.test_gpu_ckv import run_loop

pytestmark = pytest.mark.gpu

MODES = [0, 0, ipv.TAR_REVERSE, ipv.VAN_REVERSE, ipv.TAR_ADJACENT, ipv.HEAD_SHARED,
         ipv.TAR_ADJACENT | ipv.HEAD_SHARED | ipv.TAR_REVERSE, ipv.UNIFORM_SELECT,
         ipv.UNIFORM_SELECT | ipv.HEAD_SHARED]


def draw(seed):
    rng = np.random.default_rng(7000 + seed)
    dtype = synth.BF16 if rng.random() < 0.7 else synth.F32
    D = int(rng.choice([32, 64, 128, 256]))
    gh, gw = int(rng.integers(1, 7)), int(rng.integers(1, 7))
    p = gh * gw
    L, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
    r = int(rng.integers(1, 4))
    cap = int(rng.integers(r + 1, r + 7)) * p + int(rng.integers(0, p))
    # the loop asks for a budget that holds the largest window a cache can have
    budget = int(rng.integers(r * p, cap))
    frames = int(rng.integers(cap // p + 1, 4 * (cap // p) + 3))
    return dict(dtype=dtype, D=D, gh=gh, gw=gw, L=L, H=H, r=r, cap=cap, budget=budget, frames=frames,
                alpha=float(rng.choice([0.0, 0.3, 0.5, 1.0])), mode=int(rng.choice(MODES)),
                tau=(0.3, 0.5, 0.7) if rng.random() < 0.3 else None,
                sigma=(0.1, 0.35, 0.55, 1.0) if rng.random() < 0.5 else (0.5,))


@pytest.mark.parametrize("seed", range(512))
def test_random_ckv_loop(seed):
    c = draw(seed)
    print("draw", seed, c, flush=True)
    passes = run_loop(c["L"], c["H"], c["D"], c["gh"], c["gw"], c["frames"], c["cap"], c["budget"], c["r"],
                      c["alpha"], c["dtype"], 11000 + seed, synth.RhoSpec(0.0, 0.99, 0.3), c["mode"], c["tau"],
                      c["sigma"])
    assert passes >= 1
