"""The selection kernel on score values that stress its keys: infinities,
the largest finite floats, subnormals, signed zeros, a single repeated value,
two values, and magnitudes spread over sixty decades. Given the same fp32
scores, the GPU's keep set must be the oracle's exactly (Alg. 1 steps (3)-(5):
higher score first, ties to the lower row)."""
import numpy as np
import pytest
import torch

import oracle
from tests import parity as P

pytestmark = pytest.mark.gpu

FMAX = np.finfo(np.float32).max
SUB = np.float32(1e-40)  # subnormal


def draw(kind, rng, shape):
    if kind == "special":
        pool = np.array([np.inf, -np.inf, FMAX, -FMAX, SUB, -SUB, 0.0, -0.0, 1.0, -1.0, 0.5, 1e-30, -1e-30],
                        np.float32)
        return rng.choice(pool, size=shape).astype(np.float32)
    if kind == "constant":
        return np.full(shape, 0.25, np.float32)
    if kind == "two":
        return np.where(rng.random(shape) < 0.3, np.float32(-0.75), np.float32(2.0)).astype(np.float32)
    if kind == "decades":
        mag = 10.0 ** rng.uniform(-30, 30, size=shape)
        return (np.where(rng.random(shape) < 0.5, -1.0, 1.0) * mag).astype(np.float32)
    raise ValueError(kind)


@pytest.mark.parametrize("kind", ["special", "constant", "two", "decades"])
@pytest.mark.parametrize("mode", [0, oracle.TAR_REVERSE | oracle.VAN_REVERSE])
def test_selection_on_extreme_score_values(kind, mode):
    from paper_2506_15745_amd import ipv
    rng = np.random.default_rng(7 + len(kind) + mode)
    B, L, H, gh, gw, frames, r = 1, 2, 3, 10, 10, 30, 2
    p = gh * gw
    n = frames * p
    S = n + 4
    fr = np.full((B, L, H, S), -1, np.int32)
    fr[..., :n] = np.arange(n, dtype=np.int32) // p
    tar = draw(kind, rng, (B, L, H, S))
    van = np.abs(draw(kind, rng, (B, L, H, S)))  # value norms are not negative
    for budget, alpha in ((n // 2, 0.5), (r * p + 1, 0.5), (n - 1, 0.3), (n // 3, 1.0), (n // 3, 0.0)):
        print("case %s mode=%d C=%d alpha=%s" % (kind, mode, budget, alpha), flush=True)
        sel = oracle.select(tar, van, fr, n, budget, alpha, r, mode=mode)
        keep = torch.zeros((B, L, H, budget), dtype=torch.int32, device="cuda:0")
        ws = ipv.alloc_workspace(ipv.Shape(B, L, H, 64, S, gh, gw, 0), "cuda:0")
        ipv.ipv_select(P.to_device(tar), P.to_device(van), P.to_device(fr), n, budget, alpha, r, keep, ws, gh, gw,
                       head_dim=64, mode=mode)
        torch.cuda.synchronize()
        assert ipv.ipv_read_device_errors(ws) == 0
        assert np.array_equal(keep.cpu().numpy(), sel.keep_idx), (kind, mode, budget, alpha)


@pytest.mark.parametrize("n", [1, 63, 64, 65, 256, 257, 4096, 4097, 6272, 8192, 8193, 16385, 65536])
def test_selection_workgroup_sizes(n):
    """The selection's workgroup is fitted to the rows (whole waves for n rows
    at 4, 8, 16, 32 or 64 rows a thread): counts on both sides of each step
    give the oracle's keep sets."""
    from paper_2506_15745_amd import ipv
    rng = np.random.default_rng(n)
    B, L, H, gh, gw, r = 1, 1, 2, 1, 1, 1
    S = n + (n % 3)
    fr = np.full((B, L, H, S), -1, np.int32)
    fr[..., :n] = np.arange(n, dtype=np.int32)  # one row per frame: the window is the last row
    tar = rng.standard_normal((B, L, H, S)).astype(np.float32)
    van = np.abs(rng.standard_normal((B, L, H, S))).astype(np.float32)
    tar[..., ::7] = 0.5  # ties
    for budget, alpha in ((max(1, n // 2), 0.5), (n, 0.5), (1, 0.0)):
        print("case n=%d C=%d alpha=%s" % (n, budget, alpha), flush=True)
        sel = oracle.select(tar, van, fr, n, budget, alpha, r)
        keep = torch.zeros((B, L, H, budget), dtype=torch.int32, device="cuda:0")
        ws = ipv.alloc_workspace(ipv.Shape(B, L, H, 64, S, gh, gw, 0), "cuda:0")
        ipv.ipv_select(P.to_device(tar), P.to_device(van), P.to_device(fr), n, budget, alpha, r, keep, ws, gh, gw,
                       head_dim=64)
        torch.cuda.synchronize()
        assert ipv.ipv_read_device_errors(ws) == 0
        assert np.array_equal(keep.cpu().numpy(), sel.keep_idx), (n, budget, alpha)
