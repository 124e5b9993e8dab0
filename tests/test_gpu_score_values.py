"""The whole pass on caches whose rows span the magnitudes the score kernels
must handle: zero rows (TaR 0 by the zero-norm rule, Sec. 3.1; a zero recent
key still counts in its position's mean), rows scaled by 2^-60 and by 2^50,
and ordinary rows, in K and V alike, past and recent. Scores, keep sets and
the compacted cache are checked against the oracle as in the other parity
tests. Row squared norms stay within fp32 range (elements up to about 1e18
in magnitude); the header states that bound."""
import numpy as np
import pytest

import synth
from synth import workloads as W
from tests.test_gpu_parity import cache_of, full_check

pytestmark = pytest.mark.gpu

SCALES = (0, -60, 50, None)  # exponent shift per row; 0 = zero row, None = unchanged


def rescale_rows(a: np.ndarray, dtype: int, shift: np.ndarray, zero: np.ndarray) -> np.ndarray:
    """Multiply whole rows of a [B, L, H, S, D] array by 2^shift exactly (bf16
    bit patterns: add to the exponent field of the non-zero elements)."""
    out = a.copy()
    if dtype == synth.BF16:
        exp = (out >> 7) & 0xFF
        nz = exp != 0
        out = np.where(nz, (out.astype(np.int32) + (shift[..., None].astype(np.int32) << 7)).astype(np.uint16), out)
    else:
        out = (out * np.exp2(shift[..., None]).astype(np.float32)).astype(np.float32)
    out[zero] = 0
    return out


@pytest.mark.parametrize("dtype,D", [(synth.BF16, 64), (synth.F32, 32)])
def test_pass_on_zero_tiny_and_huge_rows(dtype, D):
    n = 16 * 12 + 5
    w = W.Workload(name="values-D%d" % D, streams=1, layers=2, kv_heads=2, head_dim=D, grid_h=4, grid_w=4,
                   n_tokens=n, budget=100, recent_frames=2, alphas=(0.5,), dtype=dtype, seeds=(41,),
                   rho_specs=(synth.RhoSpec(0.0, 0.99, static_frac=0.3, static_rho=0.999),))
    K, V, fr, pa = cache_of(w)
    rng = np.random.default_rng(5 + D)
    for name in ("K", "V"):
        pick = rng.choice(len(SCALES), size=K.shape[:4], p=(0.15, 0.15, 0.15, 0.55))
        shift = np.array([s if s is not None else 0 for s in SCALES])[pick]
        zero = pick == 0
        shift[zero] = 0
        if name == "K":
            K = rescale_rows(K, dtype, shift, zero)
        else:
            V = rescale_rows(V, dtype, shift, zero)
    for alpha in (0.5, 1.0, 0.0):
        full_check(w, K, V, fr, pa, alpha)
