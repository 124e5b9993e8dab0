"""Hand-built tiny caches for the oracle's pins (test helper)."""
import numpy as np


def slice_cache(rows_k, rows_v=None, grid_h=1, grid_w=1, frames=None, patches=None, capacity=None):
    """One stream, one layer, one head; fp32 rows. Row x holds frame x // p and
    patch x % p unless frames/patches are given."""
    K = np.asarray(rows_k, np.float32)
    n, D = K.shape
    V = np.ones_like(K) if rows_v is None else np.asarray(rows_v, np.float32)
    p = grid_h * grid_w
    S = capacity or n
    Kc = np.zeros((1, 1, 1, S, D), np.float32)
    Vc = np.zeros((1, 1, 1, S, V.shape[1]), np.float32)
    Kc[0, 0, 0, :n] = K
    Vc[0, 0, 0, :n] = V
    fr = np.full((1, 1, 1, S), -1, np.int32)
    pa = np.full((1, 1, 1, S), -1, np.int32)
    fr[0, 0, 0, :n] = np.arange(n) // p if frames is None else np.asarray(frames)
    pa[0, 0, 0, :n] = np.arange(n) % p if patches is None else np.asarray(patches)
    return Kc, Vc, fr, pa, n
