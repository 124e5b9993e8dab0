"""Seeded synthetic KV caches (input generation only).

This package draws random caches shaped like a streaming video MLLM's KV cache
and holds none of the compression method's arithmetic. The CPU oracle and the
GPU path both consume the byte arrays it returns, so neither side's inputs come
from the other.

Layout of a cache for one stream: K and V are ``[L, H, S, D]`` (bf16 stored as
``uint16`` bit patterns, or float32), ``frame_idx`` and ``patch_idx`` are int32
``[L, H, S]``; rows ``[0, n)`` are valid. A batch of B streams stacks these on a
leading axis, giving ``[B, L, H, S, D]``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")

BF16, F32 = 0, 1

_lib = None


def build(force: bool = True) -> str:
    """Compile the generator with gcc (OpenMP) into ``synth/libsynth.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        vp, dp, i32, i64, u64, f64 = (ctypes.c_void_p, ctypes.POINTER(ctypes.c_double), ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_uint64, ctypes.c_double)
        L.synth_rho.argtypes = [u64, i32, f64, f64, f64, f64, dp]
        L.synth_rho.restype = None
        L.synth_keys.argtypes = [u64, i32, i32, i32, dp, i32, i32, i64, dp, vp, i64, i64, i32]
        L.synth_keys.restype = ctypes.c_int
        L.synth_values.argtypes = [u64, i32, i32, i32, i32, dp, i32, i32, i64, vp, i64, i64, i32]
        L.synth_values.restype = ctypes.c_int
        L.synth_fresh_meta.argtypes = [i32, i64, i64, i32, vp, vp]
        L.synth_fresh_meta.restype = None
        L.synth_normals.argtypes = [u64, u64, u64, i64, dp]
        L.synth_normals.restype = None
        _lib = L
    return _lib


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


@dataclass(frozen=True)
class RhoSpec:
    """Per-patch AR(1) coefficient: static with probability ``static_frac``
    (rho = ``static_rho``), else ``U(lo, hi)``."""
    lo: float = 0.0
    hi: float = 0.99
    static_frac: float = 0.0
    static_rho: float = 0.999


def rho(seed: int, p: int, spec: RhoSpec) -> np.ndarray:
    out = np.empty(p, np.float64)
    lib().synth_rho(seed, p, spec.static_frac, spec.static_rho, spec.lo, spec.hi, _dp(out))
    return out


def normals(seed: int, tag: int, count: int, c0: int = 0) -> np.ndarray:
    out = np.empty(count, np.float64)
    lib().synth_normals(seed, tag, c0, count, _dp(out))
    return out


@dataclass
class Stream:
    """A single stream's cache, filled frame by frame.

    ``append(nf)`` draws the next ``nf`` frames' keys and values for every
    (layer, head) and writes them after the ``n`` valid rows of each slice
    (the harness sets the metadata of appended rows to the stream's frame id
    and patch position). The AR(1) state is carried across calls, so a cache
    filled in several appends equals one filled at once.
    """
    seed: int
    L: int
    H: int
    S: int
    D: int
    grid_h: int
    grid_w: int
    dtype: int = BF16
    rho_spec: RhoSpec = field(default_factory=RhoSpec)
    value_sigma: tuple = (0.5,)  # LogNormal sigma of the per-row value scale, cycled over layers

    def __post_init__(self):
        self.p = self.grid_h * self.grid_w
        edt = np.uint16 if self.dtype == BF16 else np.float32
        self.K = np.zeros((self.L, self.H, self.S, self.D), edt)
        self.V = np.zeros((self.L, self.H, self.S, self.D), edt)
        self.frame_idx = np.full((self.L, self.H, self.S), -1, np.int32)
        self.patch_idx = np.full((self.L, self.H, self.S), -1, np.int32)
        self.n = 0
        self.next_frame = 0
        self.rho = rho(self.seed, self.p, self.rho_spec)
        self.sigma = np.array([self.value_sigma[l % len(self.value_sigma)] for l in range(self.L)], np.float64)
        self._state = np.zeros((self.L * self.H, self.p, self.D), np.float64)

    def append(self, nf: int = 1, rows_in_last: int | None = None):
        """Append ``nf`` frames; the last one may be cut to ``rows_in_last`` rows."""
        p = self.p
        total = nf * p if rows_in_last is None else (nf - 1) * p + rows_in_last
        if self.n + total > self.S:
            raise ValueError("stream capacity exceeded")
        f0 = self.next_frame
        limit = f0 * p + total  # stream-position limit for the partial last frame
        LH = self.L * self.H
        L = lib()
        rc = L.synth_keys(self.seed, LH, p, self.D, _dp(self.rho), f0, nf, limit, _dp(self._state),
                          self.K.ctypes.data, self.S, self.n, self.dtype)
        rc |= L.synth_values(self.seed, self.L, self.H, p, self.D, _dp(self.sigma), f0, nf, limit,
                             self.V.ctypes.data, self.S, self.n, self.dtype)
        if rc != 0:
            raise ValueError("generator rejected its arguments")
        rows = np.arange(total)
        self.frame_idx[:, :, self.n:self.n + total] = (f0 + rows // p).astype(np.int32)
        self.patch_idx[:, :, self.n:self.n + total] = (rows % p).astype(np.int32)
        self.n += total
        self.next_frame += nf


def fresh_cache(seed: int, L: int, H: int, S: int, D: int, grid_h: int, grid_w: int, n: int,
                dtype: int = BF16, rho_spec: RhoSpec = RhoSpec(), value_sigma=(0.5,)) -> Stream:
    """A cache holding the first ``n`` rows of a stream (whole frames, plus a
    partial last frame when ``n`` is not a multiple of the frame size)."""
    st = Stream(seed, L, H, S, D, grid_h, grid_w, dtype, rho_spec, tuple(value_sigma))
    p = st.p
    nf, rem = divmod(n, p)
    if rem:
        st.append(nf + 1, rows_in_last=rem)
    elif nf:
        st.append(nf)
    return st


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)
