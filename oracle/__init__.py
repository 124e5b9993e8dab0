"""CPU oracle of the InfiniPot-V compression pass -- TEST INFRASTRUCTURE.

Only ``tests/``, the package smoke check (``__graft_entry__.smoke``) and the
CPU-baseline leg of ``bench.py`` may import this package. The GPU library never
calls it, and the two share no code: the oracle is plain C (``ipv_oracle.c``,
built with gcc) computing every step of the pass in fp64 straight from the
paper's definitions, one slice at a time.

Functions take numpy arrays in the cache layout (K, V ``[B, L, H, S, D]`` as
bf16 bit patterns in ``uint16`` or as float32; metadata int32 ``[B, L, H, S]``)
and return numpy results.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ipv_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, ERR_ARG, ERR_META, ERR_BUDGET, ERR_NAN = 0, -1, -2, -3, -4
# variant bits (the ablation rows of Tab. 5, the head-shared reading, and the
# Uniform Select baseline of the KV-compression comparison)
TAR_REVERSE, VAN_REVERSE, TAR_ADJACENT, HEAD_SHARED, UNIFORM = 1, 2, 4, 8, 16


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so`` (IEEE math, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("streams", "layers", "kv_heads", "head_dim", "capacity", "grid_h", "grid_w", "dtype")]


class SelectInfo(ctypes.Structure):
    _fields_ = [("n_recent", ctypes.c_int32), ("b_tar", ctypes.c_int32), ("b_van", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("cut_tar", ctypes.c_float), ("cut_van", ctypes.c_float)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        L = ctypes.CDLL(_LIB)
        vp, i32 = ctypes.c_void_p, ctypes.c_int32
        sp = ctypes.POINTER(Shape)
        u32 = ctypes.c_uint32
        L.ipvo_tar_scores.argtypes = [sp, vp, vp, vp, i32, i32, u32, vp]
        L.ipvo_van_scores.argtypes = [sp, vp, vp, vp, i32, vp, vp, vp]
        L.ipvo_select.argtypes = [sp, vp, vp, vp, i32, i32, i32, i32, u32, vp, vp]
        L.ipvo_compact.argtypes = [sp, vp, vp, vp, vp, i32, vp, i32]
        L.ipvo_compress.argtypes = [sp, vp, vp, vp, vp, i32, i32, i32, i32, u32, vp, vp, vp, vp, vp]
        for f in (L.ipvo_tar_scores, L.ipvo_van_scores, L.ipvo_select, L.ipvo_compact, L.ipvo_compress):
            f.restype = ctypes.c_int
        L.ipvo_max_threads.restype = ctypes.c_int32
        L.ipvo_set_threads.argtypes = [i32]
        L.ipvo_set_threads.restype = None
        _lib = L
    return _lib


def max_threads() -> int:
    return int(lib().ipvo_max_threads())


def set_threads(threads: int) -> None:
    """Threads of the oracle's slice loops from now on (results do not depend on it)."""
    lib().ipvo_set_threads(int(threads))


def tar_budget_total(alpha: float, budget: int) -> int:
    """floor(alpha * C), taken in double precision."""
    return int(math.floor(float(alpha) * float(budget)))


def _shape(K: np.ndarray, grid_h: int, grid_w: int) -> Shape:
    if K.ndim != 5:
        raise ValueError("K must be [B, L, H, S, D]")
    if K.dtype == np.uint16:
        dt = 0
    elif K.dtype == np.float32:
        dt = 1
    else:
        raise ValueError("K must hold bf16 bits (uint16) or float32")
    B, L, H, S, D = K.shape
    return Shape(B, L, H, D, S, grid_h, grid_w, dt)


def _c(a: np.ndarray, dtype) -> np.ndarray:
    if a.dtype != dtype or not a.flags.c_contiguous:
        raise ValueError("expected a C-contiguous %s array" % np.dtype(dtype).name)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc: int, what: str):
    if rc != OK:
        raise OracleError("%s failed with code %d" % (what, rc))


def tar_scores(K, frame_idx, patch_idx, n, recent_frames, grid_h, grid_w, mode=0) -> np.ndarray:
    """TaR scores in fp64, [B, L, H, S] (rows >= n left at 0). mode & TAR_ADJACENT:
    against the previous frame's key at the same position instead of the recent window."""
    s = _shape(K, grid_h, grid_w)
    out = np.zeros(K.shape[:4], np.float64)
    _check(lib().ipvo_tar_scores(ctypes.byref(s), _ptr(K), _ptr(_c(frame_idx, np.int32)),
                                 _ptr(_c(patch_idx, np.int32)), n, recent_frames, mode, _ptr(out)), "tar_scores")
    return out


def van_scores(V, frame_idx, patch_idx, n, grid_h, grid_w, cv_tau=None):
    """VaN scores in fp64 [B, L, H, S] and the per-(stream, layer) pooling size [B, L]."""
    s = _shape(V, grid_h, grid_w)
    out = np.zeros(V.shape[:4], np.float64)
    pool = np.zeros(V.shape[:2], np.int32)
    tau = None if cv_tau is None else np.asarray(cv_tau, np.float64)
    _check(lib().ipvo_van_scores(ctypes.byref(s), _ptr(V), _ptr(_c(frame_idx, np.int32)),
                                 _ptr(_c(patch_idx, np.int32)), n, _ptr(tau), _ptr(out), _ptr(pool)),
           "van_scores")
    return out, pool


@dataclass
class Selection:
    keep_idx: np.ndarray  # [B, L, H, C] int32, ascending
    n_recent: np.ndarray  # [B, L, H]
    b_tar: np.ndarray
    b_van: np.ndarray
    cut_tar: np.ndarray   # fp32 score of the last TaR pick (NaN if none)
    cut_van: np.ndarray


def select(tar32, van32, frame_idx, n, budget, alpha, recent_frames, grid_h=1, grid_w=1, mode=0) -> Selection:
    """Keep set from fp32 scores (the precision the decision is taken in). mode:
    TAR_REVERSE / VAN_REVERSE take a stage's lowest scores; HEAD_SHARED ranks
    the fp32 sum over each layer's heads and gives every head the same rows;
    UNIFORM takes past frames at regular intervals and reads no scores (the
    score arrays may then be None)."""
    frame_idx = _c(frame_idx, np.int32)
    if mode & UNIFORM and tar32 is None:
        tar32 = van32 = None
    else:
        tar32 = _c(tar32, np.float32)
        van32 = _c(van32, np.float32)
    B, L, H, S = frame_idx.shape
    s = Shape(B, L, H, 1, S, grid_h, grid_w, 1)
    keep = np.zeros((B, L, H, budget), np.int32)
    info = (SelectInfo * (B * L * H))()
    _check(lib().ipvo_select(ctypes.byref(s), _ptr(tar32), _ptr(van32), _ptr(frame_idx), n,
                             budget, tar_budget_total(alpha, budget), recent_frames, mode, _ptr(keep),
                             ctypes.addressof(info)), "select")
    f = lambda name, dt: np.array([getattr(i, name) for i in info], dt).reshape(B, L, H)
    return Selection(keep, f("n_recent", np.int32), f("b_tar", np.int32), f("b_van", np.int32),
                     f("cut_tar", np.float32), f("cut_van", np.float32))


def compact(K, V, frame_idx, patch_idx, n, keep_idx, grid_h=1, grid_w=1):
    """In-place compaction of copies; returns (K, V, frame_idx, patch_idx)."""
    K, V, fr, pa = K.copy(), V.copy(), frame_idx.copy(), patch_idx.copy()
    s = _shape(K, grid_h, grid_w)
    budget = keep_idx.shape[-1]
    _check(lib().ipvo_compact(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(fr), _ptr(pa), n,
                              _ptr(_c(keep_idx, np.int32)), budget), "compact")
    return K, V, fr, pa


def compress_inplace(K, V, frame_idx, patch_idx, n, budget, alpha, recent_frames, grid_h, grid_w, cv_tau=None,
                     mode=0):
    """The whole pass, in place on the given arrays; returns (tar32, van32, keep_idx)."""
    s = _shape(K, grid_h, grid_w)
    tar = np.zeros(K.shape[:4], np.float32)
    van = np.zeros(K.shape[:4], np.float32)
    keep = np.zeros(K.shape[:3] + (budget,), np.int32)
    tau = None if cv_tau is None else np.asarray(cv_tau, np.float64)
    _check(lib().ipvo_compress(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(_c(frame_idx, np.int32)),
                               _ptr(_c(patch_idx, np.int32)), n, budget, tar_budget_total(alpha, budget),
                               recent_frames, mode, _ptr(tau), _ptr(tar), _ptr(van), _ptr(keep), None),
           "compress")
    return tar, van, keep


def append(K, V, frame_idx, patch_idx, n, K_new, V_new, frame_id, first_patch=0) -> int:
    """Algorithm 1 step (1), in place: rows [n, n + rows) of every slice take
    the new rows, frame id `frame_id` and patch ids first_patch, first_patch+1,
    ...; returns the new row count."""
    rows = K_new.shape[3]
    if K_new.shape != V_new.shape or K_new.shape[:3] != K.shape[:3] or n + rows > K.shape[3]:
        raise OracleError("append: rows do not fit")
    K[:, :, :, n:n + rows] = K_new
    V[:, :, :, n:n + rows] = V_new
    frame_idx[:, :, :, n:n + rows] = frame_id
    patch_idx[:, :, :, n:n + rows] = first_patch + np.arange(rows, dtype=np.int32)
    return n + rows


def ckv_step(K, V, frame_idx, patch_idx, n, K_new, V_new, frame_id, first_patch, mem_cap, budget, alpha,
             recent_frames, grid_h, grid_w, cv_tau=None, mode=0):
    """One iteration of Algorithm 1, in place: append; if the cache then holds
    len >= mem_cap rows, run the pass to `budget` rows. Returns
    (new n, (tar32, van32, keep_idx) of the pass or None)."""
    n = append(K, V, frame_idx, patch_idx, n, K_new, V_new, frame_id, first_patch)
    if n < mem_cap:
        return n, None
    out = compress_inplace(K, V, frame_idx, patch_idx, n, budget, alpha, recent_frames, grid_h, grid_w, cv_tau,
                           mode)
    return budget, out
