"""Python binding of ``libipv.so`` (ctypes; argument marshalling only).

Every function here passes device pointers of torch tensors, sizes and the
current HIP stream to the C ABI declared in ``include/ipv.h``; all of the
pass's work runs in the library's HIP kernels. Importing works anywhere, but
the first call loads ``libipv.so`` and raises :class:`IpvError` when it has
not been built -- there is no fallback implementation.

Tensor layouts (all contiguous, on the same GPU):
  K, V        [B, L, H, S, D]  torch.bfloat16 or torch.float32
  frame_idx   [B, L, H, S]     torch.int32
  patch_idx   [B, L, H, S]     torch.int32
  tar, van    [B, L, H, S]     torch.float32
  keep_idx    [B, L, H, C]     torch.int32
  pool_size   [B, L]           torch.int32
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libipv.so")

OK, ERR_NULL, ERR_ALIGN, ERR_SHAPE, ERR_DTYPE, ERR_BUDGET, ERR_ARG, ERR_WORKSPACE, ERR_HIP = range(9)
BF16, F32 = 0, 1
DEV_BAD_PATCH, DEV_BAD_FRAMES, DEV_RECENT_OVER, DEV_BAD_KEEP, DEV_NAN, DEV_WAIT_TIMEOUT = 1, 2, 4, 8, 16, 32
# `mode` bits: reversed TaR / VaN stages, consecutive-frame TaR, head-shared
# selection, Uniform Select (frames at regular intervals, no scores)
TAR_REVERSE, VAN_REVERSE, TAR_ADJACENT, HEAD_SHARED, UNIFORM_SELECT = 1, 2, 4, 8, 16

EXPORTS = ("ipv_workspace_bytes", "ipv_tar_scores", "ipv_van_scores", "ipv_select", "ipv_compact",
           "ipv_compress", "ipv_compress_timed", "ipv_compress_noalloc", "ipv_append", "ipv_ckv_step", "ipv_ckv_stream",
           "ipv_clear_device_errors",
           "ipv_read_device_errors", "ipv_status_str")


class IpvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s: %s (status %d)" % (what, status_str(status), status))


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("streams", "layers", "kv_heads", "head_dim", "capacity", "grid_h", "grid_w", "dtype")]


class Events(ctypes.Structure):
    """hipEvent_t handles recorded at the pass's step boundaries (see ipv.h)."""
    _fields_ = [("at", ctypes.c_void_p * 6)]

    def __init__(self, *handles):
        super().__init__()
        for i, h in enumerate(handles):
            self.at[i] = h


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library (raises IpvError if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise IpvError(ERR_HIP, "libipv.so is not built (run paper_2506_15745_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, f64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double, ctypes.c_size_t
        sp = ctypes.POINTER(Shape)
        L.ipv_workspace_bytes.argtypes = [sp, ctypes.POINTER(ctypes.c_size_t)]
        u32 = ctypes.c_uint32
        ns = ctypes.POINTER(i32)  # host array of B row counts
        L.ipv_tar_scores.argtypes = [sp, vp, vp, vp, ns, i32, u32, vp, vp, sz, vp]
        L.ipv_van_scores.argtypes = [sp, vp, vp, vp, ns, vp, vp, vp, vp, sz, vp]
        L.ipv_select.argtypes = [sp, vp, vp, vp, ns, i32, f64, i32, u32, vp, vp, sz, vp]
        L.ipv_compact.argtypes = [sp, vp, vp, vp, vp, ns, vp, i32, vp, sz, vp]
        L.ipv_compress.argtypes = [sp, vp, vp, vp, vp, ns, i32, f64, i32, u32, vp, vp, vp, vp, vp, sz, vp]
        L.ipv_compress_timed.argtypes = [sp, vp, vp, vp, vp, ns, i32, f64, i32, u32, vp, vp, vp, vp, vp, sz, vp,
                                         ctypes.POINTER(Events)]
        L.ipv_compress_noalloc.argtypes = [sp, vp, vp, vp, vp, ns, i32, f64, i32, u32, vp, vp, vp, vp, vp, vp]
        L.ipv_append.argtypes = [sp, vp, vp, vp, vp, ns, vp, vp, i32, i32, i32, vp]
        L.ipv_ckv_step.argtypes = [sp, vp, vp, vp, vp, ns, vp, vp, i32, i32, i32, i32, i32, f64, i32, u32, vp, vp, vp,
                                   vp, vp, sz, ns, ns, vp]
        L.ipv_ckv_stream.argtypes = [sp, vp, vp, vp, vp, ns, vp, vp, i32, i32, i32, i32, i32, f64, i32, u32, vp, vp,
                                     vp, vp, vp, sz, ns, vp]
        L.ipv_clear_device_errors.argtypes = [vp, sz, vp]
        L.ipv_read_device_errors.argtypes = [vp, sz, vp, ctypes.POINTER(ctypes.c_uint32)]
        L.ipv_status_str.argtypes = [ctypes.c_int]
        L.ipv_status_str.restype = ctypes.c_char_p
        for name in EXPORTS[:-1]:
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def status_str(status: int) -> str:
    if _lib is None and not os.path.exists(LIB_PATH):
        return "status %d" % status
    return lib().ipv_status_str(status).decode()


def _check(rc: int, what: str):
    if rc != OK:
        raise IpvError(rc, what)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise IpvError(ERR_DTYPE, "K/V dtype %s" % t.dtype)


def shape_of(K: torch.Tensor, grid_h: int, grid_w: int) -> Shape:
    if K.dim() != 5:
        raise IpvError(ERR_SHAPE, "K must be [B, L, H, S, D]")
    B, L, H, S, D = K.shape
    return Shape(B, L, H, D, S, grid_h, grid_w, _dtype_code(K))


def _ptr(t):
    if t is None:
        return None
    if t.device.type != "cuda":
        raise IpvError(ERR_ARG, "tensors must be in GPU memory (got %s)" % t.device)
    if not t.is_contiguous():
        raise IpvError(ERR_SHAPE, "tensors must be contiguous")
    return t.data_ptr()


def _expect(what, t, shape, dtype, device, optional=False):
    """Refuse a companion tensor whose shape, dtype or device does not match
    the cache: the library only sees pointers, so a smaller buffer would be
    written past its end."""
    if t is None:
        if optional:
            return
        raise IpvError(ERR_NULL, "%s is required" % what)
    if t.dtype != dtype:
        raise IpvError(ERR_DTYPE, "%s must be %s (got %s)" % (what, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise IpvError(ERR_SHAPE, "%s must have shape %s (got %s)" % (what, tuple(shape), tuple(t.shape)))
    if t.device != device:
        raise IpvError(ERR_ARG, "%s is on %s, the cache on %s" % (what, t.device, device))


def _check_meta(K, frame_idx, patch_idx):
    """frame_idx / patch_idx: int32 [B, L, H, S] beside K [B, L, H, S, D]."""
    rows = tuple(K.shape[:4])
    _expect("frame_idx", frame_idx, rows, torch.int32, K.device)
    _expect("patch_idx", patch_idx, rows, torch.int32, K.device)


def _check_scores(ref, device, tar=None, van=None, optional=False):
    """tar / van: fp32 [B, L, H, S]."""
    _expect("tar", tar, ref, torch.float32, device, optional)
    _expect("van", van, ref, torch.float32, device, optional)


def _check_keep(keep_idx, rows, budget, device, optional=False):
    """keep_idx: int32 [B, L, H, budget]."""
    _expect("keep_idx", keep_idx, tuple(rows[:3]) + (int(budget),), torch.int32, device, optional)


def _check_ws(ws, device, optional=False):
    if ws is None:
        if optional:
            return
        raise IpvError(ERR_WORKSPACE, "a workspace is required")
    if ws.device != device:
        raise IpvError(ERR_ARG, "the workspace is on %s, the cache on %s" % (ws.device, device))


def _ws_bytes(ws):
    return 0 if ws is None else ws.numel() * ws.element_size()


def _check_cache(K, V, frame_idx, patch_idx):
    """V like K; the metadata beside them."""
    _expect("V", V, tuple(K.shape), K.dtype, K.device)
    _check_meta(K, frame_idx, patch_idx)


def _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, ws, optional=False,
                        need_ws=True, mode=0):
    """Every buffer of a whole pass against the cache K [B, L, H, S, D];
    optional: the score, keep and workspace buffers may be None (the
    continual-compression calls need them only when a pass runs)."""
    _check_cache(K, V, frame_idx, patch_idx)
    _check_scores(K.shape[:4], K.device, tar, van, optional or bool(mode & UNIFORM_SELECT))
    _check_keep(keep_idx, K.shape, budget, K.device, optional)
    if need_ws:
        _check_ws(ws, K.device, optional)


def _check_new_rows(K, K_new, V_new):
    """K_new / V_new: [B, L, H, rows, D] with the cache's dtype."""
    if K_new.dtype != K.dtype or V_new.dtype != K.dtype:
        raise IpvError(ERR_DTYPE, "K_new/V_new must have the cache's dtype")
    if K_new.shape != V_new.shape or K_new.dim() != 5 or K_new.shape[:3] != K.shape[:3] \
            or K_new.shape[4] != K.shape[4]:
        raise IpvError(ERR_SHAPE, "K_new/V_new must be [B, L, H, rows, D] like the cache")


def counts(n_tokens, streams: int):
    """Host array of per-stream row counts from an int (every stream) or a sequence."""
    if isinstance(n_tokens, int):
        vals = [n_tokens] * streams
    else:
        vals = [int(v) for v in n_tokens]
        if len(vals) != streams:
            raise IpvError(ERR_SHAPE, "n_tokens needs one count per stream (%d)" % streams)
    return (ctypes.c_int32 * streams)(*vals)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def workspace_bytes(shape: Shape) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().ipv_workspace_bytes(ctypes.byref(shape), ctypes.byref(out)), "ipv_workspace_bytes")
    return out.value


def alloc_workspace(shape: Shape, device) -> torch.Tensor:
    """A zeroed workspace tensor (uint8) for calls on `shape`."""
    return torch.zeros(workspace_bytes(shape), dtype=torch.uint8, device=device)


def ipv_tar_scores(K, frame_idx, patch_idx, n_tokens, recent_frames, tar, ws, grid_h, grid_w, stream=None, mode=0):
    s = shape_of(K, grid_h, grid_w)
    _check_meta(K, frame_idx, patch_idx)
    _expect("tar", tar, K.shape[:4], torch.float32, K.device)
    _check_ws(ws, K.device)
    _check(lib().ipv_tar_scores(ctypes.byref(s), _ptr(K), _ptr(frame_idx), _ptr(patch_idx), counts(n_tokens, s.streams),
                                recent_frames, mode, _ptr(tar), _ptr(ws), _ws_bytes(ws), _stream(stream)),
           "ipv_tar_scores")


def ipv_van_scores(V, frame_idx, patch_idx, n_tokens, cv_tau, van, pool_size, ws, grid_h, grid_w, stream=None):
    s = shape_of(V, grid_h, grid_w)
    _check_meta(V, frame_idx, patch_idx)
    _expect("van", van, V.shape[:4], torch.float32, V.device)
    _expect("pool_size", pool_size, V.shape[:2], torch.int32, V.device, optional=True)
    _check_ws(ws, V.device)
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    _check(lib().ipv_van_scores(ctypes.byref(s), _ptr(V), _ptr(frame_idx), _ptr(patch_idx), counts(n_tokens, s.streams),
                                None if tau is None else ctypes.addressof(tau), _ptr(van), _ptr(pool_size),
                                _ptr(ws), _ws_bytes(ws), _stream(stream)), "ipv_van_scores")


def ipv_select(tar, van, frame_idx, n_tokens, budget, alpha, recent_frames, keep_idx, ws, grid_h, grid_w,
               head_dim=128, dtype=BF16, stream=None, mode=0):
    """The select step needs only the slice geometry: (B, L, H, S) from
    frame_idx and the patch grid; head_dim/dtype only size the workspace.
    With UNIFORM_SELECT in mode, tar and van may be None."""
    if frame_idx.dim() != 4:
        raise IpvError(ERR_SHAPE, "frame_idx must be [B, L, H, S]")
    B, L, H, S = frame_idx.shape
    s = Shape(B, L, H, head_dim, S, grid_h, grid_w, dtype)
    _expect("frame_idx", frame_idx, frame_idx.shape, torch.int32, frame_idx.device)
    _check_scores(frame_idx.shape, frame_idx.device, tar, van, optional=bool(mode & UNIFORM_SELECT))
    _check_keep(keep_idx, frame_idx.shape, budget, frame_idx.device)
    _check_ws(ws, frame_idx.device)
    _check(lib().ipv_select(ctypes.byref(s), _ptr(tar), _ptr(van), _ptr(frame_idx), counts(n_tokens, B), budget,
                            float(alpha), recent_frames, mode, _ptr(keep_idx), _ptr(ws), _ws_bytes(ws),
                            _stream(stream)),
           "ipv_select")


def ipv_compact(K, V, frame_idx, patch_idx, n_tokens, keep_idx, budget, ws, grid_h, grid_w, stream=None):
    s = shape_of(K, grid_h, grid_w)
    _check_cache(K, V, frame_idx, patch_idx)
    _check_keep(keep_idx, K.shape, budget, K.device)
    _check_ws(ws, K.device)
    _check(lib().ipv_compact(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx),
                             counts(n_tokens, s.streams),
                             _ptr(keep_idx), budget, _ptr(ws), _ws_bytes(ws), _stream(stream)),
           "ipv_compact")


def ipv_compress(K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, cv_tau, tar, van, keep_idx,
                 ws, grid_h, grid_w, stream=None, mode=0):
    s = shape_of(K, grid_h, grid_w)
    _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, ws, mode=mode)
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    _check(lib().ipv_compress(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx),
                              counts(n_tokens, s.streams),
                              budget, float(alpha), recent_frames, mode, None if tau is None else ctypes.addressof(tau),
                              _ptr(tar), _ptr(van), _ptr(keep_idx), _ptr(ws), _ws_bytes(ws), _stream(stream)),
           "ipv_compress")


def ipv_compress_timed(K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, cv_tau, tar, van,
                       keep_idx, ws, grid_h, grid_w, events: Events, stream=None, mode=0):
    s = shape_of(K, grid_h, grid_w)
    _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, ws, mode=mode)
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    _check(lib().ipv_compress_timed(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx),
                                    counts(n_tokens, s.streams),
                                    budget, float(alpha), recent_frames, mode,
                                    None if tau is None else ctypes.addressof(tau), _ptr(tar), _ptr(van),
                                    _ptr(keep_idx), _ptr(ws), _ws_bytes(ws), _stream(stream), ctypes.byref(events)),
           "ipv_compress_timed")


def ipv_compress_noalloc(K, V, frame_idx, patch_idx, n_tokens, budget, alpha, recent_frames, cv_tau, tar, van,
                         keep_idx, grid_h, grid_w, device_errors=None, stream=None, mode=0):
    """ipv_compress with the library's own per-GPU workspace (no workspace
    argument, nothing allocated by the call); device_errors: an int32/uint32
    device tensor of one element that receives the pass's error word, or None."""
    s = shape_of(K, grid_h, grid_w)
    _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, None, need_ws=False, mode=mode)
    if device_errors is not None and (device_errors.numel() != 1 or device_errors.element_size() != 4
                                      or device_errors.device != K.device):
        raise IpvError(ERR_SHAPE, "device_errors must be one 4-byte element on the cache's device")
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    _check(lib().ipv_compress_noalloc(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx),
                                      counts(n_tokens, s.streams), budget, float(alpha), recent_frames, mode,
                                      None if tau is None else ctypes.addressof(tau), _ptr(tar), _ptr(van),
                                      _ptr(keep_idx), _ptr(device_errors), _stream(stream)),
           "ipv_compress_noalloc")


def ipv_append(K, V, frame_idx, patch_idx, n_tokens, K_new, V_new, frame_id, first_patch, grid_h, grid_w,
               stream=None):
    """Append K_new/V_new ([B, L, H, rows, D]) after row n_tokens[b] of every
    slice of stream b; returns the new row count(s) (an int for an int
    n_tokens, else a list)."""
    s = shape_of(K, grid_h, grid_w)
    _check_cache(K, V, frame_idx, patch_idx)
    _check_new_rows(K, K_new, V_new)
    rows = K_new.shape[3]
    ns = counts(n_tokens, s.streams)
    _check(lib().ipv_append(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx), ns,
                            _ptr(K_new), _ptr(V_new), rows, frame_id, first_patch, _stream(stream)), "ipv_append")
    return n_tokens + rows if isinstance(n_tokens, int) else [v + rows for v in ns]


def ipv_ckv_step(K, V, frame_idx, patch_idx, n_tokens, K_new, V_new, frame_id, first_patch, mem_cap, budget,
                 alpha, recent_frames, cv_tau, tar, van, keep_idx, ws, grid_h, grid_w, stream=None, mode=0):
    """Append, then compress to `budget` every stream that holds >= mem_cap
    rows. Returns (row counts, whether each stream's pass ran): ints for an
    int n_tokens (every stream then behaves alike), else lists."""
    s = shape_of(K, grid_h, grid_w)
    _check_cache(K, V, frame_idx, patch_idx)
    _check_new_rows(K, K_new, V_new)
    _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, ws, optional=True, mode=mode)
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    n_out, comp = (ctypes.c_int32 * s.streams)(), (ctypes.c_int32 * s.streams)()
    _check(lib().ipv_ckv_step(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx),
                              counts(n_tokens, s.streams),
                              _ptr(K_new), _ptr(V_new), K_new.shape[3], frame_id, first_patch, mem_cap, budget,
                              float(alpha), recent_frames, mode, None if tau is None else ctypes.addressof(tau),
                              _ptr(tar),
                              _ptr(van), _ptr(keep_idx), _ptr(ws), _ws_bytes(ws),
                              n_out, comp, _stream(stream)), "ipv_ckv_step")
    if isinstance(n_tokens, int):
        return n_out[0], bool(comp[0])
    return list(n_out), [bool(c) for c in comp]


def ipv_ckv_stream(K, V, frame_idx, patch_idx, n_tokens, frames_K, frames_V, first_frame_id, mem_cap, budget,
                   alpha, recent_frames, cv_tau, tar, van, keep_idx, ws, grid_h, grid_w, stream=None, mode=0):
    """Frames frames_K/V[f] ([F, B, L, H, rows, D]) through ipv_ckv_step one
    after another in one library call. Returns (row counts, passes per
    stream): ints for an int n_tokens, else lists."""
    s = shape_of(K, grid_h, grid_w)
    _check_cache(K, V, frame_idx, patch_idx)
    if frames_K.dtype != K.dtype or frames_V.dtype != K.dtype:
        raise IpvError(ERR_DTYPE, "frames_K/V must have the cache's dtype")
    if frames_K.shape != frames_V.shape or frames_K.dim() != 6 or frames_K.shape[1:4] != K.shape[:3] \
            or frames_K.shape[5] != K.shape[4]:
        raise IpvError(ERR_SHAPE, "frames_K/V must be [F, B, L, H, rows, D] like the cache")
    _check_pass_buffers(K, V, frame_idx, patch_idx, tar, van, keep_idx, budget, ws, optional=True, mode=mode)
    tau = None if cv_tau is None else (ctypes.c_double * 3)(*cv_tau)
    ns = counts(n_tokens, s.streams)
    passes = (ctypes.c_int32 * s.streams)()
    _check(lib().ipv_ckv_stream(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(frame_idx), _ptr(patch_idx), ns,
                                _ptr(frames_K), _ptr(frames_V), frames_K.shape[0], frames_K.shape[4], first_frame_id,
                                mem_cap, budget, float(alpha), recent_frames, mode,
                                None if tau is None else ctypes.addressof(tau), _ptr(tar), _ptr(van), _ptr(keep_idx),
                                _ptr(ws), _ws_bytes(ws), passes, _stream(stream)), "ipv_ckv_stream")
    if isinstance(n_tokens, int):
        return ns[0], passes[0]
    return list(ns), list(passes)


def ipv_clear_device_errors(ws, stream=None):
    _check(lib().ipv_clear_device_errors(_ptr(ws), _ws_bytes(ws), _stream(stream)), "ipv_clear_device_errors")


def ipv_read_device_errors(ws, stream=None) -> int:
    out = ctypes.c_uint32(0)
    _check(lib().ipv_read_device_errors(_ptr(ws), _ws_bytes(ws), _stream(stream), ctypes.byref(out)),
           "ipv_read_device_errors")
    return out.value


class Compressor:
    """Buffers for repeated passes over caches of one shape.

    Holds the score, keep-index and workspace tensors so a pass allocates
    nothing; ``compress`` runs the whole pass on the current stream.
    """

    def __init__(self, K: torch.Tensor, grid_h: int, grid_w: int, budget: int):
        self.grid_h, self.grid_w, self.budget = grid_h, grid_w, budget
        self.shape = shape_of(K, grid_h, grid_w)
        B, L, H, S, D = K.shape
        dev = K.device
        self.tar = torch.zeros((B, L, H, S), dtype=torch.float32, device=dev)
        self.van = torch.zeros((B, L, H, S), dtype=torch.float32, device=dev)
        self.keep_idx = torch.zeros((B, L, H, budget), dtype=torch.int32, device=dev)
        self.ws = alloc_workspace(self.shape, dev)

    def compress(self, K, V, frame_idx, patch_idx, n_tokens, alpha, recent_frames, cv_tau=None, stream=None,
                 mode=0):
        ipv_compress(K, V, frame_idx, patch_idx, n_tokens, self.budget, alpha, recent_frames, cv_tau, self.tar,
                     self.van, self.keep_idx, self.ws, self.grid_h, self.grid_w, stream, mode)

    def device_errors(self) -> int:
        return ipv_read_device_errors(self.ws)
