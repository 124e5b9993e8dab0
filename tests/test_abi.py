"""The C ABI on the host: the library loads, exports every function the
header declares, and rejects bad arguments before anything is launched.

Every call here carries at least one argument the host checks reject, so no
kernel is ever enqueued (these tests run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2506_15745_amd import ipv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    with open(os.path.join(ROOT, "include", "ipv.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ipv_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert "ipv_compress" in names and len(names) >= 10
    L = ipv.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(ipv.EXPORTS)


def test_status_strings():
    for s in range(9):
        assert ipv.status_str(s) and ipv.status_str(s) != "unknown status"
    assert ipv.lib().ipv_status_str(1234) == b"unknown status"


SEVEN_B = dict(streams=1, layers=28, kv_heads=4, head_dim=128, capacity=6272, grid_h=14, grid_w=14, dtype=0)
FAKE = 0x10000  # a 256-aligned non-null address; never dereferenced because another argument is rejected


def N(*vals):
    """Host array of per-stream row counts."""
    return (ctypes.c_int32 * len(vals))(*vals)


def shape(**kw):
    d = dict(SEVEN_B)
    d.update(kw)
    return ipv.Shape(*[d[k] for k in ("streams", "layers", "kv_heads", "head_dim", "capacity", "grid_h", "grid_w",
                                      "dtype")])


def ws_bytes(s):
    return ipv.workspace_bytes(s)


def test_workspace_size_covers_the_recent_table():
    s = shape()
    assert ws_bytes(s) >= 256 + 28 * 4 * 196 * 128 * 4
    with pytest.raises(ipv.IpvError) as e:
        ipv.workspace_bytes(shape(head_dim=96))
    assert e.value.status == ipv.ERR_SHAPE
    with pytest.raises(ipv.IpvError) as e:
        ipv.workspace_bytes(shape(dtype=7))
    assert e.value.status == ipv.ERR_DTYPE


def call_compress(s, n=6272, budget=3136, alpha=0.5, r=4, tau=None, ptrs=None, ws=FAKE, wsb=None, K=FAKE, mode=0):
    p = dict(K=K, V=FAKE, fr=FAKE, pa=FAKE, tar=FAKE, van=FAKE, keep=FAKE)
    if ptrs:
        p.update(ptrs)
    t = None if tau is None else (ctypes.c_double * 3)(*tau)
    wsb = wsb if wsb is not None else 0  # default: workspace too small
    ns = N(*([n] * s.streams)) if isinstance(n, int) else N(*n)
    return ipv.lib().ipv_compress(ctypes.byref(s), p["K"], p["V"], p["fr"], p["pa"], ns, budget, alpha, r, mode,
                                  None if t is None else ctypes.addressof(t), p["tar"], p["van"], p["keep"], ws,
                                  wsb, None)


@pytest.mark.parametrize("case,status", [
    (dict(ptrs=dict(K=None)), ipv.ERR_NULL),
    (dict(ptrs=dict(keep=None)), ipv.ERR_NULL),
    (dict(ptrs=dict(V=FAKE + 8)), ipv.ERR_ALIGN),
    (dict(ptrs=dict(tar=FAKE + 4)), ipv.ERR_ALIGN),
    (dict(n=-1), ipv.ERR_SHAPE),
    (dict(n=6273), ipv.ERR_SHAPE),                # n > capacity
    (dict(budget=6273), ipv.ERR_BUDGET),          # budget > n
    (dict(budget=0), ipv.ERR_BUDGET),
    # below r * p passes the host's budget check (only the device sees the
    # window's size); the zero-byte workspace is what is refused here
    (dict(budget=783), ipv.ERR_WORKSPACE),
    (dict(alpha=1.5), ipv.ERR_ARG),
    (dict(alpha=float("nan")), ipv.ERR_ARG),
    (dict(r=0), ipv.ERR_ARG),
    (dict(r=257), ipv.ERR_ARG),
    (dict(tau=(0.5, 0.3, 0.7)), ipv.ERR_ARG),
    (dict(tau=(0.1, float("inf"), 0.7)), ipv.ERR_ARG),
    (dict(ws=None), ipv.ERR_WORKSPACE),
    (dict(ws=FAKE + 16), ipv.ERR_ALIGN),
    (dict(), ipv.ERR_WORKSPACE),                  # ws_bytes = 0
    (dict(mode=32, wsb=1 << 40), ipv.ERR_ARG),    # unknown mode bit
    (dict(mode=0xffffffff, wsb=1 << 40), ipv.ERR_ARG),
])
def test_compress_rejects_before_launch(case, status):
    assert call_compress(shape(), **case) == status


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=100), ipv.ERR_SHAPE),
    (dict(streams=0), ipv.ERR_SHAPE),
    (dict(grid_w=0), ipv.ERR_SHAPE),
    (dict(grid_h=100, grid_w=100), ipv.ERR_SHAPE),   # more patches than the pooling grid holds
    (dict(dtype=3), ipv.ERR_DTYPE),
])
def test_bad_shapes(kw, status):
    assert call_compress(shape(**kw), wsb=1 << 40) == status


def test_slice_bytes_beyond_32_bit_offsets_rejected():
    # buffer loads address a slice with 32-bit byte offsets: S * D * elem must fit
    s = shape(capacity=(1 << 22) + 1, head_dim=256, dtype=ipv.F32)
    assert call_compress(s, wsb=1 << 50) == ipv.ERR_SHAPE


def test_rows_above_select_limit_rejected():
    s = shape(capacity=70000)
    assert call_compress(s, n=70000, budget=35000, wsb=1 << 40) == ipv.ERR_SHAPE
    assert call_compress(s, n=65537, budget=35000, wsb=1 << 40) == ipv.ERR_SHAPE  # one above the limit


def test_entry_points_validate_their_own_arguments():
    L, s = ipv.lib(), shape()
    big = 1 << 40
    assert L.ipv_tar_scores(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 0, 0, FAKE, FAKE, big, None) == ipv.ERR_ARG
    assert L.ipv_tar_scores(ctypes.byref(s), FAKE, None, FAKE, N(6272), 4, 0, FAKE, FAKE, big, None) == ipv.ERR_NULL
    assert L.ipv_tar_scores(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 4, 32, FAKE, FAKE, big, None) == ipv.ERR_ARG
    assert L.ipv_van_scores(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), None, FAKE, FAKE + 2, FAKE, big,
                            None) == ipv.ERR_ALIGN
    assert L.ipv_select(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 3136, -0.1, 4, 0, FAKE, FAKE, big,
                        None) == ipv.ERR_ARG
    assert L.ipv_select(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 0, 0.5, 4, 0, FAKE, FAKE, big,
                        None) == ipv.ERR_BUDGET
    assert L.ipv_select(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 6273, 0.5, 4, 0, FAKE, FAKE, big,
                        None) == ipv.ERR_BUDGET
    # a budget below r * p is the device's to judge: here the small workspace is refused
    assert L.ipv_select(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 100, 0.5, 4, 0, FAKE, FAKE, 8,
                        None) == ipv.ERR_WORKSPACE
    assert L.ipv_select(ctypes.byref(s), FAKE, FAKE, FAKE, N(6272), 3136, 0.5, 4, 64, FAKE, FAKE, big,
                        None) == ipv.ERR_ARG
    assert L.ipv_compact(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(6272), FAKE, 0, None, 0, None) == ipv.ERR_BUDGET
    assert L.ipv_compact(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(6272), FAKE + 4, 10, None, 0,
                         None) == ipv.ERR_ALIGN
    assert L.ipv_compact(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(6272), FAKE, 10, FAKE, 8, None) == ipv.ERR_WORKSPACE
    assert L.ipv_clear_device_errors(None, 256, None) == ipv.ERR_NULL
    assert L.ipv_clear_device_errors(FAKE, 8, None) == ipv.ERR_WORKSPACE
    out = ctypes.c_uint32()
    assert L.ipv_read_device_errors(FAKE + 1, 256, None, ctypes.byref(out)) == ipv.ERR_ALIGN
    assert L.ipv_workspace_bytes(None, None) == ipv.ERR_NULL


def test_binding_fails_loudly_without_the_library(monkeypatch):
    monkeypatch.setattr(ipv, "_lib", None)
    monkeypatch.setattr(ipv, "LIB_PATH", "/nonexistent/libipv.so")
    with pytest.raises(ipv.IpvError):
        ipv.lib()


def test_append_and_ckv_step_validate_before_launch():
    L, s = ipv.lib(), shape()
    big = 1 << 40
    # ipv_append(shape, K, V, fr, pa, n, K_new, V_new, rows, frame_id, first_patch, stream)
    assert L.ipv_append(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(0), None, FAKE, 196, 0, 0, None) == ipv.ERR_NULL
    assert L.ipv_append(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(0), FAKE + 4, FAKE, 196, 0, 0, None) == ipv.ERR_ALIGN
    assert L.ipv_append(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(6200), FAKE, FAKE, 196, 0, 0, None) == ipv.ERR_SHAPE
    assert L.ipv_append(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(0), FAKE, FAKE, 0, 0, 0, None) == ipv.ERR_SHAPE
    assert L.ipv_append(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(0), FAKE, FAKE, 100, 0, 97, None) == ipv.ERR_ARG
    n_out, comp = N(0), N(0)

    def step(n=6076, rows=196, cap=6272, budget=3136, tar=FAKE, ws=FAKE, wsb=big, nout=True, mode=0):
        return L.ipv_ckv_step(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(n), FAKE, FAKE, rows, 30, 0, cap, budget, 0.5,
                              4, mode, None, tar, FAKE, FAKE, ws, wsb, n_out if nout else None, comp, None)

    assert step(nout=False) == ipv.ERR_NULL
    assert step(n=6272) == ipv.ERR_SHAPE          # the previous step left the cache at the cap
    assert step(cap=7000) == ipv.ERR_SHAPE        # cap beyond the capacity
    assert step(budget=6300) == ipv.ERR_BUDGET    # budget above the cap
    assert step(tar=None) == ipv.ERR_NULL         # the pass would run: its arguments are checked first
    assert step(wsb=0) == ipv.ERR_WORKSPACE
    assert step(budget=700) == ipv.ERR_BUDGET     # smaller than any window the loop may meet (r * p = 784)
    assert step(mode=128) == ipv.ERR_ARG          # unknown mode bit


def test_per_stream_row_counts_are_validated_before_launch():
    s = shape(streams=3)
    big = 1 << 40
    assert call_compress(s, n=[6272, 6272, 7000], wsb=big) == ipv.ERR_SHAPE     # a count above the capacity
    assert call_compress(s, n=[6272, -1, 6272], wsb=big) == ipv.ERR_SHAPE
    assert call_compress(s, n=[6272, 3000, 6272], wsb=big) == ipv.ERR_BUDGET    # budget above one stream's rows
    L = ipv.lib()
    assert L.ipv_compress(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, None, 3136, 0.5, 4, 0, None, FAKE, FAKE, FAKE,
                          FAKE, big, None) == ipv.ERR_NULL


def test_every_stream_empty_is_a_no_op():
    # no stream has rows: every argument is checked, nothing is launched
    s = shape(streams=2)
    assert call_compress(s, n=[0, 0], wsb=1 << 40) == ipv.OK


def test_binding_row_counts():
    assert list(ipv.counts(6272, 3)) == [6272, 6272, 6272]
    assert list(ipv.counts([1, 2, 3], 3)) == [1, 2, 3]
    with pytest.raises(ipv.IpvError):
        ipv.counts([1, 2], 3)


def test_ckv_step_checks_every_stream():
    s = shape(streams=2)
    L, big = ipv.lib(), 1 << 40
    n_out, comp = N(0, 0), N(0, 0)

    def step(counts, budget=3136):
        return L.ipv_ckv_step(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(*counts), FAKE, FAKE, 196, 30, 0, 6272,
                              budget, 0.5, 4, 0, None, FAKE, FAKE, FAKE, FAKE, big, n_out, comp, None)

    assert step([100, 6272]) == ipv.ERR_SHAPE        # one stream is already at the cap
    assert step([100, -4]) == ipv.ERR_SHAPE
    assert step([6076, 100], budget=700) == ipv.ERR_BUDGET  # stream 0 would run the pass: its budget is checked


def test_ckv_stream_checks_every_step_before_launch():
    s = shape(streams=1)
    L, big = ipv.lib(), 1 << 40
    passes = N(0)

    def run(n=0, frames=40, tar=FAKE, budget=3136, wsb=big, cap=6272, counts=True):
        return L.ipv_ckv_stream(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, N(n) if counts else None, FAKE, FAKE,
                                frames, 196, 0, cap, budget, 0.5, 4, 0, None, tar, FAKE, FAKE, FAKE, wsb, passes,
                                None)

    assert run(counts=False) == ipv.ERR_NULL
    assert run(tar=None) == ipv.ERR_NULL          # the pass at step 31 would need it: rejected up front
    assert run(wsb=0) == ipv.ERR_WORKSPACE
    assert run(budget=600) == ipv.ERR_BUDGET      # below the recent window at the first pass
    assert run(n=6272) == ipv.ERR_SHAPE           # already at the cap
    assert run(cap=7000) == ipv.ERR_SHAPE
    assert run(frames=0) == ipv.OK and passes[0] == 0    # nothing to do, nothing launched


def test_binding_rejects_host_tensors():
    # a host tensor would hand the kernels a host address: the binding refuses it
    import torch
    with pytest.raises(ipv.IpvError) as e:
        ipv._ptr(torch.zeros(4))
    assert e.value.status == ipv.ERR_ARG


def test_budget_from_the_window_up_passes_the_host_checks():
    # the 72B-class layout: 14x14 grid, r = 8, 36 rows in the last frame, so the
    # window holds 1408 rows while r * p = 1568; a budget of 1408 is legal and
    # only the zero-byte workspace is refused here
    s = shape(layers=80, kv_heads=8, capacity=32768)
    assert call_compress(s, n=32768, budget=1408, r=8) == ipv.ERR_WORKSPACE
    assert call_compress(s, n=32768, budget=0, r=8) == ipv.ERR_BUDGET


def test_noalloc_refuses_shapes_beyond_its_workspace():
    # 16 7B-class streams need about 180 MB of workspace, above the 96 MiB array
    L = ipv.lib()
    s = shape(streams=16)
    assert ipv.workspace_bytes(s) > (96 << 20) >= ipv.workspace_bytes(shape(layers=80, kv_heads=8, capacity=32768))
    ns = N(*([6272] * 16))
    args = (FAKE, FAKE, FAKE, FAKE, ns, 3136, 0.5, 4, 0, None, FAKE, FAKE, FAKE, None, None)
    assert L.ipv_compress_noalloc(ctypes.byref(s), *args) == ipv.ERR_WORKSPACE
    # its other arguments are checked like ipv_compress's, before anything else
    s1 = shape()
    assert L.ipv_compress_noalloc(ctypes.byref(s1), FAKE, FAKE, FAKE, FAKE, N(6272), 0, 0.5, 4, 0, None, FAKE, FAKE,
                                  FAKE, None, None) == ipv.ERR_BUDGET
    assert L.ipv_compress_noalloc(ctypes.byref(s1), FAKE, None, FAKE, FAKE, N(6272), 3136, 0.5, 4, 0, None, FAKE,
                                  FAKE, FAKE, None, None) == ipv.ERR_NULL
    assert L.ipv_compress_noalloc(ctypes.byref(s1), FAKE, FAKE, FAKE, FAKE, N(6272), 3136, 0.5, 4, 0, None, FAKE,
                                  FAKE, FAKE, FAKE + 2, None) == ipv.ERR_ALIGN
