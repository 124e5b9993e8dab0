"""The Python binding refuses companion tensors that do not match the cache.

The C ABI only sees pointers, so a score, keep-index or metadata tensor
smaller than the cache implies would be written past its end; the binding
checks shape, dtype and device of every tensor first. These checks run before
any pointer is taken, so host tensors exercise them without a GPU (a fully
consistent set of host tensors is then refused for not being in GPU memory).
"""
import pytest
import torch

from paper_2506_15745_amd import ipv

B, L, H, S, D, GH, GW, C = 1, 2, 2, 64, 32, 4, 4, 32


def bufs(dtype=torch.bfloat16):
    K = torch.zeros(B, L, H, S, D, dtype=dtype)
    return dict(K=K, V=torch.zeros_like(K), fr=torch.zeros(B, L, H, S, dtype=torch.int32),
                pa=torch.zeros(B, L, H, S, dtype=torch.int32), tar=torch.zeros(B, L, H, S),
                van=torch.zeros(B, L, H, S), keep=torch.zeros(B, L, H, C, dtype=torch.int32),
                ws=torch.zeros(1 << 16, dtype=torch.uint8), pool=torch.zeros(B, L, dtype=torch.int32))


def compress(b, budget=C):
    ipv.ipv_compress(b["K"], b["V"], b["fr"], b["pa"], S, budget, 0.5, 1, None, b["tar"], b["van"], b["keep"],
                     b["ws"], GH, GW)


def status(fn, *a, **kw):
    with pytest.raises(ipv.IpvError) as e:
        fn(*a, **kw)
    return e.value.status


@pytest.mark.parametrize("key,bad,st", [
    ("keep", torch.zeros(B, L, H, C - 1, dtype=torch.int32), ipv.ERR_SHAPE),   # shorter than the budget
    ("keep", torch.zeros(B, L, H, C, dtype=torch.int64), ipv.ERR_DTYPE),
    ("tar", torch.zeros(B, L, H, S - 1), ipv.ERR_SHAPE),                       # fewer rows than the cache
    ("van", torch.zeros(B, L, 1, S), ipv.ERR_SHAPE),
    ("van", torch.zeros(B, L, H, S, dtype=torch.float64), ipv.ERR_DTYPE),
    ("V", torch.zeros(B, L, H, S, D, dtype=torch.float32), ipv.ERR_DTYPE),     # fp32 V with a bf16 K
    ("V", torch.zeros(B, L, H, S - 8, D, dtype=torch.bfloat16), ipv.ERR_SHAPE),
    ("fr", torch.zeros(B, L, H, S, dtype=torch.int64), ipv.ERR_DTYPE),
    ("pa", torch.zeros(B, L, H, S // 2, dtype=torch.int32), ipv.ERR_SHAPE),
    ("keep", None, ipv.ERR_NULL),
    ("ws", None, ipv.ERR_WORKSPACE),
])
def test_compress_refuses_mismatched_tensors(key, bad, st):
    b = bufs()
    b[key] = bad
    assert status(compress, b) == st


def test_consistent_host_tensors_reach_the_device_check():
    assert status(compress, bufs()) == ipv.ERR_ARG


def test_keep_width_follows_the_budget():
    b = bufs()
    assert status(compress, b, budget=C - 1) == ipv.ERR_SHAPE


def test_step_entry_points_check_their_tensors():
    b = bufs()
    assert status(ipv.ipv_tar_scores, b["K"], b["fr"], b["pa"], S, 1, torch.zeros(B, L, H, 8), b["ws"], GH,
                  GW) == ipv.ERR_SHAPE
    assert status(ipv.ipv_van_scores, b["V"], b["fr"], b["pa"], S, None, b["van"], torch.zeros(B, L + 1,
                  dtype=torch.int32), b["ws"], GH, GW) == ipv.ERR_SHAPE
    assert status(ipv.ipv_select, b["tar"], b["van"], b["fr"], S, C, 0.5, 1, torch.zeros(B, L, H, 8,
                  dtype=torch.int32), b["ws"], GH, GW) == ipv.ERR_SHAPE
    assert status(ipv.ipv_select, b["tar"], torch.zeros(B, L, H, S, dtype=torch.float16), b["fr"], S, C, 0.5, 1,
                  b["keep"], b["ws"], GH, GW) == ipv.ERR_DTYPE
    assert status(ipv.ipv_compact, b["K"], b["V"], b["fr"], b["pa"], S, b["keep"], C + 1, b["ws"], GH,
                  GW) == ipv.ERR_SHAPE


def test_append_and_loop_check_new_rows():
    b = bufs()
    Kn = torch.zeros(B, L, H, 16, D, dtype=torch.float32)   # fp32 rows into a bf16 cache
    assert status(ipv.ipv_append, b["K"], b["V"], b["fr"], b["pa"], 0, Kn, Kn, 0, 0, GH, GW) == ipv.ERR_DTYPE
    Kn = torch.zeros(B, L, H + 1, 16, D, dtype=torch.bfloat16)
    assert status(ipv.ipv_append, b["K"], b["V"], b["fr"], b["pa"], 0, Kn, Kn, 0, 0, GH, GW) == ipv.ERR_SHAPE
    Kn = torch.zeros(B, L, H, 16, D, dtype=torch.bfloat16)
    assert status(ipv.ipv_ckv_step, b["K"], b["V"], b["fr"], b["pa"], 0, Kn, Kn, 0, 0, 48, C, 0.5, 1, None,
                  b["tar"], b["van"], torch.zeros(B, L, H, C + 4, dtype=torch.int32), b["ws"], GH,
                  GW) == ipv.ERR_SHAPE
    Fk = torch.zeros(3, B, L, H, 16, D, dtype=torch.float32)
    assert status(ipv.ipv_ckv_stream, b["K"], b["V"], b["fr"], b["pa"], 0, Fk, Fk, 0, 48, C, 0.5, 1, None,
                  b["tar"], b["van"], b["keep"], b["ws"], GH, GW) == ipv.ERR_DTYPE
