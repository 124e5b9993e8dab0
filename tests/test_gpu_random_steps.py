"""Seeded random configurations through the four step entry points one after
another (ipv_tar_scores, ipv_van_scores, ipv_select, ipv_compact), which run
kernels of their own (the table alone, the VaN-only sweep, a compaction that
clears its flags itself), checked against the oracle with the same rules as
the whole pass; the draws are those of the whole-pass random test."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2506_15745_amd import ipv
from tests import parity as P
from tests.test_gpu_random import draw

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seed", range(1024))
def test_random_configuration_by_steps(seed):
    c = draw(seed)
    print("draw", seed, c, flush=True)
    sts = [synth.fresh_cache(7000 + 31 * seed + b, c["L"], c["H"], c["S"], c["D"], c["gh"], c["gw"], n, c["dtype"],
                             synth.RhoSpec(0.0, 0.99, 0.3), (0.1, 0.55, 1.0)) for b, n in enumerate(c["counts"])]
    st = lambda a: np.ascontiguousarray(np.stack([getattr(x, a) for x in sts]))
    K, V, fr, pa = st("K"), st("V"), st("frame_idx"), st("patch_idx")
    kind = "bf16" if c["dtype"] == synth.BF16 else "raw"
    Kd, Vd, frd, pad = P.to_device(K, kind), P.to_device(V, kind), P.to_device(fr), P.to_device(pa)
    gh, gw, mode, counts = c["gh"], c["gw"], c["mode"], c["counts"]
    comp = ipv.Compressor(Kd, gh, gw, c["budget"])
    pool = torch.zeros(K.shape[:2], dtype=torch.int32, device="cuda:0")
    if not mode & ipv.UNIFORM_SELECT:
        ipv.ipv_tar_scores(Kd, frd, pad, counts, c["r"], comp.tar, comp.ws, gh, gw, mode=mode & ipv.TAR_ADJACENT)
        ipv.ipv_van_scores(Vd, frd, pad, counts, c["tau"], comp.van, pool, comp.ws, gh, gw)
    ipv.ipv_select(comp.tar, comp.van, frd, counts, c["budget"], c["alpha"], c["r"], comp.keep_idx, comp.ws, gh, gw,
                   head_dim=c["D"], dtype=c["dtype"], mode=mode)
    ipv.ipv_compact(Kd, Vd, frd, pad, counts, comp.keep_idx, c["budget"], comp.ws, gh, gw)
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    tar, van, keep = comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy()
    Kg, Vg, fg, pg = P.to_host(Kd), P.to_host(Vd), frd.cpu().numpy(), pad.cpu().numpy()
    for b, n in enumerate(counts):
        sl = slice(b, b + 1)
        if n == 0:
            assert np.array_equal(Kg[sl].view(np.uint8), K[sl].view(np.uint8))
            continue
        got = P.GpuPass(tar[sl], van[sl], keep[sl], Kg[sl], Vg[sl], fg[sl], pg[sl], 0)
        near = P.check_pass("seed %d stream %d" % (seed, b), K[sl], V[sl], fr[sl], pa[sl], n, c["budget"],
                            c["alpha"], c["r"], gh, gw, mode, got, c["tau"])
        if c["tau"] is not None and not mode & ipv.UNIFORM_SELECT:
            # the layer-adaptive pooling windows the VaN step chose
            _, opool = oracle.van_scores(V[sl], fr[sl], pa[sl], n, gh, gw, c["tau"])
            assert np.array_equal(pool.cpu().numpy()[sl], opool), "pooling windows differ"
        print("  stream %d: n=%d near-threshold rows %d" % (b, n, near), flush=True)
