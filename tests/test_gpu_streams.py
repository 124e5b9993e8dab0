"""GPU parity with per-stream row counts: a batch whose streams are at
different fill levels, compressed in one call, against the oracle stream by
stream; a stream with 0 rows must come out untouched."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu

GH = GW = 14
P_ROWS = GH * GW


def batch(counts, L=4, H=2, D=128, S=None, seed=300):
    """[B, L, H, S, D] bf16 caches, stream b holding counts[b] rows of its own stream."""
    S = S or max(counts)
    sts = [synth.fresh_cache(seed + b, L, H, S, D, GH, GW, n, synth.BF16, synth.RhoSpec(0.0, 0.99, 0.3))
           for b, n in enumerate(counts)]
    st = lambda a: np.ascontiguousarray(np.stack([getattr(x, a) for x in sts]))
    return st("K"), st("V"), st("frame_idx"), st("patch_idx")


@pytest.mark.parametrize("mode", [0, ipv.TAR_ADJACENT | ipv.HEAD_SHARED])
def test_streams_at_different_fill_levels(mode):
    counts = [6272, 5000, 5000, 0, 4900]  # runs: {0}, {1, 2}, {3} left alone, {4}
    budget, alpha, r = 2400, 0.5, 4
    K, V, fr, pa = batch(counts)
    print("counts %s budget %d mode %d" % (counts, budget, mode), flush=True)
    Kd, Vd = P.to_device(K, "bf16"), P.to_device(V, "bf16")
    frd, pad = P.to_device(fr), P.to_device(pa)
    comp = ipv.Compressor(Kd, GH, GW, budget)
    comp.tar.fill_(-7.0)
    comp.van.fill_(-7.0)
    comp.keep_idx.fill_(-7)
    ipv.ipv_compress(Kd, Vd, frd, pad, counts, budget, alpha, r, None, comp.tar, comp.van, comp.keep_idx, comp.ws,
                     GH, GW, mode=mode)
    torch.cuda.synchronize()
    assert comp.device_errors() == 0
    got_all = P.GpuPass(comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy(), P.to_host(Kd),
                        P.to_host(Vd), frd.cpu().numpy(), pad.cpu().numpy(), 0)
    for b, n in enumerate(counts):
        sl = slice(b, b + 1)
        if n == 0:
            assert np.array_equal(got_all.K[sl].view(np.uint8), K[sl].view(np.uint8))
            assert np.array_equal(got_all.V[sl].view(np.uint8), V[sl].view(np.uint8))
            assert np.array_equal(got_all.frame_idx[sl], fr[sl]) and np.array_equal(got_all.patch_idx[sl], pa[sl])
            assert np.all(got_all.tar[sl] == -7.0) and np.all(got_all.keep[sl] == -7)
            continue
        got = P.GpuPass(got_all.tar[sl], got_all.van[sl], got_all.keep[sl], got_all.K[sl], got_all.V[sl],
                        got_all.frame_idx[sl], got_all.patch_idx[sl], 0)
        near = P.check_pass("stream %d" % b, K[sl], V[sl], fr[sl], pa[sl], n, budget, alpha, r, GH, GW, mode, got)
        print("  stream %d (n=%d): near-threshold rows %d" % (b, n, near), flush=True)


def test_ckv_step_streams_trigger_independently():
    # three streams start at different fill levels, so their passes fire at different steps
    L, H, D = 2, 2, 64
    cap, budget, r, alpha = 12 * P_ROWS, 6 * P_ROWS + 10, 2, 0.5
    S = cap + P_ROWS
    frames = 30
    start = [0, 3, 7]
    B = len(start)
    src = [synth.fresh_cache(400 + b, L, H, (frames + 8) * P_ROWS, D, GH, GW, (frames + 8) * P_ROWS, synth.BF16,
                             synth.RhoSpec(0.0, 0.95)) for b in range(B)]
    Ko = np.zeros((B, L, H, S, D), np.uint16)
    Vo = np.zeros_like(Ko)
    fo = np.full((B, L, H, S), -1, np.int32)
    po = np.full((B, L, H, S), -1, np.int32)
    n = [0] * B
    for b in range(B):  # stream b starts with its first start[b] frames in the cache
        rows = start[b] * P_ROWS
        Ko[b, :, :, :rows], Vo[b, :, :, :rows] = src[b].K[:, :, :rows], src[b].V[:, :, :rows]
        fo[b, :, :, :rows], po[b, :, :, :rows] = src[b].frame_idx[:, :, :rows], src[b].patch_idx[:, :, :rows]
        n[b] = rows
    Kd, Vd, fd, pd = P.to_device(Ko, "bf16"), P.to_device(Vo, "bf16"), P.to_device(fo), P.to_device(po)
    comp = ipv.Compressor(Kd, GH, GW, budget)
    fired_at = [[] for _ in range(B)]
    for step in range(frames):
        # every stream receives its own next frame; one frame id per call, above every id in the caches
        fid = 100 + step
        rows_of = lambda a, b: a[:, :, (start[b] + step) * P_ROWS:(start[b] + step + 1) * P_ROWS]
        kn = np.ascontiguousarray(np.stack([rows_of(src[b].K, b) for b in range(B)]))
        vn = np.ascontiguousarray(np.stack([rows_of(src[b].V, b) for b in range(B)]))
        before = (Ko.copy(), Vo.copy(), fo.copy(), po.copy())
        n_gpu, fired = ipv.ipv_ckv_step(Kd, Vd, fd, pd, list(n), P.to_device(kn, "bf16"), P.to_device(vn, "bf16"),
                                        fid, 0, cap, budget, alpha, r, None, comp.tar, comp.van, comp.keep_idx,
                                        comp.ws, GH, GW)
        torch.cuda.synchronize()
        assert comp.device_errors() == 0
        for b in range(B):
            sl = slice(b, b + 1)
            n_prev = n[b]
            nb, out = oracle.ckv_step(Ko[sl], Vo[sl], fo[sl], po[sl], n_prev, kn[sl], vn[sl], fid, 0, cap, budget,
                                      alpha, r, GH, GW)
            assert n_gpu[b] == nb and fired[b] == (out is not None), "step %d stream %d" % (step, b)
            n[b] = nb
            if not fired[b]:
                continue
            fired_at[b].append(step)
            Kb, Vb, fb, pb = (np.ascontiguousarray(a[sl]) for a in before)
            n_full = oracle.append(Kb, Vb, fb, pb, n_prev, kn[sl], vn[sl], fid)
            got = P.GpuPass(comp.tar[sl].cpu().numpy(), comp.van[sl].cpu().numpy(), comp.keep_idx[sl].cpu().numpy(),
                            P.to_host(Kd[sl]), P.to_host(Vd[sl]), fd[sl].cpu().numpy(), pd[sl].cpu().numpy(), 0)
            P.check_pass("step %d stream %d" % (step, b), Kb, Vb, fb, pb, n_full, budget, alpha, r, GH, GW, 0, got)
        # teacher forcing: the oracle's state becomes the device state
        Kd.copy_(P.to_device(Ko, "bf16"))
        Vd.copy_(P.to_device(Vo, "bf16"))
        fd.copy_(P.to_device(fo))
        pd.copy_(P.to_device(po))
    print("passes at steps %s" % fired_at, flush=True)
    assert all(fired_at) and len({tuple(x) for x in fired_at}) == B  # every stream fired, at different steps
