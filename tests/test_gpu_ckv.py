"""GPU continual-compression loop (Algorithm 1) through ipv_append /
ipv_ckv_step against the oracle's loop, teacher-forced at every pass."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2506_15745_amd import ipv
from tests import parity as P

pytestmark = pytest.mark.gpu


def run_loop(L, H, D, gh, gw, frames, cap, budget, r, alpha, dtype, seed, rho_spec, mode=0, cv_tau=None,
             value_sigma=(0.5,)):
    p = gh * gw
    S = cap + p
    full = synth.fresh_cache(seed, L, H, frames * p, D, gh, gw, frames * p, dtype, rho_spec, value_sigma)
    kind = "bf16" if dtype == synth.BF16 else "raw"
    edt = np.uint16 if dtype == synth.BF16 else np.float32
    # oracle state
    Ko = np.zeros((1, L, H, S, D), edt)
    Vo = np.zeros_like(Ko)
    fo = np.full((1, L, H, S), -1, np.int32)
    po = np.full((1, L, H, S), -1, np.int32)
    # device state
    Kd, Vd, fd, pd = P.to_device(Ko, kind), P.to_device(Vo, kind), P.to_device(fo), P.to_device(po)
    comp = ipv.Compressor(Kd, gh, gw, budget)
    n = n_gpu = 0
    passes = near = 0
    for f in range(frames):
        kn = np.ascontiguousarray(full.K[None, :, :, f * p:(f + 1) * p])
        vn = np.ascontiguousarray(full.V[None, :, :, f * p:(f + 1) * p])
        before, n_prev = (Ko.copy(), Vo.copy(), fo.copy(), po.copy()), n
        n_gpu, fired = ipv.ipv_ckv_step(Kd, Vd, fd, pd, n_gpu, P.to_device(kn, kind), P.to_device(vn, kind), f, 0,
                                        cap, budget, alpha, r, cv_tau, comp.tar, comp.van, comp.keep_idx, comp.ws,
                                        gh, gw, mode=mode)
        n, out = oracle.ckv_step(Ko, Vo, fo, po, n, kn, vn, f, 0, cap, budget, alpha, r, gh, gw, cv_tau,
                                 mode=P.oracle_mode(mode))
        assert n_gpu == n and fired == (out is not None), "frame %d" % f
        torch.cuda.synchronize()
        assert comp.device_errors() == 0
        if not fired:
            # the appended rows arrive bit for bit
            got = P.to_host(Kd)
            assert np.array_equal(got[..., :n, :].view(np.uint8), Ko[..., :n, :].view(np.uint8))
            assert np.array_equal(fd.cpu().numpy()[..., :n], fo[..., :n])
            assert np.array_equal(pd.cpu().numpy()[..., :n], po[..., :n])
            continue
        # a pass ran on the appended cache: compare it like the single-pass parity tests
        Kb, Vb, fb, pb = before
        n_full = oracle.append(Kb, Vb, fb, pb, n_prev, kn, vn, f)
        got = P.GpuPass(comp.tar.cpu().numpy(), comp.van.cpu().numpy(), comp.keep_idx.cpu().numpy(), P.to_host(Kd),
                        P.to_host(Vd), fd.cpu().numpy(), pd.cpu().numpy(), 0)
        near += P.check_pass("pass %d" % passes, Kb, Vb, fb, pb, n_full, budget, alpha, r, gh, gw, mode, got,
                             cv_tau)
        # teacher forcing: the oracle's state becomes the device state
        Kd.copy_(P.to_device(Ko, kind))
        Vd.copy_(P.to_device(Vo, kind))
        fd.copy_(P.to_device(fo))
        pd.copy_(P.to_device(po))
        passes += 1
    print("passes %d, near-threshold rows %d" % (passes, near), flush=True)
    return passes


@pytest.mark.parametrize("dtype,D,gh,gw,cap_frames,budget_extra,r,mode", [
    (synth.BF16, 64, 3, 4, 6, 2, 2, 0),     # budget not a whole number of frames: appends overshoot the cap
    (synth.F32, 32, 2, 5, 8, 0, 1, 0),
    (synth.BF16, 128, 4, 4, 5, 5, 3, 0),
    # the variants over many passes: gappy old frames, heads kept aligned
    (synth.BF16, 128, 3, 4, 6, 2, 2, ipv.HEAD_SHARED | ipv.TAR_ADJACENT),
    (synth.F32, 64, 2, 5, 8, 3, 1, ipv.TAR_ADJACENT | ipv.VAN_REVERSE),
    (synth.BF16, 64, 3, 4, 6, 2, 2, ipv.UNIFORM_SELECT),
])
def test_ckv_loop_matches_oracle(dtype, D, gh, gw, cap_frames, budget_extra, r, mode):
    p = gh * gw
    cap = cap_frames * p
    budget = max(r * p + 1, cap // 2) + budget_extra
    passes = run_loop(2, 2, D, gh, gw, 24, cap, budget, r, 0.5, dtype, 41, synth.RhoSpec(0.0, 0.95), mode)
    assert passes >= 3


def test_ckv_loop_with_layer_adaptive_pooling():
    # value spread cycling over the layers so that different pooling windows occur
    p, r = 16, 2
    cap, budget = 6 * p, 3 * p + 5
    passes = run_loop(4, 2, 64, 4, 4, 20, cap, budget, r, 0.5, synth.BF16, 43, synth.RhoSpec(0.0, 0.95),
                      0, (0.3, 0.5, 0.7), (0.1, 0.35, 0.55, 1.0))
    assert passes >= 3


@pytest.mark.parametrize("mode,dtype,tau", [(0, synth.BF16, None),
                                            (ipv.TAR_ADJACENT | ipv.HEAD_SHARED, synth.BF16, None),
                                            (ipv.VAN_REVERSE, synth.F32, (0.3, 0.5, 0.7)),
                                            (ipv.UNIFORM_SELECT | ipv.HEAD_SHARED, synth.F32, None)])
def test_ckv_stream_equals_step_by_step(mode, dtype, tau):
    # the library-driven loop against the same loop driven from Python, bit for bit,
    # over three streams that start at different fill levels, in two stretches
    L, H, D, gh, gw = 2, 2, 64, 4, 4
    p = gh * gw
    cap, budget, r, frames = 8 * p, 4 * p + 3, 2, 30
    S = cap + p
    B = 3
    src = [synth.fresh_cache(500 + b, L, H, frames * p, D, gh, gw, frames * p, dtype, synth.RhoSpec(0.0, 0.95))
           for b in range(B)]
    kind = "bf16" if dtype == synth.BF16 else "raw"
    tdt, bits = (torch.bfloat16, torch.int16) if dtype == synth.BF16 else (torch.float32, torch.int32)
    fK = np.ascontiguousarray(np.stack([np.stack([s.K[:, :, f * p:(f + 1) * p] for s in src]) for f in range(frames)]))
    fV = np.ascontiguousarray(np.stack([np.stack([s.V[:, :, f * p:(f + 1) * p] for s in src]) for f in range(frames)]))
    fKd, fVd = P.to_device(fK, kind), P.to_device(fV, kind)
    start = [0, 2 * p, 5 * p]

    def fresh():
        K = torch.zeros((B, L, H, S, D), dtype=tdt, device="cuda:0")
        V = torch.zeros_like(K)
        fr = torch.full((B, L, H, S), -1, dtype=torch.int32, device="cuda:0")
        pa = torch.full_like(fr, -1)
        for b in range(B):  # some rows already present: frames -10.. of their own
            if start[b]:
                K[b, :, :, :start[b]] = fKd[0, b, :, :, :1].expand(L, H, start[b], D)
                V[b, :, :, :start[b]] = fVd[0, b, :, :, :1].expand(L, H, start[b], D)
                fr[b, :, :, :start[b]] = torch.arange(start[b], device="cuda:0", dtype=torch.int32) // p - 10
                pa[b, :, :, :start[b]] = torch.arange(start[b], device="cuda:0", dtype=torch.int32) % p
        return K, V, fr, pa, ipv.Compressor(K, gh, gw, budget)

    # step by step from Python
    K1, V1, f1, p1, c1 = fresh()
    n1, passes1 = list(start), [0] * B
    for f in range(frames):
        n1, fired = ipv.ipv_ckv_step(K1, V1, f1, p1, n1, fKd[f], fVd[f], f, 0, cap, budget, 0.5, r, tau, c1.tar,
                                     c1.van, c1.keep_idx, c1.ws, gh, gw, mode=mode)
        passes1 = [a + int(x) for a, x in zip(passes1, fired)]
    # the library's loop, in two stretches
    K2, V2, f2, p2, c2 = fresh()
    n2, pa_ = ipv.ipv_ckv_stream(K2, V2, f2, p2, list(start), fKd[:11], fVd[:11], 0, cap, budget, 0.5, r, tau,
                                 c2.tar, c2.van, c2.keep_idx, c2.ws, gh, gw, mode=mode)
    # problems only the device sees accumulate in the error word over a call's passes
    assert c2.device_errors() == 0
    n2, pb_ = ipv.ipv_ckv_stream(K2, V2, f2, p2, n2, fKd[11:], fVd[11:], 11, cap, budget, 0.5, r, tau,
                                 c2.tar, c2.van, c2.keep_idx, c2.ws, gh, gw, mode=mode)
    torch.cuda.synchronize()
    assert c1.device_errors() == 0 and c2.device_errors() == 0
    assert n2 == n1 and [a + b for a, b in zip(pa_, pb_)] == passes1 and min(passes1) >= 2
    for b in range(B):
        m = n1[b]
        assert torch.equal(K1[b, :, :, :m].view(bits), K2[b, :, :, :m].view(bits))
        assert torch.equal(V1[b, :, :, :m].view(bits), V2[b, :, :, :m].view(bits))
        assert torch.equal(f1[b, :, :, :m], f2[b, :, :, :m]) and torch.equal(p1[b, :, :, :m], p2[b, :, :, :m])
    print("passes per stream %s, final rows %s" % (passes1, n1), flush=True)
