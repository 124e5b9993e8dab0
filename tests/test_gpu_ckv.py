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
