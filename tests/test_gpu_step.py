"""GPU parity of the single-token decode step (bla_step) against the float64 oracle."""
import math

import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle
from test_gpu_parity import TOL, _bla, _say, assert_close, gauss, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,d,M,S,T,L", [
    (3, 2, 32, 8, 15, (15.0, 30.0), 40),
    (2, 3, 64, 24, 40, (47.0, 94.0, 60.5), 100),
    (4, 1, 128, 16, 31, (31.0,), 10),
    (2, 2, 64, 64, 64, (127.0, 254.0), 300),
    (2, 2, 128, 128, 256, (255.0, 510.0), 20),        # largest modes and slots (512-thread workgroup)
    (2, 1, 32, 100, 120, (199.0,), 50),               # padded modes and slots, d = 32
])
def test_step_small(dtype, B, H, d, M, S, T, L):
    bla = _bla()
    q, k, v = gauss(B * 100 + M, B, H, L + 1, d, dtype)
    _, sk, sv = oracle.forward(q[:, :, :L], k[:, :, :L], v[:, :, :L], T, M, S)
    sk32 = sk.astype(np.float32)
    sv32 = sv.astype(np.float32)
    pos = np.array([L + 3 * b for b in range(B)], np.int64)   # per-row positions
    ref_o, ref_k, ref_v = oracle.step(q[:, :, L], k[:, :, L], v[:, :, L], T, M, S, sk32, sv32, pos)
    tsk = torch.from_numpy(sk32).cuda()
    tsv = torch.from_numpy(sv32).cuda()
    o = bla.step(to_dev(q[:, :, L], dtype), to_dev(k[:, :, L], dtype), to_dev(v[:, :, L], dtype), T, M, S,
                 tsk, tsv, pos=torch.from_numpy(pos).cuda())
    torch.cuda.synchronize()
    tol = TOL[dtype]
    assert_close(o.float().cpu().numpy(), ref_o, tol, "o")
    assert_close(tsk.cpu().numpy(), ref_k, 1e-5, "state_k")
    assert_close(tsv.cpu().numpy(), ref_v, 1e-5, "state_v")


def test_step_first_token_mask():
    """At position 0 only slot 0 is visible: o = v for any q, k (start mask, Eq. output)."""
    bla = _bla()
    B, H, d, M, S = 2, 2, 32, 6, 11
    q, k, v = gauss(3, B, H, 1, d, torch.float32)
    tsk = torch.zeros(B, H, 2, M, d, device="cuda")
    tsv = torch.zeros(B, H, 2, M, d, device="cuda")
    o = bla.step(to_dev(q[:, :, 0], torch.float32), to_dev(k[:, :, 0], torch.float32),
                 to_dev(v[:, :, 0], torch.float32), (11.0, 20.0), M, S, tsk, tsv, t0=0)
    torch.cuda.synchronize()
    assert_close(o.cpu().numpy(), v[:, :, 0], 1e-5, "o at position 0")


def test_workload5_decode():
    """Decode workload: B=512, H=16, d=M=S=64.  Prefill 2048 tokens with bla_forward, then
    bla_step at position 2048.  Checked on three batch rows (all heads): (a) the whole GPU path
    against the oracle's prefill + step; (b) the step alone from the oracle's prefill state."""
    bla = _bla()
    w = bi.WORKLOADS[5]
    T = bi.periods(w.M, w.H)
    L = w.L
    _say("workload 5: generating inputs on the device")
    q, k, v = bi.generate_decode_device("cuda")
    pq, pk, pv = (x[:, :, :L].contiguous() for x in (q, k, v))
    sq, sk_, sv_ = (x[:, :, L].contiguous() for x in (q, k, v))
    _, gk, gv = bla.forward(pq, pk, pv, T, w.M, w.S)
    del pq, pk, pv
    o = bla.step(sq, sk_, sv_, T, w.M, w.S, gk, gv, t0=L)
    torch.cuda.synchronize()
    for b in (0, w.B // 2 + 1, w.B - 1):
        hq = q[b:b + 1].float().cpu().numpy()
        hk = k[b:b + 1].float().cpu().numpy()
        hv = v[b:b + 1].float().cpu().numpy()
        ro, rk, rv = oracle.forward(hq, hk, hv, T, w.M, w.S)
        assert_close(o[b:b + 1].float().cpu().numpy(), ro[:, :, L], 2e-2, f"step o row {b}")
        assert_close(gk[b:b + 1].cpu().numpy(), rk, 2e-2, f"state_k row {b}")
        assert_close(gv[b:b + 1].cpu().numpy(), rv, 2e-2, f"state_v row {b}")
        # (b) the step alone, from the oracle's prefill state cast to float32
        _, pk64, pv64 = oracle.forward(hq[:, :, :L], hk[:, :, :L], hv[:, :, :L], T, w.M, w.S)
        tsk = torch.from_numpy(pk64.astype(np.float32)).cuda()
        tsv = torch.from_numpy(pv64.astype(np.float32)).cuda()
        o2 = bla.step(sq[b:b + 1], sk_[b:b + 1], sv_[b:b + 1], T, w.M, w.S, tsk, tsv, t0=L)
        torch.cuda.synchronize()
        ro2, _, _ = oracle.step(hq[:, :, L], hk[:, :, L], hv[:, :, L], T, w.M, w.S,
                                pk64.astype(np.float32), pv64.astype(np.float32), [L])
        assert_close(o2.float().cpu().numpy(), ro2, 2e-2, f"step-only o row {b}")
