"""GPU parity of the state-decay form (Sec. 3.4): bla_decay_forward / bla_decay_step
through the C ABI against the oracle's token-by-token decayed slot recurrence.

Bars as for the other forms: rel-L2 <= 1e-4 (float32 inputs) and <= 2e-2 (bfloat16),
on the outputs and on the slot states.
"""
import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle
from test_gpu_parity import TOL, _bla, _say, assert_close, gauss, to_dev

pytestmark = pytest.mark.gpu


def run_decay(q, k, v, T, M, S, dtype, t0=0, sk=None, sv=None, label=""):
    bla = _bla()
    _say(f"decay case {label}: shape {q.shape} M={M} S={S} T={list(T)} t0={t0} dtype={dtype}")
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    tsk = None if sk is None else torch.from_numpy(np.ascontiguousarray(sk, np.float32)).cuda()
    tsv = None if sv is None else torch.from_numpy(np.ascontiguousarray(sv, np.float32)).cuda()
    o, ok, ov = bla.decay_forward(tq, tk, tv, T, M, S, t0=t0, slot_k=tsk, slot_v=tsv)
    torch.cuda.synchronize()
    ref_o, ref_k, ref_v = oracle.forward_decay(q, k, v, T, M, S, t0=t0, slot_k=sk, slot_v=sv)
    tol = TOL[dtype]
    assert_close(o.float().cpu().numpy(), ref_o, tol, "O")
    assert_close(ok.cpu().numpy(), ref_k, tol, "slot_k")
    assert_close(ov.cpu().numpy(), ref_v, tol, "slot_v")
    return o, ok, ov


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,L,d,M,S,T,t0", [
    (2, 3, 100, 32, 16, 16, (31.0, 62.0, 40.5), 0),     # ragged last sub-block, non-integer T
    (1, 2, 200, 64, 24, 40, (47.0, 94.0), 0),            # padded slots (40 -> 64)
    (2, 2, 70, 32, 5, 9, (9.0, 9.0), 0),                 # T = S = 2M-1: sliding window, 9-token sub-blocks
    (1, 2, 150, 64, 16, 20, (31.0, 77.25), 1000),        # absolute start far from 0
    (1, 2, 20, 64, 1, 5, (1.0, 6.5), 0),                 # M = 1: every gate flushes (two-token sub-blocks)
    (1, 2, 100, 64, 2, 8, (500.0, 300.0), 0),            # wide main lobe: many small gates in a row
    (1, 2, 90, 128, 32, 64, (63.0, 126.0), 0),           # d = 128: two waves reduce the softmax
    (1, 1, 40, 128, 100, 200, (199.0,), 0),              # 256 padded slots: eight waves
    (1, 1, 1, 64, 4, 4, (7.0,), 5),                      # a single token
])
def test_decay_small_shapes(dtype, B, H, L, d, M, S, T, t0):
    q, k, v = gauss(L * 3 + M + 7, B, H, L, d, dtype)
    run_decay(q, k, v, T, M, S, dtype, t0=t0, label=f"{B}x{H}x{L}x{d}")


def test_decay_many_heads_shared_periods():
    """70 heads whose clamped periods repeat (heads of one period share a gate table; more
    than 64 heads take two table launches), including a period below 2M-1 that clamps onto
    another head's."""
    B, H, L, d, M, S = 2, 70, 45, 32, 4, 7
    base = (7.0, 14.0, 9.5, 3.0)  # 3.0 clamps to 2M-1 = 7, the first period
    T = tuple(base[h % 4] if h != 66 else 11.25 for h in range(H))
    q, k, v = gauss(L + H, B, H, L, d, torch.float32)
    run_decay(q, k, v, T, M, S, torch.float32, t0=13, label=f"{B}x{H}x{L}x{d} shared periods")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decay_is_sliding_window_on_the_gpu(dtype):
    """T = S = 2M-1 (Sec. 3.4): the GPU decay form equals sliding-window attention with
    window 2M-1 (torch float32 attention with a banded causal mask on the CPU)."""
    bla = _bla()
    B, H, L, d, M = 2, 2, 200, 64, 8
    W = 2 * M - 1
    q, k, v = gauss(51, B, H, L, d, dtype)
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    o, _, _ = bla.decay_forward(tq, tk, tv, [float(W)] * H, M, W)
    torch.cuda.synchronize()
    i = torch.arange(L)
    mask = (i[None, :] <= i[:, None]) & (i[None, :] > i[:, None] - W)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).float(), torch.from_numpy(k).float(), torch.from_numpy(v).float(),
        attn_mask=mask, scale=d ** -0.5).numpy()
    assert_close(o.float().cpu().numpy(), ref, TOL[dtype], "O vs sliding-window attention")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_decay_continuation(dtype):
    """Two calls: the second continues from the first one's slot states at t0 = L1."""
    B, H, L1, L2, d, M, S, T = 2, 2, 130, 170, 64, 16, 20, (31.0, 77.25)
    q, k, v = gauss(52, B, H, L1 + L2, d, dtype)
    _, k1, v1 = run_decay(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], T, M, S, dtype, label="part 1")
    o2, _, _ = run_decay(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], T, M, S, dtype, t0=L1,
                         sk=k1.cpu().numpy(), sv=v1.cpu().numpy(), label="part 2")
    ref_o, _, _ = oracle.forward_decay(q, k, v, T, M, S)
    assert_close(o2.float().cpu().numpy(), ref_o[:, :, L1:], TOL[dtype], "O (second call)")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,d,M,S,T,L", [
    (3, 2, 32, 8, 15, (15.0, 30.0), 40),
    (2, 2, 64, 64, 64, (127.0, 254.0), 300),
    (2, 2, 128, 128, 256, (255.0, 510.0), 20),
])
def test_decay_step(dtype, B, H, d, M, S, T, L):
    """Decode step at position L from the oracle's slot states after L tokens, against row L
    of the decay form over L + 1 tokens."""
    bla = _bla()
    q, k, v = gauss(B * 13 + M, B, H, L + 1, d, dtype)
    _say(f"decay step B={B} H={H} d={d} M={M} S={S} L={L} dtype={dtype}")
    _, pk, pv = oracle.forward_decay(q[:, :, :L], k[:, :, :L], v[:, :, :L], T, M, S)
    sk = torch.from_numpy(pk.astype(np.float32)).cuda()
    sv = torch.from_numpy(pv.astype(np.float32)).cuda()
    o = bla.decay_step(to_dev(q[:, :, L], dtype), to_dev(k[:, :, L], dtype), to_dev(v[:, :, L], dtype), T, M,
                       S, sk, sv, t0=L)
    torch.cuda.synchronize()
    ref_o, ref_k, ref_v = oracle.forward_decay(q, k, v, T, M, S)
    assert_close(o.float().cpu().numpy(), ref_o[:, :, L], TOL[dtype], "o")
    assert_close(sk.cpu().numpy(), ref_k, 1e-5, "slot_k")
    assert_close(sv.cpu().numpy(), ref_v, 1e-5, "slot_v")


def test_decay_step_far_positions():
    """Per-row positions up to 2^31 + 7 from a zero state (the gate phase is reduced in
    double precision)."""
    bla = _bla()
    B, H, d, M, S, T = 4, 2, 64, 16, 31, (31.0, 45.5)
    pos = np.array([0, 5, 1_000_003, 2 ** 31 + 7], np.int64)
    q, k, v = gauss(53, B, H, 1, d, torch.float32)
    sk = torch.zeros(B, H, S, d, device="cuda")
    sv = torch.zeros(B, H, S, d, device="cuda")
    o = bla.decay_step(to_dev(q[:, :, 0], torch.float32), to_dev(k[:, :, 0], torch.float32),
                       to_dev(v[:, :, 0], torch.float32), T, M, S, sk, sv, pos=torch.from_numpy(pos).cuda())
    torch.cuda.synchronize()
    for b in range(B):
        ref, _, _ = oracle.forward_decay(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, M, S, t0=int(pos[b]))
        assert_close(o[b:b + 1].cpu().numpy(), ref[:, :, 0], 1e-4, f"o row {b} (pos {pos[b]})")


def test_decay_workload3_sampled_rows():
    """LM-layer shape (B=8, H=16, L=4096, d=M=S=64, bf16) in the decay form; every head of
    the first and last batch row against the oracle."""
    bla = _bla()
    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    q, k, v = bi.generate(3)
    _say(f"workload 3 decay form, full size {q.shape}")
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    o, sk, _ = bla.decay_forward(tq, tk, tv, T, w.M, w.S)
    torch.cuda.synchronize()
    for b in (0, w.B - 1):
        ref_o, ref_k, _ = oracle.forward_decay(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, w.M, w.S)
        assert_close(o[b:b + 1].float().cpu().numpy(), ref_o, 2e-2, f"O row {b}")
        assert_close(sk[b:b + 1].cpu().numpy(), ref_k, 2e-2, f"slot_k row {b}")
