"""GPU parity of the anchored-slot form (Sec. 3.3; Alg. 1 recurrent, Alg. 3 chunked).

The HIP path runs with phase_anchor=1 through the C ABI and is compared with the
oracle's token-by-token Alg. 1 (slot states as cumulative sums).  The state buffers
hold the same mode state in both forms, so the final states are compared with the
rotating oracle's states.  Same bars as the rotating form: rel-L2 <= 1e-4 (float32)
and <= 2e-2 (bfloat16).
"""
import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle
from test_gpu_parity import TOL, _bla, _say, assert_close, gauss, to_dev

pytestmark = pytest.mark.gpu


def run_anchored(q, k, v, T, M, S, dtype, t0=0, sk=None, sv=None, label="", chunk=0):
    bla = _bla()
    _say(f"anchored case {label}: shape {q.shape} M={M} S={S} T={list(T)} t0={t0} dtype={dtype} chunk={chunk}")
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    tsk = None if sk is None else torch.from_numpy(np.ascontiguousarray(sk, np.float32)).cuda()
    tsv = None if sv is None else torch.from_numpy(np.ascontiguousarray(sv, np.float32)).cuda()
    o, ok, ov = bla.forward(tq, tk, tv, T, M, S, t0=t0, state_k=tsk, state_v=tsv, phase_anchor=True,
                            chunk=chunk)
    torch.cuda.synchronize()
    return o.float().cpu().numpy(), ok.cpu().numpy(), ov.cpu().numpy()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,L,d,M,S,T,t0", [
    (2, 3, 100, 32, 16, 16, (31.0, 62.0, 40.5), 0),    # ragged last chunk, non-integer T
    (1, 2, 200, 64, 24, 40, (47.0, 94.0), 0),           # padded modes and slots
    (2, 2, 7, 32, 5, 9, (9.0, 9.0), 0),                 # L < chunk, T = S = 2M-1
    (1, 2, 150, 64, 16, 20, (31.0, 77.25), 1000),       # absolute start far from 0
    (1, 1, 1, 64, 4, 4, (7.0,), 5),                     # a single token
])
def test_anchor_small_shapes(dtype, B, H, L, d, M, S, T, t0):
    q, k, v = gauss(L * 5 + M + 1, B, H, L, d, dtype)
    o, ok, ov = run_anchored(q, k, v, T, M, S, dtype, t0=t0, label=f"{B}x{H}x{L}x{d}")
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S, t0=t0)
    _, ref_k, ref_v = oracle.forward(q, k, v, T, M, S, t0=t0)
    tol = TOL[dtype]
    assert_close(o, ref_o, tol, "O")
    assert_close(ok, ref_k, tol, "state_k")
    assert_close(ov, ref_v, tol, "state_v")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (1, 2, 64 * 37 + 5, 32, 16, 31, (31.0, 62.0)),     # many segments, ragged tail
    (1, 1, 64 * 8 + 20, 64, 64, 64, (127.0,)),         # bf16: idle partner unit in the last workgroup
    (2, 1, 64 * 30 + 33, 64, 64, 64, (127.0, 254.0)),  # several chunks per segment
])
def test_anchor_segments(dtype, B, H, L, d, M, S, T):
    """Segments start at absolute positions far from 0: each unit's twiddle row uses its own
    chunk start, while the entering state comes from the (unchanged) summaries."""
    q, k, v = gauss(L + 17, B, H, L, d, dtype)
    o, ok, ov = run_anchored(q, k, v, T[:H], M, S, dtype, label=f"segments {B}x{H}x{L}")
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T[:H], M, S)
    _, ref_k, ref_v = oracle.forward(q, k, v, T[:H], M, S)
    tol = TOL[dtype]
    assert_close(o, ref_o, tol, "O")
    assert_close(ok, ref_k, tol, "state_k")
    assert_close(ov, ref_v, tol, "state_v")


@pytest.mark.parametrize("chunk", [16, 32, 128])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_anchor_chunk_lengths(dtype, chunk):
    """Anchored slots with chunks of 16, 32 and 128 tokens: each chunk's twiddle row at its own
    absolute start; several segments, ragged tail, t0 > 0."""
    B, H, L, d, M, S, T, t0 = 1, 2, 64 * 21 + 11, 32, 16, 31, (31.0, 45.5), 333
    q, k, v = gauss(L + chunk, B, H, L, d, dtype)
    o, ok, ov = run_anchored(q, k, v, T, M, S, dtype, t0=t0, label=f"chunk {chunk}", chunk=chunk)
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S, t0=t0)
    _, ref_k, ref_v = oracle.forward(q, k, v, T, M, S, t0=t0)
    tol = TOL[dtype]
    assert_close(o, ref_o, tol, "O")
    assert_close(ok, ref_k, tol, "state_k")
    assert_close(ov, ref_v, tol, "state_v")


def test_anchor_eight_waves():
    """bf16, d = M = 128 (eight waves per workgroup), several segments, ragged tail."""
    B, H, L, d, M, S, T = 1, 2, 64 * 11 + 9, 128, 128, 128, (255.0, 510.0)
    q, k, v = gauss(L + 29, B, H, L, d, torch.bfloat16)
    o, ok, ov = run_anchored(q, k, v, T, M, S, torch.bfloat16, label=f"eight waves {B}x{H}x{L}")
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S)
    _, ref_k, ref_v = oracle.forward(q, k, v, T, M, S)
    tol = TOL[torch.bfloat16]
    assert_close(o, ref_o, tol, "O")
    assert_close(ok, ref_k, tol, "state_k")
    assert_close(ov, ref_v, tol, "state_v")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_anchor_continuation(dtype):
    """Two calls: the second continues from the first one's state at t0 = L1 (the state
    handed over is the mode state), against Alg. 1 run once over the whole sequence."""
    B, H, L1, L2, d, M, S, T = 2, 2, 130, 170, 64, 16, 20, (31.0, 77.25)
    q, k, v = gauss(21, B, H, L1 + L2, d, dtype)
    o1, k1, v1 = run_anchored(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], T, M, S, dtype, label="part 1")
    o2, _, _ = run_anchored(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], T, M, S, dtype, t0=L1, sk=k1, sv=v1,
                            label="part 2")
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S)
    assert_close(np.concatenate([o1, o2], axis=2), ref_o, TOL[dtype], "O (two calls)")


def test_anchor_equals_rotating_on_the_integer_grid():
    """T = S = 2M-1: the anchored slots are a permutation of the rotating ones (Sec. 3.3), so
    the two GPU forms agree with each other (and each with its oracle)."""
    bla = _bla()
    B, H, L, d, M = 2, 2, 64 * 5 + 9, 64, 8
    W = 2 * M - 1
    q, k, v = gauss(22, B, H, L, d, torch.float32)
    tq, tk, tv = (to_dev(x, torch.float32) for x in (q, k, v))
    a, _, _ = bla.forward(tq, tk, tv, [float(W)] * H, M, W, phase_anchor=True)
    r, _, _ = bla.forward(tq, tk, tv, [float(W)] * H, M, W)
    torch.cuda.synchronize()
    assert_close(a.cpu().numpy(), r.cpu().numpy(), 1e-4, "anchored vs rotating")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,d,M,S,T,L", [
    (3, 2, 32, 8, 15, (15.0, 30.0), 40),
    (2, 2, 64, 64, 64, (127.0, 254.0), 300),
    (2, 2, 128, 128, 256, (255.0, 510.0), 20),
])
def test_anchor_step(dtype, B, H, d, M, S, T, L):
    """Decode step with anchored slots at position L from the mode state after L tokens (the
    oracle's prefill state: the same state in both forms), against row L of Alg. 1 over L + 1
    tokens."""
    bla = _bla()
    q, k, v = gauss(B * 10 + M + 3, B, H, L + 1, d, dtype)
    _say(f"anchored step B={B} H={H} d={d} M={M} S={S} L={L} dtype={dtype}")
    _, pk, pv = oracle.forward(q[:, :, :L], k[:, :, :L], v[:, :, :L], T, M, S)
    sk = torch.from_numpy(pk.astype(np.float32)).cuda()
    sv = torch.from_numpy(pv.astype(np.float32)).cuda()
    o = bla.step(to_dev(q[:, :, L], dtype), to_dev(k[:, :, L], dtype), to_dev(v[:, :, L], dtype), T, M, S,
                 sk, sv, t0=L, phase_anchor=True)
    torch.cuda.synchronize()
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S)
    _, ref_k, ref_v = oracle.forward(q, k, v, T, M, S)
    assert_close(o.float().cpu().numpy(), ref_o[:, :, L], TOL[dtype], "o")
    assert_close(sk.cpu().numpy(), ref_k, 1e-5, "state_k")
    assert_close(sv.cpu().numpy(), ref_v, 1e-5, "state_v")


def test_anchor_prefill_then_step():
    """The whole anchored GPU path: bla_forward over L tokens, then bla_step at position L."""
    bla = _bla()
    B, H, d, M, S, T, L = 2, 2, 64, 64, 64, (127.0, 254.0), 300
    q, k, v = gauss(24, B, H, L + 1, d, torch.bfloat16)
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    _, sk, sv = bla.forward(tq[:, :, :L].contiguous(), tk[:, :, :L].contiguous(), tv[:, :, :L].contiguous(),
                            T, M, S, phase_anchor=True)
    o = bla.step(tq[:, :, L].contiguous(), tk[:, :, L].contiguous(), tv[:, :, L].contiguous(), T, M, S, sk, sv,
                 t0=L, phase_anchor=True)
    torch.cuda.synchronize()
    ref_o, _, _ = oracle.forward_anchored(q, k, v, T, M, S)
    _, ref_k, ref_v = oracle.forward(q, k, v, T, M, S)
    assert_close(o.float().cpu().numpy(), ref_o[:, :, L], 2e-2, "o")
    assert_close(sk.cpu().numpy(), ref_k, 2e-2, "state_k")
    assert_close(sv.cpu().numpy(), ref_v, 2e-2, "state_v")


def test_anchor_step_far_positions():
    """Per-row positions up to 2^31 + 7 from a zero state: the phase m w p is reduced in
    double precision before the sincos (Alg. 1 with t0 = p and a single token)."""
    bla = _bla()
    B, H, d, M, S, T = 4, 2, 64, 16, 31, (31.0, 45.5)
    pos = np.array([0, 5, 1_000_003, 2 ** 31 + 7], np.int64)
    q, k, v = gauss(23, B, H, 1, d, torch.float32)
    tsk = torch.zeros(B, H, 2, M, d, device="cuda")
    tsv = torch.zeros(B, H, 2, M, d, device="cuda")
    o = bla.step(to_dev(q[:, :, 0], torch.float32), to_dev(k[:, :, 0], torch.float32),
                 to_dev(v[:, :, 0], torch.float32), T, M, S, tsk, tsv, pos=torch.from_numpy(pos).cuda(),
                 phase_anchor=True)
    torch.cuda.synchronize()
    for b in range(B):
        ref, _, _ = oracle.forward_anchored(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, M, S, t0=int(pos[b]))
        assert_close(o[b:b + 1].cpu().numpy(), ref[:, :, 0], 1e-4, f"o row {b} (pos {pos[b]})")


def test_anchor_workload3_sampled_rows():
    """LM-layer workload (B=8, H=16, L=4096, d=M=S=64, bf16) with anchored slots, in the
    benchmark's launch configuration; every head of the first and last batch row is checked
    against Alg. 1."""
    bla = _bla()
    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    q, k, v = bi.generate(3)
    _say(f"workload 3 anchored, full size {q.shape}")
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    o, sk, _ = bla.forward(tq, tk, tv, T, w.M, w.S, phase_anchor=True)
    torch.cuda.synchronize()
    for b in (0, w.B - 1):
        ref_o, _, _ = oracle.forward_anchored(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, w.M, w.S)
        _, ref_k, _ = oracle.forward(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, w.M, w.S)
        assert_close(o[b:b + 1].float().cpu().numpy(), ref_o, 2e-2, f"O row {b}")
        assert_close(sk[b:b + 1].cpu().numpy(), ref_k, 2e-2, f"state_k row {b}")
