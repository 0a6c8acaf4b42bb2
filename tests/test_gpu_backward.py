"""GPU parity of the backward pass: bla_backward through the C ABI against the float64 oracle's
reverse pass through Alg. 2 (itself pinned by finite differences, autograd through causal
softmax attention and closed forms).

Bars as for the forward: rel-L2 <= 1e-4 (float32 inputs) and <= 2e-2 (bfloat16 inputs), on
dq, dk, dv and the input-state gradients; with the same per-element guard, and a per-row
guard at 10x the rel-L2 bar.  The bf16 bar
holds with margin: every operand of the backward's contractions is rounded to bf16 once, as
in the forward, and the measured errors sit near the forward's (a few 1e-3).
"""
import math

import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle
from test_gpu_parity import TOL, _bla, _say, assert_close, to_dev

pytestmark = pytest.mark.gpu


def tensors(seed, B, H, L, d, M, dtype, with_states=False):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(4):
        x = (rng.standard_normal((B, H, L, d)) / math.sqrt(d)).astype(np.float32)
        out.append(bi.round_bf16(x) if dtype == torch.bfloat16 else x)
    states = [None] * 4
    if with_states:
        states = [(rng.standard_normal((B, H, 2, M, d)) * 0.3).astype(np.float32) for _ in range(4)]
        for s in states:
            s[:, :, 1, 0, :] = 0.0      # the m = 0 sin row of a state is identically zero
    return out, states


def run_bwd(q, k, v, g, T, M, S, dtype, t0=0, sk=None, sv=None, gk=None, gv=None, label="",
            rows=None):
    """rows: optional list of (b, h) sequences the oracle checks (the GPU runs the whole batch)."""
    bla = _bla()
    _say(f"backward case {label}: shape {q.shape} M={M} S={S} T={list(T)} t0={t0} dtype={dtype}")
    tq, tk, tv, tg = (to_dev(x, dtype) for x in (q, k, v, g))
    dev = lambda x: None if x is None else torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    dq, dk, dv, rsk, rsv = bla.backward(tq, tk, tv, tg, T, M, S, t0=t0, state_k=dev(sk), state_v=dev(sv),
                                        dstate_k=dev(gk), dstate_v=dev(gv))
    torch.cuda.synchronize()
    got = [x.float().cpu().numpy() for x in (dq, dk, dv, rsk, rsv)]
    sel = (lambda x: x) if rows is None else (lambda x: None if x is None else
                                              np.stack([x[b, h] for b, h in rows])[None])
    Tsel = list(T) if rows is None else [T[h] for _, h in rows]
    if rows is not None:
        # the oracle takes one "batch row" of len(rows) heads with their own periods
        ref = oracle.backward(sel(q), sel(k), sel(v), sel(g), Tsel, M, S, t0=t0, state_k=sel(sk),
                              state_v=sel(sv), dstate_k=sel(gk), dstate_v=sel(gv), nthreads=len(rows))
    else:
        ref = oracle.backward(q, k, v, g, T, M, S, t0=t0, state_k=sk, state_v=sv, dstate_k=gk, dstate_v=gv)
    tol = TOL[dtype]
    scale = math.sqrt(float(np.mean(ref[2] ** 2))) if ref[2].size else 1.0
    for name, a, b in zip(("dq", "dk", "dv", "dstate_k", "dstate_v"), got, ref):
        if b.size and math.sqrt(float(np.mean(b ** 2))) <= 1e-12 * scale:
            # a vanishing gradient (M = 1: zero up to the oracle's rounding), bounded against the
            # gradient scale of v
            emax = float(np.abs(sel(a)).max())
            _say(f"  {name}: zero reference, max-abs {emax:.3e} (scale {scale:.3e})")
            assert emax <= tol * scale, name
        else:
            # gradients of the softmax are differences of nearly equal terms (dz = P o (dP -
            # rowsum(P o dP))), so single rows carry more relative rounding than the forward's
            assert_close(sel(a), b, tol, name, row_tol=10 * tol)
    return got


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,L,d,M,S,T,t0", [
    (2, 3, 100, 32, 16, 16, (31.0, 62.0, 40.5), 0),   # ragged last chunk, non-integer T
    (1, 2, 64, 32, 8, 15, (15.0, 30.0), 0),            # exactly one chunk, S = 2M-1
    (2, 2, 7, 32, 5, 9, (9.0, 9.0), 0),                # L < chunk, T = S = 2M-1
    (1, 2, 200, 32, 24, 40, (47.0, 94.0), 3),          # padded modes and slots, t0 > 0
    (1, 1, 1, 32, 4, 4, (7.0,), 5),                    # a single token
    (1, 2, 33, 32, 1, 3, (1.0, 5.5), 0),               # M = 1: dq = dk = 0
])
def test_backward_small_shapes(dtype, B, H, L, d, M, S, T, t0):
    (q, k, v, g), _ = tensors(L + 7 * M, B, H, L, d, M, dtype)
    run_bwd(q, k, v, g, T, M, S, dtype, t0=t0, label=f"{B}x{H}x{L}x{d}")


@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (2, 2, 150, 64, 64, 64, (127.0, 254.0)),           # the LM-layer head shape, ragged
    (1, 3, 130, 64, 32, 64, (63.0, 126.0, 70.0)),      # S = 2 M
    (2, 1, 96, 32, 64, 128, (127.0,)),                 # d = 32 with 128 padded slots
    (1, 2, 70, 64, 16, 32, (31.0, 62.0)),
])
def test_backward_bf16_shapes(B, H, L, d, M, S, T):
    (q, k, v, g), _ = tensors(L + M + S, B, H, L, d, M, torch.bfloat16)
    run_bwd(q, k, v, g, T, M, S, torch.bfloat16, label=f"{B}x{H}x{L}x{d}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_backward_state_gradients_and_offset(dtype):
    """Input states, final-state gradients and t0 > 0: the chain through a split call."""
    B, H, L, d, M, S = 2, 2, 170, 32, 12, 20
    (q, k, v, g), (sk, sv, gk, gv) = tensors(77, B, H, L, d, M, dtype, with_states=True)
    run_bwd(q, k, v, g, (23.0, 41.5), M, S, dtype, t0=37, sk=sk, sv=sv, gk=gk, gv=gv, label="states")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_backward_many_segments(dtype):
    """Few sequences and many chunks: the sequence is cut into segments whose end states and
    end adjoints come from the forward and adjoint summaries."""
    B, H, L, d, M, S = 1, 2, 1100, 32, 16, 31
    (q, k, v, g), (sk, sv, gk, gv) = tensors(78, B, H, L, d, M, dtype, with_states=True)
    run_bwd(q, k, v, g, (31.0, 45.25), M, S, dtype, sk=sk, sv=sv, gk=gk, gv=gv, label="segments")


def test_backward_empty_and_deterministic():
    bla = _bla()
    B, H, d, M, S = 1, 2, 32, 4, 7
    gk = torch.randn(B, H, 2, M, d, device="cuda")
    gv = torch.randn(B, H, 2, M, d, device="cuda")
    z = torch.zeros(B, H, 0, d, device="cuda")
    _, _, _, rk, rv = bla.backward(z, z, z, z, [7.0, 9.0], M, S, dstate_k=gk, dstate_v=gv)
    torch.cuda.synchronize()
    assert torch.equal(rk, gk) and torch.equal(rv, gv)
    (q, k, v, g), _ = tensors(5, 2, 2, 300, 64, 64, torch.bfloat16)
    args = [to_dev(x, torch.bfloat16) for x in (q, k, v, g)]
    r1 = bla.backward(*args, [127.0, 254.0], 64, 64)
    r2 = bla.backward(*args, [127.0, 254.0], 64, 64)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)


def test_backward_unsupported_shapes_are_rejected():
    bla = _bla()
    q = torch.zeros(1, 1, 8, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(bla.BlaError):
        bla.backward(q, q, q, q, [255.0], 128, 128)


@pytest.mark.parametrize("d,M,S", [(64, 32, 64), (32, 16, 32)])
def test_backward_summary_blocks(d, M, S):
    """64 sequences of 8 chunks, the last one ragged: 4 segments of 2 chunks on the 256 compute
    units of an MI355X, and the adjoint summaries split into 2 blocks per segment (8 blocks of one
    chunk), so the forward states and the adjoint of every segment are Horner sums over blocks;
    with input states, final-state gradients and a position offset.  The oracle checks four
    sequences."""
    B, H, L = 16, 4, 64 * 7 + 13
    (q, k, v, g), (sk, sv, gk, gv) = tensors(91 + d, B, H, L, d, M, torch.bfloat16, with_states=True)
    T = bi.periods(M, H)
    run_bwd(q, k, v, g, T, M, S, torch.bfloat16, t0=5, sk=sk, sv=sv, gk=gk, gv=gv, label="summary blocks",
            rows=[(0, 0), (5, 1), (10, 2), (15, 3)])


def test_backward_workload3_sampled_rows():
    """The LM-layer workload at full size (B=8, H=16, L=4096, d=M=S=64, bf16) in the launch
    configuration the benchmark times; the oracle checks four whole sequences."""
    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    q, k, v = bi.generate(3)
    g = bi.generate_grad(3)
    rows = [(0, 0), (3, 5), (7, 14), (7, 15)]
    run_bwd(q, k, v, g, T, w.M, w.S, torch.bfloat16, label="workload 3", rows=rows)
