"""The sub-block regrouping of the decay form (Sec. 3.4) that the HIP kernels compute,
checked in float64 against the oracle's token-by-token decayed slot recurrence.

Per sub-block of c <= 16 tokens (local index i, j) at absolute start P, with the
anchored interpolation weights g_j[s] = D_M(P + j - tau_s) (Eq. compressed_simplified,
obtained as the absolute phase rows times [A | B]) and the gates a_j[s] = 1 - g_j[s]:

  E_i[s] = prod_{l <= i} max(a_l[s], eps)        (prefix product inside the sub-block)
  Bq[j, s] = g_j[s] / E_j[s]
  K~_i = E_i o (K~_b + sum_{j <= i} Bq[j] k_j)   (the decayed slot state after token i)

so that, with G = tril(Q K^T) and Y = Q K~_b^T,

  z   = scale E o (Y + G Bq),  masked, P = softmax
  O   = (P o E) V~_b + tril((P o E) Bq^T) V
  K~  <- E_{c-1} o (K~_b + Bq^T K)               (V~ likewise)

Clamping a gate at eps keeps E_j > 0 where the decay flushes a slot exactly (a = 0 at
T = S = 2M-1); the state left before a flush is then scaled by eps instead of 0.
A sequence split into segments combines per-segment summaries: a segment maps its
entering state X to A_g o X + S_g (A_g = product of the segment's gates), so the state
entering segment g is the Horner combination of the earlier summaries.
"""
import math

import numpy as np
import pytest

import oracle

EPS = 1e-12


def _relerr(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300)


def gates(P, c, M, S, T):
    """g [c, S] at absolute positions P..P+c-1: [cos | sin](m w p) rows times [A | B]^T."""
    A, B, _ = oracle.interp(M, S, T)
    Tc = max(T, 2 * M - 1)
    w = 2 * np.pi / Tc
    p = P + np.arange(c)
    ph = w * np.fmod(np.outer(p, np.arange(M)).astype(np.float64), Tc)
    return np.cos(ph) @ A.T + np.sin(ph) @ B.T


def cut_length(P, cmax, M, S, T, eps=EPS, floor_log2=-100.0):
    """Sub-block length the kernels take at P: at most cmax tokens, ending before any slot's
    gate product drops below 2^floor_log2, and at least one token."""
    g = gates(P, cmax, M, S, T)
    lg = np.cumsum(np.log2(np.maximum(1.0 - g, eps)), axis=0)     # [cmax, S]
    bad = np.nonzero((lg < floor_log2).any(axis=1))[0]
    return max(1, int(bad[0]) if bad.size else cmax)


def subblock_sequence(q, k, v, T, M, S, sub=16, t0=0, scale=None, kt=None, vt=None, eps=EPS,
                      out=True, adaptive=False):
    """One (b,h) sequence through the sub-block form; returns (o, K~, V~, A_total).  The
    sub-blocks tile windows of `sub` tokens from the sequence start (with adaptive cuts, a
    window may hold several), as the kernels schedule them."""
    L, d = q.shape
    Tc = max(T, 2 * M - 1)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    _, _, theta = oracle.interp(M, S, Tc)
    kt = np.zeros((S, d)) if kt is None else kt.copy()
    vt = np.zeros((S, v.shape[1])) if vt is None else vt.copy()
    o = np.zeros((L, v.shape[1]))
    a_total = np.ones(S)
    b0 = 0
    while b0 < L:
        c = min(sub - b0 % sub, L - b0)  # sub-blocks never cross a window of `sub` tokens
        if adaptive:
            c = cut_length(t0 + b0, c, M, S, T, eps)
        g = gates(t0 + b0, c, M, S, T)                           # [c, S]
        E = np.cumprod(np.maximum(1.0 - g, eps), axis=0)         # [c, S]
        Bq = g / E
        Qb, Kb, Vb = q[b0:b0 + c], k[b0:b0 + c], v[b0:b0 + c]
        if out:
            G = np.tril(Qb @ Kb.T)
            z = scale * E * (Qb @ kt.T + G @ Bq)
            pos = t0 + b0 + np.arange(c)
            z = np.where(pos[:, None] >= theta[None, :], z, -np.inf)
            P = np.exp(z - z.max(axis=1, keepdims=True))
            P /= P.sum(axis=1, keepdims=True)
            PE = P * E
            o[b0:b0 + c] = PE @ vt + np.tril(PE @ Bq.T) @ Vb
        kt = E[-1][:, None] * (kt + Bq.T @ Kb)
        vt = E[-1][:, None] * (vt + Bq.T @ Vb)
        a_total *= E[-1]
        b0 += c
    return o, kt, vt, a_total


@pytest.mark.parametrize("M,S,T,L,t0", [(4, 7, 7.0, 70, 0), (4, 7, 14.0, 53, 0), (5, 9, 18.5, 61, 3),
                                        (8, 15, 15.0, 100, 0), (6, 6, 22.0, 47, 9), (1, 5, 6.5, 20, 0),
                                        (16, 16, 62.0, 90, 0)])
def test_subblock_form_matches_oracle(M, S, T, L, t0):
    rng = np.random.default_rng(40)
    q = rng.standard_normal((1, 1, L, 6)) / math.sqrt(6)
    k = rng.standard_normal((1, 1, L, 6)) / math.sqrt(6)
    v = rng.standard_normal((1, 1, L, 4))
    ref_o, ref_k, ref_v = oracle.forward_decay(q, k, v, [T], M, S, t0=t0)
    o, kt, vt, _ = subblock_sequence(q[0, 0], k[0, 0], v[0, 0], T, M, S, t0=t0)
    # the clamp leaves eps of a flushed state behind: far below float32 rounding
    assert _relerr(o, ref_o[0, 0]) < 1e-9
    assert _relerr(kt, ref_k[0, 0]) < 1e-9 and _relerr(vt, ref_v[0, 0]) < 1e-9


@pytest.mark.parametrize("sub", [4, 8, 16])
def test_subblock_length_is_free(sub):
    rng = np.random.default_rng(41)
    M, S, T, L = 5, 9, 18.5, 45
    q = rng.standard_normal((L, 4))
    k = rng.standard_normal((L, 4))
    v = rng.standard_normal((L, 3))
    a = subblock_sequence(q, k, v, T, M, S, sub=sub)
    b = subblock_sequence(q, k, v, T, M, S, sub=1)
    for x, y in zip(a[:3], b[:3]):
        assert _relerr(x, y) < 1e-10


def test_segments_combine_by_summaries():
    """Segments of 32 tokens: summary = the state reached from zero plus the product of the
    segment's gates; the entering state is the Horner combination of the earlier ones."""
    rng = np.random.default_rng(42)
    M, S, T, L, Ls = 4, 7, 14.0, 128, 32
    q = rng.standard_normal((L, 5)) / math.sqrt(5)
    k = rng.standard_normal((L, 5)) / math.sqrt(5)
    v = rng.standard_normal((L, 3))
    ref_o, _, _ = oracle.forward_decay(q[None, None], k[None, None], v[None, None], [T], M, S)
    kin = rng.standard_normal((S, 5))
    vin = rng.standard_normal((S, 3))
    ref_o2, _, _ = oracle.forward_decay(q[None, None], k[None, None], v[None, None], [T], M, S,
                                        slot_k=kin[None, None], slot_v=vin[None, None])
    summ = []
    for g0 in range(0, L - Ls, Ls):
        _, sk, sv, a = subblock_sequence(q[g0:g0 + Ls], k[g0:g0 + Ls], v[g0:g0 + Ls], T, M, S, t0=g0,
                                         out=False)
        summ.append((sk, sv, a))
    for state_in, ref in (((None, None), ref_o), ((kin, vin), ref_o2)):
        outs = []
        for gi, g0 in enumerate(range(0, L, Ls)):
            xk = np.zeros((S, 5)) if state_in[0] is None else state_in[0].copy()
            xv = np.zeros((S, 3)) if state_in[1] is None else state_in[1].copy()
            for sk, sv, a in summ[:gi]:
                xk = a[:, None] * xk + sk
                xv = a[:, None] * xv + sv
            o, _, _, _ = subblock_sequence(q[g0:g0 + Ls], k[g0:g0 + Ls], v[g0:g0 + Ls], T, M, S, t0=g0,
                                           kt=xk, vt=xv)
            outs.append(o)
        assert _relerr(np.concatenate(outs), ref[0, 0]) < 1e-9


@pytest.mark.parametrize("M,S,T,L", [(2, 8, 500.0, 80), (1, 5, 6.5, 30), (3, 5, 300.0, 64), (64, 64, 127.0, 64)])
def test_adaptive_cut_keeps_the_range(M, S, T, L):
    """Small M against a long period makes many consecutive gates small (the main lobe of
    D_M is T / (2M - 1) tokens wide); the gate-driven cut keeps every E above 2^-100 and the
    result equal to the recurrence.  On the workload shapes (M = 64) the cut stays at 16."""
    rng = np.random.default_rng(43)
    q = rng.standard_normal((1, 1, L, 4)) / 2
    k = rng.standard_normal((1, 1, L, 4)) / 2
    v = rng.standard_normal((1, 1, L, 3))
    ref_o, ref_k, _ = oracle.forward_decay(q, k, v, [T], M, S)
    o, kt, _, _ = subblock_sequence(q[0, 0], k[0, 0], v[0, 0], T, M, S, adaptive=True)
    assert _relerr(o, ref_o[0, 0]) < 1e-9 and _relerr(kt, ref_k[0, 0]) < 1e-9
    if M == 64:
        assert all(cut_length(p, 16, M, S, T) == 16 for p in range(0, 4096, 16))
