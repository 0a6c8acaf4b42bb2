"""The chunkwise-parallel regrouping that the HIP kernels compute, checked in float64.

This is the algebra of the chunked form, written as a plain numpy reference and
compared with the oracle's token-by-token recurrence (Sec. 3.1 Eq. recurrence,
Eq. compressed, Eq. output; Alg. 2).  It fixes the regrouping before any kernel
implements it: the pre-rotated state, the intra-chunk Gram terms with their
causal masks, the local phase tables, the ragged last chunk, the start mask at
absolute positions, and the split of a sequence into segments whose carried-in
states come from per-block summaries.

Per chunk of c tokens (local index j), with rho_m = exp(i m w), pre-rotated state
Z' = rho Z (Z = Kcos + i Ksin), E[j,m] = rho_m^j and G = (Q K^T) lower-triangular:

  U    = E o (Q Z'_k^T + G conj(E))                      u_j = <q_j, Z_k after token j>
  z    = scale (Re U A^T + Im U B^T), masked, P = softmax
  W''  = (P A - i P B) o E
  O    = Re(W'' Z'_v) + (Re(W'' conj(E)^T) o tril) V
  Z'  <- rho^c o Z' + sum_i rho^{c-i} [k_i | v_i]
"""
import math

import numpy as np
import pytest

import oracle


def _relerr(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300)


def chunked_sequence(q, k, v, T, M, S, C, t0=0, scale=None, zk_in=None, zv_in=None):
    """One (b,h) sequence.  q,k [L,dk], v [L,dv]; states complex [M,d] (Z = cos + i sin)."""
    L, dk = q.shape
    dv = v.shape[1]
    Tc = max(T, 2 * M - 1)
    w = 2 * np.pi / Tc
    scale = 1.0 / math.sqrt(dk) if scale is None else scale
    A, B, theta = oracle.interp(M, S, Tc)
    m = np.arange(M)
    E = np.exp(1j * w * np.outer(np.arange(C + 1), m))       # [C+1, M]
    rho = E[1]
    zk = np.zeros((M, dk), complex) if zk_in is None else zk_in.copy()
    zv = np.zeros((M, dv), complex) if zv_in is None else zv_in.copy()
    zk = rho[:, None] * zk                                     # pre-rotated
    zv = rho[:, None] * zv
    o = np.zeros((L, dv))
    for n0 in range(0, L, C):
        c = min(C, L - n0)
        Q, K, V = q[n0:n0 + c], k[n0:n0 + c], v[n0:n0 + c]
        Ec = E[:c]
        tril = np.tril(np.ones((c, c)))
        G = (Q @ K.T) * tril
        U = Ec * (Q @ zk.T + G @ np.conj(Ec))
        z = scale * (U.real @ A.T + U.imag @ B.T)
        pos = t0 + n0 + np.arange(c)
        z = np.where(pos[:, None] >= theta[None, :], z, -np.inf)
        P = np.exp(z - z.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        W2 = (P @ A - 1j * (P @ B)) * Ec
        Hm = (W2 @ np.conj(Ec).T).real * tril
        o[n0:n0 + c] = (W2 @ zv).real + Hm @ V
        Erev = E[c - np.arange(c)]                              # rho^{c-i}
        zk = E[c][:, None] * zk + Erev.T @ K
        zv = E[c][:, None] * zv + Erev.T @ V
    return o, np.conj(rho)[:, None] * zk, np.conj(rho)[:, None] * zv


def block_summary(k, v, T, M, C):
    """Pre-rotated state after a block of tokens, starting from zero."""
    _, zk, zv = chunked_sequence(np.zeros_like(k), k, v, T, M, 1, C)
    Tc = max(T, 2 * M - 1)
    rho = np.exp(1j * 2 * np.pi / Tc * np.arange(M))
    return rho[:, None] * zk, rho[:, None] * zv


def segmented_sequence(q, k, v, T, M, S, C, blk, nseg_blocks, t0=0):
    """Split into segments of nseg_blocks blocks of blk tokens; carry states by a scan over
    block summaries; each segment then runs the chunked form from its carry."""
    L = q.shape[0]
    Tc = max(T, 2 * M - 1)
    rho = np.exp(1j * 2 * np.pi / Tc * np.arange(M))
    seg = blk * nseg_blocks
    nseg = -(-L // seg)
    sums = []
    for j in range((nseg - 1) * nseg_blocks):
        sums.append(block_summary(k[j * blk:(j + 1) * blk], v[j * blk:(j + 1) * blk], T, M, C))
    rot = np.exp(1j * 2 * np.pi / Tc * ((np.arange(M) * blk) % Tc))    # rho^blk
    carries = [(np.zeros((M, q.shape[1]), complex), np.zeros((M, v.shape[1]), complex))]
    zk, zv = carries[0]
    for j, (sk, sv) in enumerate(sums):
        zk = rot[:, None] * zk + sk
        zv = rot[:, None] * zv + sv
        if (j + 1) % nseg_blocks == 0:
            carries.append((zk, zv))
    outs = []
    fk = fv = None
    for g in range(nseg):
        a, b = g * seg, min(L, (g + 1) * seg)
        ck, cv = carries[g]
        o, fk, fv = chunked_sequence(q[a:b], k[a:b], v[a:b], T, M, S, C, t0=t0 + a,
                                     zk_in=np.conj(rho)[:, None] * ck,
                                     zv_in=np.conj(rho)[:, None] * cv)
        outs.append(o)
    return np.concatenate(outs), fk, fv


def _case(seed, L, dk, dv):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((1, 1, L, dk)) / math.sqrt(dk)
    k = rng.standard_normal((1, 1, L, dk)) / math.sqrt(dk)
    v = rng.standard_normal((1, 1, L, dv))
    return q, k, v


@pytest.mark.parametrize("M,S,T,C,L", [(4, 7, 7.0, 8, 40), (5, 5, 18.5, 7, 33), (6, 4, 22.0, 16, 16),
                                       (8, 8, 30.0, 16, 100), (16, 16, 62.0, 64, 256),
                                       (3, 9, 5.0, 1, 12), (5, 6, 14.0, 64, 50)])
def test_p7_chunked_equals_recurrence(M, S, T, C, L):
    q, k, v = _case(M * 100 + L, L, 5, 3)
    ref_o, ref_k, ref_v = oracle.forward(q, k, v, [T], M, S)
    o, zk, zv = chunked_sequence(q[0, 0], k[0, 0], v[0, 0], T, M, S, C)
    assert _relerr(o, ref_o[0, 0]) < 1e-12
    assert _relerr(zk.real, ref_k[0, 0, 0]) < 1e-12 and _relerr(zk.imag, ref_k[0, 0, 1]) < 1e-12
    assert _relerr(zv.real, ref_v[0, 0, 0]) < 1e-12 and _relerr(zv.imag, ref_v[0, 0, 1]) < 1e-12


def test_p7_chunked_with_state_in_and_offset():
    M, S, T, C, L, t0 = 6, 9, 13.5, 8, 45, 21
    q, k, v = _case(7, L + t0, 4, 4)
    _, sk, sv = oracle.forward(q[..., :t0, :], k[..., :t0, :], v[..., :t0, :], [T], M, S)
    ref_o, ref_k, ref_v = oracle.forward(q[..., t0:, :], k[..., t0:, :], v[..., t0:, :], [T], M, S,
                                         t0=t0, state_k=sk, state_v=sv)
    o, zk, zv = chunked_sequence(q[0, 0, t0:], k[0, 0, t0:], v[0, 0, t0:], T, M, S, C, t0=t0,
                                 zk_in=sk[0, 0, 0] + 1j * sk[0, 0, 1],
                                 zv_in=sv[0, 0, 0] + 1j * sv[0, 0, 1])
    assert _relerr(o, ref_o[0, 0]) < 1e-12
    assert _relerr(zk.real, ref_k[0, 0, 0]) < 1e-12 and _relerr(zv.imag, ref_v[0, 0, 1]) < 1e-12


@pytest.mark.parametrize("blk,nsb,L", [(8, 2, 100), (16, 1, 64), (8, 3, 61), (32, 2, 300)])
def test_segments_from_block_summaries(blk, nsb, L):
    M, S, T, C = 5, 8, 14.0, 8
    q, k, v = _case(blk + L, L, 4, 3)
    ref_o, ref_k, ref_v = oracle.forward(q, k, v, [T], M, S)
    o, zk, zv = segmented_sequence(q[0, 0], k[0, 0], v[0, 0], T, M, S, C, blk, nsb)
    assert _relerr(o, ref_o[0, 0]) < 1e-12
    assert _relerr(zk.real, ref_k[0, 0, 0]) < 1e-12 and _relerr(zv.real, ref_v[0, 0, 0]) < 1e-12
