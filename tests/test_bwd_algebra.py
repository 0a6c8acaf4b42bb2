"""The chunked regrouping of the backward pass that the HIP kernels compute, checked in
float64 against the oracle's token-by-token reverse pass through Alg. 2.

Per chunk of c tokens (local index i), with rho_m = exp(i m w), E[i,m] = rho_m^i, the
pre-rotated forward state Z' = rho Z entering the chunk, G = tril(Q K^T), Gd = tril(dO V^T),
and the pre-rotated adjoint Gam' = rho dLoss/dZ of the state after the chunk's last token:

  forward quantities:  U = E o (Q Z'_k^T + G conj(E)),  z = scale(Re U A^T + Im U B^T) masked,
                       P = softmax(z),  W'' = (P A - i P B) o E
  readout gradient:    Y = E o (dO Z'_v^T + Gd conj(E))          (y_i[m] = <dO_i, Z_v after i>)
                       dP = Re Y A^T + Im Y B^T,  dz = P o (dP - rowsum(P o dP))
  score gradient:      Wq'' = (dz A - i dz B) o E * scale          (conj(du) o E)
  dq = Re(Wq'' Z'_k) + tril(Re(Wq'' conj(E)^T)) K
  dk = tril(Re(Wq'' conj(E)^T))^T Q + Re(conj(Erev) Gam'_k)      (Erev[j] = rho^{c-j})
  dv = tril(Re(W'' conj(E)^T))^T dO + Re(conj(Erev) Gam'_v)
  adjoint:  Gam'_k <- conj(rho^c) o Gam'_k + conj(Wq'')^T Q,   Gam'_v <- ... + conj(W'')^T dO
  forward state, walked backwards:  Z'_in = conj(rho^c) o (Z'_out - Erev^T [K | V])

A sequence is cut into segments: the forward states at the segment ends come from forward
summaries (Z'_end(g) = rho^{len_g} Z'_end(g-1) + S_g), the adjoints at the segment ends from
adjoint summaries (the adjoint at a segment's start from a zero adjoint at its end; then
Gam'_end(g) = A_{g+1} + conj(rho^{len_{g+1}}) Gam'_end(g+1)).
"""
import math

import numpy as np
import pytest

import oracle


def _relerr(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / max(np.linalg.norm(np.asarray(b)), 1e-300)


def _tables(T, M, S, C):
    Tc = max(T, 2 * M - 1)
    w = 2 * np.pi / Tc
    A, B, theta = oracle.interp(M, S, Tc)
    E = np.exp(1j * w * np.outer(np.arange(C + 1), np.arange(M)))
    return w, A, B, theta, E


def fwd_summary(k, v, T, M, C):
    """Pre-rotated state after the tokens k, v from a zero state: sum_t rho^{len - t} x_t."""
    w, _, _, _, E = _tables(T, M, 1, C)
    L = k.shape[0]
    ph = np.exp(1j * w * np.outer(L - np.arange(L), np.arange(M)))   # rho^{L-t}
    return ph.T @ k, ph.T @ v


def chunked_backward_segment(q, k, v, g, T, M, S, C, n0, n1, zk_end, zv_end, gk_end, gv_end,
                             t0=0, scale=None, outputs=True):
    """Reverse walk over the chunks of tokens [n0, n1) of one sequence (chunk starts at
    multiples of C from n0).  zk_end, zv_end: pre-rotated forward states after token n1-1;
    gk_end, gv_end: pre-rotated adjoints of that state.  Returns (dq, dk, dv) of the tokens
    and the pre-rotated adjoints at the start of the range."""
    dk_ = q.shape[1]
    scale = 1.0 / math.sqrt(dk_) if scale is None else scale
    w, A, B, theta, E = _tables(T, M, S, C)
    zk, zv, gk, gv = zk_end.copy(), zv_end.copy(), gk_end.copy(), gv_end.copy()
    dq = np.zeros((n1 - n0, q.shape[1]))
    dk = np.zeros_like(dq)
    dv = np.zeros((n1 - n0, v.shape[1]))
    starts = list(range(n0, n1, C))
    for s0 in reversed(starts):
        c = min(C, n1 - s0)
        Q, K, V, Gd_o = q[s0:s0 + c], k[s0:s0 + c], v[s0:s0 + c], g[s0:s0 + c]
        Ec = E[:c]
        Erev = E[c - np.arange(c)]                       # rho^{c-j}
        tril = np.tril(np.ones((c, c)))
        # forward state entering the chunk, from the state after it
        zk = np.conj(E[c])[:, None] * (zk - Erev.T @ K)
        zv = np.conj(E[c])[:, None] * (zv - Erev.T @ V)
        Gq = (Q @ K.T) * tril
        Gd = (Gd_o @ V.T) * tril
        U = Ec * (Q @ zk.T + Gq @ np.conj(Ec))
        z = scale * (U.real @ A.T + U.imag @ B.T)
        pos = t0 + s0 + np.arange(c)
        z = np.where(pos[:, None] >= theta[None, :], z, -np.inf)
        P = np.exp(z - z.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        W2 = (P @ A - 1j * (P @ B)) * Ec
        Y = Ec * (Gd_o @ zv.T + Gd @ np.conj(Ec))
        dP = Y.real @ A.T + Y.imag @ B.T
        dz = P * (dP - (P * dP).sum(axis=1, keepdims=True))
        Wq = scale * (dz @ A - 1j * (dz @ B)) * Ec
        Hq = (Wq @ np.conj(Ec).T).real * tril
        Hv = (W2 @ np.conj(Ec).T).real * tril
        r0 = s0 - n0
        dq[r0:r0 + c] = (Wq @ zk).real + Hq @ K
        dk[r0:r0 + c] = Hq.T @ Q + (np.conj(Erev) @ gk).real
        dv[r0:r0 + c] = Hv.T @ Gd_o + (np.conj(Erev) @ gv).real
        gk = np.conj(E[c])[:, None] * gk + np.conj(Wq).T @ Q
        gv = np.conj(E[c])[:, None] * gv + np.conj(W2).T @ Gd_o
    return dq, dk, dv, gk, gv


def chunked_backward(q, k, v, g, T, M, S, C, seg_chunks, t0=0, zk_in=None, zv_in=None, gz_k=None,
                     gz_v=None):
    """Whole sequence, cut into segments of seg_chunks chunks, combined by summaries."""
    L, d = q.shape
    Tc = max(T, 2 * M - 1)
    w = 2 * np.pi / Tc
    rho = np.exp(1j * w * np.arange(M))
    zk_in = np.zeros((M, d), complex) if zk_in is None else zk_in
    zv_in = np.zeros((M, v.shape[1]), complex) if zv_in is None else zv_in
    gz_k = np.zeros((M, d), complex) if gz_k is None else gz_k
    gz_v = np.zeros((M, v.shape[1]), complex) if gz_v is None else gz_v
    bounds = [(a, min(L, a + seg_chunks * C)) for a in range(0, L, seg_chunks * C)]
    rot = lambda n: np.exp(1j * w * n * np.arange(M))[:, None]
    # forward states at the segment ends
    zk_end, zv_end = [], []
    zk, zv = rho[:, None] * zk_in, rho[:, None] * zv_in
    for a, b in bounds:
        sk, sv = fwd_summary(k[a:b], v[a:b], T, M, C)
        zk, zv = rot(b - a) * zk + sk, rot(b - a) * zv + sv
        zk_end.append(zk)
        zv_end.append(zv)
    # adjoint summaries of every segment but the first, from a zero adjoint at the end
    zeros_k, zeros_v = np.zeros_like(gz_k), np.zeros_like(gz_v)
    summ = [None] * len(bounds)
    for s in range(1, len(bounds)):
        a, b = bounds[s]
        _, _, _, ak, av = chunked_backward_segment(q, k, v, g, T, M, S, C, a, b, zk_end[s], zv_end[s],
                                                   zeros_k, zeros_v, t0=t0)
        summ[s] = (ak, av)
    # adjoints at the segment ends (Horner from the last segment down)
    gk_end = [None] * len(bounds)
    gv_end = [None] * len(bounds)
    gk, gv = rho[:, None] * gz_k, rho[:, None] * gz_v
    for s in range(len(bounds) - 1, -1, -1):
        gk_end[s], gv_end[s] = gk, gv
        if s > 0:
            a, b = bounds[s]
            gk = summ[s][0] + np.conj(rot(b - a)) * gk
            gv = summ[s][1] + np.conj(rot(b - a)) * gv
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for s, (a, b) in enumerate(bounds):
        dq[a:b], dk[a:b], dv[a:b], gk, gv = chunked_backward_segment(
            q, k, v, g, T, M, S, C, a, b, zk_end[s], zv_end[s], gk_end[s], gv_end[s], t0=t0)
        if s == 0:
            gin_k, gin_v = np.conj(rho)[:, None] * gk, np.conj(rho)[:, None] * gv
    return dq, dk, dv, gin_k, gin_v


def _split(z):
    return np.stack([z.real, z.imag])


@pytest.mark.parametrize("M,S,T,L,C,seg,t0", [
    (5, 9, 18.5, 70, 16, 100, 0),      # one segment, ragged last chunk
    (4, 7, 7.0, 64, 8, 2, 0),          # T = S = 2M-1, four segments
    (6, 6, 22.0, 91, 16, 2, 3),        # S = M, segments with a ragged tail, t0 > 0
    (3, 5, 7.25, 40, 8, 1, 0),         # a segment per chunk
])
def test_chunked_backward_matches_oracle(M, S, T, L, C, seg, t0):
    rng = np.random.default_rng(50)
    d = 5
    q, k, v, g = (rng.standard_normal((L, d)) / math.sqrt(d) for _ in range(4))
    zk, zv, gzk, gzv = ((rng.standard_normal((M, d)) + 1j * rng.standard_normal((M, d))) * 0.3
                        for _ in range(4))
    zk[0].imag = zv[0].imag = gzk[0].imag = gzv[0].imag = 0.0   # the m = 0 sin row is identically 0
    dq, dk, dv, gk, gv = chunked_backward(q, k, v, g, T, M, S, C, seg, t0=t0, zk_in=zk, zv_in=zv,
                                          gz_k=gzk, gz_v=gzv)
    rq, rk, rv, rgk, rgv = oracle.backward(q[None, None], k[None, None], v[None, None], g[None, None],
                                           [T], M, S, t0=t0, state_k=_split(zk)[None, None],
                                           state_v=_split(zv)[None, None], dstate_k=_split(gzk)[None, None],
                                           dstate_v=_split(gzv)[None, None])
    assert _relerr(dq, rq[0, 0]) < 1e-11
    assert _relerr(dk, rk[0, 0]) < 1e-11
    assert _relerr(dv, rv[0, 0]) < 1e-11
    assert _relerr(_split(gk), rgk[0, 0]) < 1e-11
    assert _relerr(_split(gv), rgv[0, 0]) < 1e-11
