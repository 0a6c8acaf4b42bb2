"""Pins of the float64 oracle against what the paper and the mathematics fix.

Each test names the passage it checks and the mistakes it would catch.  None of
them re-types the oracle's own formula: they use closed forms, brute force on
tiny inputs, textbook special cases and invariants.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _relerr(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (den if den > 0 else 1.0)


def dirichlet_closed(x, M, T):
    """Textbook closed form of the normalised Dirichlet kernel of period T.

    (1 + 2 sum_{m=1}^{M-1} cos(m w x)) / (2M-1) = sin((2M-1) w x / 2) / ((2M-1) sin(w x / 2)),
    with value 1 where sin(w x / 2) = 0 (x a multiple of T).
    """
    x = np.asarray(x, np.float64)
    y = np.pi * x / T
    num = np.sin((2 * M - 1) * y)
    den = (2 * M - 1) * np.sin(y)
    near = np.abs(den) < 1e-12
    safe = np.where(near, 1.0, den)
    return np.where(near, 1.0, num / safe)


def _inputs(rng, B, H, L, d, dv=None):
    dv = d if dv is None else dv
    q = rng.standard_normal((B, H, L, d)) / math.sqrt(d)
    k = rng.standard_normal((B, H, L, d)) / math.sqrt(d)
    v = rng.standard_normal((B, H, L, dv))
    return q, k, v


# ---------------------------------------------------------------- P1, P2: tables
@pytest.mark.parametrize("M,T", [(2, 3.0), (4, 7.0), (5, 9.0), (5, 18.0), (6, 18.5), (16, 62.0),
                                 (64, 254.0)])
def test_p1_dirichlet_closed_form(M, T):
    """Sec. 3.1 Eq. dirichlet: the slot-0 row of A holds the Dirichlet coefficients c_m.

    Catches a wrong c_0 / c_m normalisation or a wrong frequency w = 2 pi / T.
    """
    A, B, _ = oracle.interp(M, 3, T)
    w = 2 * np.pi / max(T, 2 * M - 1)
    x = np.linspace(-3 * T, 3 * T, 997) + 0.123
    series = sum(A[0, m] * np.cos(m * w * x) for m in range(M))
    assert np.max(np.abs(series - dirichlet_closed(x, M, max(T, 2 * M - 1)))) < 1e-12
    assert np.all(B[0] == 0.0)


def test_p1_golden_integer_points():
    """Sec. 3.1 / Appendix B: at T = 2M-1, D_M(0) = 1 and D_M(t) = 0 for t = 1..2M-2."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "dirichlet_integer_points.txt"))
            if l.strip() and not l.startswith("#")]
    assert rows
    for M, T, t, val in rows:
        M, T, t, val = int(M), float(T), float(t), float(val)
        A, _, _ = oracle.interp(M, 2 * M - 1, T)
        w = 2 * np.pi / T
        series = sum(A[0, m] * np.cos(m * w * t) for m in range(M))
        assert abs(series - val) < 1e-13, (M, T, t)


@pytest.mark.parametrize("M,S,T", [(4, 7, 7.0), (4, 7, 14.0), (4, 4, 7.0), (5, 9, 18.5),
                                   (8, 8, 30.0), (16, 16, 62.0), (3, 11, 5.0)])
def test_p2_translated_kernels(M, S, T):
    """Sec. 3.1 Eq. translated / Appendix B: row s of (A, B) is D_M translated by tau_s = sT/S.

    sum_m A[s,m] cos(m w x) + B[s,m] sin(m w x) = D_M(x - tau_s).  Catches a wrong sign of B,
    a wrong slot grid or a transposed A/B.
    """
    A, B, _ = oracle.interp(M, S, T)
    Tc = max(T, 2 * M - 1)
    w = 2 * np.pi / Tc
    x = np.linspace(-2 * Tc, 2 * Tc, 401) + 0.37
    for s in range(S):
        series = sum(A[s, m] * np.cos(m * w * x) + B[s, m] * np.sin(m * w * x) for m in range(M))
        assert np.max(np.abs(series - dirichlet_closed(x - s * Tc / S, M, Tc))) < 1e-12


def test_mask_grid_readings():
    """Alg. 1/2 dilated time grid: at T = S = 2M-1 the thresholds are the integer lags s.

    Also documents the rounding reading (ties to even) on two ties that the
    workloads' period rule produces: S=16,T=62,s=12 -> 46.5 -> 46 and
    S=64,T=254,s=48 -> 190.5 -> 190.
    """
    for M in (2, 4, 16):
        _, _, th = oracle.interp(M, 2 * M - 1, 2 * M - 1)
        assert list(th) == list(range(2 * M - 1))
    _, _, th = oracle.interp(16, 16, 62.0)
    assert th[12] == 46 and th[2] == 8 and th[3] == 12  # 7.75 -> 8, 11.625 -> 12
    _, _, th = oracle.interp(64, 64, 254.0)
    assert th[48] == 190
    # the period is clamped to 2M-1 (Alg. 1 "clamp period")
    _, _, th = oracle.interp(8, 15, 3.0)
    assert list(th) == list(range(15))


# ---------------------------------------------------------------- P3: closed-form states
@pytest.mark.parametrize("M,S,T,L", [(4, 7, 7.0, 30), (5, 5, 18.5, 41), (6, 11, 22.0, 64)])
def test_p3_closed_form_states(M, S, T, L):
    """Sec. 3.1 Eq. states (proof in Appendix B): after tokens 0..L-1,
    Kcos[m] = sum_t' cos(m w (L-1-t')) k_t', Ksin[m] = sum_t' sin(m w (L-1-t')) k_t'.

    Catches an off-by-one in the update order, a sign error in the rotation and a
    wrong w.
    """
    rng = np.random.default_rng(1)
    q, k, v = _inputs(rng, 2, 2, L, 5, 3)
    Ts = [T, 2 * T]
    _, sk, sv = oracle.forward(q, k, v, Ts, M, S)
    for h in range(2):
        Tc = max(Ts[h], 2 * M - 1)
        w = 2 * np.pi / Tc
        lag = (L - 1 - np.arange(L))[:, None] * np.arange(M)[None, :] * w   # [L, M]
        for b in range(2):
            ref_kc = np.cos(lag).T @ k[b, h]
            ref_ks = np.sin(lag).T @ k[b, h]
            ref_vc = np.cos(lag).T @ v[b, h]
            ref_vs = np.sin(lag).T @ v[b, h]
            assert _relerr(sk[b, h, 0], ref_kc) < 1e-12
            assert _relerr(sk[b, h, 1], ref_ks) < 1e-12
            assert _relerr(sv[b, h, 0], ref_vc) < 1e-12
            assert _relerr(sv[b, h, 1], ref_vs) < 1e-12


# ---------------------------------------------------------------- P4: O(L^2) brute force
def brute_force(q, k, v, M, S, T, t0=0, scale=None):
    """Sec. 3.1 Eqs. conv, translated, compressed, output written as a direct sum:
    slot s at time t holds sum_{t'<=t} D_M(t - t' - tau_s) k_t' (and likewise for v),
    z_s = scale <q_t, slot_s> masked where t0+t < rint(tau_s), o_t = sum_s softmax(z)_s vslot_s.
    Uses the closed-form Dirichlet kernel, never the mode states.
    """
    L, d = q.shape
    Tc = max(T, 2 * M - 1)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    tau = np.arange(S) * Tc / S
    theta = np.rint(tau)
    o = np.zeros((L, v.shape[1]))
    for t in range(L):
        lags = t - np.arange(t + 1)                                  # [t+1]
        W = dirichlet_closed(lags[None, :] - tau[:, None], M, Tc)    # [S, t+1]
        ks = W @ k[: t + 1]
        vs = W @ v[: t + 1]
        z = scale * (ks @ q[t])
        z = np.where(t0 + t >= theta, z, -np.inf)
        p = np.exp(z - z.max())
        p /= p.sum()
        o[t] = p @ vs
    return o


@pytest.mark.parametrize("M,S,T,L,t0", [(4, 7, 7.0, 23, 0), (4, 4, 9.0, 30, 0), (5, 9, 18.5, 40, 0),
                                        (6, 6, 22.0, 37, 5), (3, 8, 5.0, 19, 0), (8, 15, 30.0, 50, 2)])
@pytest.mark.parametrize("literal", [True, False])
def test_p4_brute_force(M, S, T, L, t0, literal):
    """Brute-force O(L^2) evaluation of the Dirichlet-weighted KV history vs the oracle.

    Catches errors in slot reconstruction, the mask, the scale, the softmax and the readout.
    """
    rng = np.random.default_rng(2)
    q, k, v = _inputs(rng, 1, 2, L, 6, 4)
    Ts = [T, T + 3.25]
    o, _, _ = oracle.forward(q, k, v, Ts, M, S, t0=t0, literal=literal)
    for h in range(2):
        ref = brute_force(q[0, h], k[0, h], v[0, h], M, S, Ts[h], t0=t0)
        assert _relerr(o[0, h], ref) < 1e-12


# ---------------------------------------------------------------- P5: SWA / full-attention limit
@pytest.mark.parametrize("M", [2, 4, 8])
def test_p5_full_attention_limit(M):
    """Sec. 3.1 (text after Eq. compressed; Fig. 2 caption): with T = S = 2M-1 and a sequence
    no longer than 2M-1, BLA is exactly causal softmax attention.  Reference: torch's
    scaled_dot_product_attention (float64, CPU, causal).
    """
    rng = np.random.default_rng(3)
    W = 2 * M - 1
    q, k, v = _inputs(rng, 2, 3, W, 8, 5)
    o, _, _ = oracle.forward(q, k, v, [float(W)] * 3, M, W)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), is_causal=True,
        scale=1.0 / math.sqrt(8)).numpy()
    assert _relerr(o, ref) < 1e-12


def test_p5_residue_class_sums():
    """Sec. 3.1 Eq. conv_key: at T = S = 2M-1 and L > 2M-1, slot s holds the sum of all keys
    (values) whose lag is congruent to s modulo 2M-1, and is valid once t >= s.
    """
    rng = np.random.default_rng(4)
    M, L, d = 4, 40, 6
    W = 2 * M - 1
    q, k, v = _inputs(rng, 1, 1, L, d, 3)
    o, _, _ = oracle.forward(q, k, v, [float(W)], M, W)
    qq, kk, vv = q[0, 0], k[0, 0], v[0, 0]
    ref = np.zeros((L, 3))
    for t in range(L):
        ks = np.zeros((W, d))
        vs = np.zeros((W, 3))
        for tp in range(t + 1):
            ks[(t - tp) % W] += kk[tp]
            vs[(t - tp) % W] += vv[tp]
        z = (ks @ qq[t]) / math.sqrt(d)
        z[np.arange(W) > t] = -np.inf
        p = np.exp(z - z.max())
        p /= p.sum()
        ref[t] = p @ vs
    assert _relerr(o[0, 0], ref) < 1e-12


# ---------------------------------------------------------------- P8: one mode
def test_p8_single_mode():
    """M = 1 (Eq. dirichlet with c_0 = 1): every slot equals the running sum, so
    o_t = sum_{t'<=t} v_t' whatever q and k are.  Pins the normalisation of softmax."""
    rng = np.random.default_rng(5)
    q, k, v = _inputs(rng, 2, 2, 33, 4, 3)
    o, _, _ = oracle.forward(q, k, v, [1.0, 6.5], 1, 5)
    assert _relerr(o, np.cumsum(v, axis=2)) < 1e-12


# ---------------------------------------------------------------- P9: state I/O and positions
@pytest.mark.parametrize("L1", [1, 17, 40])
def test_p9_split_call(L1):
    """Recurrent mode (Sec. 3.2, last paragraph): running L tokens at once equals running
    L1 tokens, then L-L1 more from the returned state with t0 = L1."""
    rng = np.random.default_rng(6)
    M, S, L = 5, 7, 57
    q, k, v = _inputs(rng, 2, 2, L, 4, 3)
    Ts = [9.0, 13.5]
    o, sk, sv = oracle.forward(q, k, v, Ts, M, S)
    o1, sk1, sv1 = oracle.forward(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], Ts, M, S)
    o2, sk2, sv2 = oracle.forward(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], Ts, M, S, t0=L1,
                                  state_k=sk1, state_v=sv1)
    assert _relerr(np.concatenate([o1, o2], axis=2), o) < 1e-13
    assert _relerr(sk2, sk) < 1e-13 and _relerr(sv2, sv) < 1e-13


def test_p9_step_matches_forward():
    """Decode step at position L from the prefill state == row L of a forward over L+1."""
    rng = np.random.default_rng(7)
    M, S, L = 6, 6, 30
    q, k, v = _inputs(rng, 3, 2, L + 1, 4, 5)
    Ts = [11.0, 22.0]
    o, sk, sv = oracle.forward(q, k, v, Ts, M, S)
    _, pk, pv = oracle.forward(q[:, :, :L], k[:, :, :L], v[:, :, :L], Ts, M, S)
    so, sk2, sv2 = oracle.step(q[:, :, L], k[:, :, L], v[:, :, L], Ts, M, S, pk, pv, [L] * 3)
    assert _relerr(so, o[:, :, L]) < 1e-13
    assert _relerr(sk2, sk) < 1e-13 and _relerr(sv2, sv) < 1e-13


def test_start_mask_first_token():
    """Eq. output / Alg. 2 mask: at position 0 only slot 0 (lag 0) is visible, so o_0 = v_0
    for any M, S, T (the slot-0 kernel takes the value D_M(0) = 1 at lag 0)."""
    rng = np.random.default_rng(8)
    q, k, v = _inputs(rng, 1, 2, 1, 4, 3)
    for (M, S, T) in [(4, 4, 14.0), (5, 9, 9.0), (7, 3, 40.0)]:
        o, _, _ = oracle.forward(q, k, v, [T, T], M, S)
        assert _relerr(o[0, :, 0], v[0, :, 0]) < 1e-13


# ---------------------------------------------------------------- P10, P11, periodicity
def test_p10_linear_in_values():
    """Eq. output: the softmax weights do not depend on V, so O is linear in V."""
    rng = np.random.default_rng(9)
    q, k, v1 = _inputs(rng, 1, 2, 29, 4, 3)
    v2 = rng.standard_normal(v1.shape)
    args = ([7.0, 10.0], 4, 6)
    o1, _, _ = oracle.forward(q, k, v1, *args)
    o2, _, _ = oracle.forward(q, k, v2, *args)
    o3, _, _ = oracle.forward(q, k, 2.5 * v1 - 0.75 * v2, *args)
    assert _relerr(o3, 2.5 * o1 - 0.75 * o2) < 1e-12


def test_p11_state_size():
    """Table 1 row BLA: the state has H (d_k + d_v)(2M-1) non-trivial reals; the m = 0 sin
    accumulators are identically zero (Sec. 3.1: K^sin, V^sin have M-1 modes)."""
    rows = [l.split() for l in open(os.path.join(GOLDEN, "state_size.txt"))
            if l.strip() and not l.startswith("#")]
    rng = np.random.default_rng(10)
    for H, dk, dv, M, n in rows:
        H, dk, dv, M, n = int(H), int(dk), int(dv), int(M), int(n)
        assert H * (dk + dv) * (2 * M - 1) == n
    H, dk, dv, M = 2, 5, 3, 6
    q, k, v = _inputs(rng, 1, H, 20, dk, dv)
    _, sk, sv = oracle.forward(q, k, v, [11.0, 17.0], M, 4)
    assert np.all(sk[:, :, 1, 0] == 0.0) and np.all(sv[:, :, 1, 0] == 0.0)
    nontrivial = np.count_nonzero(sk) + np.count_nonzero(sv)
    assert nontrivial == H * (dk + dv) * (2 * M - 1)


def test_periodicity_of_the_rotation():
    """w = 2 pi / T: T further zero tokens rotate every mode by a full turn, so the state
    after L + T tokens (the last T zero) equals the state after L tokens."""
    rng = np.random.default_rng(11)
    M, T, L = 5, 13, 21
    q, k, v = _inputs(rng, 1, 1, L + T, 3, 2)
    k[:, :, L:] = 0.0
    v[:, :, L:] = 0.0
    _, sk1, sv1 = oracle.forward(q[:, :, :L], k[:, :, :L], v[:, :, :L], [float(T)], M, 9)
    _, sk2, sv2 = oracle.forward(q, k, v, [float(T)], M, 9)
    assert _relerr(sk2, sk1) < 1e-12 and _relerr(sv2, sv1) < 1e-12


def test_scale_argument():
    """Eq. output scale: an explicit scale equal to 1/sqrt(d) reproduces the default, and
    scale 0 gives uniform weights over the visible slots."""
    rng = np.random.default_rng(12)
    q, k, v = _inputs(rng, 1, 1, 12, 4, 2)
    a, _, _ = oracle.forward(q, k, v, [7.0], 4, 7)
    b, _, _ = oracle.forward(q, k, v, [7.0], 4, 7, scale=0.5)
    assert _relerr(a, b) < 1e-15
    c, _, _ = oracle.forward(q, k, v, [7.0], 4, 7, scale=0.0)
    # uniform weights over the min(t+1, 7) visible slots at T = S = 2M-1; the slots partition
    # the history into residue classes (Eq. conv_key), so the average is cumsum / min(t+1, 7)
    csum = np.cumsum(v[0, 0], axis=0)
    ref = np.stack([csum[t] / min(t + 1, 7) for t in range(12)])
    assert _relerr(c[0, 0], ref) < 1e-13


def test_empty_sequence():
    """L = 0 is an empty call: no outputs, the state passes through unchanged."""
    rng = np.random.default_rng(13)
    sk = rng.standard_normal((1, 2, 2, 4, 3))
    sv = rng.standard_normal((1, 2, 2, 4, 2))
    z = np.zeros((1, 2, 0, 3))
    o, sk2, sv2 = oracle.forward(z, z, np.zeros((1, 2, 0, 2)), [7.0, 9.0], 4, 5, state_k=sk,
                                 state_v=sv)
    assert o.shape == (1, 2, 0, 2)
    assert np.array_equal(sk2, sk) and np.array_equal(sv2, sv)


# ---------------------------------------------------------------- P6: absolute-phase form
def brute_force_anchored(q, k, v, M, S, T, t0=0, scale=None):
    """Sec. 3.3 Eq. permuted written as a direct sum: at absolute position p = t0 + t,
    slot s holds sum_{t'<=t} D_M(t0 + t' - tau_s) k_t' (the Dirichlet kernel translated to
    the slot's lag and evaluated at the key's own absolute position); masked where
    p < rint(tau_s).  Uses the closed-form Dirichlet kernel, never mode or slot states.
    """
    L, d = q.shape
    Tc = max(T, 2 * M - 1)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    tau = np.arange(S) * Tc / S
    theta = np.rint(tau)
    W = dirichlet_closed((t0 + np.arange(L))[None, :] - tau[:, None], M, Tc)   # [S, L]
    o = np.zeros((L, v.shape[1]))
    for t in range(L):
        ks = W[:, : t + 1] @ k[: t + 1]
        vs = W[:, : t + 1] @ v[: t + 1]
        z = scale * (ks @ q[t])
        z = np.where(t0 + t >= theta, z, -np.inf)
        p = np.exp(z - z.max())
        p /= p.sum()
        o[t] = p @ vs
    return o


@pytest.mark.parametrize("M,S,T,L,t0", [(4, 7, 7.0, 23, 0), (4, 4, 9.0, 30, 0), (5, 9, 18.5, 40, 3),
                                        (3, 8, 5.0, 19, 0), (8, 15, 30.0, 50, 2), (6, 6, 22.0, 37, 5)])
def test_p6_anchored_brute_force(M, S, T, L, t0):
    """Alg. 1 against the O(L^2) direct sum of Eq. permuted with the closed-form kernel.

    Catches a wrong sign of the sine table (D is even in the lag, so a flipped B evaluates
    the kernel at p + tau_s), a phase origin off by one token or by t0, and mask errors.
    """
    rng = np.random.default_rng(20)
    q, k, v = _inputs(rng, 1, 2, L, 6, 4)
    Ts = [T, T + 3.25]
    o, _, _ = oracle.forward_anchored(q, k, v, Ts, M, S, t0=t0)
    for h in range(2):
        ref = brute_force_anchored(q[0, h], k[0, h], v[0, h], M, S, Ts[h], t0=t0)
        assert _relerr(o[0, h], ref) < 1e-12


@pytest.mark.parametrize("M,T,t0", [(2, 3, 0), (4, 7, 0), (5, 9, 4), (8, 15, 0), (4, 12, 0),
                                    (5, 20, 7)])
def test_p6_anchored_equals_rotating_at_integer_period(M, T, t0):
    """Sec. 3.3: with one slot per integer lag (S = T, the paper's case being T = S = 2M-1)
    the anchored slots are a permutation of the rotating ones at every step (slot s holds
    lag (p - s) mod T), the start mask maps onto itself, and softmax ignores the order, so
    Alg. 1 gives exactly the output of Alg. 2.  At S = T > 2M-1 this is the same
    permutation on a finer grid.
    """
    rng = np.random.default_rng(21)
    L = 3 * T + 5
    q, k, v = _inputs(rng, 2, 2, L, 5, 3)
    o_a, _, _ = oracle.forward_anchored(q, k, v, [float(T)] * 2, M, T, t0=t0)
    o_r, _, _ = oracle.forward(q, k, v, [float(T)] * 2, M, T, t0=t0)
    assert _relerr(o_a, o_r) < 1e-12


def test_p6_anchored_differs_off_the_integer_grid():
    """The permutation argument needs integer slot lags: at T = 2(2M-1) with S = 2M-1 the
    two forms give different outputs (the rotating form is the operator of Sec. 3.1)."""
    rng = np.random.default_rng(22)
    M, L = 4, 40
    q, k, v = _inputs(rng, 1, 1, L, 5, 3)
    o_a, _, _ = oracle.forward_anchored(q, k, v, [14.0], M, 7)
    o_r, _, _ = oracle.forward(q, k, v, [14.0], M, 7)
    assert _relerr(o_a, o_r) > 1e-2


@pytest.mark.parametrize("M,S,T,L,t0", [(4, 7, 14.0, 33, 0), (5, 9, 18.5, 41, 6), (3, 5, 7.25, 20, 0)])
def test_p6_anchored_slots_are_rotating_slots_at_moving_lags(M, S, T, L, t0):
    """Sec. 3.3's derivation: after the token at absolute position p, anchored slot s holds
    the rotating operator's blurry slot at lag p - tau_s, i.e. the Dirichlet-weighted
    history read from the Alg. 2 mode state with coefficients c_m (Eq. dirichlet) at that
    lag.  This is the identity that lets one mode state serve both forms.
    """
    rng = np.random.default_rng(23)
    q, k, v = _inputs(rng, 1, 2, L, 5, 3)
    Ts = [T, T + 1.5]
    _, kt, vt = oracle.forward_anchored(q, k, v, Ts, M, S, t0=t0)
    _, sk, sv = oracle.forward(q, k, v, Ts, M, S, t0=t0)
    p = t0 + L - 1
    c = np.array([1.0] + [2.0] * (M - 1)) / (2 * M - 1)
    for h in range(2):
        Tc = max(Ts[h], 2 * M - 1)
        w = 2 * np.pi / Tc
        lag = p - np.arange(S) * Tc / S
        cosm = c[None, :] * np.cos(np.outer(lag, np.arange(M)) * w)   # [S, M]
        sinm = c[None, :] * np.sin(np.outer(lag, np.arange(M)) * w)
        assert _relerr(kt[0, h], cosm @ sk[0, h, 0] + sinm @ sk[0, h, 1]) < 1e-12
        assert _relerr(vt[0, h], cosm @ sv[0, h, 0] + sinm @ sv[0, h, 1]) < 1e-12


@pytest.mark.parametrize("L1", [1, 17, 40])
def test_p6_anchored_split_call(L1):
    """Alg. 1 carries K_prev / V_prev across tokens: a run over L tokens equals L1 tokens,
    then L - L1 more from the returned slot states with t0 = L1."""
    rng = np.random.default_rng(24)
    M, S, L = 5, 7, 57
    q, k, v = _inputs(rng, 2, 2, L, 4, 3)
    Ts = [9.0, 13.5]
    o, kt, vt = oracle.forward_anchored(q, k, v, Ts, M, S)
    o1, kt1, vt1 = oracle.forward_anchored(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], Ts, M, S)
    o2, kt2, vt2 = oracle.forward_anchored(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], Ts, M, S,
                                           t0=L1, slot_k=kt1, slot_v=vt1)
    assert _relerr(np.concatenate([o1, o2], axis=2), o) < 1e-13
    assert _relerr(kt2, kt) < 1e-13 and _relerr(vt2, vt) < 1e-13


def test_p6_anchored_single_mode_and_attention_limit():
    """M = 1: every weight g_s is D_1 = 1, so o_t = sum_{t'<=t} v_t'.  T = S = 2M-1 with
    L <= 2M-1: causal softmax attention (torch's float64 CPU attention as reference)."""
    rng = np.random.default_rng(25)
    q, k, v = _inputs(rng, 2, 2, 33, 4, 3)
    o, _, _ = oracle.forward_anchored(q, k, v, [1.0, 6.5], 1, 5)
    assert _relerr(o, np.cumsum(v, axis=2)) < 1e-12
    M = 5
    W = 2 * M - 1
    q, k, v = _inputs(rng, 2, 3, W, 8, 5)
    o, _, _ = oracle.forward_anchored(q, k, v, [float(W)] * 3, M, W)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), is_causal=True,
        scale=1.0 / math.sqrt(8)).numpy()
    assert _relerr(o, ref) < 1e-12


def test_p6_anchored_long_positions():
    """Phases at large absolute positions: the period of the anchored weights is T, so
    shifting t0 by a multiple of an integer T leaves the output unchanged (the oracle
    reduces m p modulo T exactly)."""
    rng = np.random.default_rng(26)
    M, S, T, L = 6, 11, 23.0, 30
    q, k, v = _inputs(rng, 1, 1, L, 4, 3)
    a, _, _ = oracle.forward_anchored(q, k, v, [T], M, S, t0=40)
    b, _, _ = oracle.forward_anchored(q, k, v, [T], M, S, t0=40 + 23 * 100003)
    assert _relerr(a, b) < 1e-13


# ---------------------------------------------------------------- P12: state decay (Sec. 3.4)
def sliding_window_attention(q, k, v, W, scale):
    """Causal softmax attention over the last W keys (torch, float64 CPU)."""
    L = q.shape[-2]
    i = torch.arange(L)
    mask = (i[None, :] <= i[:, None]) & (i[None, :] > i[:, None] - W)
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), attn_mask=mask,
        scale=scale).numpy()


@pytest.mark.parametrize("M", [2, 4, 8])
def test_p12_decay_is_sliding_window_attention(M):
    """Sec. 3.4: with the decay 1 - D and T = S = 2M-1, each write replaces the slot of
    the current residue class, so BLA is exactly sliding-window softmax attention with
    window 2M-1 (torch's float64 CPU attention with a banded causal mask as reference)."""
    rng = np.random.default_rng(30)
    W = 2 * M - 1
    L = 4 * W + 3
    q, k, v = _inputs(rng, 2, 2, L, 6, 4)
    o, _, _ = oracle.forward_decay(q, k, v, [float(W)] * 2, M, W)
    ref = sliding_window_attention(q, k, v, W, 1.0 / math.sqrt(6))
    assert _relerr(o, ref) < 1e-12


def brute_force_decay(q, k, v, M, S, T, t0=0, scale=None):
    """Sec. 3.4 written as a direct sum: slot s at absolute position p holds
    sum_{t'<=t} D(p' - tau_s) prod_{t'<l<=t} (1 - D(p_l - tau_s)) k_t' with the closed-form
    Dirichlet kernel; no recursion over a state."""
    L, d = q.shape
    Tc = max(T, 2 * M - 1)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    tau = np.arange(S) * Tc / S
    theta = np.rint(tau)
    Dk = dirichlet_closed((t0 + np.arange(L))[None, :] - tau[:, None], M, Tc)   # [S, L]
    o = np.zeros((L, v.shape[1]))
    for t in range(L):
        Wt = np.zeros((S, t + 1))
        for tp in range(t + 1):
            Wt[:, tp] = Dk[:, tp] * np.prod(1.0 - Dk[:, tp + 1: t + 1], axis=1)
        ks = Wt @ k[: t + 1]
        vs = Wt @ v[: t + 1]
        z = scale * (ks @ q[t])
        z = np.where(t0 + t >= theta, z, -np.inf)
        p = np.exp(z - z.max())
        p /= p.sum()
        o[t] = p @ vs
    return o


@pytest.mark.parametrize("M,S,T,L,t0", [(4, 7, 14.0, 30, 0), (5, 9, 18.5, 36, 3), (3, 8, 5.0, 19, 0),
                                        (6, 6, 22.0, 31, 7), (4, 7, 7.0, 25, 0)])
def test_p12_decay_brute_force(M, S, T, L, t0):
    """The decayed slot states against the O(L^2 S) product form with the closed-form kernel.

    Catches a decay applied after the write instead of before, a gate 1 - D on the wrong
    token, and the phase origin."""
    rng = np.random.default_rng(31)
    q, k, v = _inputs(rng, 1, 2, L, 5, 3)
    Ts = [T, T + 2.75]
    o, _, _ = oracle.forward_decay(q, k, v, Ts, M, S, t0=t0)
    for h in range(2):
        ref = brute_force_decay(q[0, h], k[0, h], v[0, h], M, S, Ts[h], t0=t0)
        assert _relerr(o[0, h], ref) < 1e-11


def test_p12_decay_single_mode():
    """M = 1: D = 1 everywhere, so every slot is overwritten by the current token and
    o_t = v_t whatever q and k are."""
    rng = np.random.default_rng(32)
    q, k, v = _inputs(rng, 2, 2, 21, 4, 3)
    o, _, _ = oracle.forward_decay(q, k, v, [1.0, 6.5], 1, 5)
    assert _relerr(o, v) < 1e-13


@pytest.mark.parametrize("L1", [1, 17, 40])
def test_p12_decay_split_call(L1):
    """The decayed slot states carry a sequence across calls: L tokens at once equal L1
    tokens, then L - L1 more from the returned slot states with t0 = L1."""
    rng = np.random.default_rng(33)
    M, S, L = 5, 7, 57
    q, k, v = _inputs(rng, 2, 2, L, 4, 3)
    Ts = [9.0, 13.5]
    o, kt, vt = oracle.forward_decay(q, k, v, Ts, M, S)
    o1, kt1, vt1 = oracle.forward_decay(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], Ts, M, S)
    o2, kt2, vt2 = oracle.forward_decay(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], Ts, M, S, t0=L1,
                                        slot_k=kt1, slot_v=vt1)
    assert _relerr(np.concatenate([o1, o2], axis=2), o) < 1e-13
    assert _relerr(kt2, kt) < 1e-13 and _relerr(vt2, vt) < 1e-13


def test_p12_decay_forgets_the_past_at_T_equal_2M_minus_1():
    """Ring-buffer property: at T = S = 2M-1 the slot states after L >= 2M-1 tokens hold
    exactly the last 2M-1 keys, each in the slot of its residue class."""
    rng = np.random.default_rng(34)
    M, L = 4, 40
    W = 2 * M - 1
    q, k, v = _inputs(rng, 1, 1, L, 5, 3)
    _, kt, _ = oracle.forward_decay(q, k, v, [float(W)], M, W)
    for tp in range(L - W, L):
        assert np.allclose(kt[0, 0, tp % W], k[0, 0, tp], atol=1e-13)


# ---------------------------------------------------------------- P13: backward of Alg. 2
def _loss(q, k, v, g, gk, gv, T, M, S, t0=0, sk=None, sv=None):
    """The scalar loss whose gradients the backward computes: <g, O> + <gk, Zk_L> + <gv, Zv_L>."""
    o, zk, zv = oracle.forward(q, k, v, T, M, S, t0=t0, state_k=sk, state_v=sv)
    return float((o * g).sum() + (zk * gk).sum() + (zv * gv).sum())


def test_p13_backward_every_element_by_finite_differences():
    """Each element of dq, dk, dv and of the state-in gradients against a central finite
    difference of the forward oracle (float64, h = 1e-6).  Brute force on a tiny problem
    with a ragged period, S != 2M-1, t0 > 0 and nonzero states in and out: catches any
    dropped term, sign or transposed index of the reverse pass."""
    rng = np.random.default_rng(40)
    B, H, L, d, M, S, t0 = 1, 2, 9, 3, 3, 4, 2
    q, k, v = _inputs(rng, B, H, L, d)
    g = rng.standard_normal((B, H, L, d))
    sk, sv = (rng.standard_normal((B, H, 2, M, d)) * 0.3 for _ in range(2))
    gk, gv = (rng.standard_normal((B, H, 2, M, d)) * 0.2 for _ in range(2))
    T = [6.5, 11.0]
    dq, dk, dv, dsk, dsv = oracle.backward(q, k, v, g, T, M, S, t0=t0, state_k=sk, state_v=sv,
                                           dstate_k=gk, dstate_v=gv)
    args = [q, k, v, sk, sv]
    grads = [dq, dk, dv, dsk, dsv]
    h = 1e-6
    for which, (x, gx) in enumerate(zip(args, grads)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            ap, am = list(args), list(args)
            ap[which], am[which] = xp, xm
            fp = _loss(ap[0], ap[1], ap[2], g, gk, gv, T, M, S, t0, ap[3], ap[4])
            fm = _loss(am[0], am[1], am[2], g, gk, gv, T, M, S, t0, am[3], am[4])
            fd[idx] = (fp - fm) / (2 * h)
        assert _relerr(gx, fd) < 1e-7, (which, _relerr(gx, fd))


@pytest.mark.parametrize("M,S,T,L,t0", [(5, 9, 18.5, 70, 0), (4, 4, 9.0, 41, 5), (8, 15, 15.0, 33, 0)])
def test_p13_backward_directional_derivative(M, S, T, L, t0):
    """Directional derivatives at larger sizes: <grad, delta> equals the central difference
    of the loss along a random direction of every input at once."""
    rng = np.random.default_rng(41)
    B, H, d = 2, 2, 5
    q, k, v = _inputs(rng, B, H, L, d)
    g = rng.standard_normal((B, H, L, d))
    gk, gv = (rng.standard_normal((B, H, 2, M, d)) * 0.1 for _ in range(2))
    Ts = [T, 2 * T]
    dq, dk, dv, _, _ = oracle.backward(q, k, v, g, Ts, M, S, t0=t0, dstate_k=gk, dstate_v=gv)
    dirs = [rng.standard_normal(x.shape) for x in (q, k, v)]
    h = 1e-5
    fp = _loss(q + h * dirs[0], k + h * dirs[1], v + h * dirs[2], g, gk, gv, Ts, M, S, t0)
    fm = _loss(q - h * dirs[0], k - h * dirs[1], v - h * dirs[2], g, gk, gv, Ts, M, S, t0)
    an = float((dq * dirs[0]).sum() + (dk * dirs[1]).sum() + (dv * dirs[2]).sum())
    assert abs((fp - fm) / (2 * h) - an) <= 1e-8 * max(1.0, abs(an))


@pytest.mark.parametrize("M", [2, 4, 8])
def test_p13_backward_full_attention_limit(M):
    """T = S = 2M-1 and L <= 2M-1: the operator is causal softmax attention (P5), so its
    gradients are those of torch's autograd through scaled_dot_product_attention (float64
    CPU math path)."""
    rng = np.random.default_rng(42)
    W = 2 * M - 1
    L, d = W, 6
    q, k, v = _inputs(rng, 2, 2, L, d)
    g = rng.standard_normal(v.shape)
    dq, dk, dv, _, _ = oracle.backward(q, k, v, g, [float(W)] * 2, M, W)
    tq, tk, tv = (torch.from_numpy(x).requires_grad_(True) for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=d ** -0.5)
    o.backward(torch.from_numpy(g))
    for a, b in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        assert _relerr(a, b.numpy()) < 1e-12


def test_p13_backward_single_mode():
    """M = 1: o_t = sum_{t' <= t} v_t' whatever q and k are (P8), so dq = dk = 0 and dv is the
    reverse cumulative sum of dO."""
    rng = np.random.default_rng(43)
    q, k, v = _inputs(rng, 1, 2, 17, 4)
    g = rng.standard_normal(v.shape)
    dq, dk, dv, _, _ = oracle.backward(q, k, v, g, [1.0, 5.5], 1, 3)
    assert np.abs(dq).max() < 1e-13 and np.abs(dk).max() < 1e-13
    assert _relerr(dv, np.cumsum(g[:, :, ::-1], axis=2)[:, :, ::-1]) < 1e-14


@pytest.mark.parametrize("L1", [1, 13, 30])
def test_p13_backward_split_call(L1):
    """The state gradients chain calls: the backward of L tokens equals the backward of the
    last L - L1 tokens (from the first part's final states, t0 = L1), whose state-in gradients
    are then the final-state gradients of the first part."""
    rng = np.random.default_rng(44)
    M, S, L = 5, 7, 45
    q, k, v = _inputs(rng, 2, 2, L, 4)
    g = rng.standard_normal(v.shape)
    Ts = [9.0, 13.5]
    dq, dk, dv, _, _ = oracle.backward(q, k, v, g, Ts, M, S)
    _, zk, zv = oracle.forward(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], Ts, M, S)
    dq2, dk2, dv2, gk, gv = oracle.backward(q[:, :, L1:], k[:, :, L1:], v[:, :, L1:], g[:, :, L1:],
                                            Ts, M, S, t0=L1, state_k=zk, state_v=zv)
    dq1, dk1, dv1, _, _ = oracle.backward(q[:, :, :L1], k[:, :, :L1], v[:, :, :L1], g[:, :, :L1],
                                          Ts, M, S, dstate_k=gk, dstate_v=gv)
    assert _relerr(np.concatenate([dq1, dq2], 2), dq) < 1e-13
    assert _relerr(np.concatenate([dk1, dk2], 2), dk) < 1e-13
    assert _relerr(np.concatenate([dv1, dv2], 2), dv) < 1e-13


# ---------------------------------------------------------------- P14: the layer around the operator
def test_p14_layer_with_identity_projections_is_the_operator():
    """One head, W_qkv = [I | I | I] and W_o = I: the layer is the operator applied to x
    itself as queries, keys and values."""
    rng = np.random.default_rng(60)
    B, L, D, M, S = 2, 37, 6, 4, 7
    x = rng.standard_normal((B, L, D))
    eye = np.eye(D)
    y, sk, _ = oracle.layer_forward(x, np.concatenate([eye, eye, eye], 1), eye, [9.5], 1, M, S)
    xh = x[:, None]
    o, rk, _ = oracle.forward(xh, xh, xh, [9.5], M, S)
    assert _relerr(y, o[:, 0]) < 1e-14 and _relerr(sk, rk) < 1e-14


@pytest.mark.parametrize("H,M", [(2, 3), (4, 2)])
def test_p14_layer_attention_limit_is_multi_head_attention(H, M):
    """T = S = 2M-1 and L <= 2M-1: every head is causal softmax attention (P5), so the layer is
    multi-head attention with the same projections (torch float64: per-head
    scaled_dot_product_attention between the projections)."""
    rng = np.random.default_rng(61)
    W = 2 * M - 1
    B, L, d = 3, W, 4
    D = H * d
    x = rng.standard_normal((B, L, D))
    wqkv = rng.standard_normal((D, 3 * D)) / math.sqrt(D)
    wo = rng.standard_normal((D, D)) / math.sqrt(D)
    y, _, _ = oracle.layer_forward(x, wqkv, wo, [float(W)] * H, H, M, W)
    tx = torch.from_numpy(x)
    q, k, v = (tx @ torch.from_numpy(wqkv[:, i * D:(i + 1) * D]) for i in range(3))
    split = lambda t: t.reshape(B, L, H, d).transpose(1, 2)
    o = torch.nn.functional.scaled_dot_product_attention(split(q), split(k), split(v), is_causal=True,
                                                         scale=d ** -0.5)
    ref = o.transpose(1, 2).reshape(B, L, D) @ torch.from_numpy(wo)
    assert _relerr(y, ref.numpy()) < 1e-12
