"""Float64 CPU oracle for the Blurry Window Attention forward operator.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package; the product package never
does.  The oracle shares no code with the HIP library.

``bla_oracle.c`` runs the paper's naive recurrent algorithm (Appendix C, Alg. 2:
the mode-state recurrence of Sec. 3.1 Eq. recurrence, the blurry slots of
Eq. compressed and the masked slot softmax of Eq. output) token by token in
double precision.  ``interp`` exposes its interpolation matrices (Eq. translated
evaluated on the dilated slot grid) so the tests can pin them.
``forward_anchored`` runs the absolute-phase form of Sec. 3.3 (Alg. 1: slots
anchored at phase 0, slot states accumulated as a cumulative sum) token by token;
``forward_decay`` the same with the state decay of Sec. 3.4 (previous slot state
multiplied by 1 - D before each write).  ``backward`` differentiates Alg. 2: the chain
rule taken through the token loop in reverse, with the forward states of every token
stored by a forward pass.  ``layer_forward`` puts the operator between the projections of
an attention layer (queries, keys and values projected from the hidden states, an output
projection after the heads), with numpy's float64 matrix products for the projections.

Parity status of each function (what pins it) is listed in the tests
(``tests/test_oracle_pins.py``); every function here is pinned.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bla_oracle.c")
_LIB = os.path.join(_HERE, "libbla_oracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_ip = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP, strict IEEE double)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                        "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.bla_oracle_interp.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double,
                                          _dp, _dp, _ip]
        lib.bla_oracle_interp.restype = None
        lib.bla_oracle_forward.argtypes = [ctypes.c_int] * 7 + [
            _dp, ctypes.c_int64, ctypes.c_double, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp,
            ctypes.c_int, ctypes.c_int]
        lib.bla_oracle_forward.restype = ctypes.c_int
        lib.bla_oracle_step.argtypes = [ctypes.c_int] * 6 + [
            _dp, _ip, ctypes.c_double, _dp, _dp, _dp, _dp, _dp, _dp, ctypes.c_int]
        lib.bla_oracle_step.restype = ctypes.c_int
        lib.bla_oracle_forward_anchored.argtypes = [ctypes.c_int] * 7 + [
            _dp, ctypes.c_int64, ctypes.c_double, _dp, _dp, _dp, _dp, _dp, _dp, _dp, _dp,
            ctypes.c_int, ctypes.c_int]
        lib.bla_oracle_forward_anchored.restype = ctypes.c_int
        lib.bla_oracle_backward.argtypes = [ctypes.c_int] * 7 + [
            _dp, ctypes.c_int64, ctypes.c_double] + [_dp] * 13 + [ctypes.c_int]
        lib.bla_oracle_backward.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(_dp)


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def interp(M: int, S: int, T: float):
    """Interpolation matrices A, B [S, M] and mask thresholds theta [S] for one head."""
    lib = _load()
    A = np.zeros((S, M), np.float64)
    B = np.zeros((S, M), np.float64)
    th = np.zeros((S,), np.int64)
    lib.bla_oracle_interp(M, S, float(T), _ptr(A), _ptr(B), th.ctypes.data_as(_ip))
    return A, B, th


def forward(q, k, v, T, M: int, S: int, t0: int = 0, scale=None, state_k=None,
            state_v=None, literal: bool = False, nthreads: int = 0):
    """Alg. 2 over q,k [B,H,L,dk], v [B,H,L,dv]; T is a per-head sequence of periods.

    Returns (o [B,H,L,dv], state_k [B,H,2,M,dk], state_v [B,H,2,M,dv]) in float64.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    Bn, H, L, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == q.shape and v.shape[:3] == (Bn, H, L)
    T = np.ascontiguousarray(np.broadcast_to(np.asarray(T, np.float64), (H,)))
    if scale is None:
        scale = 1.0 / np.sqrt(dk)
    sk_in, sv_in = _f64(state_k), _f64(state_v)
    o = np.zeros((Bn, H, L, dv), np.float64)
    sk = np.zeros((Bn, H, 2, M, dk), np.float64)
    sv = np.zeros((Bn, H, 2, M, dv), np.float64)
    rc = _load().bla_oracle_forward(Bn, H, L, dk, dv, M, S, _ptr(T), int(t0), float(scale),
                                    _ptr(q), _ptr(k), _ptr(v), _ptr(sk_in), _ptr(sv_in),
                                    _ptr(o), _ptr(sk), _ptr(sv), 1 if literal else 0,
                                    int(nthreads))
    if rc != 0:
        raise ValueError("bla_oracle_forward rejected its arguments")
    return o, sk, sv


def step(q, k, v, T, M: int, S: int, state_k, state_v, pos, scale=None, nthreads: int = 0):
    """One recurrent decode step at absolute positions pos [B]; q,k [B,H,dk], v [B,H,dv].

    Returns (o [B,H,dv], new state_k, new state_v) without modifying the inputs.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    Bn, H, dk = q.shape
    dv = v.shape[-1]
    T = np.ascontiguousarray(np.broadcast_to(np.asarray(T, np.float64), (H,)))
    if scale is None:
        scale = 1.0 / np.sqrt(dk)
    sk = np.array(state_k, dtype=np.float64, copy=True, order="C")
    sv = np.array(state_v, dtype=np.float64, copy=True, order="C")
    pos = np.ascontiguousarray(np.broadcast_to(np.asarray(pos, np.int64), (Bn,)))
    o = np.zeros((Bn, H, dv), np.float64)
    rc = _load().bla_oracle_step(Bn, H, dk, dv, M, S, _ptr(T), pos.ctypes.data_as(_ip),
                                 float(scale), _ptr(q), _ptr(k), _ptr(v), _ptr(sk), _ptr(sv),
                                 _ptr(o), int(nthreads))
    if rc != 0:
        raise ValueError("bla_oracle_step rejected its arguments")
    return o, sk, sv


def forward_anchored(q, k, v, T, M: int, S: int, t0: int = 0, scale=None, slot_k=None,
                     slot_v=None, nthreads: int = 0, decay: bool = False):
    """Alg. 1 (absolute-phase slots, Sec. 3.3) over q,k [B,H,L,dk], v [B,H,L,dv].

    slot_k / slot_v [B,H,S,d] are the slot states before token 0 (None = zero).
    decay applies the state decay of Sec. 3.4.
    Returns (o [B,H,L,dv], slot_k [B,H,S,dk], slot_v [B,H,S,dv]) in float64.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    Bn, H, L, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == q.shape and v.shape[:3] == (Bn, H, L)
    T = np.ascontiguousarray(np.broadcast_to(np.asarray(T, np.float64), (H,)))
    if scale is None:
        scale = 1.0 / np.sqrt(dk)
    kt_in, vt_in = _f64(slot_k), _f64(slot_v)
    o = np.zeros((Bn, H, L, dv), np.float64)
    kt = np.zeros((Bn, H, S, dk), np.float64)
    vt = np.zeros((Bn, H, S, dv), np.float64)
    rc = _load().bla_oracle_forward_anchored(Bn, H, L, dk, dv, M, S, _ptr(T), int(t0),
                                             float(scale), _ptr(q), _ptr(k), _ptr(v),
                                             _ptr(kt_in), _ptr(vt_in), _ptr(o), _ptr(kt),
                                             _ptr(vt), 1 if decay else 0, int(nthreads))
    if rc != 0:
        raise ValueError("bla_oracle_forward_anchored rejected its arguments")
    return o, kt, vt


def forward_decay(q, k, v, T, M: int, S: int, t0: int = 0, scale=None, slot_k=None,
                  slot_v=None, nthreads: int = 0):
    """Anchored slots with the state decay of Sec. 3.4; same arguments and results as
    forward_anchored."""
    return forward_anchored(q, k, v, T, M, S, t0=t0, scale=scale, slot_k=slot_k, slot_v=slot_v,
                            nthreads=nthreads, decay=True)


def backward(q, k, v, dO, T, M: int, S: int, t0: int = 0, scale=None, state_k=None, state_v=None,
             dstate_k=None, dstate_v=None, nthreads: int = 0):
    """Gradients of Alg. 2 (the operator of ``forward``) for the loss whose gradients are
    dO = dLoss/dO [B,H,L,dv] and dstate_k / dstate_v = dLoss/d(final states) [B,H,2,M,d]
    (None = zero).  state_k / state_v are the forward's input states (None = zero).

    Returns (dq [B,H,L,dk], dk [B,H,L,dk], dv [B,H,L,dv], dLoss/d(state_k in),
    dLoss/d(state_v in)) in float64.
    """
    q, k, v, dO = _f64(q), _f64(k), _f64(v), _f64(dO)
    Bn, H, L, dk = q.shape
    dv = v.shape[-1]
    assert k.shape == q.shape and v.shape[:3] == (Bn, H, L) and dO.shape == v.shape
    T = np.ascontiguousarray(np.broadcast_to(np.asarray(T, np.float64), (H,)))
    if scale is None:
        scale = 1.0 / np.sqrt(dk)
    dq = np.zeros_like(q)
    dkk = np.zeros_like(k)
    dvv = np.zeros_like(v)
    gsk = np.zeros((Bn, H, 2, M, dk), np.float64)
    gsv = np.zeros((Bn, H, 2, M, dv), np.float64)
    rc = _load().bla_oracle_backward(Bn, H, L, dk, dv, M, S, _ptr(T), int(t0), float(scale),
                                     _ptr(q), _ptr(k), _ptr(v), _ptr(dO), _ptr(_f64(state_k)),
                                     _ptr(_f64(state_v)), _ptr(_f64(dstate_k)), _ptr(_f64(dstate_v)),
                                     _ptr(dq), _ptr(dkk), _ptr(dvv), _ptr(gsk), _ptr(gsv),
                                     int(nthreads))
    if rc != 0:
        raise ValueError("bla_oracle_backward rejected its arguments")
    return dq, dkk, dvv, gsk, gsv


def layer_forward(x, w_qkv, w_o, T, H: int, M: int, S: int, t0: int = 0, scale=None, state_k=None,
                  state_v=None, nthreads: int = 0):
    """A BLA layer on hidden states x [B, L, D] (D = H d): [q | k | v] = x W_qkv (W_qkv [D, 3D],
    head h's columns h d .. h d + d - 1 of each block), the operator (``forward``) per head,
    y = concat_h(o_h) W_o (W_o [D, D]).  Everything in float64.

    Returns (y [B, L, D], state_k, state_v) as ``forward`` does.
    """
    x = _f64(x)
    Bn, L, D = x.shape
    d = D // H
    qkv = x @ _f64(w_qkv)                                     # [B, L, 3D]
    heads = qkv.reshape(Bn, L, 3, H, d).transpose(2, 0, 3, 1, 4)  # [3, B, H, L, d]
    o, sk, sv = forward(heads[0], heads[1], heads[2], T, M, S, t0=t0, scale=scale, state_k=state_k,
                        state_v=state_v, nthreads=nthreads)
    y = o.transpose(0, 2, 1, 3).reshape(Bn, L, D) @ _f64(w_o)
    return y, sk, sv
