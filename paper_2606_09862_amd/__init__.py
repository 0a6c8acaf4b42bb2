"""Blurry Window Attention forward operator (and its backward pass) on MI355X (gfx950).

A thin ctypes binding over ``libbla.so`` (the C ABI in ``include/bla.h``).  It
only marshals arguments: every step of the operator runs in the library's HIP
kernels.  torch is used for device buffers and the current stream.  If the
library has not been built, importing works but every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbla.so")

BLA_F32, BLA_BF16 = 0, 1
STATUS = {0: "BLA_OK", 1: "BLA_ERR_INVALID_ARG", 2: "BLA_ERR_UNSUPPORTED", 3: "BLA_ERR_WORKSPACE",
          4: "BLA_ERR_HIP"}


class BlaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what} failed: {STATUS.get(status, status)}")
        self.status = status


class Params(ctypes.Structure):
    """Mirror of ``bla_params``."""
    _fields_ = [("B", ctypes.c_int32), ("H", ctypes.c_int32), ("L", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("M", ctypes.c_int32),
                ("S", ctypes.c_int32), ("chunk", ctypes.c_int32), ("t0", ctypes.c_int64),
                ("scale", ctypes.c_float), ("io_dtype", ctypes.c_int32),
                ("phase_anchor", ctypes.c_int32), ("reuse_tables", ctypes.c_int32)]


_lib = None
_dp = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p


def lib():
    """The loaded library; raises if it is missing (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2606_09862_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(Params)
        L.bla_status_string.argtypes = [ctypes.c_int]
        L.bla_status_string.restype = ctypes.c_char_p
        L.bla_supported.argtypes = [P]
        L.bla_supported.restype = ctypes.c_int
        L.bla_workspace_size.argtypes = [P]
        L.bla_workspace_size.restype = ctypes.c_size_t
        L.bla_step_workspace_size.argtypes = [P]
        L.bla_step_workspace_size.restype = ctypes.c_size_t
        L.bla_forward.argtypes = [P, _dp] + [_vp] * 9 + [ctypes.c_size_t, _vp]
        L.bla_forward.restype = ctypes.c_int
        L.bla_step.argtypes = [P, _dp] + [_vp] * 8 + [ctypes.c_size_t, _vp]
        L.bla_forward_noalloc.argtypes = [P, _dp] + [_vp] * 8 + [_vp]
        L.bla_forward_noalloc.restype = ctypes.c_int
        L.bla_interp_tables.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_double, _dp, _dp,
                                        ctypes.POINTER(ctypes.c_int32)]
        L.bla_interp_tables.restype = ctypes.c_int
        L.bla_step.restype = ctypes.c_int
        L.bla_decay_workspace_size.argtypes = [P]
        L.bla_decay_workspace_size.restype = ctypes.c_size_t
        L.bla_decay_forward.argtypes = [P, _dp] + [_vp] * 9 + [ctypes.c_size_t, _vp]
        L.bla_decay_forward.restype = ctypes.c_int
        L.bla_decay_step.argtypes = [P, _dp] + [_vp] * 8 + [ctypes.c_size_t, _vp]
        L.bla_decay_step.restype = ctypes.c_int
        L.bla_backward_workspace_size.argtypes = [P]
        L.bla_backward_workspace_size.restype = ctypes.c_size_t
        L.bla_backward.argtypes = [P, _dp] + [_vp] * 14 + [ctypes.c_size_t, _vp]
        L.bla_backward.restype = ctypes.c_int
        L.bla_backward_timed.argtypes = [P, _dp] + [_vp] * 14 + [ctypes.c_size_t, _vp,
                                                                  ctypes.POINTER(ctypes.c_void_p)]
        L.bla_backward_timed.restype = ctypes.c_int
        L.bla_layer_workspace_size.argtypes = [P]
        L.bla_layer_workspace_size.restype = ctypes.c_size_t
        L.bla_layer_forward.argtypes = [P, _dp] + [_vp] * 9 + [ctypes.c_size_t, _vp]
        L.bla_layer_forward.restype = ctypes.c_int
        L.bla_layer_forward_timed.argtypes = [P, _dp] + [_vp] * 9 + [ctypes.c_size_t, _vp,
                                                                       ctypes.POINTER(ctypes.c_void_p)]
        L.bla_layer_forward_timed.restype = ctypes.c_int
        _lib = L
    return _lib


def make_params(B, H, L, d, M, S, dtype, t0=0, scale=0.0, chunk=0, phase_anchor=False,
                reuse_tables=False) -> Params:
    io = BLA_BF16 if dtype == torch.bfloat16 else BLA_F32
    return Params(B, H, L, d, d, M, S, chunk, int(t0), float(scale), io, int(phase_anchor),
                  int(reuse_tables))


def _periods(T, H):
    arr = (ctypes.c_double * max(H, 1))()
    vals = list(T) if hasattr(T, "__len__") else [T] * H
    if len(vals) != H:
        raise ValueError("T must have one period per head")
    for i, x in enumerate(vals):
        arr[i] = float(x)
    return arr


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def interp_tables(M: int, S: int, T: float):
    """Float64 slot tables of one head from the library: A, B [S, M] and thresholds [S]."""
    import numpy as np
    A = np.zeros((S, M), np.float64)
    B = np.zeros((S, M), np.float64)
    th = np.zeros((S,), np.int32)
    st = lib().bla_interp_tables(M, S, float(T), A.ctypes.data_as(_dp), B.ctypes.data_as(_dp),
                                 th.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    if st != 0:
        raise BlaError(st, "bla_interp_tables")
    return A, B, th


def supported(p: Params) -> int:
    return lib().bla_supported(ctypes.byref(p))


def workspace_size(p: Params) -> int:
    return lib().bla_workspace_size(ctypes.byref(p))


def step_workspace_size(p: Params) -> int:
    return lib().bla_step_workspace_size(ctypes.byref(p))


def _check(t, shape, dtype, name):
    if t.shape != tuple(shape) or t.dtype != dtype or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected contiguous {dtype} cuda tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def _out(out, like, shape):
    """A fresh output like `like`, or the caller's `out` after the same checks as the inputs
    (shape, dtype, contiguity, device), so that a wrong buffer fails before any launch."""
    if out is None:
        return torch.empty_like(like)
    _check(out, shape, like.dtype, "out")
    if out.device != like.device:
        raise ValueError(f"out: expected a tensor on {like.device}, got {out.device}")
    return out


def forward(q, k, v, T, M: int, S: int, t0: int = 0, scale: float | None = None,
            state_k=None, state_v=None, want_state: bool = True, workspace=None, out=None,
            phase_anchor: bool = False, reuse_tables: bool = False, chunk: int = 0):
    """bla_forward on q, k, v [B,H,L,d] (float32 or bfloat16 cuda tensors).

    Returns (o, state_k_out, state_v_out); the states are float32 [B,H,2,M,d]
    (None when want_state is False).  phase_anchor selects the anchored slots of
    Sec. 3.3 (Alg. 1 / Alg. 3); the state is the same mode state in both forms.
    reuse_tables: keep the tables an earlier call built in the same `workspace`
    (bla_params.reuse_tables; only meaningful with a caller-kept workspace).  chunk: tokens
    per chunk of the parallel form (16, 32, 64 or 128; 0 = 64).
    """
    B, H, L, d = q.shape
    dt = q.dtype
    for name, t in (("k", k), ("v", v)):
        _check(t, (B, H, L, d), dt, name)
    _check(q, (B, H, L, d), dt, "q")
    p = make_params(B, H, L, d, M, S, dt, t0, 0.0 if scale is None else scale, chunk=chunk,
                    phase_anchor=phase_anchor, reuse_tables=reuse_tables)
    for name, t in (("state_k", state_k), ("state_v", state_v)):
        if t is not None:
            _check(t, (B, H, 2, M, d), torch.float32, name)
    dev = q.device
    o = _out(out, q, (B, H, L, d))
    sk = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state else None
    sv = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state else None
    need = workspace_size(p)
    if need == 0 and supported(p) != 0:
        raise BlaError(supported(p), "bla_forward (shape check)")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().bla_forward(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(state_k),
                           _ptr(state_v), _ptr(o), _ptr(sk), _ptr(sv), _ptr(workspace),
                           workspace.numel(), _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_forward")
    return o, sk, sv


def forward_noalloc(q, k, v, T, M: int, S: int, t0: int = 0, scale: float | None = None,
                    state_k=None, state_v=None, out=None, state_k_out=None, state_v_out=None,
                    phase_anchor: bool = False, reuse_tables: bool = False):
    """bla_forward_noalloc: bla_forward with the library's own fixed device workspace.  The
    library allocates nothing; the caller passes every output (`out`, and `state_k_out` /
    `state_v_out` float32 [B,H,2,M,d], None = not wanted).  Returns (o, state_k_out, state_v_out)."""
    B, H, L, d = q.shape
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, (B, H, L, d), dt, name)
    if out is None:
        raise ValueError("out: bla_forward_noalloc needs the caller's output buffer")
    o = _out(out, q, (B, H, L, d))
    for name, t in (("state_k", state_k), ("state_v", state_v), ("state_k_out", state_k_out),
                    ("state_v_out", state_v_out)):
        if t is not None:
            _check(t, (B, H, 2, M, d), torch.float32, name)
    p = make_params(B, H, L, d, M, S, dt, t0, 0.0 if scale is None else scale,
                    phase_anchor=phase_anchor, reuse_tables=reuse_tables)
    st = lib().bla_forward_noalloc(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(state_k),
                                   _ptr(state_v), _ptr(o), _ptr(state_k_out), _ptr(state_v_out),
                                   _stream(q.device))
    if st != 0:
        raise BlaError(st, "bla_forward_noalloc")
    return o, state_k_out, state_v_out


def step(q, k, v, T, M: int, S: int, state_k, state_v, pos=None, t0: int = 0,
         scale: float | None = None, workspace=None, out=None, phase_anchor: bool = False,
         reuse_tables: bool = False):
    """bla_step: one decode token per row; q,k,v [B,H,d]; updates state_k/state_v in place."""
    B, H, d = q.shape
    dt = q.dtype
    _check(q, (B, H, d), dt, "q")
    _check(k, (B, H, d), dt, "k")
    _check(v, (B, H, d), dt, "v")
    _check(state_k, (B, H, 2, M, d), torch.float32, "state_k")
    _check(state_v, (B, H, 2, M, d), torch.float32, "state_v")
    if pos is not None:
        _check(pos, (B,), torch.int64, "pos")
    p = make_params(B, H, 1, d, M, S, dt, t0, 0.0 if scale is None else scale,
                    phase_anchor=phase_anchor, reuse_tables=reuse_tables)
    dev = q.device
    o = _out(out, q, (B, H, d))
    need = step_workspace_size(p)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().bla_step(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(pos),
                        _ptr(state_k), _ptr(state_v), _ptr(o), _ptr(workspace), workspace.numel(),
                        _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_step")
    return o


def decay_workspace_size(p: Params) -> int:
    return lib().bla_decay_workspace_size(ctypes.byref(p))


def decay_forward(q, k, v, T, M: int, S: int, t0: int = 0, scale: float | None = None,
                  slot_k=None, slot_v=None, want_state: bool = True, workspace=None, out=None):
    """bla_decay_forward (state-decay form, Sec. 3.4) on q, k, v [B,H,L,d].

    Returns (o, slot_k_out, slot_v_out); slot states are float32 [B,H,S,d].
    """
    B, H, L, d = q.shape
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, (B, H, L, d), dt, name)
    for name, t in (("slot_k", slot_k), ("slot_v", slot_v)):
        if t is not None:
            _check(t, (B, H, S, d), torch.float32, name)
    p = make_params(B, H, L, d, M, S, dt, t0, 0.0 if scale is None else scale)
    dev = q.device
    o = _out(out, q, (B, H, L, d))
    sk = torch.empty((B, H, S, d), dtype=torch.float32, device=dev) if want_state else None
    sv = torch.empty((B, H, S, d), dtype=torch.float32, device=dev) if want_state else None
    need = decay_workspace_size(p)
    if need == 0 and supported(p) != 0:
        raise BlaError(supported(p), "bla_decay_forward (shape check)")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().bla_decay_forward(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(slot_k),
                                 _ptr(slot_v), _ptr(o), _ptr(sk), _ptr(sv), _ptr(workspace),
                                 workspace.numel(), _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_decay_forward")
    return o, sk, sv


def decay_step(q, k, v, T, M: int, S: int, slot_k, slot_v, pos=None, t0: int = 0,
               scale: float | None = None, workspace=None, out=None):
    """bla_decay_step: one decode token per row; q,k,v [B,H,d]; updates slot_k/slot_v in place."""
    B, H, d = q.shape
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v)):
        _check(t, (B, H, d), dt, name)
    _check(slot_k, (B, H, S, d), torch.float32, "slot_k")
    _check(slot_v, (B, H, S, d), torch.float32, "slot_v")
    if pos is not None:
        _check(pos, (B,), torch.int64, "pos")
    p = make_params(B, H, 1, d, M, S, dt, t0, 0.0 if scale is None else scale)
    dev = q.device
    o = _out(out, q, (B, H, d))
    need = decay_workspace_size(p)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    st = lib().bla_decay_step(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(pos),
                              _ptr(slot_k), _ptr(slot_v), _ptr(o), _ptr(workspace), workspace.numel(),
                              _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_decay_step")
    return o


def backward_workspace_size(p: Params) -> int:
    return lib().bla_backward_workspace_size(ctypes.byref(p))


def backward(q, k, v, dO, T, M: int, S: int, t0: int = 0, scale: float | None = None,
             state_k=None, state_v=None, dstate_k=None, dstate_v=None, want_state_grad: bool = True,
             workspace=None):
    """bla_backward: gradients of ``forward`` (rotating slots) for dO = dLoss/dO [B,H,L,d] and
    dstate_k / dstate_v = dLoss/d(final states) [B,H,2,M,d] (None = zero).  state_k / state_v
    are the forward's input states.  Returns (dq, dk, dv, dLoss/d(state_k in),
    dLoss/d(state_v in)); the last two are None when want_state_grad is False.
    """
    B, H, L, d = q.shape
    dt = q.dtype
    for name, t in (("q", q), ("k", k), ("v", v), ("dO", dO)):
        _check(t, (B, H, L, d), dt, name)
    for name, t in (("state_k", state_k), ("state_v", state_v), ("dstate_k", dstate_k),
                    ("dstate_v", dstate_v)):
        if t is not None:
            _check(t, (B, H, 2, M, d), torch.float32, name)
    p = make_params(B, H, L, d, M, S, dt, t0, 0.0 if scale is None else scale)
    dev = q.device
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    gsk = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state_grad else None
    gsv = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state_grad else None
    need = backward_workspace_size(p)
    if need == 0:
        raise BlaError(2, "bla_backward (shape check)")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    st = lib().bla_backward(ctypes.byref(p), _periods(T, H), _ptr(q), _ptr(k), _ptr(v), _ptr(dO),
                            _ptr(state_k), _ptr(state_v), _ptr(dstate_k), _ptr(dstate_v), _ptr(dq),
                            _ptr(dk), _ptr(dv), _ptr(gsk), _ptr(gsv), _ptr(workspace), workspace.numel(),
                            _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_backward")
    return dq, dk, dv, gsk, gsv


def layer_workspace_size(p: Params) -> int:
    return lib().bla_layer_workspace_size(ctypes.byref(p))


def layer_forward(x, w_qkv, w_o, T, H: int, M: int, S: int, t0: int = 0, scale: float | None = None,
                  state_k=None, state_v=None, want_state: bool = True, workspace=None, out=None,
                  phase_anchor: bool = False):
    """bla_layer_forward: y = BLA(x W_qkv) W_o on hidden states x [B, L, D] (bf16, D = H d);
    w_qkv [D, 3D] and w_o [D, D] bf16.  Returns (y [B, L, D], state_k_out, state_v_out)."""
    B, L, D = x.shape
    d = D // H
    dt = x.dtype
    if dt != torch.bfloat16 or d * H != D:
        raise ValueError("layer_forward: bf16 hidden states with D = H * d")
    _check(x, (B, L, D), dt, "x")
    _check(w_qkv, (D, 3 * D), dt, "w_qkv")
    _check(w_o, (D, D), dt, "w_o")
    for name, t in (("state_k", state_k), ("state_v", state_v)):
        if t is not None:
            _check(t, (B, H, 2, M, d), torch.float32, name)
    p = make_params(B, H, L, d, M, S, dt, t0, 0.0 if scale is None else scale, phase_anchor=phase_anchor)
    dev = x.device
    y = _out(out, x, (B, L, D))
    sk = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state else None
    sv = torch.empty((B, H, 2, M, d), dtype=torch.float32, device=dev) if want_state else None
    need = layer_workspace_size(p)
    if need == 0:
        raise BlaError(supported(p) or 2, "bla_layer_forward (shape check)")
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    st = lib().bla_layer_forward(ctypes.byref(p), _periods(T, H), _ptr(x), _ptr(w_qkv), _ptr(w_o), _ptr(state_k),
                                 _ptr(state_v), _ptr(y), _ptr(sk), _ptr(sv), _ptr(workspace), workspace.numel(),
                                 _stream(dev))
    if st != 0:
        raise BlaError(st, "bla_layer_forward")
    return y, sk, sv
