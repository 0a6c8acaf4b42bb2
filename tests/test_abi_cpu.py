"""The C ABI on the host (no GPU needed): exports, shape rules, workspace sizes, and every
argument error path, which must return before any kernel is launched."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import paper_2606_09862_amd as bla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bla.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(bla.LIB_PATH):
        from paper_2606_09862_amd import build
        build.build()
    return bla.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bla_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"bla_forward", "bla_step", "bla_workspace_size"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"libbla.so does not export {n}"


def test_params_struct_layout():
    # int32 x8, then int64 t0 (8-aligned), float, int32, int32 (+4 tail pad) -> 56 bytes as in bla.h
    assert ctypes.sizeof(bla.Params) == 56
    assert bla.Params.t0.offset == 32 and bla.Params.io_dtype.offset == 44
    assert bla.Params.phase_anchor.offset == 48 and bla.Params.reuse_tables.offset == 52


def test_reuse_tables_flag(lib):
    """reuse_tables is 0 or 1 (anything else is an argument error); it does not change the
    workspace size."""
    p = P()
    base = bla.workspace_size(p)
    for val, expect in ((0, OK), (1, OK), (2, INVALID), (-1, INVALID)):
        p.reuse_tables = val
        assert bla.supported(p) == expect
    p.reuse_tables = 1
    assert bla.workspace_size(p) == base


def test_phase_anchor_flag(lib):
    """phase_anchor selects the anchored slots (1) or the rotating ones (0); anything else is
    an argument error.  The workspace does not depend on the form."""
    p = P()
    for val, expect in ((0, OK), (1, OK), (2, INVALID), (-1, INVALID)):
        p.phase_anchor = val
        assert bla.supported(p) == expect
    p.phase_anchor = 1
    a = bla.workspace_size(p)
    p.phase_anchor = 0
    assert a == bla.workspace_size(p) and a > 0


def test_status_strings(lib):
    for s in range(5):
        assert lib.bla_status_string(s).decode().startswith(bla.STATUS[s])
    assert lib.bla_status_string(99) == b"BLA_ERR_UNKNOWN"


def P(**kw):
    base = dict(B=2, H=2, L=100, d=64, M=16, S=16, dtype=None, t0=0, scale=0.0, chunk=0)
    base.update(kw)
    import torch
    dt = torch.bfloat16 if base.pop("dtype") in (None, "bf16") else torch.float32
    return bla.make_params(base["B"], base["H"], base["L"], base["d"], base["M"], base["S"], dt,
                           base["t0"], base["scale"], base["chunk"])


@pytest.mark.parametrize("kw,expect", [
    ({}, OK),
    (dict(d=32, M=16, S=16, dtype="f32"), OK),
    (dict(d=128, M=128, S=128), OK),
    (dict(M=64, S=127), OK),                 # S = 2M-1
    (dict(M=1, S=1), OK),
    (dict(M=128, S=255), OK),
    (dict(d=48), UNSUPPORTED),
    (dict(M=129), UNSUPPORTED),
    (dict(M=16, S=33), UNSUPPORTED),        # S beyond 2 * padded M
    (dict(S=257), UNSUPPORTED),
    (dict(chunk=16), OK),
    (dict(chunk=32), OK),
    (dict(chunk=64), OK),
    (dict(chunk=128), OK),
    (dict(chunk=128, d=32, dtype="f32"), OK),
    (dict(chunk=48), UNSUPPORTED),
    (dict(chunk=8), UNSUPPORTED),
    (dict(chunk=32, M=100, S=100), UNSUPPORTED),   # chunks other than 64 need P(M) <= 64
    (dict(chunk=128, d=64, M=64, S=64, dtype="f32"), UNSUPPORTED),  # float32 tiles exceed the LDS
    (dict(d=128, M=128, S=128, dtype="f32"), UNSUPPORTED),  # float32 tiles exceed the LDS
    (dict(M=0), INVALID),
    (dict(S=0), INVALID),
    (dict(L=-1), INVALID),
    (dict(B=-1), INVALID),
    (dict(t0=-5), INVALID),
    (dict(scale=float("nan")), INVALID),
])
def test_supported(lib, kw, expect):
    p = P(**kw)
    assert bla.supported(p) == expect


def test_dk_dv_mismatch_unsupported(lib):
    p = P()
    p.d_v = 32
    assert bla.supported(p) == UNSUPPORTED
    p = P()
    p.io_dtype = 7
    assert bla.supported(p) == INVALID


def test_workspace_sizes(lib):
    small = bla.workspace_size(P(B=64, H=4, L=512, d=64, M=32, S=32))
    assert small > 0
    assert bla.workspace_size(P(M=0)) == 0
    assert bla.step_workspace_size(P(B=512, H=16, L=1, d=64, M=64, S=64)) > 0
    # workloads that split sequences into segments need room for the block summaries
    seg = bla.workspace_size(P(B=1, H=16, L=65536, d=128, M=128, S=128))
    assert seg > 16 * 4 * 128 * 128 * 4


def _fake(addr):
    return ctypes.c_void_p(addr)


def call_forward(lib, p, T=None, q=0x10000, k=0x20000, v=0x30000, o=0x40000, ski=None, svi=None,
                 sko=None, svo=None, ws=0x100000, nbytes=1 << 40):
    H = max(p.H, 1)
    arr = (ctypes.c_double * H)(*([31.0] * H if T is None else T))
    return lib.bla_forward(ctypes.byref(p), arr, _fake(q), _fake(k), _fake(v), _fake(ski), _fake(svi),
                           _fake(o), _fake(sko), _fake(svo), _fake(ws), nbytes, None)


@pytest.mark.parametrize("T", [[float("nan"), 31.0], [0.0, 31.0], [-3.0, 31.0], [float("inf"), 31.0],
                               [1e10, 31.0]])
def test_bad_periods(lib, T):
    assert call_forward(lib, P(), T=T) == INVALID


def test_pointer_errors(lib):
    assert call_forward(lib, P(), q=0) == INVALID
    assert call_forward(lib, P(), o=0) == INVALID
    assert call_forward(lib, P(), v=0x30008) == INVALID            # misaligned
    assert call_forward(lib, P(), ski=0x50004) == INVALID          # misaligned state
    assert call_forward(lib, P(), ski=0x50000, sko=0x50000) == INVALID  # output aliases input
    assert call_forward(lib, P(), ws=0) == WORKSPACE
    assert call_forward(lib, P(), nbytes=16) == WORKSPACE
    assert call_forward(lib, P(), ws=0x100004) == WORKSPACE        # misaligned workspace
    assert lib.bla_forward(None, None, *([None] * 9), 0, None) == INVALID


def test_empty_batch_is_a_noop(lib):
    # B = 0: nothing to compute, null data pointers are fine, no workspace needed
    p = P(B=0)
    assert call_forward(lib, p, q=0, k=0, v=0, o=0, ws=0, nbytes=0) == OK


def test_step_errors(lib):
    p = P(L=1)
    H = 2
    arr = (ctypes.c_double * H)(31.0, 62.0)
    args = [_fake(0x10000), _fake(0x20000), _fake(0x30000), None, _fake(0x40000), _fake(0x50000),
            _fake(0x60000)]
    assert lib.bla_step(ctypes.byref(p), arr, *args, _fake(0x100000), 16, None) == WORKSPACE
    bad = list(args)
    bad[3] = _fake(0x70004)   # pos not 8-byte aligned
    assert lib.bla_step(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    bad = list(args)
    bad[4] = None             # state_k missing
    assert lib.bla_step(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    nan = (ctypes.c_double * H)(math.nan, 1.0)
    assert lib.bla_step(ctypes.byref(p), nan, *args, _fake(0x100000), 1 << 40, None) == INVALID


def test_decay_errors(lib):
    """Argument checks of the decay entry points run before any launch (no GPU needed)."""
    p = P(L=10)
    H = 2
    arr = (ctypes.c_double * H)(31.0, 62.0)
    assert bla.decay_workspace_size(p) > 0
    fwd = [_fake(0x10000), _fake(0x20000), _fake(0x30000), None, None, _fake(0x40000), None, None]
    assert lib.bla_decay_forward(ctypes.byref(p), arr, *fwd, _fake(0x100000), 16, None) == WORKSPACE
    bad = list(fwd)
    bad[0] = None              # q missing
    assert lib.bla_decay_forward(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    bad = list(fwd)
    bad[2] = _fake(0x30008)    # v not 16-byte aligned
    assert lib.bla_decay_forward(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    bad = list(fwd)
    bad[3] = _fake(0x50000)    # slot_k_out aliasing slot_k_in
    bad[6] = _fake(0x50000)
    assert lib.bla_decay_forward(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    nan = (ctypes.c_double * H)(math.nan, 1.0)
    assert lib.bla_decay_forward(ctypes.byref(p), nan, *fwd, _fake(0x100000), 1 << 40, None) == INVALID
    step = [_fake(0x10000), _fake(0x20000), _fake(0x30000), None, _fake(0x40000), _fake(0x50000),
            _fake(0x60000)]
    assert lib.bla_decay_step(ctypes.byref(p), arr, *step, _fake(0x100000), 16, None) == WORKSPACE
    bad = list(step)
    bad[4] = None              # slot_k missing
    assert lib.bla_decay_step(ctypes.byref(p), arr, *bad, _fake(0x100000), 1 << 40, None) == INVALID
    q = P(d=48)
    assert bla.decay_workspace_size(q) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(bla, "LIB_PATH", str(tmp_path / "nope.so"))
    monkeypatch.setattr(bla, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        bla.lib()


@pytest.mark.parametrize("M,S,T", [(16, 16, 31.0), (8, 15, 15.0), (64, 64, 254.0), (5, 9, 3.0), (24, 40, 47.5),
                                   (16, 16, 62.0)])
def test_interp_tables_match_oracle(lib, M, S, T):
    """The library's host slot tables against the oracle's (independent code, same formulas);
    T = 3 is clamped to 2M-1 = 9, and S = 16, T = 62 hits a rounding tie (s = 12: 46.5 -> 46)."""
    import oracle
    A, B, th = bla.interp_tables(M, S, T)
    A2, B2, th2 = oracle.interp(M, S, T)
    assert np.max(np.abs(A - A2)) < 1e-13 and np.max(np.abs(B - B2)) < 1e-13
    assert np.array_equal(th.astype(np.int64), th2)


def test_interp_tables_errors(lib):
    A = np.zeros(16, np.float64)
    th = np.zeros(4, np.int32)
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int32)
    f = lib.bla_interp_tables
    ok = f(4, 4, 7.0, A.ctypes.data_as(dp), A.ctypes.data_as(dp), th.ctypes.data_as(ip))
    assert ok == 0
    for args in [(0, 4, 7.0), (4, 0, 7.0), (4, 4, 0.0), (4, 4, float("nan")), (4, 4, float("inf"))]:
        assert f(*args, A.ctypes.data_as(dp), A.ctypes.data_as(dp), th.ctypes.data_as(ip)) == INVALID
    assert f(4, 4, 7.0, None, A.ctypes.data_as(dp), th.ctypes.data_as(ip)) == INVALID


def test_backward_errors(lib):
    """Argument and shape checks of bla_backward run before any launch (no GPU needed)."""
    p = P(L=10)
    H = 2
    arr = (ctypes.c_double * H)(31.0, 62.0)
    assert bla.backward_workspace_size(p) > 0
    # q, k, v, dO, state_k_in, state_v_in, dstate_k_out, dstate_v_out, dq, dk, dv, dstate_k_in, dstate_v_in
    args = [_fake(0x10000), _fake(0x20000), _fake(0x30000), _fake(0x40000), None, None, None, None,
            _fake(0x50000), _fake(0x60000), _fake(0x70000), None, None]
    call = lambda a, nbytes=1 << 40, params=p, T=arr: lib.bla_backward(
        ctypes.byref(params), T, *a, _fake(0x100000), nbytes, None)
    assert call(args, nbytes=16) == WORKSPACE
    for i in (0, 3, 8, 10):              # q, dO, dq, dv missing
        bad = list(args)
        bad[i] = None
        assert call(bad) == INVALID
    bad = list(args)
    bad[9] = _fake(0x60008)              # dk not 16-byte aligned
    assert call(bad) == INVALID
    bad = list(args)
    bad[6] = bad[11] = _fake(0x80000)    # dstate_k_in aliasing dstate_k_out
    assert call(bad) == INVALID
    nan = (ctypes.c_double * H)(math.nan, 1.0)
    assert call(args, T=nan) == INVALID
    # outside the backward's shapes: d = 128, M > 64, the anchored form
    assert bla.backward_workspace_size(P(d=128)) == 0
    assert bla.backward_workspace_size(P(M=100, S=100)) == 0
    pa = P(L=10)
    pa.phase_anchor = 1
    assert bla.backward_workspace_size(pa) == 0
    assert call(args, params=pa) == UNSUPPORTED
    assert bla.backward_workspace_size(P(dtype="f32", d=32, M=32, S=64)) > 0
    assert bla.backward_workspace_size(P(dtype="f32", d=64)) == 0
    # the backward runs 64-token chunks only
    assert bla.backward_workspace_size(P(chunk=64)) > 0
    assert bla.backward_workspace_size(P(chunk=32)) == 0
    assert call(args, params=P(L=10, chunk=32)) == UNSUPPORTED


def test_layer_errors(lib):
    """Shape and argument checks of bla_layer_forward before any launch (no GPU needed)."""
    p = P(L=10, d=64, H=2)
    arr = (ctypes.c_double * 2)(31.0, 62.0)
    assert bla.layer_workspace_size(p) > 0
    assert bla.layer_workspace_size(P(dtype="f32")) == 0          # the layer is bf16 only
    args = [_fake(0x10000), _fake(0x20000), _fake(0x30000), None, None, _fake(0x40000), None, None]
    call = lambda a, nbytes=1 << 40: lib.bla_layer_forward(ctypes.byref(p), arr, *a, _fake(0x100000), nbytes, None)
    assert call(args, nbytes=16) == WORKSPACE
    for i in (0, 1, 2, 5):                                      # x, W_qkv, W_o, y missing
        bad = list(args)
        bad[i] = None
        assert call(bad) == INVALID
    bad = list(args)
    bad[1] = _fake(0x20008)                                      # misaligned W_qkv
    assert call(bad) == INVALID


def test_binding_argument_counts_match_the_header(lib):
    """Every entry point the binding declares argument types for takes as many arguments as
    its C declaration in include/bla.h."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    seen = 0
    for m in re.finditer(r"\b(bla_[a-z_]+)\s*\(([^;{]*?)\)\s*;", text):
        name, params = m.group(1), m.group(2).strip()
        n = 0 if params in ("", "void") else params.count(",") + 1
        at = getattr(getattr(lib, name), "argtypes", None)
        if at is not None:
            seen += 1
            assert len(at) == n, f"{name}: binding has {len(at)} argument types, the header {n} parameters"
    assert seen >= 10
