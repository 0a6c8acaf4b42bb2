"""bla_forward_noalloc (the forward with the library's own fixed device workspace, for callers
that cannot allocate) against bla_forward with a caller workspace: two calls in a row, the
second on a smaller input, each bitwise equal to bla_forward's result (the same kernels on the
same plan) and within the parity bar of the oracle."""
import numpy as np
import pytest
import torch

import oracle
from test_gpu_parity import _bla, _say, assert_close, gauss, to_dev

pytestmark = pytest.mark.gpu


def _one(bla, B, H, L, d, M, S, T, dtype, t0, seed, with_state):
    q, k, v = gauss(seed, B, H, L, d, dtype)
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    sk_in = sv_in = None
    if with_state:
        rng = np.random.default_rng(seed + 1)
        sk_in = torch.from_numpy((rng.standard_normal((B, H, 2, M, d)) * 0.3).astype(np.float32)).cuda()
        sv_in = torch.from_numpy((rng.standard_normal((B, H, 2, M, d)) * 0.3).astype(np.float32)).cuda()
        sk_in[:, :, 1, 0] = 0.0
        sv_in[:, :, 1, 0] = 0.0
    _say(f"no-alloc case {B}x{H}x{L}x{d} M={M} S={S} t0={t0} {dtype}")
    o = torch.empty_like(tq)
    sk = torch.empty(B, H, 2, M, d, device="cuda")
    sv = torch.empty_like(sk)
    bla.forward_noalloc(tq, tk, tv, T, M, S, t0=t0, state_k=sk_in, state_v=sv_in, out=o, state_k_out=sk,
                        state_v_out=sv)
    ro, rk, rv = bla.forward(tq, tk, tv, T, M, S, t0=t0, state_k=sk_in, state_v=sv_in)
    torch.cuda.synchronize()
    assert torch.equal(o, ro) and torch.equal(sk, rk) and torch.equal(sv, rv)
    to = lambda x: None if x is None else x.cpu().numpy().astype(np.float64)
    eo, ek, ev = oracle.forward(q, k, v, T, M, S, t0=t0, state_k=to(sk_in), state_v=to(sv_in))
    tol = 2e-2 if dtype == torch.bfloat16 else 1e-4
    assert_close(o.float().cpu().numpy(), eo, tol, "O (no-alloc)")
    assert_close(sk.cpu().numpy(), ek, tol, "state_k (no-alloc)")
    assert_close(sv.cpu().numpy(), ev, tol, "state_v (no-alloc)")


def test_noalloc_matches_forward_twice():
    bla = _bla()
    # first call: several segments, state in, t0 > 0; second call smaller, another dtype and shape
    _one(bla, 2, 4, 64 * 13 + 7, 64, 64, 64, (127.0, 254.0, 127.0, 254.0), torch.bfloat16, 100, 31, True)
    _one(bla, 1, 2, 150, 32, 16, 20, (31.0, 77.25), torch.float32, 0, 32, False)


def test_noalloc_rejects_oversized_workspace():
    bla = _bla()
    # a shape whose workspace exceeds the fixed array: an error before any launch
    B, H, L, d, M, S = 1, 16, 65536, 128, 128, 128
    p = bla.make_params(B, H, L, d, M, S, torch.bfloat16)
    assert bla.workspace_size(p) > (64 << 20)
    x = torch.empty(B, H, L, d, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(bla.BlaError) as e:
        bla.forward_noalloc(x, x, x, [255.0] * H, M, S, out=torch.empty_like(x))
    assert e.value.status == 3
