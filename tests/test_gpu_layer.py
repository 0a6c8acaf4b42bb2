"""GPU parity of the whole layer: bla_layer_forward (hipBLASLt projections around the operator,
which reads q, k, v in place from the projection output and writes o in the output projection's
layout) against the oracle's float64 layer (numpy projections around the token-by-token
operator).  Bar: rel-L2 <= 2e-2 (bf16), with the per-element guard; the
projected q, k, v and the operator's output are rounded to bf16 on the GPU path only.
"""
import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle
from test_gpu_parity import TOL, _bla, _say, assert_close

pytestmark = pytest.mark.gpu


def run_layer(x, wqkv, wo, T, H, M, S, t0=0, rows=None, label="", phase_anchor=False):
    bla = _bla()
    _say(f"layer case {label}: x {x.shape} H={H} M={M} S={S} t0={t0}")
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda().to(torch.bfloat16)
    y, sk, sv = bla.layer_forward(dev(x), dev(wqkv), dev(wo), T, H, M, S, t0=t0, phase_anchor=phase_anchor)
    torch.cuda.synchronize()
    sel = slice(None) if rows is None else list(rows)
    ry, rk, rv = oracle.layer_forward(x[sel], wqkv, wo, T, H, M, S, t0=t0)
    tol = TOL[torch.bfloat16]
    assert_close(y.float().cpu().numpy()[sel], ry, tol, "y")
    assert_close(sk.cpu().numpy()[sel], rk, tol, "state_k")
    assert_close(sv.cpu().numpy()[sel], rv, tol, "state_v")


@pytest.mark.parametrize("B,L,H,d,M,S,T", [
    (2, 100, 2, 64, 16, 16, (31.0, 62.0)),        # ragged chunk
    (1, 300, 4, 32, 8, 15, (15.0, 30.0, 15.0, 40.5)),
    (3, 64, 1, 64, 32, 32, (63.0,)),
])
def test_layer_small_shapes(B, L, H, d, M, S, T):
    x, wqkv, wo = bi.generate_layer(2, B=B, L=L, H=H, d=d)
    run_layer(x, wqkv, wo, T, H, M, S, label=f"{B}x{L}x{H}x{d}")


def test_layer_workload2_recall_shape_sampled_rows():
    """The recall workload's shape (B=64, H=4, L=512, d=64, M=S=32; D = 256) at full size; the
    oracle checks three batch rows."""
    w = bi.WORKLOADS[2]
    x, wqkv, wo = bi.generate_layer(2)
    run_layer(x, wqkv, wo, bi.periods(w.M, w.H), w.H, w.M, w.S, rows=[0, 31, 63], label="workload 2 shape")


def test_layer_rejects_float32():
    bla = _bla()
    x = torch.zeros(1, 8, 64, device="cuda")
    with pytest.raises(ValueError):
        bla.layer_forward(x, torch.zeros(64, 192, device="cuda"), torch.zeros(64, 64, device="cuda"), [7.0], 1, 4, 7)
