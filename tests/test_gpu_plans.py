"""GPU checks of the launch plan's choices and of the call conventions around the kernels:

* few long sequences (B*H small): the pair kernel's segments are capped and the one-unit
  kernels with per-block summaries and the scan run instead, against the oracle;
* reuse_tables: tables kept in a workspace across calls, rebuilt when the record of the
  workspace does not match the call (other periods, another entry point in between);
* the binding rejects a wrong `out` buffer before any launch.
"""
import numpy as np
import pytest
import torch

import oracle
from test_gpu_parity import _bla, _say, assert_close, gauss, run_case, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (1, 2, 64 * 64, 64, 64, 64, (127.0, 254.0)),      # 64 segments of one chunk on the one-unit kernels
    (1, 1, 64 * 40 + 17, 32, 16, 31, (31.0,)),        # ragged tail, d = 32
])
def test_few_long_sequences_bf16(B, H, L, d, M, S, T):
    q, k, v = gauss(L + d, B, H, L, d, torch.bfloat16)
    run_case(q, k, v, T, M, S, torch.bfloat16, label=f"few long sequences {B}x{H}x{L}x{d}")


def test_one_sequence_64k_tokens():
    """B = H = 1, L = 65536, d = M = S = 64 in bf16: one sequence split over the whole device
    (the regime where the pair kernel's summary combination would grow with nseg^2)."""
    B, H, L, d, M, S, T = 1, 1, 65536, 64, 64, 64, (127.0,)
    q, k, v = gauss(65536, B, H, L, d, torch.bfloat16)
    run_case(q, k, v, T, M, S, torch.bfloat16, label="one sequence of 65536 tokens")


def test_reuse_tables():
    bla = _bla()
    B, H, L, d, M, S = 2, 2, 64 * 9 + 5, 64, 32, 32
    T1, T2 = (63.0, 126.0), (70.5, 90.0)
    q, k, v = gauss(21, B, H, L, d, torch.bfloat16)
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    p = bla.make_params(B, H, L, d, M, S, torch.bfloat16)
    ws = torch.empty(bla.workspace_size(p), dtype=torch.uint8, device="cuda")
    ref1 = bla.forward(tq, tk, tv, T1, M, S, workspace=ws)
    again = bla.forward(tq, tk, tv, T1, M, S, workspace=ws, reuse_tables=True)   # tables kept
    torch.cuda.synchronize()
    for a, b in zip(ref1, again):
        assert torch.equal(a, b)
    # other periods with the flag set: the record does not match, so the tables are rebuilt
    got2 = bla.forward(tq, tk, tv, T2, M, S, workspace=ws, reuse_tables=True)
    torch.cuda.synchronize()
    ro, rk, rv = oracle.forward(q, k, v, T2, M, S)
    assert_close(got2[0].float().cpu().numpy(), ro, 2e-2, "O, new periods")
    assert_close(got2[1].cpu().numpy(), rk, 2e-2, "state_k, new periods")
    # a decode step writes its own tables into the same workspace; the next forward with the
    # flag must notice and rebuild
    sk, sv = got2[1].clone(), got2[2].clone()
    bla.step(tq[:, :, 0].contiguous(), tk[:, :, 0].contiguous(), tv[:, :, 0].contiguous(), T1, M, S, sk, sv,
             t0=L, workspace=ws)
    got1 = bla.forward(tq, tk, tv, T1, M, S, workspace=ws, reuse_tables=True)
    torch.cuda.synchronize()
    for a, b in zip(ref1, got1):
        assert torch.equal(a, b)


def test_reuse_tables_wide():
    """The d = M = 128 plan keeps fragment-ordered copies of its tables next to the row-major
    ones: kept with the tables, rebuilt with them when the periods change."""
    bla = _bla()
    B, H, L, d, M, S = 1, 2, 64 * 5 + 11, 128, 128, 128
    T1, T2 = (255.0, 300.0), (400.0, 260.5)
    q, k, v = gauss(41, B, H, L, d, torch.bfloat16)
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    p = bla.make_params(B, H, L, d, M, S, torch.bfloat16)
    ws = torch.empty(bla.workspace_size(p), dtype=torch.uint8, device="cuda")
    ref1 = bla.forward(tq, tk, tv, T1, M, S, workspace=ws)
    again = bla.forward(tq, tk, tv, T1, M, S, workspace=ws, reuse_tables=True)
    torch.cuda.synchronize()
    for a, b in zip(ref1, again):
        assert torch.equal(a, b)
    got2 = bla.forward(tq, tk, tv, T2, M, S, workspace=ws, reuse_tables=True)
    torch.cuda.synchronize()
    ro, rk, rv = oracle.forward(q, k, v, T2, M, S)
    assert_close(got2[0].float().cpu().numpy(), ro, 2e-2, "O, new periods")
    assert_close(got2[2].cpu().numpy(), rv, 2e-2, "state_v, new periods")
    got1 = bla.forward(tq, tk, tv, T1, M, S, workspace=ws, reuse_tables=True)
    torch.cuda.synchronize()
    for a, b in zip(ref1, got1):
        assert torch.equal(a, b)


def test_out_buffer_is_checked():
    bla = _bla()
    q, k, v = (to_dev(x, torch.bfloat16) for x in gauss(3, 1, 2, 70, 32, torch.bfloat16))
    for bad in (torch.empty(1, 2, 69, 32, dtype=torch.bfloat16, device="cuda"),      # too small
                torch.empty(1, 2, 70, 32, dtype=torch.float32, device="cuda"),       # wrong dtype
                torch.empty(1, 2, 32, 70, dtype=torch.bfloat16, device="cuda").transpose(2, 3)):  # strided
        with pytest.raises(ValueError, match="out"):
            bla.forward(q, k, v, (31.0, 62.0), 16, 16, out=bad)
    sk = torch.zeros(1, 2, 2, 16, 32, device="cuda")
    sv = torch.zeros_like(sk)
    with pytest.raises(ValueError, match="out"):
        bla.step(q[:, :, 0].contiguous(), k[:, :, 0].contiguous(), v[:, :, 0].contiguous(), (31.0, 62.0), 16, 16,
                 sk, sv, out=torch.empty(1, 2, 16, dtype=torch.bfloat16, device="cuda"))
    good = torch.empty_like(q)
    o, _, _ = bla.forward(q, k, v, (31.0, 62.0), 16, 16, out=good)
    torch.cuda.synchronize()
    assert o.data_ptr() == good.data_ptr()
    _say("out buffers checked")
