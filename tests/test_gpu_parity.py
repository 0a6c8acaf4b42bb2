"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Bar (from the operator's specification): relative L2 error <= 1e-4 for float32
inputs and <= 2e-2 for bfloat16 inputs, on the outputs and on the final states.
Two local guards catch errors confined to a few tokens (one chunk boundary, one
segment start) that an L2 norm over the whole tensor would dilute:
  * per row (one token's output vector, one mode's state row): the relative error
    of the row, ||got_t - ref_t|| / ||ref_t||, at most 2.5x the bar for bfloat16
    (5e-2) and 10x the bar for float32 (1e-3); rows whose reference norm is below
    a tenth of the typical (RMS) row norm are measured against that floor instead
    (a row that is zero in exact arithmetic carries rounding noise of the size of
    the terms that cancel in it);
  * per element: max |err| <= 25 x bar x RMS.
"""
import math
import sys

import numpy as np
import pytest
import torch

import bla_inputs as bi
import oracle

pytestmark = pytest.mark.gpu

TOL = {torch.float32: 1e-4, torch.bfloat16: 2e-2}


def _bla():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    import paper_2606_09862_amd as bla
    bla.lib()  # raises if the library is not built
    return bla


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def relerr(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def row_tolerance(tol):
    """Bar on the worst row's relative error for a rel-L2 bar `tol`."""
    return 10 * tol if tol <= 1e-4 else 2.5 * tol


def worst_row_error(got, ref):
    """(max over rows of ||got_r - ref_r|| / max(||ref_r||, floor), index of that row); a row
    is the last axis (one token's output, one mode's state row)."""
    d = ref.shape[-1] if ref.ndim else 1
    g = got.reshape(-1, d)
    r = ref.reshape(-1, d)
    rn = np.linalg.norm(r, axis=1)
    en = np.linalg.norm(g - r, axis=1)
    floor = 0.1 * math.sqrt(float(np.mean(rn ** 2))) if rn.size else 0.0
    rel = en / np.maximum(rn, max(floor, 1e-300))
    i = int(np.argmax(rel)) if rel.size else 0
    return (float(rel[i]) if rel.size else 0.0), i


def assert_close(got, ref, tol, what, row_tol=None):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    e = relerr(got, ref)
    rms = math.sqrt(float(np.mean(ref ** 2))) if ref.size else 0.0
    emax = float(np.max(np.abs(got - ref))) if ref.size else 0.0
    row_tol = row_tolerance(tol) if row_tol is None else row_tol
    er, ir = worst_row_error(got, ref)
    _say(f"  {what}: rel-L2 {e:.3e} (bar {tol:.0e}), worst row {er:.3e} at row {ir} (bar {row_tol:.1e}), "
         f"max-abs {emax:.3e}, rms {rms:.3e}")
    assert e <= tol, f"{what}: rel-L2 {e:.3e} > {tol:.0e}"
    assert er <= row_tol, f"{what}: row {ir} relative error {er:.3e} > {row_tol:.1e}"
    assert emax <= 25 * tol * max(rms, 1e-30), f"{what}: max-abs {emax:.3e}"


def to_dev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to("cuda").to(dtype)


def run_case(q, k, v, T, M, S, dtype, t0=0, sk=None, sv=None, literal=False, label="", chunk=0):
    """q,k,v float32 numpy holding dtype-representable values; returns errors dict."""
    bla = _bla()
    _say(f"case {label}: shape {q.shape} M={M} S={S} T={list(T)} t0={t0} dtype={dtype} chunk={chunk}")
    tq, tk, tv = (to_dev(x, dtype) for x in (q, k, v))
    tsk = None if sk is None else torch.from_numpy(np.ascontiguousarray(sk, np.float32)).cuda()
    tsv = None if sv is None else torch.from_numpy(np.ascontiguousarray(sv, np.float32)).cuda()
    o, ok, ov = bla.forward(tq, tk, tv, T, M, S, t0=t0, state_k=tsk, state_v=tsv, chunk=chunk)
    torch.cuda.synchronize()
    ref_o, ref_k, ref_v = oracle.forward(q, k, v, T, M, S, t0=t0,
                                         state_k=None if sk is None else np.asarray(sk, np.float64),
                                         state_v=None if sv is None else np.asarray(sv, np.float64),
                                         literal=literal)
    tol = TOL[dtype]
    assert_close(o.float().cpu().numpy(), ref_o, tol, "O")
    assert_close(ok.cpu().numpy(), ref_k, tol, "state_k")
    assert_close(ov.cpu().numpy(), ref_v, tol, "state_v")
    return o, ok, ov


def gauss(seed, B, H, L, d, dtype):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(3):
        x = (rng.standard_normal((B, H, L, d)) / math.sqrt(d)).astype(np.float32)
        out.append(bi.round_bf16(x) if dtype == torch.bfloat16 else x)
    return out


# ------------------------------------------------------------------ the tiny workload (id 1)
def test_workload1_tiny_fp32():
    w = bi.WORKLOADS[1]
    q, k, v = bi.generate(1)
    run_case(q, k, v, bi.periods(w.M, w.H), w.M, w.S, torch.float32, literal=True, label="workload 1")


# ------------------------------------------------------------------ small shapes, ragged, edge cases
def rejected_chunk(B, H, L, d, M, S, dtype, chunk):
    """float32 tiles of 128-token chunks at d = 64 exceed the LDS: the library rejects the
    shape (BLA_ERR_UNSUPPORTED) before any launch."""
    if not (dtype == torch.float32 and chunk == 128 and d == 64):
        return False
    bla = _bla()
    assert bla.supported(bla.make_params(B, H, L, d, M, S, dtype, chunk=chunk)) == 2
    return True


CHUNKS = [16, 32, 64, 128]   # Alg. 3's chunk length (64 is the default)


@pytest.mark.parametrize("chunk", CHUNKS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (2, 3, 100, 32, 16, 16, (31.0, 62.0, 40.5)),     # ragged last chunk, non-integer T
    (1, 2, 64, 64, 8, 15, (15.0, 30.0)),              # exactly one chunk, S = 2M-1
    (2, 2, 7, 32, 5, 9, (9.0, 9.0)),                  # L < chunk, T = S = 2M-1 (SWA limit)
    (1, 2, 200, 64, 24, 40, (47.0, 94.0)),            # padded modes (24 -> 32) and slots (40 -> 64)
    (3, 1, 130, 32, 32, 63, (3.0,)),                  # T below 2M-1 is clamped
    (1, 1, 1, 64, 4, 4, (7.0,)),                      # a single token
])
def test_small_shapes(dtype, B, H, L, d, M, S, T, chunk):
    if rejected_chunk(B, H, L, d, M, S, dtype, chunk):
        return
    q, k, v = gauss(L * 7 + M, B, H, L, d, dtype)
    run_case(q, k, v, T, M, S, dtype, label=f"small {B}x{H}x{L}x{d}", chunk=chunk)


@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (1, 2, 300, 128, 20, 30, (41.0, 82.5)),           # d = 128: one sequence unit per workgroup
    (1, 1, 200, 32, 100, 120, (199.0,)),              # M = 128 padded: two owned mode tiles per wave
    (1, 1, 64 * 8 + 20, 64, 64, 64, (127.0,)),        # 9 segments: an idle partner unit in the last workgroup
    (2, 1, 64 * 30 + 33, 64, 64, 64, (127.0, 254.0)), # several chunks per segment, ragged last segment
])
def test_bf16_unit_layouts(B, H, L, d, M, S, T):
    """Layouts of the bf16 kernels: one or two units per workgroup, one or two owned mode
    tiles per wave, idle units, segments of several chunks."""
    q, k, v = gauss(L * 3 + d + M, B, H, L, d, torch.bfloat16)
    run_case(q, k, v, T[:H], M, S, torch.bfloat16, label=f"layout {B}x{H}x{L}x{d} M={M}")


@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (8, 4, 64 * 8 + 5, 32, 16, 16, (31.0, 62.0, 31.0, 62.0)),     # d = 32: one 32-column summary slice
    (4, 4, 64 * 6 + 17, 128, 32, 32, (63.0, 126.0, 63.0, 126.0)),  # d = 128: four slices, one unit per workgroup
    (8, 4, 64 * 5 + 40, 64, 8, 15, (15.0, 30.0, 15.0, 30.0)),     # 16 modes: two-wave summary workgroups
])
def test_pair_summary_layouts(B, H, L, d, M, S, T):
    """bf16 sequences numerous enough for the pair kernels (at least 16 units per workgroup slot)
    yet split into several segments on 256 compute units, so that the summary kernel runs its
    32-column slices (one per d/32), its mode-tile split and its XCD-grouped indexing at
    d = 32, 128 and 16 modes (the LM-layer and recall workloads cover d = 64)."""
    q, k, v = gauss(L + 3 * d + M, B, H, L, d, torch.bfloat16)
    run_case(q, k, v, T[:H], M, S, torch.bfloat16, label=f"pair summaries {B}x{H}x{L}x{d} M={M}")


@pytest.mark.parametrize("B,H,L,d,M,S,T", [
    (1, 2, 64 * 11 + 9, 128, 128, 128, (255.0, 510.0)),  # d = M = 128: eight waves, one mode tile each
    (2, 1, 300, 128, 100, 256, (199.0,)),                 # modes padded 100 -> 128, slots 256
    (1, 2, 64 * 6 + 23, 128, 128, 64, (127.0, 300.0)),     # 64 slots: 32 per wave of a token tile
])
def test_wide_state_eight_waves(B, H, L, d, M, S, T):
    """bf16, d = M = 128 runs eight waves per workgroup.  With 64 or 128 slots the two waves
    of a token tile split the chain (slot halves, whose softmax statistics are combined; mode
    halves; head-dim halves), the upper slot half fully masked at the first positions; with 256
    slots the chain runs on the first four waves.  float32 I/O at this size does not fit the
    LDS tiles and is rejected."""
    q, k, v = gauss(L + 5 * M + S, B, H, L, d, torch.bfloat16)
    run_case(q, k, v, T[:H], M, S, torch.bfloat16, label=f"eight waves {B}x{H}x{L}x{d} M={M} S={S}")
    bla = _bla()
    assert bla.supported(bla.make_params(B, H, L, d, M, S, torch.float32)) != 0


@pytest.mark.parametrize("S", [128, 64])
def test_wide_state_in_offset_segments(S):
    """d = M = 128 (eight waves, the column-split chain and its fragment-ordered tables) with
    input states, t0 > 0 and a ragged tail, cut into many segments: the carries from the block
    summaries and the scan enter every segment but the first."""
    B, H, L, d, M, T = 1, 2, 64 * 13 + 29, 128, 128, (300.0, 511.0)
    q, k, v = gauss(31 + S, B, H, L, d, torch.bfloat16)
    rng = np.random.default_rng(32)
    sk = rng.standard_normal((B, H, 2, M, d)).astype(np.float32) * 0.1
    sv = rng.standard_normal((B, H, 2, M, d)).astype(np.float32) * 0.1
    sk[:, :, 1, 0] = 0.0
    sv[:, :, 1, 0] = 0.0
    run_case(q, k, v, T, M, S, torch.bfloat16, t0=777, sk=sk, sv=sv, label=f"wide continuation S={S}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_state_in_and_offset(dtype):
    """Continue a sequence: state_in from the oracle, t0 > 0 (start mask at absolute positions)."""
    B, H, L, d, M, S, T = 2, 2, 150, 64, 16, 20, (31.0, 77.25)
    q, k, v = gauss(11, B, H, 2 * L, d, dtype)
    _, sk, sv = oracle.forward(q[:, :, :L], k[:, :, :L], v[:, :, :L], T, M, S)
    run_case(q[:, :, L:], k[:, :, L:], v[:, :, L:], T, M, S, dtype, t0=L, sk=sk, sv=sv,
             label="continuation")


@pytest.mark.parametrize("chunk", CHUNKS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_many_segments(dtype, chunk):
    """Few sequences and many chunks: the sequence is split into segments whose entering
    states come from per-block summaries and the scan; ragged tail included."""
    B, H, L, d, M, S, T = 1, 2, 64 * 37 + 5, 32, 16, 31, (31.0, 62.0)
    q, k, v = gauss(12, B, H, L, d, dtype)
    run_case(q, k, v, T, M, S, dtype, label="segments", chunk=chunk)


@pytest.mark.parametrize("chunk", CHUNKS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_segments_with_state_in(dtype, chunk):
    B, H, L, d, M, S, T = 1, 1, 64 * 20 + 7, 64, 16, 16, (50.0,)
    if rejected_chunk(B, H, L, d, M, S, dtype, chunk):
        return
    q, k, v = gauss(13, B, H, L, d, dtype)
    rng = np.random.default_rng(14)
    sk = rng.standard_normal((B, H, 2, M, d)).astype(np.float32)
    sv = rng.standard_normal((B, H, 2, M, d)).astype(np.float32)
    sk[:, :, 1, 0] = 0.0
    sv[:, :, 1, 0] = 0.0
    run_case(q, k, v, T, M, S, dtype, t0=1000, sk=sk, sv=sv, label="segments+state_in", chunk=chunk)


@pytest.mark.parametrize("chunk", [16, 32, 128])
def test_chunk_lengths_lm_shape(chunk):
    """The LM-layer head shape (d = M = S = 64, bf16, periods 127 and 254) with the other
    chunk lengths, against the oracle and against the default 64-token chunks."""
    bla = _bla()
    B, H, L, d, M, S, T = 2, 2, 64 * 12 + 29, 64, 64, 64, (127.0, 254.0)
    q, k, v = gauss(17 + chunk, B, H, L, d, torch.bfloat16)
    o, sk, sv = run_case(q, k, v, T, M, S, torch.bfloat16, label=f"LM shape chunk {chunk}", chunk=chunk)
    o64, sk64, sv64 = bla.forward(*(to_dev(x, torch.bfloat16) for x in (q, k, v)), T, M, S)
    torch.cuda.synchronize()
    assert_close(o.float().cpu().numpy(), o64.float().cpu().numpy(), 2e-2, "O against chunk 64")


def test_empty_and_degenerate():
    bla = _bla()
    M, d = 8, 32
    # L = 0 passes the state through
    sk = torch.randn(2, 3, 2, M, d, device="cuda")
    sv = torch.randn(2, 3, 2, M, d, device="cuda")
    z = torch.zeros(2, 3, 0, d, device="cuda")
    o, ok, ov = bla.forward(z, z, z, [15.0] * 3, M, 15, state_k=sk, state_v=sv)
    torch.cuda.synchronize()
    assert o.shape == (2, 3, 0, d)
    assert torch.equal(ok, sk) and torch.equal(ov, sv)
    # L = 0 without a state gives zeros
    _, ok, ov = bla.forward(z, z, z, [15.0] * 3, M, 15)
    torch.cuda.synchronize()
    assert torch.count_nonzero(ok) == 0 and torch.count_nonzero(ov) == 0
    # B = 0: nothing to do
    e = torch.zeros(0, 3, 10, d, device="cuda")
    o, _, _ = bla.forward(e, e, e, [15.0] * 3, M, 15)
    assert o.shape == (0, 3, 10, d)


def test_deterministic():
    """No atomics in any reduction: two runs give bitwise-identical results."""
    bla = _bla()
    q, k, v = gauss(15, 2, 4, 64 * 9 + 3, 64, torch.bfloat16)
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    a = bla.forward(tq, tk, tv, [63.0, 126.0] * 2, 32, 32)
    b = bla.forward(tq, tk, tv, [63.0, 126.0] * 2, 32, 32)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)


# ------------------------------------------------------------------ the full workloads
def test_workload2_recall_bf16():
    w = bi.WORKLOADS[2]
    q, k, v = bi.generate(2)
    run_case(q, k, v, bi.periods(w.M, w.H), w.M, w.S, torch.bfloat16, label="workload 2")


def test_workload3_lm_layer_sampled_rows():
    """Full LM-layer workload on the GPU (the benchmark's launch configuration); the oracle
    checks every head and every token of three batch rows: first, middle and last.  The
    sequences run as several segments (their entering states combined from the preceding
    segments' summaries); the tokens around every quarter of the sequence and every chunk
    start are also checked on their own."""
    bla = _bla()
    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    q, k, v = bi.generate(3)
    _say(f"workload 3 full size {q.shape}")
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    o, sk, sv = bla.forward(tq, tk, tv, T, w.M, w.S)
    torch.cuda.synchronize()
    starts = sorted({t for j in range(4) for t in (j * w.L // 4 - 1, j * w.L // 4, j * w.L // 4 + 1) if t >= 0} |
                    set(range(0, w.L, w.chunk)))
    for b in (0, w.B // 2, w.B - 1):
        ref_o, ref_k, ref_v = oracle.forward(q[b:b + 1], k[b:b + 1], v[b:b + 1], T, w.M, w.S)
        got = o[b:b + 1].float().cpu().numpy()
        assert_close(got, ref_o, 2e-2, f"O row {b}")
        assert_close(got[:, :, starts], ref_o[:, :, starts], 2e-2, f"O row {b}, segment and chunk starts")
        assert_close(sk[b:b + 1].cpu().numpy(), ref_k, 2e-2, f"state_k row {b}")
        assert_close(sv[b:b + 1].cpu().numpy(), ref_v, 2e-2, f"state_v row {b}")


def test_workload4_long_context():
    """B=1, H=16, L=65536, d=M=S=128: every head against the oracle (threads over heads)."""
    bla = _bla()
    w = bi.WORKLOADS[4]
    T = bi.periods(w.M, w.H)
    q, k, v = bi.generate(4)
    _say(f"workload 4 full size {q.shape}")
    tq, tk, tv = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    o, sk, sv = bla.forward(tq, tk, tv, T, w.M, w.S)
    torch.cuda.synchronize()
    ref_o, ref_k, ref_v = oracle.forward(q, k, v, T, w.M, w.S)
    assert_close(o.float().cpu().numpy(), ref_o, 2e-2, "O")
    assert_close(sk.cpu().numpy(), ref_k, 2e-2, "state_k")
    assert_close(sv.cpu().numpy(), ref_v, 2e-2, "state_v")
