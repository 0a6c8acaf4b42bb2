"""Benchmark of the BLA forward operator on one MI355X.

Workload: the LM-layer shape (B=8, H=16, L=4096, d=64, M=S=64, chunk 64, bf16 inputs,
fp32 state), periods T_h = (1 + h mod 2)(2M-1), synthetic seeded inputs resident in
HBM.  One step = one bla_forward call (segment summaries and the chunked forward kernel;
the phase and slot tables are built by the first call and kept in the caller's workspace,
reuse_tables = 1, as Alg. 1 / Alg. 3 take A and B as precomputed inputs) producing O and
the final states.

Prints ONE JSON line: tokens/s (B*L per step); `roofline` of the dominant kernel (chunked
forward: algorithmic bytes / its average duration from HIP events recorded between the
library's launches on the same stream) and `operator_roofline` of the whole step
(algorithmic bytes / step time, HBM traffic of every kernel of the step); the float64 CPU
oracle timed on the host on the same workload; the recall and long-context workloads
(B=64 H=4 L=512 d=64 M=S=32, and B=1 H=16 L=65536 d=M=S=128) measured the same way with
their own rooflines and oracle baselines; and the decode step (bla_step) on the decode
workload (B=512, H=16, d=M=S=64 after a 2048-token prefill).

The headline is the operator with slots at lags behind the current token (Sec. 3.1).
The anchored-slot form (Sec. 3.3, Alg. 1/3; phase_anchor = 1) and the state-decay form
(Sec. 3.4, bla_decay_forward) are measured the same way on the same workload and reported
under "anchored" and "decay", each with its own oracle timed on the host.  --form
anchored / --form decay makes that form the only forward that runs (for profiling it
alone); --workload recall / long_context runs only that workload's forward.  The backward
pass (bla_backward: dq, dk, dv from dO on the same workload) is measured under "backward"
with the matrix-core roofline of its reverse-walk kernel and the oracle's backward timed on
a sample of the sequences; --form backward runs only it.  The whole layer
(bla_layer_forward: projections, operator, output projection) is measured under "layer" at
the recall workload's shape.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16 matrix cores
METRIC = "BLA forward tokens/sec at L=4096 (1 MI355X) + % of MFMA/HBM roofline"


def forward_flops_per_token_head(C, d, M, S):
    """Algorithmic flops of the chunked form per (token, head); the C x C terms count their
    causal half with the diagonal: 2(C+1)d + 4(C+1)M + 8MS + 16Md."""
    return 2 * (C + 1) * d + 4 * (C + 1) * M + 8 * M * S + 16 * M * d


def decay_flops_per_token_head(d, S, sub=16):
    """Algorithmic flops of the decay form's sub-block contractions per (token, head):
    K~ Q^T and the readout against V~ (2 S d each), the state update of K~ and V~ (4 S d),
    and the causal sub-block terms Bq^T G^T, tril(Bq P^T), G and V H (about S + d each per
    token pair, (sub + 1) / 2 pairs)."""
    return 8 * S * d + (sub + 1) * (2 * S + 2 * d)


def backward_flops_per_token_head(C, d, M, S):
    """Algorithmic flops of the backward's reverse walk per (token, head), causal halves of the
    C x C terms with the diagonal: the Gram tiles Q K^T, dO V^T and the tril(H) products for dq,
    dk, dv (5(C+1)d); G conj(E), Gd conj(E), H_q, H_v (8(C+1)M); scores, dP, W'' and Wq''
    (16MS); Q Z'_k^T, dO Z'_v^T, Re(Wq'' Z'_k), the two adjoint terms of dk and dv, the state
    rebuilt by subtraction and the adjoint update (36Md)."""
    return 5 * (C + 1) * d + 8 * (C + 1) * M + 16 * M * S + 36 * M * d


def forward_bytes(B, H, L, d, M, io_bytes):
    """q, k, v read + o written (io dtype) + final fp32 states written."""
    return B * H * L * d * io_bytes * 4 + B * H * 2 * (2 * M * d * 4)


KERNEL_SOURCES = {
    "rotating": ("bla_device.h", "bla_forward.h", "bla_forward_pair.h", "bla_plan.h"),
    "anchored": ("bla_device.h", "bla_forward.h", "bla_forward_pair.h", "bla_plan.h"),
    "decay": ("bla_device.h", "bla_plan.h", "bla_decay.hip"),
    "backward": ("bla_device.h", "bla_forward.h", "bla_forward_pair.h", "bla_plan.h", "bla_backward.h",
                 "bla_backward_bf16.h"),
    "step": ("bla_device.h", "bla_plan.h", "bla_step.hip"),
}


def kernel_sources_digest(form):
    """Digest of the sources the form's forward kernels are built from; a committed traffic
    figure is used only while it matches."""
    csrc = os.path.join(ROOT, "paper_2606_09862_amd", "csrc")
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[form]:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(path, digest, key="hbm_bytes_per_launch"):
    """HBM bytes from a committed rocprofv3 --pmc summary: `hbm_bytes_per_launch` of the
    dominant kernel, or `hbm_bytes_per_step` of every kernel of a step; None if the file or
    the key is absent or the figures were taken on a different kernel source."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_sources_sha") != digest:
        return None
    try:
        return float(vals[key])
    except (KeyError, ValueError):
        return None


def host_cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def oracle_threads(n_seq):
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    return max(1, min(threads, n_seq))


class Hip:
    """Minimal HIP event API through the runtime library (timing plumbing only)."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")
        self.lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.lib.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def event(self):
        e = ctypes.c_void_p()
        assert self.lib.hipEventCreate(ctypes.byref(e)) == 0
        return e

    def record(self, e, stream):
        assert self.lib.hipEventRecord(e, stream) == 0

    def elapsed_ms(self, a, b):
        assert self.lib.hipEventSynchronize(b) == 0
        ms = ctypes.c_float()
        assert self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) == 0
        return ms.value


WORKLOAD_IDS = {"recall": 2, "lm_layer": 3, "long_context": 4}
PROFILE_STEM = {  # committed rocprofv3 summaries of each measured forward
    ("rotating", 3): "forward_pair_kernel_lm_layer",
    ("anchored", 3): "forward_pair_kernel_lm_layer_anchored",
    ("decay", 3): "decay_forward_kernel_lm_layer",
    ("rotating", 2): "forward_pair_kernel_recall",
    ("rotating", 4): "forward_kernel_long_context",
}
KERNEL_NAME = {
    ("rotating", 3): "forward_pair_kernel<64,64,64,false>",
    ("anchored", 3): "forward_pair_kernel<64,64,64,true>",
    ("decay", 3): "decay_forward_kernel<bf16,64,64,false>",
    ("rotating", 2): "forward_pair_kernel<64,32,32,false>",
    ("rotating", 4): "forward_kernel<bf16,128,128,128,false>",
}


def bench_forward(args, hip, inputs, form, cid=3):
    """One workload's forward: whole steps timed back to back, then the same steps with events
    between the library's launches for the per-phase durations."""
    import numpy as np
    import torch

    import bla_inputs as bi
    import paper_2606_09862_amd as bla

    w = bi.WORKLOADS[cid]
    T = bi.periods(w.M, w.H)
    q, k, v = inputs
    dev = torch.device("cuda:0")
    tq, tk, tv = (torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v))
    decay = form == "decay"
    p = bla.make_params(w.B, w.H, w.L, w.d, w.M, w.S, torch.bfloat16, phase_anchor=form == "anchored",
                        reuse_tables=True)
    ws_bytes = bla.decay_workspace_size(p) if decay else bla.workspace_size(p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    o = torch.empty_like(tq)
    state_shape = (w.B, w.H, w.S, w.d) if decay else (w.B, w.H, 2, w.M, w.d)
    sk = torch.empty(state_shape, dtype=torch.float32, device=dev)
    sv = torch.empty_like(sk)
    stream = torch.cuda.current_stream(dev)
    sptr = ctypes.c_void_p(stream.cuda_stream)
    Tarr = (ctypes.c_double * w.H)(*T)
    L = bla.lib()
    fn = L.bla_decay_forward_timed if decay else L.bla_forward_timed
    fn.argtypes = [ctypes.POINTER(bla.Params), ctypes.POINTER(ctypes.c_double)] + \
        [ctypes.c_void_p] * 9 + [ctypes.c_size_t, ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    fn.restype = ctypes.c_int
    ptrs = [ctypes.c_void_p(t.data_ptr()) if t is not None else None
            for t in (tq, tk, tv, None, None, o, sk, sv, ws)]

    def call(evs):
        arr = None if evs is None else (ctypes.c_void_p * 5)(*[e.value for e in evs])
        st = fn(ctypes.byref(p), Tarr, *ptrs, ws.numel(), sptr, arr)
        if st != 0:
            raise RuntimeError(f"bla_forward failed: {bla.STATUS.get(st, st)}")

    for _ in range(args.warmup):
        call(None)
    # whole steps, nothing recorded between the launches of a step
    t_start, t_stop = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(t_start, sptr)
    for i in range(args.steps):
        call(None)
    hip.record(t_stop, sptr)
    torch.cuda.synchronize(dev)
    ms = hip.elapsed_ms(t_start, t_stop) / args.steps
    # the same steps again with events between the library's launches: the forward kernel's
    # duration for its roofline.  Events 1-3 bracket the segment summaries (and, on the
    # one-unit kernels, the scan of the summaries into carried states), reported as one phase.
    evs = [[hip.event() for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    for i in range(args.steps):
        call(evs[i])
    torch.cuda.synchronize(dev)
    # the tables are recorded by the first call, so the first span launches nothing: its
    # figure is the cost of the events themselves
    spans = {"tables_cached_event_gap": (0, 1), "segment_summaries": (1, 3), "forward": (3, 4)}
    if decay:
        spans = {"tables_and_schedule": (0, 1), "summaries_and_scan": (1, 3), "forward": (3, 4)}
    phase_ms = {ph: float(np.mean([hip.elapsed_ms(e[a], e[b]) for e in evs])) for ph, (a, b) in spans.items()}
    # per-call durations of the same pass (first to last event of a call): their median
    call_ms = float(np.median([hip.elapsed_ms(e[0], e[4]) for e in evs]))
    tokens = w.B * w.L
    if decay:
        flops = decay_flops_per_token_head(w.d, w.S) * w.B * w.H * w.L
        nbytes = w.B * w.H * w.L * w.d * 2 * 4 + w.B * w.H * 2 * w.S * w.d * 4
    else:
        flops = forward_flops_per_token_head(w.chunk, w.d, w.M, w.S) * w.B * w.H * w.L
        nbytes = forward_bytes(w.B, w.H, w.L, w.d, w.M, 2)
    t_fwd = phase_ms["forward"] * 1e-3
    digest = kernel_sources_digest(form)
    stem = PROFILE_STEM.get((form, cid))
    tpath = os.path.join(ROOT, "profiles", f"{stem}_traffic.txt") if stem else ""
    t_mfma, t_hbm = flops / (BF16_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)
    if t_mfma > t_hbm:   # a contraction-bound workload (the long-context shape)
        achieved = flops / t_fwd / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                    "traffic": read_traffic(tpath, digest) if stem else None}
        op_achieved = flops / (ms * 1e-3) / 1e12
        operator = {"bound": "mfma", "achieved": round(op_achieved, 1), "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(op_achieved / BF16_PEAK_TFLOPS, 4)}
    else:
        achieved = nbytes / t_fwd / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": read_traffic(tpath, digest) if stem else None}
        op_achieved = nbytes / (ms * 1e-3) / 1e9
        operator = {"bound": "hbm", "achieved": round(op_achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(op_achieved / HBM_PEAK_GBS, 4)}
    operator["traffic"] = read_traffic(tpath, digest, "hbm_bytes_per_step") if stem else None
    operator["scope"] = "the whole step (every kernel of one call): algorithmic bytes or flops / ms_per_step"
    roofline["scope"] = f"{KERNEL_NAME.get((form, cid), 'forward kernel')} alone: algorithmic bytes or flops / " \
                        "its average duration from events between the launches"
    extra = {
        "kernel": KERNEL_NAME.get((form, cid)),
        "algorithmic_bytes_per_launch": nbytes,
        "algorithmic_flops_per_launch": flops,
        "forward_kernel_us": round(phase_ms["forward"] * 1e3, 2),
        "forward_kernel_mfma_tflops": round(flops / t_fwd / 1e12, 1),
        "forward_kernel_mfma_frac": round(flops / t_fwd / 1e12 / BF16_PEAK_TFLOPS, 4),
        "forward_kernel_hbm_gbs": round(nbytes / t_fwd / 1e9, 1),
        "phase_us": {k2: round(v2 * 1e3, 2) for k2, v2 in phase_ms.items()},
        "ideal_us": round(max(t_mfma, t_hbm) * 1e6, 2),
        "median_call_us_with_events": round(call_ms * 1e3, 2),
        "kernel_sources_sha": digest,
    }
    del tq, tk, tv, o, sk, sv, ws
    return w, T, ms, tokens / (ms * 1e-3), roofline, operator, extra


def bench_backward(args, hip, inputs):
    """bla_backward on the LM-layer workload: dq, dk, dv and the input-state gradients from
    q, k, v and dO (all resident in HBM).  One step = one bla_backward call (tables, forward
    summaries, adjoint summaries, reverse walk)."""
    import numpy as np
    import torch

    import bla_inputs as bi
    import paper_2606_09862_amd as bla

    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    dev = torch.device("cuda:0")
    q, k, v = inputs
    g = bi.generate_grad(3)
    tq, tk, tv, tg = (torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v, g))
    p = bla.make_params(w.B, w.H, w.L, w.d, w.M, w.S, torch.bfloat16, reuse_tables=True)
    ws = torch.empty(bla.backward_workspace_size(p), dtype=torch.uint8, device=dev)
    dq, dk, dv = torch.empty_like(tq), torch.empty_like(tk), torch.empty_like(tv)
    gsk = torch.empty((w.B, w.H, 2, w.M, w.d), dtype=torch.float32, device=dev)
    gsv = torch.empty_like(gsk)
    sptr = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    Tarr = (ctypes.c_double * w.H)(*T)
    ptrs = [ctypes.c_void_p(t.data_ptr()) if t is not None else None
            for t in (tq, tk, tv, tg, None, None, None, None, dq, dk, dv, gsk, gsv, ws)]
    fn = bla.lib().bla_backward_timed

    def call(evs):
        arr = None if evs is None else (ctypes.c_void_p * 5)(*[e.value for e in evs])
        st = fn(ctypes.byref(p), Tarr, *ptrs, ws.numel(), sptr, arr)
        if st != 0:
            raise RuntimeError(f"bla_backward failed: {bla.STATUS.get(st, st)}")

    for _ in range(args.warmup):
        call(None)
    t0, t1 = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(t0, sptr)
    for _ in range(args.steps):
        call(None)
    hip.record(t1, sptr)
    torch.cuda.synchronize(dev)
    ms = hip.elapsed_ms(t0, t1) / args.steps
    evs = [[hip.event() for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    for i in range(args.steps):
        call(evs[i])
    torch.cuda.synchronize(dev)
    # first span: tables recorded by the first call, nothing launched (the events' own cost)
    phases = ["tables_cached_event_gap", "forward_summaries", "adjoint_summaries", "reverse_walk"]
    phase_ms = {ph: float(np.mean([hip.elapsed_ms(e[j], e[j + 1]) for e in evs])) for j, ph in enumerate(phases)}
    flops = backward_flops_per_token_head(w.chunk, w.d, w.M, w.S) * w.B * w.H * w.L
    nbytes = w.B * w.H * w.L * w.d * 2 * 7 + w.B * w.H * 2 * (2 * w.M * w.d * 4)
    t_walk = phase_ms["reverse_walk"] * 1e-3
    tflops = flops / t_walk / 1e12
    digest = kernel_sources_digest("backward")
    traffic = read_traffic(os.path.join(ROOT, "profiles", "bwd_kernel_lm_layer_traffic.txt"), digest)
    roofline = {"bound": "mfma", "achieved": round(tflops, 1), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tflops / BF16_PEAK_TFLOPS, 4), "traffic": traffic}
    t_ideal = max(flops / (BF16_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9))
    detail = {
        "kernel": "bwd16_kernel<64,64,64,false>",
        "algorithmic_flops_per_launch": flops,
        "algorithmic_bytes_per_launch": nbytes,
        "reverse_walk_us": round(phase_ms["reverse_walk"] * 1e3, 2),
        "reverse_walk_hbm_gbs": round(nbytes / t_walk / 1e9, 1),
        "phase_us": {k2: round(v2 * 1e3, 2) for k2, v2 in phase_ms.items()},
        "operator_roofline_frac": round(t_ideal / (ms * 1e-3), 4),
        "kernel_sources_sha": digest,
    }
    del tq, tk, tv, tg, dq, dk, dv, gsk, gsv, ws
    return ms, w.B * w.L / (ms * 1e-3), roofline, detail, g


def cpu_baseline_backward(w, T, inputs, g, nseq=16):
    """The oracle's backward (token by token, per-token states kept) on a bounded sample: the
    first nseq of the workload's sequences, one per host thread."""
    import numpy as np

    import oracle

    q, k, v = inputs
    H = w.H
    rows = [(i // H, i % H) for i in range(nseq)]
    pick = lambda x: np.stack([x[b, h] for b, h in rows])[None]
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    threads = max(1, min(threads, nseq))
    t = time.perf_counter()
    oracle.backward(pick(q), pick(k), pick(v), pick(g), [T[h] for _, h in rows], w.M, w.S, nthreads=threads)
    dt = time.perf_counter() - t
    return {"value": round(nseq * w.L / H / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{nseq} of the LM-layer workload's {w.B * w.H} sequences (L={w.L}), float64 reverse pass "
                      f"through Alg. 2, one sequence per thread; {dt:.2f} s wall; tokens/s counts a token with "
                      f"all {H} heads, as the GPU figure does"}


def bench_layer(args, hip):
    """bla_layer_forward at the recall workload's shape (B=64, H=4, L=512, d=64, D=256, M=S=32):
    x [B, L, D] -> y [B, L, D] through the QKV projection, the operator and the output
    projection.  One step = one layer call."""
    import numpy as np
    import torch

    import bla_inputs as bi
    import paper_2606_09862_amd as bla

    w = bi.WORKLOADS[2]
    T = bi.periods(w.M, w.H)
    D = w.H * w.d
    dev = torch.device("cuda:0")
    x, wqkv, wo = bi.generate_layer(2)
    tx, tw, to = (torch.from_numpy(a).to(dev).to(torch.bfloat16) for a in (x, wqkv, wo))
    p = bla.make_params(w.B, w.H, w.L, w.d, w.M, w.S, torch.bfloat16, reuse_tables=True)
    ws = torch.empty(bla.layer_workspace_size(p), dtype=torch.uint8, device=dev)
    y = torch.empty_like(tx)
    sk = torch.empty((w.B, w.H, 2, w.M, w.d), dtype=torch.float32, device=dev)
    sv = torch.empty_like(sk)
    sptr = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    Tarr = (ctypes.c_double * w.H)(*T)
    ptrs = [ctypes.c_void_p(t.data_ptr()) if t is not None else None for t in (tx, tw, to, None, None, y, sk, sv, ws)]
    fn = bla.lib().bla_layer_forward_timed

    def call(evs):
        arr = None if evs is None else (ctypes.c_void_p * 4)(*[e.value for e in evs])
        st = fn(ctypes.byref(p), Tarr, *ptrs, ws.numel(), sptr, arr)
        if st != 0:
            raise RuntimeError(f"bla_layer_forward failed: {bla.STATUS.get(st, st)}")

    for _ in range(args.warmup):
        call(None)
    e0, e1 = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(e0, sptr)
    for _ in range(args.steps):
        call(None)
    hip.record(e1, sptr)
    torch.cuda.synchronize(dev)
    ms = hip.elapsed_ms(e0, e1) / args.steps
    evs = [[hip.event() for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    for i in range(args.steps):
        call(evs[i])
    torch.cuda.synchronize(dev)
    phases = ["qkv_projection", "operator", "output_projection"]
    phase_us = {ph: round(float(np.mean([hip.elapsed_ms(e[j], e[j + 1]) for e in evs])) * 1e3, 2)
                for j, ph in enumerate(phases)}
    tokens = w.B * w.L
    gemm_flops = 8 * tokens * D * D
    op_flops = forward_flops_per_token_head(w.chunk, w.d, w.M, w.S) * w.B * w.H * w.L
    # the layer's own inputs and outputs: x, y, the weights and the final states
    nbytes = 2 * tokens * D * 2 + 4 * D * D * 2 + w.B * w.H * 2 * (2 * w.M * w.d * 4)
    t_ideal = max((gemm_flops + op_flops) / (BF16_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9))
    gemm_s = (phase_us["qkv_projection"] + phase_us["output_projection"]) * 1e-6
    out = {"workload": f"recall shape: B={w.B} H={w.H} L={w.L} d={w.d} (D={D}) M={w.M} S={w.S}, bf16",
           "value": round(tokens / (ms * 1e-3), 1), "unit": "tokens/s", "ms_per_step": round(ms, 5),
           "phase_us": phase_us, "flops_per_launch": gemm_flops + op_flops,
           "projection_tflops": round(gemm_flops / gemm_s / 1e12, 1),
           "layer_roofline_frac": round(t_ideal / (ms * 1e-3), 4)}
    if not args.no_cpu_baseline:
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
        t = time.perf_counter()
        oracle.layer_forward(x, wqkv, wo, T, w.H, w.M, w.S, nthreads=threads)
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": round(tokens / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
                               "sample": f"the whole layer workload: float64 numpy projections and the "
                                         f"token-by-token operator over {w.B * w.H} sequences; {dt:.2f} s wall"}
    del tx, tw, to, y, sk, sv, ws
    return out


def bench_decode(args, hip):
    import torch

    import bla_inputs as bi
    import paper_2606_09862_amd as bla

    w = bi.WORKLOADS[5]
    T = bi.periods(w.M, w.H)
    dev = torch.device("cuda:0")
    q, k, v = bi.generate_decode_device(dev)
    pq, pk, pv = (x[:, :, :w.L].contiguous() for x in (q, k, v))
    sq, sk_, sv_ = (x[:, :, w.L].contiguous() for x in (q, k, v))
    del q, k, v
    _, gk, gv = bla.forward(pq, pk, pv, T, w.M, w.S)
    del pq, pk, pv
    p = bla.make_params(w.B, w.H, 1, w.d, w.M, w.S, torch.bfloat16, t0=w.L)
    ws = torch.empty(bla.step_workspace_size(p), dtype=torch.uint8, device=dev)
    o = torch.empty_like(sq)
    for _ in range(args.warmup):
        bla.step(sq, sk_, sv_, T, w.M, w.S, gk, gv, t0=w.L, workspace=ws, out=o, reuse_tables=True)
    sptr = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    e0, e1 = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(e0, sptr)
    for i in range(args.steps):
        bla.step(sq, sk_, sv_, T, w.M, w.S, gk, gv, t0=w.L + i, workspace=ws, out=o, reuse_tables=True)
    hip.record(e1, sptr)
    torch.cuda.synchronize(dev)
    ms = hip.elapsed_ms(e0, e1) / args.steps
    state_bytes = w.B * w.H * 2 * (2 * w.M * w.d * 4)        # k and v states
    nbytes = 2 * state_bytes + w.B * w.H * w.d * 2 * 4       # read + write states, q,k,v,o
    gbs = nbytes / (ms * 1e-3) / 1e9
    # a plain device-to-device copy of the same state size (read + write), for the rate a
    # streaming read-modify-write can reach on this device
    src = torch.empty(state_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    c0, c1 = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(c0, sptr)
    for _ in range(args.steps):
        dst.copy_(src)
    hip.record(c1, sptr)
    torch.cuda.synchronize(dev)
    copy_gbs = 2 * state_bytes / (hip.elapsed_ms(c0, c1) / args.steps * 1e-3) / 1e9
    del src, dst
    traffic = read_traffic(os.path.join(ROOT, "profiles", "step_kernel_decode_traffic.txt"),
                           kernel_sources_digest("step"))
    return {"workload": "decode", "B": w.B, "H": w.H, "d": w.d, "M": w.M, "S": w.S, "position": w.L,
            "ms_per_step": round(ms, 4), "tokens_per_s": round(w.B / (ms * 1e-3), 1),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic},
            "device_copy_gbs": round(copy_gbs, 1), "frac_of_device_copy": round(gbs / copy_gbs, 4)}


def cpu_baseline_anchored(w, T, inputs):
    """Alg. 1 oracle (token by token, slot states as cumulative sums) on the whole workload."""
    import oracle

    q, k, v = inputs
    threads = oracle_threads(w.B * w.H)
    t = time.perf_counter()
    oracle.forward_anchored(q, k, v, T, w.M, w.S, nthreads=threads)
    dt = time.perf_counter() - t
    return {"value": round(w.B * w.L / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu": host_cpu_model(),
            "sample": f"the whole LM-layer workload ({w.B}x{w.H} sequences of {w.L} tokens), float64 "
                      f"Alg. 1 with slot states, OpenMP over (b,h); {dt:.2f} s wall"}


def cpu_baseline_decay(w, T, inputs):
    """Decay-form oracle (token by token, decayed slot states) on the whole workload."""
    import oracle

    q, k, v = inputs
    threads = oracle_threads(w.B * w.H)
    t = time.perf_counter()
    oracle.forward_decay(q, k, v, T, w.M, w.S, nthreads=threads)
    dt = time.perf_counter() - t
    return {"value": round(w.B * w.L / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu": host_cpu_model(),
            "sample": f"the whole LM-layer workload ({w.B}x{w.H} sequences of {w.L} tokens), float64 "
                      f"decayed slot recurrence, OpenMP over (b,h); {dt:.2f} s wall"}


def _oracle_rate(w, T, q, k, v, literal, L=None, nseq=None):
    """tokens/s (a token with all H heads) of the float64 oracle on the first `nseq` sequences
    (b, h in order) and the first L tokens of the workload; (rate, threads, seconds, what)."""
    import numpy as np

    import oracle

    L = w.L if L is None else L
    total = w.B * w.H
    nseq = total if nseq is None else min(nseq, total)
    if nseq == total:
        qs, ks, vs, Ts = q[:, :, :L], k[:, :, :L], v[:, :, :L], T
    else:
        rows = [(i // w.H, i % w.H) for i in range(nseq)]
        pick = lambda x: np.stack([x[b, h, :L] for b, h in rows])[None]
        qs, ks, vs, Ts = pick(q), pick(k), pick(v), [T[h] for _, h in rows]
    threads = oracle_threads(nseq)
    t = time.perf_counter()
    oracle.forward(qs, ks, vs, Ts, w.M, w.S, literal=literal, nthreads=threads)
    dt = time.perf_counter() - t
    what = (f"{'all' if nseq == total else nseq} of the {total} sequences" +
            ("" if L == w.L else f", first {L} of {w.L} tokens"))
    return nseq * L / w.H / dt, threads, dt, what


def cpu_baseline(w, T, inputs, literal_sample=None, factored_sample=None):
    """The float64 oracle (Alg. 2 token by token, OpenMP over (b,h)) on the host: the factored
    readout (the same sums regrouped) on the workload or `factored_sample` = (nseq, L), and the
    literal readout (slots materialised per token, as Eq. compressed writes them) on
    `literal_sample` = (nseq, L) (None: the whole workload)."""
    q, k, v = inputs
    fs = factored_sample or (None, None)
    rate, threads, dt, what = _oracle_rate(w, T, q, k, v, False, L=fs[1], nseq=fs[0])
    ls = literal_sample or (None, None)
    lrate, lthreads, ldt, lwhat = _oracle_rate(w, T, q, k, v, True, L=ls[1], nseq=ls[0])
    return {"value": round(rate, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu": host_cpu_model(),
            "sample": f"{what} ({w.name} workload, B={w.B} H={w.H} L={w.L} d={w.d} M={w.M} S={w.S}), float64 "
                      f"recurrence with the factored readout, OpenMP over (b,h); {dt:.2f} s wall; tokens/s "
                      f"counts a token with all {w.H} heads",
            "literal_readout": {"value": round(lrate, 1), "unit": "tokens/s", "cores": lthreads,
                                "sample": f"{lwhat}, slots materialised per token; {ldt:.2f} s wall"}}


def bench_workload(args, hip, name):
    """The rotating form's forward on the recall or long-context workload, with its oracle."""
    import bla_inputs as bi

    cid = WORKLOAD_IDS[name]
    inputs = bi.generate(cid)
    w, T, ms, value, roof, op, extra = bench_forward(args, hip, inputs, "rotating", cid)
    out = {"workload": name, "B": w.B, "H": w.H, "L": w.L, "d": w.d, "M": w.M, "S": w.S, "chunk": w.chunk,
           "value": round(value, 1), "unit": "tokens/s", "ms_per_step": round(ms, 5), "roofline": roof,
           "operator_roofline": op, "forward_detail": extra}
    if not args.no_cpu_baseline:
        if cid == 4:
            # a bounded sample: every head over the first 4096 tokens (the recurrence costs the
            # same per token at any position)
            out["cpu_baseline"] = cpu_baseline(w, T, inputs, literal_sample=(16, 256), factored_sample=(16, 4096))
        else:
            out["cpu_baseline"] = cpu_baseline(w, T, inputs)
    del inputs
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-anchored", action="store_true", help="skip the anchored-slot measurement")
    ap.add_argument("--no-decay", action="store_true", help="skip the state-decay measurement")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward measurement")
    ap.add_argument("--no-layer", action="store_true", help="skip the whole-layer measurement")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the recall and long-context workloads")
    ap.add_argument("--form", choices=("rotating", "anchored", "decay", "backward"), default="rotating",
                    help="the form of the headline forward; otherwise no other forward runs "
                         "(backward: only the backward pass runs, for profiling it alone)")
    ap.add_argument("--workload", choices=("recall", "long_context"), default=None,
                    help="run only this workload's forward (rotating slots), for profiling it alone")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="first run one plain device copy of this many bytes (reference kernel for "
                         "scaling the HBM byte counters of a rocprofv3 --pmc run)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the library has no multi-GPU path); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    hip = Hip()
    if args.copy_bytes > 0:
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    import bla_inputs as bi
    if args.workload is not None:
        out = bench_workload(args, hip, args.workload)
        print(json.dumps(out), flush=True)
        return
    inputs = bi.generate(3)
    if args.form == "backward":
        b_ms, b_value, b_roof, b_detail, _ = bench_backward(args, hip, inputs)
        print(json.dumps({"metric": "BLA backward tokens/sec at L=4096 (1 MI355X)", "value": round(b_value, 1),
                          "unit": "tokens/s", "ms_per_step": round(b_ms, 5), "roofline": b_roof,
                          "detail": b_detail}), flush=True)
        return
    head = args.form
    w, T, ms, value, roofline, operator, extra = bench_forward(args, hip, inputs, head)
    titles = {"anchored": "anchored slots (Sec. 3.3, Alg. 1/3), phase_anchor=1",
              "decay": "state decay (Sec. 3.4), bla_decay_forward, float32 slot states [B,H,S,d]"}
    baselines = {"anchored": cpu_baseline_anchored, "decay": cpu_baseline_decay}
    others = {}
    for form, skip in (("anchored", args.no_anchored), ("decay", args.no_decay)):
        if head != "rotating" or skip:
            others[form] = None
            continue
        _, _, f_ms, f_value, f_roof, f_op, f_extra = bench_forward(args, hip, inputs, form)
        others[form] = {"form": titles[form], "value": round(f_value, 1), "unit": "tokens/s",
                        "ms_per_step": round(f_ms, 5), "roofline": f_roof, "operator_roofline": f_op,
                        "forward_detail": f_extra,
                        "cpu_baseline": None if args.no_cpu_baseline else baselines[form](w, T, inputs)}
    backward = None
    if head == "rotating" and not args.no_backward:
        b_ms, b_value, b_roof, b_detail, g = bench_backward(args, hip, inputs)
        w3 = bi.WORKLOADS[3]
        backward = {"form": "gradients of the rotating form (Alg. 2): dq, dk, dv and the input-state gradients",
                    "value": round(b_value, 1), "unit": "tokens/s", "ms_per_step": round(b_ms, 5),
                    "roofline": b_roof, "detail": b_detail,
                    "cpu_baseline": None if args.no_cpu_baseline else
                    cpu_baseline_backward(w3, bi.periods(w3.M, w3.H), inputs, g)}
    layer = None if args.no_layer or head != "rotating" else bench_layer(args, hip)
    decode = None if args.no_decode or head != "rotating" else bench_decode(args, hip)
    cpu = None
    if not args.no_cpu_baseline:
        if head == "rotating":
            cpu = cpu_baseline(w, T, inputs, literal_sample=(16, 512))
        else:
            cpu = baselines[head](w, T, inputs)
    workloads = {}
    if head == "rotating" and not args.no_workloads:
        del inputs
        for name in ("recall", "long_context"):
            workloads[name] = bench_workload(args, hip, name)
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "lm_layer", "B": w.B, "H": w.H, "L": w.L, "d": w.d, "M": w.M, "S": w.S,
                   "chunk": w.chunk, "periods": "T_h=(1+h%2)(2M-1)", "state": "fp32",
                   "form": head},
        "roofline": roofline, "operator_roofline": operator, "cpu_baseline": cpu, "forward_detail": extra,
        "recall": workloads.get("recall"), "long_context": workloads.get("long_context"),
        "decode_step": decode, "anchored": others["anchored"], "decay": others["decay"], "backward": backward,
        "layer": layer,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
