"""Benchmark of the BLA forward operator on one MI355X.

Workload: the LM-layer shape (B=8, H=16, L=4096, d=64, M=S=64, chunk 64, bf16 inputs,
fp32 state), periods T_h = (1 + h mod 2)(2M-1), synthetic seeded inputs resident in
HBM.  One step = one bla_forward call (tables, block summaries, summary scan and the
chunked forward kernel) producing O and the final states.

Prints ONE JSON line: tokens/s (B*L per step), the roofline of the dominant kernel
(chunked forward: algorithmic bytes / its average duration from HIP events recorded
between the library's launches on the same stream), the float64 CPU oracle timed on
the host on the same workload, and the decode step (bla_step) on the decode
workload (B=512, H=16, d=M=S=64 after a 2048-token prefill).

The headline is the operator with slots at lags behind the current token (Sec. 3.1).
The anchored-slot form (Sec. 3.3, Alg. 1/3; phase_anchor = 1) is measured the same way
on the same workload and reported under "anchored", with its own oracle timed on a
bounded sample.  --form anchored makes the anchored form the only forward that runs
(for profiling it alone).
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


def forward_bytes(B, H, L, d, M, io_bytes):
    """q, k, v read + o written (io dtype) + final fp32 states written."""
    return B * H * L * d * io_bytes * 4 + B * H * 2 * (2 * M * d * 4)


def kernel_sources_digest():
    csrc = os.path.join(ROOT, "paper_2606_09862_amd", "csrc")
    h = hashlib.sha256()
    for name in ("bla_device.h", "bla_forward.h", "bla_forward_pair.h", "bla_plan.h"):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(path, digest):
    """HBM bytes per launch of the forward kernel from a committed rocprofv3 --pmc summary,
    or None if absent or taken on a different kernel source."""
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
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


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


def bench_forward(args, hip, inputs, anchor):
    import numpy as np
    import torch

    import bla_inputs as bi
    import paper_2606_09862_amd as bla

    w = bi.WORKLOADS[3]
    T = bi.periods(w.M, w.H)
    q, k, v = inputs
    dev = torch.device("cuda:0")
    tq, tk, tv = (torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (q, k, v))
    p = bla.make_params(w.B, w.H, w.L, w.d, w.M, w.S, torch.bfloat16, phase_anchor=anchor)
    ws = torch.empty(bla.workspace_size(p), dtype=torch.uint8, device=dev)
    o = torch.empty_like(tq)
    sk = torch.empty((w.B, w.H, 2, w.M, w.d), dtype=torch.float32, device=dev)
    sv = torch.empty_like(sk)
    stream = torch.cuda.current_stream(dev)
    sptr = ctypes.c_void_p(stream.cuda_stream)
    Tarr = (ctypes.c_double * w.H)(*T)
    L = bla.lib()
    L.bla_forward_timed.argtypes = [ctypes.POINTER(bla.Params), ctypes.POINTER(ctypes.c_double)] + \
        [ctypes.c_void_p] * 9 + [ctypes.c_size_t, ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]
    L.bla_forward_timed.restype = ctypes.c_int
    ptrs = [ctypes.c_void_p(t.data_ptr()) if t is not None else None
            for t in (tq, tk, tv, None, None, o, sk, sv, ws)]

    def call(evs):
        arr = None if evs is None else (ctypes.c_void_p * 5)(*[e.value for e in evs])
        st = L.bla_forward_timed(ctypes.byref(p), Tarr, *ptrs, ws.numel(), sptr, arr)
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
    # the same steps again with events between the phases (the forward kernel's duration
    # for the roofline; the intervals of the other phases include the event overhead)
    evs = [[hip.event() for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize(dev)
    for i in range(args.steps):
        call(evs[i])
    torch.cuda.synchronize(dev)
    phases = ["tables", "summary", "scan", "forward"]
    phase_ms = {ph: float(np.mean([hip.elapsed_ms(e[j], e[j + 1]) for e in evs]))
                for j, ph in enumerate(phases)}
    tokens = w.B * w.L
    flops = forward_flops_per_token_head(w.chunk, w.d, w.M, w.S) * w.B * w.H * w.L
    nbytes = forward_bytes(w.B, w.H, w.L, w.d, w.M, 2)
    t_fwd = phase_ms["forward"] * 1e-3
    achieved_gbs = nbytes / t_fwd / 1e9
    digest = kernel_sources_digest()
    tname = "forward_pair_kernel_lm_layer_anchored_traffic.txt" if anchor else "forward_pair_kernel_lm_layer_traffic.txt"
    traffic = read_traffic(os.path.join(ROOT, "profiles", tname), digest)
    roofline = {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": traffic}
    t_ideal = max(flops / (BF16_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9))
    extra = {
        "kernel": "forward_pair_kernel<64,64,64>",
        "algorithmic_bytes_per_launch": nbytes,
        "algorithmic_flops_per_launch": flops,
        "forward_kernel_us": round(phase_ms["forward"] * 1e3, 2),
        "forward_kernel_mfma_tflops": round(flops / t_fwd / 1e12, 1),
        "forward_kernel_mfma_frac": round(flops / t_fwd / 1e12 / BF16_PEAK_TFLOPS, 4),
        "phase_us": {k2: round(v2 * 1e3, 2) for k2, v2 in phase_ms.items()},
        "operator_roofline_frac": round(t_ideal / (ms * 1e-3), 4),
        "kernel_sources_sha": digest,
    }
    del tq, tk, tv, o, sk, sv, ws
    return w, T, ms, tokens / (ms * 1e-3), roofline, extra


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
        bla.step(sq, sk_, sv_, T, w.M, w.S, gk, gv, t0=w.L, workspace=ws, out=o)
    sptr = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    e0, e1 = hip.event(), hip.event()
    torch.cuda.synchronize(dev)
    hip.record(e0, sptr)
    for i in range(args.steps):
        bla.step(sq, sk_, sv_, T, w.M, w.S, gk, gv, t0=w.L + i, workspace=ws, out=o)
    hip.record(e1, sptr)
    torch.cuda.synchronize(dev)
    ms = hip.elapsed_ms(e0, e1) / args.steps
    state_bytes = w.B * w.H * 2 * (2 * w.M * w.d * 4)        # k and v states
    nbytes = 2 * state_bytes + w.B * w.H * w.d * 2 * 4       # read + write states, q,k,v,o
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"workload": "decode", "B": w.B, "H": w.H, "d": w.d, "M": w.M, "S": w.S, "position": w.L,
            "ms_per_step": round(ms, 4), "tokens_per_s": round(w.B / (ms * 1e-3), 1),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None}}


def cpu_baseline_anchored(w, T, inputs):
    """Alg. 1 oracle (token by token, slot states as cumulative sums) on the whole workload."""
    import oracle

    q, k, v = inputs
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    threads = max(1, min(threads, w.B * w.H))
    t = time.perf_counter()
    oracle.forward_anchored(q, k, v, T, w.M, w.S, nthreads=threads)
    dt = time.perf_counter() - t
    return {"value": round(w.B * w.L / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"the whole LM-layer workload ({w.B}x{w.H} sequences of {w.L} tokens), float64 "
                      f"Alg. 1 with slot states, OpenMP over (b,h); {dt:.2f} s wall"}


def cpu_baseline(w, T, inputs):
    import oracle

    q, k, v = inputs
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    threads = max(1, min(threads, w.B * w.H))
    t = time.perf_counter()
    oracle.forward(q, k, v, T, w.M, w.S, nthreads=threads)
    dt = time.perf_counter() - t
    return {"value": round(w.B * w.L / dt, 1), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"the whole LM-layer workload ({w.B}x{w.H} sequences of {w.L} tokens), float64 "
                      f"recurrence with the factored readout, OpenMP over (b,h); {dt:.2f} s wall"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-anchored", action="store_true", help="skip the anchored-slot measurement")
    ap.add_argument("--form", choices=("rotating", "anchored"), default="rotating",
                    help="the form of the headline forward; with 'anchored' no other forward runs")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="first run one plain device copy of this many bytes (reference kernel for "
                         "scaling the HBM byte counters of a rocprofv3 --pmc run)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build has no multi-GPU path); got --gpus {args.gpus}",
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
    inputs = bi.generate(3)
    head_anchor = args.form == "anchored"
    w, T, ms, value, roofline, extra = bench_forward(args, hip, inputs, head_anchor)
    anchored = None
    if not head_anchor and not args.no_anchored:
        _, _, a_ms, a_value, a_roof, a_extra = bench_forward(args, hip, inputs, True)
        anchored = {"form": "anchored slots (Sec. 3.3, Alg. 1/3), phase_anchor=1", "value": round(a_value, 1),
                    "unit": "tokens/s", "ms_per_step": round(a_ms, 5), "roofline": a_roof,
                    "forward_detail": a_extra,
                    "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline_anchored(w, T, inputs)}
    decode = None if args.no_decode or head_anchor else bench_decode(args, hip)
    if args.no_cpu_baseline:
        cpu = None
    else:
        cpu = cpu_baseline_anchored(w, T, inputs) if head_anchor else cpu_baseline(w, T, inputs)
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "lm_layer", "B": w.B, "H": w.H, "L": w.L, "d": w.d, "M": w.M, "S": w.S,
                   "chunk": w.chunk, "periods": "T_h=(1+h%2)(2M-1)", "state": "fp32",
                   "phase_anchor": head_anchor},
        "roofline": roofline, "cpu_baseline": cpu, "forward_detail": extra, "decode_step": decode,
        "anchored": anchored,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
