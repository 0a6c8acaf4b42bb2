"""Seeded synthetic inputs for the BLA forward operator.

This module is shared by the tests, the benchmark and the smoke check, and by
both sides of every parity comparison.  It holds no part of the operator's
arithmetic: it only draws q, k, v (and, for the decode workload, the token at
the decode position) with the shapes and value distributions of the paper's
workloads, and rounds them to the dtype the GPU receives.

Workloads (the paper evaluates on MQAR and RegBench, Sec. 4 and Appendix D,
Tables 2-3; those datasets are not used -- these synthetic inputs stand in for
them with the same shapes and structure):

  id 1  tiny:        B=1,  H=2,  L=256,   d=32,  M=S=16,  fp32, q,k,v ~ N(0,1)/sqrt(d)
  id 2  recall:      B=64, H=4,  L=512,   d=64,  M=S=32,  bf16; per-head codebook of 256
                     unit vectors, q and k pick codebook rows by independent uniform
                     token ids (MQAR shape: L=512, Table 2), v ~ N(0,1)
  id 3  LM layer:    B=8,  H=16, L=4096,  d=64,  M=S=64,  bf16; X ~ N(0,1)^{L x 1024},
                     W_{q,k,v} ~ N(0,1/1024), q = X W_q / sqrt(d) (then split in heads)
  id 4  long ctx:    B=1,  H=16, L=65536, d=128, M=S=128, bf16, q,k,v ~ N(0,1)/sqrt(d)
  id 5  decode:      B=512,H=16, d=64, M=S=64; an LM-layer style sequence of 2049 tokens:
                     the first 2048 are prefilled, token 2048 is the decode step.

Periods: T_h = (1 + h mod 2) (2M-1), i.e. heads alternate between token
resolution 1 and 2 (Sec. 4.1 Eq. tok_res; Appendix D uses T = 2(2M-1) and
T in {1,2,4}(2M-1)).

Host generation uses numpy PCG64 with SeedSequence([0, cfg, tensor, b]), one
stream per batch row so that any subset of rows can be regenerated alone.
Values are drawn in float64, rounded to float32, then (bf16 workloads) rounded
to bfloat16 with round-to-nearest-even; both sides receive those exact values.
The decode workload (id 5) is too large to draw on the host in seconds, so its
LM-layer projection runs on the torch device from a seeded torch generator;
the oracle then receives a host copy of the sampled rows' generated values.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    B: int
    H: int
    L: int
    d: int
    M: int
    S: int
    chunk: int
    dtype: str  # "f32" or "bf16"
    kind: str   # "gauss", "recall", "lm", "decode"


WORKLOADS = {
    1: Workload(1, "tiny", 1, 2, 256, 32, 16, 16, 64, "f32", "gauss"),
    2: Workload(2, "recall", 64, 4, 512, 64, 32, 32, 64, "bf16", "recall"),
    3: Workload(3, "lm_layer", 8, 16, 4096, 64, 64, 64, 64, "bf16", "lm"),
    4: Workload(4, "long_context", 1, 16, 65536, 128, 128, 128, 64, "bf16", "gauss"),
    5: Workload(5, "decode", 512, 16, 2048, 64, 64, 64, 64, "bf16", "decode"),
}

HIDDEN = 1024          # model width of the LM-layer workloads (D = H*d = 16*64)
CODEBOOK = 256         # recall workload: codebook size per head


def periods(M: int, H: int):
    """Per-head periods T_h = (1 + h mod 2)(2M-1) as a float64 array [H]."""
    return np.array([(1 + (h % 2)) * (2 * M - 1) for h in range(H)], np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    return (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)


def _cast(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    return round_bf16(x32) if dtype == "bf16" else x32


def _rng(cid: int, tensor: int, b: int = -1):
    key = [0, cid, tensor] + ([b] if b >= 0 else [])
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(key)))


def _proj_weights(cid: int, H: int, d: int):
    """W_q, W_k, W_v ~ N(0, 1/HIDDEN), each [HIDDEN, H*d]."""
    return [_rng(cid, 10 + i).standard_normal((HIDDEN, H * d)) / math.sqrt(HIDDEN)
            for i in range(3)]


def generate(cid: int, rows=None, L=None, B=None, H=None, d=None):
    """q, k, v as float32 arrays [len(rows), H, L, d] holding io-dtype values.

    rows: batch rows to draw (default: all).  L, B, H, d override the workload's
    sizes (used for smaller parity cases with the same distribution).
    """
    w = WORKLOADS[cid]
    Bn = w.B if B is None else B
    Hn = w.H if H is None else H
    Ln = w.L if L is None else L
    dn = w.d if d is None else d
    rows = list(range(Bn)) if rows is None else list(rows)
    n = len(rows)
    q = np.empty((n, Hn, Ln, dn), np.float32)
    k = np.empty_like(q)
    v = np.empty_like(q)
    if w.kind == "gauss":
        for i, b in enumerate(rows):
            for t, arr in enumerate((q, k, v)):
                x = _rng(cid, t, b).standard_normal((Hn, Ln, dn)) / math.sqrt(dn)
                arr[i] = _cast(x, w.dtype)
    elif w.kind == "recall":
        books = []
        for h in range(Hn):
            e = _rng(cid, 20 + h).standard_normal((CODEBOOK, dn))
            books.append(e / np.linalg.norm(e, axis=1, keepdims=True))
        for i, b in enumerate(rows):
            ids_k = _rng(cid, 0, b).integers(0, CODEBOOK, size=Ln)
            ids_q = _rng(cid, 1, b).integers(0, CODEBOOK, size=Ln)
            vv = _rng(cid, 2, b).standard_normal((Hn, Ln, dn))
            for h in range(Hn):
                k[i, h] = _cast(books[h][ids_k], w.dtype)
                q[i, h] = _cast(books[h][ids_q], w.dtype)
            v[i] = _cast(vv, w.dtype)
    elif w.kind in ("lm", "decode"):
        Ws = _proj_weights(cid, Hn, dn)
        for i, b in enumerate(rows):
            X = _rng(cid, 0, b).standard_normal((Ln, HIDDEN))
            for t, arr in enumerate((q, k, v)):
                y = (X @ Ws[t]) / math.sqrt(dn)                      # [L, H*d]
                arr[i] = _cast(y.reshape(Ln, Hn, dn).transpose(1, 0, 2), w.dtype)
    else:
        raise ValueError(w.kind)
    return q, k, v


def generate_grad(cid: int, rows=None, L=None, B=None, H=None, d=None):
    """dLoss/dO for the backward pass: [len(rows), H, L, d] float32 holding io-dtype values,
    N(0, 1)/sqrt(d) from the stream of tensor 3 of each batch row (an upstream gradient of the
    same scale as the inputs; the loss itself is not modelled)."""
    w = WORKLOADS[cid]
    Bn = w.B if B is None else B
    Hn = w.H if H is None else H
    Ln = w.L if L is None else L
    dn = w.d if d is None else d
    rows = list(range(Bn)) if rows is None else list(rows)
    g = np.empty((len(rows), Hn, Ln, dn), np.float32)
    for i, b in enumerate(rows):
        g[i] = _cast(_rng(cid, 3, b).standard_normal((Hn, Ln, dn)) / math.sqrt(dn), w.dtype)
    return g


def generate_layer(cid: int, rows=None, L=None, B=None, H=None, d=None):
    """Hidden states and projections of a whole layer: x [len(rows), L, D] ~ N(0, 1) and
    W_qkv [D, 3D], W_o [D, D] ~ N(0, 1/D) (D = H d), float32 arrays holding bf16 values."""
    w = WORKLOADS[cid]
    Bn = w.B if B is None else B
    Hn = w.H if H is None else H
    Ln = w.L if L is None else L
    dn = w.d if d is None else d
    D = Hn * dn
    rows = list(range(Bn)) if rows is None else list(rows)
    x = np.empty((len(rows), Ln, D), np.float32)
    for i, b in enumerate(rows):
        x[i] = _cast(_rng(cid, 30, b).standard_normal((Ln, D)), "bf16")
    w_qkv = _cast(_rng(cid, 31).standard_normal((D, 3 * D)) / math.sqrt(D), "bf16")
    w_o = _cast(_rng(cid, 32).standard_normal((D, D)) / math.sqrt(D), "bf16")
    return x, w_qkv, w_o


def generate_decode_device(device, B=None, L=None, seed: int = 5):
    """Decode workload on a torch device: LM-layer style q,k,v [B,H,L,d] in bf16.

    X ~ N(0,1) from a seeded torch generator on `device`; W_{q,k,v} from the host
    streams of `_proj_weights`.  Returns bf16 torch tensors.
    """
    import torch

    w = WORKLOADS[5]
    Bn = w.B if B is None else B
    Ln = (w.L + 1) if L is None else L
    Ws = [torch.from_numpy(x.astype(np.float32)).to(device) for x in _proj_weights(5, w.H, w.d)]
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = [torch.empty((Bn, w.H, Ln, w.d), dtype=torch.bfloat16, device=device) for _ in range(3)]
    step = 16
    for b0 in range(0, Bn, step):
        nb = min(step, Bn - b0)
        X = torch.randn((nb, Ln, HIDDEN), generator=gen, device=device, dtype=torch.float32)
        for t in range(3):
            y = torch.matmul(X, Ws[t]) / math.sqrt(w.d)
            out[t][b0:b0 + nb] = y.view(nb, Ln, w.H, w.d).permute(0, 2, 1, 3).to(torch.bfloat16)
        del X
    return out
