"""Algorithmic byte and FLOP model of decode attention over the chunk tree.

The model follows the paper's cost breakdown of decode self-attention
(Table 1: per layer and decoded token, reading K and V of n context tokens
for h heads of size d costs 2*h*n*d elements and 4*h*n*d FLOPs). With a
prefix tree each chunk is read once, so the bytes a call must move are the
shared chunks once, every row's private chunks once, q in and o out.

Peaks are MI355X's published figures.
"""
from __future__ import annotations

import numpy as np

PEAK_HBM_GBPS = 8000.0
PEAK_MFMA_TFLOPS = {"f16": 2500.0, "bf16": 2500.0, "f32": 157.3}


def table1_self_attention(b: int, n: int, h: int = 32, d: int = 128, esize: int = 2):
    """Dense decode attention without sharing: (FLOPs, bytes) per layer."""
    flops = 4 * b * h * n * d
    mem = 2 * b * h * n * d * esize
    return flops, mem


def call_model(tab: dict, H: int, d: int, esize: int) -> dict:
    """Bytes and FLOPs of one attention call over exported canonical tables."""
    rb, re = tab["node_row_begin"], tab["node_row_end"]
    lens = tab["node_len"].astype(np.int64)
    rows = (re - rb).astype(np.int64)
    shared = rows >= 2
    B = int(tab["row_seq"].shape[0])
    row_bytes = H * d * esize          # one token's K (or V) for all heads
    shared_kv = 2 * int(lens[shared].sum()) * row_bytes
    private_kv = 2 * int(lens[~shared].sum()) * row_bytes
    q_bytes = B * H * d * esize
    o_bytes = B * H * d * esize
    ctx = int((lens * rows).sum())     # sum over rows of their context length
    flops = 4 * H * d * ctx
    kcf_flops = 4 * H * d * int((lens[shared] * rows[shared]).sum())
    return dict(
        B=B, shared_kv=shared_kv, private_kv=private_kv, q=q_bytes, o=o_bytes,
        total=shared_kv + private_kv + q_bytes + o_bytes,
        dense_equivalent=2 * ctx * row_bytes + q_bytes + o_bytes,
        flops=flops, kcf_flops=kcf_flops,
        ksf_bytes=private_kv + q_bytes + o_bytes,
        kcf_bytes=shared_kv + int(rows[shared].max(initial=0) > 0) * q_bytes,
    )
