"""Shared helpers for the GPU parity tests: build the same tree in the HIP
library and in the oracle from one seeded workload, run the library's
attention, and measure the error against the oracle's float64 result."""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

from oracle import OracleTree, dense_attention_rows, tables
from paper_2402_15220_amd.cache import Cache

# parity bar for fp16 inputs with fp32 accumulation (max-abs and relative L2)
FP16_MAX_ABS = 2e-3
FP16_REL_L2 = 1e-3
# fp32 inputs: fp32 products and sums over at most a few thousand terms
FP32_MAX_ABS = 2e-5
FP32_REL_L2 = 1e-5

TORCH_DT = {np.dtype(np.float16): torch.float16, np.dtype(np.float32): torch.float32}


def tol(dtype):
    if np.dtype(dtype) == np.float16:
        return FP16_MAX_ABS, FP16_REL_L2
    return FP32_MAX_ABS, FP32_REL_L2


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def errors(o, ref):
    """max-abs over everything, rel-L2 over the whole tensor, worst row."""
    o = np.asarray(o, np.float64)
    ref = np.asarray(ref, np.float64)
    diff = o - ref
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    rel = float(np.linalg.norm(diff) / max(np.linalg.norm(ref), 1e-300)) if diff.size else 0.0
    worst = int(np.abs(diff).reshape(diff.shape[0], -1).max(axis=1).argmax()) if diff.size else -1
    return max_abs, rel, worst


def assert_close(o, ref, dtype, what=""):
    ma, rel, worst = errors(o, ref)
    amax, rmax = tol(dtype)
    print(f"[parity] {what} max_abs={ma:.3e} rel_l2={rel:.3e} worst_row={worst}", flush=True)
    assert ma <= amax and rel <= rmax, f"{what}: max_abs {ma:.3e} rel_l2 {rel:.3e} (worst row {worst})"
    return ma, rel


class Pair:
    """The same cache on both sides: the HIP library and the oracle. Pools
    are the wrapper's default (K|V-interleaved) unless a layout is named."""

    def __init__(self, c, H, d, dtype, num_slots, oracle_kv=True, layout="interleaved"):
        self.dtype = np.dtype(dtype)
        self.cache = Cache(c, H, d, num_slots, dtype=TORCH_DT[self.dtype], layout=layout)
        self.tree = OracleTree(c=c, with_kv=oracle_kv)
        self.H, self.d, self.c = H, d, c

    def insert(self, sid, tokens, k, v, dev_k=None, dev_v=None):
        dk = to_dev(k) if dev_k is None else dev_k
        dv = to_dev(v) if dev_v is None else dev_v
        m1 = self.cache.insert(sid, tokens, dk, dv)
        m2 = self.tree.insert(sid, tokens, k, v)
        assert m1 == m2
        return m1

    def extend(self, sid, tokens, k, v):
        m1 = self.cache.extend(sid, tokens, to_dev(k), to_dev(v))
        m2 = self.tree.extend(sid, tokens, k, v)
        assert m1 == m2

    def append(self, sids, tokens, k, v, dev_k=None, dev_v=None):
        self.cache.append(sids, tokens, to_dev(k) if dev_k is None else dev_k,
                          to_dev(v) if dev_v is None else dev_v)
        self.tree.append_batch(sids, tokens, k, v)

    def remove(self, sid):
        self.cache.remove(sid)
        self.tree.remove(sid)

    def check_tables(self):
        lib = self.cache.tables()
        ora = tables(self.tree).as_dict()
        for k in ora:
            assert np.array_equal(lib[k], ora[k]), k
        return ora

    def check_pool(self, max_nodes=None, rng=None):
        """Pool rows of every (or a sample of) node equal the oracle's K/V."""
        torch.cuda.synchronize()
        nodes = self.tree.nodes()
        if max_nodes is not None and len(nodes) > max_nodes:
            rng = rng or np.random.default_rng(0)
            nodes = [nodes[i] for i in rng.choice(len(nodes), max_nodes, replace=False)]
        for n in nodes:
            L = len(n)
            kp = self.cache.k_pool[n.slot, :, :L, :].cpu().numpy()
            vp = self.cache.v_pool[n.slot, :, :L, :].cpu().numpy()
            assert np.array_equal(kp, n.k.transpose(1, 0, 2)), f"K of slot {n.slot}"
            assert np.array_equal(vp, n.v.transpose(1, 0, 2)), f"V of slot {n.slot}"

    def attention(self, q_by_sid, scale=0.0):
        """q_by_sid: dict or callable sid -> q[H, d]. Returns (o rows, row_seq)."""
        row_seq = self.cache.seq_order()
        q = np.stack([q_by_sid[int(s)] for s in row_seq]).astype(self.dtype)
        o = self.cache.attention(to_dev(q), scale=scale)
        torch.cuda.synchronize()
        return o.cpu().numpy(), q, row_seq

    def reference(self, row_seq, q, scale, rows=None):
        sc = scale if scale else 1.0 / np.sqrt(self.d)
        return reference_rows(self.tree, row_seq, q, sc, rows=rows)


def host_threads():
    """Threads for the oracle: the CPUs this process may use, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def reference_rows(tree, row_seq, q, scale, rows=None, threads=None):
    """The oracle's dense_attention_rows for `rows`, the rows split over a
    thread pool (NumPy releases the GIL in its copies and reductions); the
    oracle code and its arithmetic are unchanged, each row is computed by one
    call on one thread."""
    rows = list(range(q.shape[0])) if rows is None else [int(r) for r in rows]
    n = threads or host_threads()
    if n <= 1 or len(rows) < 4:
        return dense_attention_rows(tree, row_seq, q, scale, rows=rows)
    per = -(-len(rows) // (2 * n))
    groups = [rows[i:i + per] for i in range(0, len(rows), per)]
    with ThreadPoolExecutor(n) as ex:
        parts = list(ex.map(lambda g: dense_attention_rows(tree, row_seq, q, scale, rows=g), groups))
    return np.concatenate(parts, axis=0)
