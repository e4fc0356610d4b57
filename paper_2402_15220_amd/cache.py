"""Torch-facing wrapper of the C ABI: torch provides device memory and the
current stream, every step of the attention path runs in the HIP library."""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B

_DT = {torch.float16: B.CA_FP16, torch.float32: B.CA_FP32}

# The current stream's raw handle without building a torch Stream object
# (~0.3 us instead of ~3 us per call; the same call torch's own kernel
# launchers use), falling back to the public API.
_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


class Cache:
    """A prefix-tree chunked KV cache on one GPU (or table-only on the host).

    Pools are allocated here with torch and lent to the library; q/o rows
    follow ``seq_order()``. ``layout="interleaved"`` (default) keeps each
    chunk-head's K and V tiles adjacent in one buffer [slot][head][K|V][c][d]
    (strided pools: a block that reads a chunk's K and then its V reads one
    contiguous region, which measured faster than two separate regions on
    every decode workload, most on calls that miss the caches); ``"split"``
    uses two buffers [slot][head][c][d] (the C ABI's dense default).
    ``k_pool``/``v_pool`` are [slot][head][c][d] views either way.
    """

    def __init__(self, chunk_size: int, num_heads: int, head_dim: int, num_slots: int,
                 dtype=torch.float16, device="cuda", table_only: bool = False,
                 layout: str = "interleaved"):
        self.c, self.H, self.d = chunk_size, num_heads, head_dim
        self.dtype = dtype
        self.num_slots = num_slots
        self.table_only = table_only
        self.layout = None if table_only else layout
        if table_only:
            self.k_pool = self.v_pool = None
            self.h = B.ca_create(chunk_size, num_heads, head_dim, _DT[dtype], num_slots)
        elif layout == "interleaved":
            self.kv_pool = torch.empty((num_slots, num_heads, 2, chunk_size, head_dim), dtype=dtype,
                                       device=device)
            self.k_pool = self.kv_pool[:, :, 0]
            self.v_pool = self.kv_pool[:, :, 1]
            tile = chunk_size * head_dim
            self.h = B.ca_create(chunk_size, num_heads, head_dim, _DT[dtype], num_slots,
                                 self.k_pool.data_ptr(), self.v_pool.data_ptr(),
                                 slot_stride=2 * num_heads * tile, head_stride=2 * tile)
        elif layout == "split":
            shape = (num_slots, num_heads, chunk_size, head_dim)
            self.k_pool = torch.empty(shape, dtype=dtype, device=device)
            self.v_pool = torch.empty(shape, dtype=dtype, device=device)
            self.h = B.ca_create(chunk_size, num_heads, head_dim, _DT[dtype], num_slots,
                                 self.k_pool.data_ptr(), self.v_pool.data_ptr())
        else:
            raise ValueError(f"unknown layout {layout!r}")
        self._ws = None
        self._dev_index = None if table_only else self.k_pool.device.index

    # -- helpers -----------------------------------------------------------
    def stream(self):
        """Handle of the current stream of the pools' device."""
        if _raw_stream is not None:
            return _raw_stream(self._dev_index)
        return torch.cuda.current_stream(self._dev_index).cuda_stream

    def _kv(self, k, v, n):
        if self.table_only:
            if k is not None or v is not None:
                raise ValueError("table-only cache takes no K/V")
            return None, None, None
        for t in (k, v):
            if not isinstance(t, torch.Tensor) or t.dtype != self.dtype \
                    or tuple(t.shape) != (n, self.H, self.d) or not t.is_contiguous() \
                    or t.device != self.k_pool.device:
                raise ValueError(f"K/V must be contiguous {self.dtype} tensors [{n},{self.H},{self.d}] "
                                 f"on {self.k_pool.device}")
        return k.data_ptr(), v.data_ptr(), self.stream()

    def _check_rows(self, t, n, name):
        """q and o: contiguous [n, H, d] of the cache's dtype on the pools'
        device (the kernels read and write exactly n*H*d elements)."""
        if not isinstance(t, torch.Tensor) or t.dtype != self.dtype or t.dim() != 3 \
                or tuple(t.shape) != (n, self.H, self.d) or not t.is_contiguous() \
                or t.device != self.k_pool.device:
            raise ValueError(f"{name} must be a contiguous {self.dtype} tensor [{n},{self.H},{self.d}] "
                             f"on {self.k_pool.device}")

    # -- tree operations ---------------------------------------------------
    def match(self, tokens) -> int:
        return B.ca_match(self.h, tokens)

    def insert(self, seq_id, tokens, k=None, v=None) -> int:
        tokens = np.asarray(tokens, np.int32)
        kp, vp, s = self._kv(k, v, tokens.shape[0])
        return B.ca_insert(self.h, seq_id, tokens, kp, vp, s)

    def extend(self, seq_id, tokens, k=None, v=None) -> int:
        tokens = np.asarray(tokens, np.int32)
        kp, vp, s = self._kv(k, v, tokens.shape[0])
        return B.ca_extend(self.h, seq_id, tokens, kp, vp, s)

    def append(self, seq_ids, tokens, k=None, v=None):
        tokens = np.asarray(tokens, np.int32)
        kp, vp, s = self._kv(k, v, tokens.shape[0])
        B.ca_append_batch(self.h, seq_ids, tokens, kp, vp, s)

    def remove(self, seq_id):
        B.ca_remove(self.h, seq_id)

    def num_seqs(self) -> int:
        return B.ca_num_seqs(self.h)

    def seq_order(self) -> np.ndarray:
        return B.ca_seq_order(self.h)

    def tables(self) -> dict:
        return B.ca_export_tables(self.h)

    def stats(self) -> dict:
        return B.ca_stats(self.h)

    def set_tuning(self, seg_chunks=0, split_chunks=-1, phase_mask=0, schedule=-1):
        B.ca_set_tuning(self.h, seg_chunks, split_chunks, phase_mask, schedule)

    def prepare(self) -> bool:
        """Build the kernel context for the current tree now and enqueue its
        upload on the current stream (True if one was needed)."""
        return B.ca_prepare(self.h, None if self.table_only else self.stream())

    # -- attention ---------------------------------------------------------
    def workspace(self):
        need = B.ca_workspace_size(self.h)
        if self._ws is None or self._ws.numel() < need:
            self._ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.k_pool.device)
        return self._ws, need

    def attention(self, q, out=None, scale: float = 0.0, seq_ids=None):
        """q: [B, H, d] in seq_order(), or in the order of ``seq_ids`` (every
        live sequence once) when given; returns o in the same row order."""
        if self.table_only:
            raise ValueError("table-only cache has no attention")
        Bn = self.num_seqs()
        self._check_rows(q, Bn, "q")
        if out is None:
            out = torch.empty_like(q)
        self._check_rows(out, Bn, "out")
        ws, need = self.workspace()
        if seq_ids is None:
            B.ca_attention(self.h, q.data_ptr(), out.data_ptr(), scale, ws.data_ptr(), ws.numel(),
                           self.stream())
        else:
            B.ca_attention_ordered(self.h, q.data_ptr(), out.data_ptr(), seq_ids, scale,
                                   ws.data_ptr(), ws.numel(), self.stream())
        return out

    def attention_noalloc(self, q, out, scale: float = 0.0):
        """ca_attention_noalloc: q and out [B, H, d] in seq_order(), both
        already allocated; the library allocates nothing for the call (its
        partials live in a static device scratch). Needs the kernel context
        on the device: call prepare() after structural tree changes."""
        if self.table_only:
            raise ValueError("table-only cache has no attention")
        Bn = self.num_seqs()
        self._check_rows(q, Bn, "q")
        self._check_rows(out, Bn, "out")
        B.ca_attention_noalloc(self.h, q.data_ptr(), out.data_ptr(), scale, self.stream())
        return out

    def prefill(self, seq_id, q, out=None, scale: float = 0.0):
        """Causal attention of sequence ``seq_id``'s last q.shape[0] tokens over
        its whole K/V (prefill after a prefix-matched insert). q: [n_q, H, d]."""
        if self.table_only:
            raise ValueError("table-only cache has no attention")
        if not isinstance(q, torch.Tensor) or q.dim() != 3:
            raise ValueError(f"q must be a tensor [n_q,{self.H},{self.d}]")
        self._check_rows(q, q.shape[0], "q")
        if out is None:
            out = torch.empty_like(q)
        self._check_rows(out, q.shape[0], "out")
        B.ca_prefill_attention(self.h, seq_id, q.data_ptr(), out.data_ptr(), q.shape[0], scale,
                               self.stream())
        return out

    def close(self):
        """Destroy the library cache. ca_destroy frees the library's device
        buffers without waiting, so the device is synchronised first (the
        calls may have been enqueued on several streams)."""
        if self.h is not None:
            if not self.table_only:
                torch.cuda.synchronize(self._dev_index)
            B.ca_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
