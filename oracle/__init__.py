"""CPU oracle for decode attention over a prefix-tree chunked KV cache.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. The HIP library
never calls it and shares no code with it.

It is a plain, slow, obviously-correct restatement of ChunkAttention
(arXiv 2402.15220):
  * ``tree``   - the prefix-aware KV cache (Section 3.1, PAKV): a forest of
                 chunks of at most ``c`` tokens with their K/V rows, insert with
                 prefix matching and chunk splitting, extend/append, remove,
                 and a pool of chunk slots with a free list;
  * ``tables`` - the kernel context of Section 3.3 / Figure 2: per chunk the
                 half-open range of query rows it covers, plus each sequence's
                 shared and private chunk lists (Algorithms 1 and 2);
  * ``attention`` - the result the two-phase partition must reach: for every
                 sequence and head, softmax(scale * K q) V over the K/V rows on
                 the sequence's root-to-leaf path, in float64; and, as a
                 self-check only, the same result assembled chunk by chunk with
                 partial_attn (Eqn 1) and attn_reduce (Eqn 2); plus causal
                 prefill attention for a sequence's last tokens over its
                 whole path (Section 3.2, prefill paragraph).
"""
from .tree import OracleTree, PoolExhausted  # noqa: F401
from .tables import tables, Tables  # noqa: F401
from .attention import (  # noqa: F401
    dense_attention,
    dense_attention_rows,
    structured_attention,
    partial_attn,
    attn_reduce,
    path_kv,
    prefill_attention,
)
