"""Decode attention over the tree, in float64 (paper Section 3.2).

Test infrastructure only (see the package docstring).

The two-phase partition (Algorithms 1 and 2) is an exact reorganisation of
plain softmax attention: for sequence r and head h, with K_r and V_r the K/V
rows stored along r's root-to-leaf path,

    o[r, h] = softmax(scale * K_r q[r, h]) V_r,   scale = 1/sqrt(d) by default.

Eqn 1 as printed has no scale factor; the comparison formula of the
experiments divides by sqrt(d), so ``scale`` is an explicit argument.
``dense_attention`` is that definition written out. ``partial_attn`` (Eqn 1)
and ``attn_reduce`` (Eqn 2) restate the paper's building blocks and
``structured_attention`` assembles the result chunk by chunk with them; it is
used only to check that the partition reaches the dense result.
"""
from __future__ import annotations

import numpy as np


def path_kv(tree, sid):
    """K, V rows of ``sid`` concatenated root -> leaf, as float64 [L, H, d]."""
    nodes = tree.path(sid)
    k = np.concatenate([n.k for n in nodes], axis=0).astype(np.float64)
    v = np.concatenate([n.v for n in nodes], axis=0).astype(np.float64)
    return k, v


def _softmax_attend(q, k, v, scale):
    """q [H, d], k/v [L, H, d] -> o [H, d] (float64)."""
    s = scale * np.einsum("lhd,hd->hl", k, q)
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    w /= w.sum(axis=1, keepdims=True)
    return np.einsum("hl,lhd->hd", w, v)


def dense_attention_rows(tree, row_seq, q, scale, rows=None, heads=None):
    """o for the given query rows (tree row order) and heads.

    q: [B, H, d] in row order. Returns float64 [len(rows), len(heads), d].
    """
    B, H, d = q.shape
    rows = range(B) if rows is None else rows
    heads = np.arange(H) if heads is None else np.asarray(heads)
    out = np.empty((len(rows), len(heads), d), np.float64)
    for i, r in enumerate(rows):
        k, v = path_kv(tree, int(row_seq[r]))
        out[i] = _softmax_attend(q[r, heads].astype(np.float64), k[:, heads], v[:, heads], scale)
    return out


def dense_attention(tree, row_seq, q, scale):
    return dense_attention_rows(tree, row_seq, q, scale)


def prefill_attention(tree, sid, q, scale, heads=None, queries=None):
    """Causal attention for the last n_q tokens of sequence ``sid`` over its
    whole K/V (Section 3.2, prefill paragraph: after the prefix lookup the
    suffix's K/V joins the tree and ordinary self-attention runs over the
    entire K/V of the sequence).

    q: [n_q, H, d], query i belongs to position p = L - n_q + i and attends
    to positions 0..p of the root-to-leaf K/V. Returns float64
    [len(queries), len(heads), d].
    """
    k, v = path_kv(tree, sid)
    L = k.shape[0]
    n_q, H, d = q.shape
    if n_q > L:
        raise ValueError("more queries than tokens")
    heads = np.arange(H) if heads is None else np.asarray(heads)
    queries = range(n_q) if queries is None else queries
    out = np.empty((len(queries), len(heads), d), np.float64)
    for j, i in enumerate(queries):
        p = L - n_q + i
        out[j] = _softmax_attend(q[i, heads].astype(np.float64), k[: p + 1, heads],
                                 v[: p + 1, heads], scale)
    return out


# -- Eqn 1 / Eqn 2, for the structural self-check only ----------------------

def partial_attn(Q, K, V, scale):
    """Eqn 1 for one chunk and one head: Q [rows, d], K/V [len, d].

    W = scale * Q K^T, m = rowmax W, E = exp(W - m), n = rowsum E, O = E V
    (O unnormalised).
    """
    W = scale * (Q @ K.T)
    m = W.max(axis=1)
    E = np.exp(W - m[:, None])
    n = E.sum(axis=1)
    O = E @ V
    return O, m, n


def attn_reduce(o_c, m_c, n_c, O, m, n):
    """Eqn 2: fold one partial (o_c, m_c, n_c) into the running (O, m, n)."""
    mx = max(m_c, m)
    x = np.exp(m_c - mx)
    y = np.exp(m - mx)
    return x * o_c + y * O, mx, x * n_c + y * n


def structured_attention(tree, row_seq, q, scale):
    """Per row and head: Eqn 1 on each chunk of the path, Eqn 2 in path
    order starting from the first chunk's partial, then O/n."""
    B, H, d = q.shape
    out = np.empty((B, H, d), np.float64)
    for r in range(B):
        nodes = tree.path(int(row_seq[r]))
        for h in range(H):
            qh = q[r, h].astype(np.float64)[None, :]
            acc = None
            for nd in nodes:
                o_c, m_c, n_c = partial_attn(qh, nd.k[:, h].astype(np.float64),
                                             nd.v[:, h].astype(np.float64), scale)
                part = (o_c[0], float(m_c[0]), float(n_c[0]))
                acc = part if acc is None else attn_reduce(*part, *acc)
            O, _, n = acc
            out[r, h] = O / n
    return out
