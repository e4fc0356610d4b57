"""Brute-force prefix lookup for the tests of the prefix lookup (paper
Section 3.2, prefill paragraph: the matched prefix of a joining sequence is
found in the tree and its K/V reused).

The tree stores every live sequence as a root-to-terminal path, and every
node lies on the path of at least one live sequence (zero-count nodes are
freed). A probe's tokens can therefore be followed down the tree exactly as
far as they agree with some live sequence: the lookup must return

    max over live sequences s of  LCP(probe, s)

where LCP is the length of the longest common prefix. This module computes
that from the sequences' token lists, which the tests keep themselves (no
tree involved), and draws probes that exercise every way a lookup ends:
inside a chunk, at a chunk boundary, at the end of a stored path, past every
stored path, and on the first token.
"""
from __future__ import annotations

import numpy as np


def lcp(a, b) -> int:
    a = np.asarray(a)
    b = np.asarray(b)
    n = min(a.shape[0], b.shape[0])
    diff = np.flatnonzero(a[:n] != b[:n])
    return int(diff[0]) if diff.size else n


def max_lcp(live_tokens, probe) -> int:
    """Longest prefix of `probe` shared with any of the live sequences."""
    return max((lcp(s, probe) for s in live_tokens), default=0)


def probes(rng, live_tokens, n, alphabet, extra=3):
    """`n` non-empty probes: prefixes of live sequences cut at every kind of
    position, extended by a few tokens (some from outside the alphabet),
    with one token changed, longer than the sequence itself, and random."""
    live = [np.asarray(s, np.int32) for s in live_tokens]
    out = []
    for _ in range(n):
        kind = int(rng.integers(0, 5))
        if not live or kind == 4:
            m = int(rng.integers(1, 8))
            out.append(rng.integers(0, alphabet + 1, m).astype(np.int32))
            continue
        s = live[int(rng.integers(0, len(live)))]
        cut = int(rng.integers(0, s.shape[0] + 1))
        tail = rng.integers(0, alphabet + 1, int(rng.integers(0, extra + 1))).astype(np.int32)
        if kind == 0:          # a cut prefix, maybe with a short random tail
            p = np.concatenate([s[:cut], tail])
        elif kind == 1:        # the whole sequence and more: past the stored path
            p = np.concatenate([s, tail, [alphabet + 7]])
        elif kind == 2:        # one token changed at the cut
            p = s.copy()
            if cut < p.shape[0]:
                p[cut] = (p[cut] + 1 + int(rng.integers(0, alphabet))) % (alphabet + 1)
        else:                  # exactly a live sequence
            p = s.copy()
        if p.shape[0] == 0:
            p = np.array([int(rng.integers(0, alphabet + 1))], np.int32)
        out.append(p.astype(np.int32))
    return out
