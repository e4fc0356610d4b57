"""Prefix-aware KV cache as a tree of chunks (paper Section 3.1, PAKV).

Test infrastructure only (see the package docstring).

What the paper fixes (Section 3.1):
  * each node is a chunk holding up to ``c`` tokens and the K and V slices of
    those tokens; every root-to-leaf path is one sequence; a forest is allowed;
  * a joining sequence searches the tree and inserts a new path, a leaving
    sequence deletes its path, and decoding appends tokens to leaf chunks,
    growing a new chunk when the leaf is full;
  * chunks come from a pool with a free list and are never returned to the OS;
    the memory lost to partly filled chunks is bounded by (c-1)/n;
  * the sequences covered by any chunk are contiguous in the batch index.

What the paper leaves open, and the reading taken here (rules R1-R10):
  R1  a virtual root without tokens; its children are the trees of the forest.
  R2  insert: from the root, descend into the child whose first token equals
      the next token. A fully matched child is descended; a mismatch inside a
      child, or the end of the sequence inside it, splits the child there
      (R4) and stops. The remaining tokens become ceil(rem/c) new chunks, all
      full except the last, chained under the node reached. Spare capacity of
      a node that someone else already uses is never filled. ``matched`` is
      the number of tokens that were already present.
  R3  extend/append: if the sequence's terminal node is private (one
      sequence, hence childless) it is filled up to ``c`` and then new chunks
      follow; otherwise R2 continues from the terminal node.
  R4  split X at p: X keeps tokens[:p] and its slot; a new node X' takes
      tokens[p:] with a fresh slot (K/V rows copied), X's children, count and
      terminal sequences; X's only child becomes X'.
  R5  a new chunk takes a slot from the pool and copies the caller's rows.
  R6  remove: decrement counts along the path; nodes reaching zero are
      detached and their slots freed from the leaf towards the root. Chains
      are never merged.
  R7  identical sequences and sequences that are prefixes of others are
      allowed; sequence ids are distinct.
  R8  pool: a LIFO free stack; when it is empty, fresh slot ids ascend from 0.
      A split takes its X' slot before any new chunk of the same operation.
      If the pool cannot supply an operation, it fails and changes nothing.
  R9  canonical order: children sorted by ascending first token (see tables).
  R10 invariants: 1 <= len <= c; sibling first tokens distinct;
      count = number of sequences through the node; the path tokens
      concatenated equal the sequence; shared nodes (count >= 2) form a prefix
      of every path; covered rows are contiguous.
"""
from __future__ import annotations

import copy

import numpy as np


class PoolExhausted(Exception):
    """Raised when the pool cannot supply the slots an operation needs."""


class Node:
    __slots__ = ("tokens", "k", "v", "slot", "count", "children", "parent", "terminals")

    def __init__(self, tokens, k, v, slot, parent):
        self.tokens = tokens          # np.int32 [len]
        self.k = k                    # [len, H, d] or None (table-only)
        self.v = v
        self.slot = slot
        self.count = 0
        self.children = {}            # first token -> Node
        self.parent = parent
        self.terminals = set()        # seq ids whose last token is in this node

    def __len__(self):
        return int(self.tokens.shape[0])


class OracleTree:
    def __init__(self, c: int, num_slots: int | None = None, with_kv: bool = True):
        if c < 1:
            raise ValueError("chunk size must be >= 1")
        self.c = c
        self.num_slots = num_slots
        self.with_kv = with_kv
        self.root = Node(np.zeros(0, np.int32), None, None, -1, None)
        self.free = []                # LIFO stack of freed slots
        self.fresh = 0                # next never-used slot id
        self.term = {}                # seq id -> terminal node
        self.length = {}              # seq id -> number of tokens

    # -- pool (R8) ---------------------------------------------------------
    def available(self) -> int:
        if self.num_slots is None:
            return 1 << 62
        return len(self.free) + (self.num_slots - self.fresh)

    def _alloc(self) -> int:
        if self.free:
            return self.free.pop()
        if self.num_slots is not None and self.fresh >= self.num_slots:
            raise PoolExhausted()
        s = self.fresh
        self.fresh += 1
        return s

    def slots_in_use(self) -> int:
        return self.fresh - len(self.free)

    # -- helpers -----------------------------------------------------------
    def _descend(self, cur, tokens, pos):
        """R2 search from ``cur``: returns (node reached, new pos, split)."""
        n = tokens.shape[0]
        while pos < n:
            child = cur.children.get(int(tokens[pos]))
            if child is None:
                return cur, pos, None
            L = len(child)
            m = min(L, n - pos)
            diff = np.flatnonzero(child.tokens[:m] != tokens[pos:pos + m])
            p = int(diff[0]) if diff.size else m
            if p == L:
                cur, pos = child, pos + L
                continue
            return cur, pos + p, (child, p)
        return cur, pos, None

    def _split(self, x, p):
        """R4: X keeps tokens[:p]; X' gets the rest, a fresh slot, X's children."""
        slot = self._alloc()
        xp = Node(x.tokens[p:].copy(),
                  None if x.k is None else x.k[p:].copy(),
                  None if x.v is None else x.v[p:].copy(), slot, x)
        xp.count = x.count
        xp.children = x.children
        for ch in xp.children.values():
            ch.parent = xp
        xp.terminals = x.terminals
        for sid in xp.terminals:
            self.term[sid] = xp
        x.tokens = x.tokens[:p].copy()
        if x.k is not None:
            x.k = x.k[:p].copy()
            x.v = x.v[:p].copy()
        x.children = {int(xp.tokens[0]): xp}
        x.terminals = set()
        return x

    def _new_chain(self, cur, tokens, k, v, pos):
        """R5: chunks of at most c tokens for tokens[pos:], chained under cur."""
        n = tokens.shape[0]
        while pos < n:
            e = min(pos + self.c, n)
            node = Node(tokens[pos:e].copy(),
                        None if k is None else np.array(k[pos:e]),
                        None if v is None else np.array(v[pos:e]),
                        self._alloc(), cur)
            cur.children[int(tokens[pos])] = node
            cur = node
            pos = e
        return cur

    def _need(self, start, tokens, pos0):
        cur, pos, split = self._descend(start, tokens, pos0)
        rem = tokens.shape[0] - pos
        return (1 if split else 0) + (-(-rem // self.c)), cur, pos, split

    def _check_kv(self, k, v, n):
        if self.with_kv:
            if k is None or v is None or k.shape[0] != n or v.shape[0] != n:
                raise ValueError("K/V rows must be given for every token")

    # -- operations --------------------------------------------------------
    def match(self, tokens) -> int:
        """Prefix lookup (Section 3.2, prefill paragraph): R2's descent
        without any change to the tree. Returns how many leading tokens are
        already stored, counting a partial match inside the chunk where the
        descent stops."""
        tokens = np.asarray(tokens, np.int32)
        _, pos, _ = self._descend(self.root, tokens, 0)
        return pos

    def insert(self, sid, tokens, k=None, v=None) -> int:
        """R2. Returns the number of already present (matched) tokens."""
        tokens = np.asarray(tokens, np.int32)
        if sid in self.term:
            raise KeyError(f"sequence {sid} exists")
        if tokens.shape[0] < 1:
            raise ValueError("empty sequence")
        self._check_kv(k, v, tokens.shape[0])
        need, cur, pos, split = self._need(self.root, tokens, 0)
        if need > self.available():
            raise PoolExhausted()
        matched = pos
        if split:
            cur = self._split(*split)
        cur = self._new_chain(cur, tokens, k, v, pos)
        self._attach(sid, cur, tokens.shape[0])
        return matched

    def _attach(self, sid, terminal, length):
        node = terminal
        while node is not self.root:
            node.count += 1
            node = node.parent
        terminal.terminals.add(sid)
        self.term[sid] = terminal
        self.length[sid] = length

    def extend(self, sid, tokens, k=None, v=None) -> int:
        """R3. Returns the number of tokens matched against existing nodes."""
        tokens = np.asarray(tokens, np.int32)
        if sid not in self.term:
            raise KeyError(f"sequence {sid} not found")
        if tokens.shape[0] < 1:
            raise ValueError("empty extension")
        self._check_kv(k, v, tokens.shape[0])
        t = self.term[sid]
        n = tokens.shape[0]
        if t.count == 1:
            f = min(self.c - len(t), n)
            need = -(-(n - f) // self.c)
            if need > self.available():
                raise PoolExhausted()
            if f > 0:
                t.tokens = np.concatenate([t.tokens, tokens[:f]])
                if t.k is not None:
                    t.k = np.concatenate([t.k, k[:f]])
                    t.v = np.concatenate([t.v, v[:f]])
            end = self._new_chain(t, tokens, k, v, f)
            t.terminals.discard(sid)
            node = end
            while node is not t:
                node.count += 1
                node = node.parent
            end.terminals.add(sid)
            self.term[sid] = end
            self.length[sid] += n
            return 0
        need, cur, pos, split = self._need(t, tokens, 0)
        if need > self.available():
            raise PoolExhausted()
        matched = pos
        if split:
            cur = self._split(*split)
            # a split of t's own child never moves t; sid still ends at t
        end = self._new_chain(cur, tokens, k, v, pos)
        t.terminals.discard(sid)
        node = end
        while node is not t:
            node.count += 1
            node = node.parent
        end.terminals.add(sid)
        self.term[sid] = end
        self.length[sid] += n
        return matched

    def append_batch(self, sids, tokens, k=None, v=None):
        """One decode token per listed sequence, applied in the listed order.

        All or nothing: when the pool may be too small for the worst case
        (one slot per sequence), the batch is first rehearsed on a copy.
        """
        sids = [int(s) for s in sids]
        tokens = np.asarray(tokens, np.int32)
        if len(set(sids)) != len(sids):
            raise ValueError("duplicate sequence id in batch")
        for s in sids:
            if s not in self.term:
                raise KeyError(f"sequence {s} not found")
        if self.with_kv and (k is None or v is None):
            raise ValueError("K/V rows must be given")
        if self.available() < len(sids):
            rehearsal = copy.deepcopy(self)
            rehearsal.with_kv = False
            rehearsal._strip_kv()
            for i, s in enumerate(sids):
                rehearsal.extend(s, tokens[i:i + 1])   # raises PoolExhausted
        for i, s in enumerate(sids):
            self.extend(s, tokens[i:i + 1],
                        None if k is None else k[i:i + 1],
                        None if v is None else v[i:i + 1])

    def _strip_kv(self):
        stack = [self.root]
        while stack:
            n = stack.pop()
            n.k = n.v = None
            stack.extend(n.children.values())

    def remove(self, sid):
        """R6: decrement counts; free zero-count nodes leaf -> root."""
        if sid not in self.term:
            raise KeyError(f"sequence {sid} not found")
        node = self.term.pop(sid)
        del self.length[sid]
        node.terminals.discard(sid)
        while node is not self.root:
            node.count -= 1
            parent = node.parent
            if node.count == 0:
                del parent.children[int(node.tokens[0])]
                self.free.append(node.slot)
            node = parent

    # -- inspection --------------------------------------------------------
    def seq_ids(self):
        return sorted(self.term)

    def path(self, sid):
        """Nodes from the root's child down to the terminal of ``sid``."""
        out = []
        node = self.term[sid]
        while node is not self.root:
            out.append(node)
            node = node.parent
        return out[::-1]

    def nodes(self):
        out = []
        stack = list(self.root.children.values())
        while stack:
            n = stack.pop()
            out.append(n)
            stack.extend(n.children.values())
        return out

    def slot_map(self):
        """slot -> node for every live node."""
        return {n.slot: n for n in self.nodes()}

    def check_invariants(self):
        """R10."""
        seen_slots = set()
        for n in self.nodes():
            assert 1 <= len(n) <= self.c, "node length out of range"
            assert n.slot not in seen_slots, "slot used twice"
            seen_slots.add(n.slot)
            firsts = [int(ch.tokens[0]) for ch in n.children.values()]
            assert len(firsts) == len(set(firsts)), "sibling first tokens collide"
            for key, ch in n.children.items():
                assert key == int(ch.tokens[0]) and ch.parent is n
            through = len(n.terminals) + sum(ch.count for ch in n.children.values())
            assert n.count == through, "count mismatch"
            if n.count == 1:
                assert len(n.children) <= 1
        for sid, t in self.term.items():
            p = self.path(sid)
            assert sum(len(x) for x in p) == self.length[sid]
            shared = [x.count >= 2 for x in p]
            # shared nodes form a prefix of the path
            assert shared == sorted(shared, reverse=True), "private node above a shared one"
        assert seen_slots.isdisjoint(self.free)
