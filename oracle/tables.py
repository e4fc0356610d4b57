"""Kernel context flattened from the tree (paper Section 3.3 and Figure 2).

Test infrastructure only (see the package docstring).

The paper's context is, per chunk C, the slice [i, j] of query rows that C
covers (Figure 2 prints the end index inclusively: C0-C2 cover rows 0..2,
C3 row 0, C4/C6 row 1, C5/C7 row 2). Ranges here are half-open [i, j), the
convention of Eqn 1's Q_{i:j} with j-i rows. Algorithm 1 walks the chunks
shared by several sequences; Algorithm 2 walks, per sequence, the partial
results of its shared chunks and then its own chunks.

Canonical order (R9): children by ascending first token. Rows follow a
depth-first pre-order in which the sequences ending at a node come first
(ascending id) before its child subtrees. Node indices follow breadth-first
level order with the same child order; this reproduces Figure 2's labels.

Tables (all int32 except row_seq):
  row_seq[B]            sequence id of each query row
  node_slot/len/row_begin/row_end/parent/start_pos [n_nodes]
  shared: nodes with row_end-row_begin >= 2 in node order, with part_base =
          running sum of their row counts (one partial result per covered row)
  priv_ptr[B+1], priv_node[]  per row, private nodes root -> leaf
  shr_ptr[B+1],  shr_part[]   per row, partial index part_base + r - row_begin
                              of each shared node on its path, root -> leaf
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class Tables:
    row_seq: np.ndarray
    node_slot: np.ndarray
    node_len: np.ndarray
    node_row_begin: np.ndarray
    node_row_end: np.ndarray
    node_parent: np.ndarray
    node_start_pos: np.ndarray
    shr_node: np.ndarray
    shr_part_base: np.ndarray
    priv_ptr: np.ndarray
    priv_node: np.ndarray
    shr_ptr: np.ndarray
    shr_part: np.ndarray

    @property
    def B(self):
        return int(self.row_seq.shape[0])

    @property
    def n_nodes(self):
        return int(self.node_slot.shape[0])

    @property
    def n_parts(self):
        if self.shr_node.shape[0] == 0:
            return 0
        last = int(self.shr_node[-1])
        return int(self.shr_part_base[-1] + self.node_row_end[last] - self.node_row_begin[last])

    def as_dict(self):
        return {f.name: getattr(self, f.name) for f in dataclasses.fields(self)}


def _children(node):
    return [node.children[k] for k in sorted(node.children)]


def tables(tree) -> Tables:
    # rows: depth-first pre-order, terminals (ascending id) before children
    row_of = {}
    rows = []
    rng = {}
    # iterative pre-order walk (chains can be long); each node's row range is
    # recorded when its subtree is finished
    stack = [(tree.root, False)]
    begins = {}
    while stack:
        node, done = stack.pop()
        if done:
            rng[id(node)] = (begins[id(node)], len(rows))
            continue
        begins[id(node)] = len(rows)
        for sid in sorted(node.terminals):
            row_of[sid] = len(rows)
            rows.append(sid)
        stack.append((node, True))
        for ch in reversed(_children(node)):
            stack.append((ch, False))

    # nodes: breadth-first level order
    order = []
    frontier = _children(tree.root)
    while frontier:
        order.extend(frontier)
        nxt = []
        for n in frontier:
            nxt.extend(_children(n))
        frontier = nxt
    index = {id(n): i for i, n in enumerate(order)}
    start = {}
    for n in order:
        p = n.parent
        start[id(n)] = 0 if p is tree.root else start[id(p)] + len(p)

    nn = len(order)
    node_slot = np.array([n.slot for n in order], np.int32).reshape(nn)
    node_len = np.array([len(n) for n in order], np.int32).reshape(nn)
    node_rb = np.array([rng[id(n)][0] for n in order], np.int32).reshape(nn)
    node_re = np.array([rng[id(n)][1] for n in order], np.int32).reshape(nn)
    node_parent = np.array([-1 if n.parent is tree.root else index[id(n.parent)] for n in order],
                           np.int32).reshape(nn)
    node_start = np.array([start[id(n)] for n in order], np.int32).reshape(nn)
    for n in order:
        assert rng[id(n)][1] - rng[id(n)][0] == n.count

    shr_node = [i for i in range(nn) if node_re[i] - node_rb[i] >= 2]
    part_base = {}
    acc = 0
    for i in shr_node:
        part_base[i] = acc
        acc += int(node_re[i] - node_rb[i])

    B = len(rows)
    priv_ptr = [0]
    priv_node = []
    shr_ptr = [0]
    shr_part = []
    for r, sid in enumerate(rows):
        for n in tree.path(sid):
            i = index[id(n)]
            if i in part_base:
                shr_part.append(part_base[i] + r - int(node_rb[i]))
            else:
                priv_node.append(i)
        priv_ptr.append(len(priv_node))
        shr_ptr.append(len(shr_part))

    return Tables(
        row_seq=np.array(rows, np.int64).reshape(B),
        node_slot=node_slot, node_len=node_len,
        node_row_begin=node_rb, node_row_end=node_re,
        node_parent=node_parent, node_start_pos=node_start,
        shr_node=np.array(shr_node, np.int32).reshape(len(shr_node)),
        shr_part_base=np.array([part_base[i] for i in shr_node], np.int32).reshape(len(shr_node)),
        priv_ptr=np.array(priv_ptr, np.int32),
        priv_node=np.array(priv_node, np.int32).reshape(len(priv_node)),
        shr_ptr=np.array(shr_ptr, np.int32),
        shr_part=np.array(shr_part, np.int32).reshape(len(shr_part)),
    )
