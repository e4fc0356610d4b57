"""Pins for the CPU oracle: facts fixed by the paper and by mathematics.

Each test ties the oracle to something other than itself: the paper's worked
example (Figure 2), a hand-derived split/remove example, closed forms for the
workload trees, the memory-loss bound of Section 3.1, an independent library
routine for softmax attention, and special cases with known answers.
"""
import os

import numpy as np
import pytest
import torch

from oracle import (OracleTree, PoolExhausted, dense_attention, dense_attention_rows,
                    path_kv, prefill_attention, structured_attention, tables)
from prefix_util import max_lcp, probes
from workloads import make_dynamic, make_static, prefix_keyed_kv, random_op_script

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fig2_tree(with_kv=False, H=1, d=4, seed=0):
    t = OracleTree(c=4, with_kv=with_kv)
    shared = list(range(10, 22))
    seqs = [shared + list(range(30, 34)), shared + list(range(40, 48)), shared + list(range(50, 58))]
    for sid, toks in enumerate(seqs):
        toks = np.array(toks, np.int32)
        if with_kv:
            k, v = prefix_keyed_kv(seed, toks, 0, H, d, np.float64)
            t.insert(sid, toks, k, v)
        else:
            t.insert(sid, toks)
    return t


def _read_fig2_golden():
    ctx, lists = {}, {}
    with open(os.path.join(GOLDEN, "fig2_kernel_context.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if not line:
                continue
            if line[0].startswith("C"):
                ctx[int(line[0][1:])] = (int(line[1]), int(line[2]))
            else:
                lists[int(line[0][1:])] = [int(x[1:]) for x in line[1:]]
    return ctx, lists


def test_fig2_kernel_context_matches_paper():
    """Figure 2: chunk -> [i, j] (inclusive) and per-sequence chunk lists."""
    tb = tables(_fig2_tree())
    ctx, lists = _read_fig2_golden()
    assert tb.n_nodes == 8
    assert list(tb.row_seq) == [0, 1, 2]
    for c, (i, j) in ctx.items():
        assert (tb.node_row_begin[c], tb.node_row_end[c]) == (i, j + 1), c
    assert list(tb.shr_node) == [0, 1, 2]
    assert list(tb.shr_part_base) == [0, 3, 6]
    for r, chunks in lists.items():
        got = list(tb.priv_node[tb.priv_ptr[r]:tb.priv_ptr[r + 1]])
        assert got == chunks
        # every row reads the partials of C0-C2 at its own offset
        assert list(tb.shr_part[tb.shr_ptr[r]:tb.shr_ptr[r + 1]]) == [r, 3 + r, 6 + r]
    # slots in allocation order: S0 takes 0-3, S1 4 (C4) and 5 (C6), S2 6 and 7
    assert list(tb.node_slot) == [0, 1, 2, 3, 4, 6, 5, 7]
    assert list(tb.node_parent) == [-1, 0, 1, 2, 2, 2, 4, 5]
    assert list(tb.node_start_pos) == [0, 4, 8, 12, 12, 12, 16, 16]
    assert list(tb.node_len) == [4] * 8


def test_split_and_remove_example():
    """c=4, A=[1..6] then B=[1,2,9]: split, slot order, LIFO reuse (R4, R6, R8)."""
    t = OracleTree(c=4, with_kv=False)
    assert t.insert(0, [1, 2, 3, 4, 5, 6]) == 0
    assert t.insert(1, [1, 2, 9]) == 2
    tb = tables(t)
    # BFS: X=[1,2] (slot 0), X'=[3,4] (slot 2), Z=[9] (slot 3), Y=[5,6] (slot 1)
    assert list(tb.node_slot) == [0, 2, 3, 1]
    assert list(tb.node_len) == [2, 2, 1, 2]
    assert list(tb.row_seq) == [0, 1]
    assert list(tb.node_row_begin) == [0, 0, 1, 0]
    assert list(tb.node_row_end) == [2, 1, 2, 1]
    assert list(tb.node_parent) == [-1, 0, 0, 1]
    assert list(tb.node_start_pos) == [0, 2, 2, 4]
    assert list(tb.shr_node) == [0]
    assert list(tb.priv_node) == [1, 3, 2]
    t.remove(0)
    t.check_invariants()
    tb = tables(t)
    assert list(tb.node_slot) == [0, 3]       # X stays, private to B; no merge
    assert list(tb.node_len) == [2, 1]
    assert t.free == [1, 2]                    # Y freed first, then X'
    t.insert(2, [7])
    assert t.term[2].slot == 2                 # LIFO: last freed slot first
    t.insert(3, [8])
    assert t.term[3].slot == 1


def test_prefix_sequences_and_identical_sequences():
    t = OracleTree(c=4, with_kv=False)
    t.insert(0, [1, 2, 3, 4, 5])
    assert t.insert(1, [1, 2, 3]) == 3          # ends inside a chunk -> split
    assert t.insert(2, [1, 2, 3, 4, 5]) == 5    # identical to seq 0
    t.check_invariants()
    tb = tables(t)
    # X=[1,2,3] shared by 3, X'=[4] by 2 (0 and 2), [5] by 2
    assert list(tb.node_len) == [3, 1, 1]
    assert list(tb.row_seq) == [1, 0, 2]
    assert list(tb.node_row_begin) == [0, 1, 1]
    assert list(tb.node_row_end) == [3, 3, 3]
    assert tb.n_parts == 3 + 2 + 2
    # extend the shared-terminal sequence 1 with [4, 7]: descends X', new [7]
    t.extend(1, [4, 7])
    t.check_invariants()
    tb = tables(t)
    assert list(tb.row_seq) == [0, 2, 1]
    # appending to seq 0 (terminal [5] shared with seq 2) grows a new chunk
    t.append_batch([0, 2], [6, 6])
    t.check_invariants()
    p0 = [len(n) for n in t.path(0)]
    assert p0 == [3, 1, 1, 1] and t.path(0)[-1] is t.path(2)[-1]


def test_pool_exhaustion_changes_nothing():
    t = OracleTree(c=2, num_slots=3, with_kv=False)
    t.insert(0, [1, 2, 3, 4])                  # 2 slots
    before = tables(t).as_dict()
    with pytest.raises(PoolExhausted):
        t.insert(1, [1, 9, 9, 9])              # split (1) + 2 new chunks
    after = tables(t).as_dict()
    for k in before:
        assert np.array_equal(before[k], after[k]), k
    assert t.free == [] and t.fresh == 2
    with pytest.raises(PoolExhausted):
        t.extend(0, [5, 6, 7])                 # needs 2 chunks, 1 available
    t.append_batch([0], [5])                   # needs exactly the last slot
    t.append_batch([0], [6])                   # terminal [5] has room: no slot
    with pytest.raises(PoolExhausted):
        t.append_batch([0], [7])               # terminal full, pool empty
    assert t.length[0] == 6


def test_append_batch_all_or_nothing():
    t = OracleTree(c=1, num_slots=4, with_kv=False)
    t.insert(0, [1])
    t.insert(1, [2])
    t.insert(2, [3])
    snap = tables(t).as_dict()
    with pytest.raises(PoolExhausted):
        t.append_batch([0, 1], [5, 5])         # needs 2, one available
    for k, v in tables(t).as_dict().items():
        assert np.array_equal(snap[k], v)
    t.append_batch([0], [5])


@pytest.mark.parametrize("seed", range(12))
def test_random_scripts_keep_invariants(seed):
    """R10 after every operation, and table consistency with the paths."""
    c = [1, 2, 3, 4][seed % 4]
    t = OracleTree(c=c, with_kv=False)
    for op in random_op_script(seed, n_ops=60):
        if op[0] == "insert":
            t.insert(op[1], op[2])
        elif op[0] == "extend":
            t.extend(op[1], op[2])
        elif op[0] == "append":
            t.append_batch(op[1], op[2])
        else:
            t.remove(op[1])
        t.check_invariants()
        tb = tables(t)
        for r in range(tb.B):
            sid = int(tb.row_seq[r])
            # nodes on the path cover row r; node ranges are contiguous
            path_len = 0
            for i in range(tb.n_nodes):
                if tb.node_row_begin[i] <= r < tb.node_row_end[i]:
                    path_len += int(tb.node_len[i])
            assert path_len == t.length[sid]


# -- prefix lookup (Section 3.2, prefill paragraph) ---------------------------

def test_match_on_fig2_tree_hand_values():
    """Figure 2's tree (c=4; shared 10..21, S0 +30..33, S1 +40..47, S2 +50..57):
    lookups that end inside a shared chunk, at chunk boundaries, inside a
    private chunk, at the end of a path, past it, and on the first token."""
    t = _fig2_tree()
    shared = list(range(10, 22))
    cases = [
        ([10, 11, 12, 99], 3),                          # inside C0
        ([10, 11, 12, 13], 4),                          # end of C0
        (list(range(10, 16)) + [99], 6),                # inside C1
        (shared, 12),                                   # end of the shared run
        (shared + [40, 41, 99], 14),                    # inside C4 (S1's first private chunk)
        (shared + list(range(40, 44)), 16),             # end of C4
        (shared + list(range(40, 48)), 20),             # exactly S1
        (shared + list(range(40, 48)) + [1, 2, 3], 20),  # past S1's path
        (shared + [50, 51, 52, 53, 54, 99], 17),        # inside C7
        (shared + [30, 31, 32, 33, 34], 16),            # past S0
        (shared + [31], 12),                            # no child starts with 31
        ([11, 12], 0),                                  # not a root prefix
        ([99], 0),
        ([10], 1),
    ]
    for probe, want in cases:
        assert t.match(probe) == want, (probe, want)


def test_match_on_split_example_hand_values():
    """c=4, A=[1..6] then B=[1,2,9]; then A leaves: lookups across the split
    node X=[1,2] / X'=[3,4], and after the removal frees X' and Y."""
    t = OracleTree(c=4, with_kv=False)
    t.insert(0, [1, 2, 3, 4, 5, 6])
    assert t.match([1, 2, 3, 7]) == 3          # inside the chunk before any split
    assert t.match([1, 2, 3, 4, 5, 6, 7]) == 6
    t.insert(1, [1, 2, 9])
    assert t.match([1, 2]) == 2                # end of X
    assert t.match([1, 2, 3]) == 3             # inside X'
    assert t.match([1, 2, 3, 4, 7]) == 4       # end of X'
    assert t.match([1, 2, 3, 4, 5, 9]) == 5    # inside Y
    assert t.match([1, 2, 9, 9]) == 3          # past B's path
    assert t.match([1, 9]) == 1
    t.remove(0)
    assert t.match([1, 2, 3]) == 2             # X' and Y were freed
    assert t.match([1, 2, 9]) == 3


def _match_script_check(t, live, rng, alphabet, n_probes=12):
    for p in probes(rng, list(live.values()), n_probes, alphabet):
        assert t.match(p) == max_lcp(live.values(), p), (p, t.match(p))


@pytest.mark.parametrize("seed", range(12))
def test_match_is_longest_common_prefix_with_live_sequences(seed):
    """After every operation of a random script, the lookup of any probe equals
    the longest common prefix of the probe with any live sequence, computed
    by brute force from the sequences' own token lists (no tree)."""
    c = [1, 2, 3, 4, 5, 7][seed % 6]
    alphabet = 2 + seed % 3
    t = OracleTree(c=c, with_kv=False)
    live = {}
    rng = np.random.default_rng(500 + seed)
    for op in random_op_script(seed, n_ops=60, alphabet=alphabet, max_len=3 * c + 4):
        if op[0] == "insert":
            t.insert(op[1], op[2])
            live[op[1]] = np.asarray(op[2], np.int32)
        elif op[0] == "extend":
            t.extend(op[1], op[2])
            live[op[1]] = np.concatenate([live[op[1]], op[2]]).astype(np.int32)
        elif op[0] == "append":
            t.append_batch(op[1], op[2])
            for sid, tok in zip(op[1], op[2]):
                live[sid] = np.concatenate([live[sid], [tok]]).astype(np.int32)
        else:
            t.remove(op[1])
            del live[op[1]]
        _match_script_check(t, live, rng, alphabet)


def _full_chunks_only_match(self, tokens):
    """A plausible mistake: count only fully matched chunks, dropping a
    partial match inside the chunk where the lookup stops."""
    tokens = np.asarray(tokens, np.int32)
    cur, pos = self.root, 0
    while pos < tokens.shape[0]:
        child = cur.children.get(int(tokens[pos]))
        if child is None:
            break
        L = len(child)
        if pos + L > tokens.shape[0] or not np.array_equal(child.tokens, tokens[pos:pos + L]):
            break
        cur, pos = child, pos + L
    return pos


@pytest.mark.parametrize("plant", ["full_chunks_only", "off_by_one"])
def test_plant_match_mistakes_are_caught(monkeypatch, plant):
    """The brute-force and hand-value pins catch a lookup that drops the
    partial match inside the last chunk, and one that is off by one."""
    import oracle.tree as T

    good = T.OracleTree.match
    bad = _full_chunks_only_match if plant == "full_chunks_only" else (
        lambda self, tokens: max(0, good(self, tokens) - 1))
    monkeypatch.setattr(T.OracleTree, "match", bad)
    with pytest.raises(AssertionError):
        test_match_on_fig2_tree_hand_values()
    with pytest.raises(AssertionError):
        test_match_is_longest_common_prefix_with_live_sequences(3)   # c = 4


def test_memory_loss_bound():
    """Section 3.1: a sequence of n tokens wastes at most c-1 slots' rows."""
    rng = np.random.default_rng(7)
    for c in (1, 3, 16, 64):
        for n in (1, 5, 63, 64, 65, 1000):
            t = OracleTree(c=c, with_kv=False)
            t.insert(0, rng.integers(0, 100, n))
            used = t.slots_in_use()
            assert 0 <= used * c - n <= c - 1
            assert used == -(-n // c)
            # decode appends keep the bound
            t.append_batch([0], [1])
            assert t.slots_in_use() * c - (n + 1) <= c - 1


def _build_static(wl, with_kv):
    t = OracleTree(c=wl.c, with_kv=with_kv)
    for s in wl.seqs:
        toks = s.tokens(wl.segments)
        if with_kv:
            k, v = s.kv(wl.segments)
            t.insert(s.seq_id, toks, k, v)
        else:
            t.insert(s.seq_id, toks)
    return t


@pytest.mark.parametrize("cfg,nodes,shared,parts", [
    (1, 16, 8, 8 * 4),
    (2, 272, 16, 16 * 32),
    (3, 320, 64, 64 * 32),
    (4, 352, 96, 2 * 16 * 32 + 4 * 16 * 16),
])
def test_static_config_closed_forms(cfg, nodes, shared, parts):
    wl = make_static(cfg)
    t = _build_static(wl, with_kv=False)
    t.check_invariants()
    tb = tables(t)
    assert tb.n_nodes == nodes
    assert tb.shr_node.shape[0] == shared
    assert tb.n_parts == parts
    assert list(tb.row_seq) == list(range(wl.B)) or sorted(tb.row_seq) == list(range(wl.B))


def test_dynamic_config_initial_closed_form():
    wl = make_dynamic()
    t = OracleTree(c=wl.c, with_kv=False)
    for s in wl.seqs:
        t.insert(s.seq_id, s.tokens(wl.segments))
    tb = tables(t)
    u = [len(wl.segments[s.segs[1]]) for s in wl.seqs]
    assert all(64 <= x <= 1024 for x in u)
    assert tb.n_nodes == 32 + sum(-(-x // 64) for x in u)
    assert tb.shr_node.shape[0] == 32
    assert tb.n_parts == 32 * 128


# -- attention pins ----------------------------------------------------------

def _sdpa(q, k, v, scale):
    """torch's scaled_dot_product_attention in float64 on the CPU: q [H,d], k/v [L,H,d]."""
    qq = torch.from_numpy(np.ascontiguousarray(q, np.float64))[:, None, :]      # H,1,d
    kk = torch.from_numpy(np.ascontiguousarray(k.transpose(1, 0, 2), np.float64))  # H,L,d
    vv = torch.from_numpy(np.ascontiguousarray(v.transpose(1, 0, 2), np.float64))
    o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=scale)
    return o[:, 0, :].numpy()


def test_dense_matches_library_attention_without_tree():
    """Brute force: per-sequence K/V straight from the generator, no tree."""
    wl = make_static(1)
    t = _build_static(wl, with_kv=True)
    tb = tables(t)
    q_rows = wl.q[tb.row_seq]
    o = dense_attention(t, tb.row_seq, q_rows, wl.scale)
    for r, sid in enumerate(tb.row_seq):
        k, v = wl.seqs[sid].kv(wl.segments)
        ref = _sdpa(wl.q[sid].astype(np.float64), k.astype(np.float64), v.astype(np.float64), wl.scale)
        np.testing.assert_allclose(o[r], ref, rtol=0, atol=1e-12)
        # the tree stores exactly the sequence's rows, in order
        pk, pv = path_kv(t, int(sid))
        assert np.array_equal(pk, k.astype(np.float64)) and np.array_equal(pv, v.astype(np.float64))


def test_default_scale_is_inverse_sqrt_d():
    """The experiments' formula divides by sqrt(d): torch's default scale."""
    wl = make_static(1)
    t = _build_static(wl, with_kv=True)
    tb = tables(t)
    sid = int(tb.row_seq[0])
    k, v = wl.seqs[sid].kv(wl.segments)
    qq = torch.from_numpy(wl.q[sid].astype(np.float64))[:, None, :]
    kk = torch.from_numpy(k.astype(np.float64).transpose(1, 0, 2).copy())
    vv = torch.from_numpy(v.astype(np.float64).transpose(1, 0, 2).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv)[:, 0].numpy()
    o = dense_attention_rows(t, tb.row_seq, wl.q[tb.row_seq], 1.0 / np.sqrt(wl.d), rows=[0])
    np.testing.assert_allclose(o[0], ref, rtol=0, atol=1e-12)


def test_chunk_size_invariance():
    wl = make_static(1)
    outs = []
    for c in (1, 2, 3, 5, 16, 64, 1000):
        t = OracleTree(c=c, with_kv=True)
        for s in wl.seqs:
            k, v = s.kv(wl.segments)
            t.insert(s.seq_id, s.tokens(wl.segments), k, v)
        tb = tables(t)
        o = dense_attention(t, tb.row_seq, wl.q[tb.row_seq], wl.scale)
        outs.append(o[np.argsort(tb.row_seq)])
    for o in outs[1:]:
        np.testing.assert_allclose(o, outs[0], rtol=0, atol=1e-12)


def test_structured_eqn1_eqn2_equals_dense():
    """Algorithms 1+2 (Eqn 1 per chunk, Eqn 2 merge, O/n) reach the dense result."""
    for c in (3, 16):
        wl = make_static(1)
        t = OracleTree(c=c, with_kv=True)
        for s in wl.seqs:
            k, v = s.kv(wl.segments)
            t.insert(s.seq_id, s.tokens(wl.segments), k, v)
        tb = tables(t)
        q = wl.q[tb.row_seq]
        np.testing.assert_allclose(structured_attention(t, tb.row_seq, q, wl.scale),
                                   dense_attention(t, tb.row_seq, q, wl.scale), rtol=1e-12, atol=1e-13)


def test_weights_sum_to_one_and_outputs_in_hull():
    wl = make_static(1)
    t = _build_static(wl, with_kv=True)
    tb = tables(t)
    q = wl.q[tb.row_seq] * 3.0
    o = dense_attention(t, tb.row_seq, q, wl.scale)
    for r, sid in enumerate(tb.row_seq):
        _, v = path_kv(t, int(sid))
        assert np.all(o[r] >= v.min(axis=0) - 1e-12) and np.all(o[r] <= v.max(axis=0) + 1e-12)
    # V = 1 everywhere -> output exactly 1 (weights sum to one)
    for n in t.nodes():
        n.v = np.ones_like(n.v)
    o1 = dense_attention(t, tb.row_seq, q, wl.scale)
    np.testing.assert_allclose(o1, 1.0, rtol=0, atol=1e-14 * 160)


def test_special_cases():
    rng = np.random.default_rng(3)
    H, d = 2, 8
    t = OracleTree(c=4)
    k = rng.standard_normal((1, H, d))
    v = rng.standard_normal((1, H, d))
    t.insert(0, [5], k, v)                      # one token: o = v
    o = dense_attention(t, np.array([0]), rng.standard_normal((1, H, d)), 0.3)
    np.testing.assert_allclose(o[0], v[0], rtol=0, atol=1e-15)

    t = OracleTree(c=4)
    L = 11
    k = rng.standard_normal((L, H, d))
    v = rng.standard_normal((L, H, d))
    t.insert(0, np.arange(L), k, v)
    o = dense_attention(t, np.array([0]), np.zeros((1, H, d)), 0.3)   # q = 0: mean of V
    np.testing.assert_allclose(o[0], v.mean(axis=0), rtol=0, atol=1e-14)

    q = rng.standard_normal((1, H, d))
    k2 = k.copy()
    # key 7 scores 60 for both heads; the others score |q||k| < 15 here, so
    # every other weight is below exp(-45) and o equals v[7] to ~1e-19
    k2[7] = q[0] * (60.0 / np.sum(q[0] ** 2, axis=1, keepdims=True))
    others = np.einsum("lhd,hd->lh", np.delete(k2, 7, axis=0), q[0])
    assert others.max() < 15.0
    t = OracleTree(c=4)
    t.insert(0, np.arange(L), k2, v)            # spike key: o ~= v[7]
    o = dense_attention(t, np.array([0]), q, 1.0)
    np.testing.assert_allclose(o[0], v[7], rtol=0, atol=1e-17)

    t = OracleTree(c=4)                          # identical sequences
    t.insert(0, np.arange(L), k, v)
    t.insert(1, np.arange(L), k, v)
    qq = np.repeat(q, 2, axis=0)
    o = dense_attention(t, tables(t).row_seq, qq, 0.3)
    assert np.array_equal(o[0], o[1])


def test_random_trees_with_prefix_keyed_kv():
    """Collisions and splits: the path K/V is always the sequence's own K/V."""
    H, d = 2, 8
    for seed in range(6):
        c = 1 + seed % 4
        t = OracleTree(c=c)
        full = {}
        for op in random_op_script(100 + seed, n_ops=40):
            if op[0] == "insert":
                toks = op[2]
                k, v = prefix_keyed_kv(seed, toks, 0, H, d, np.float64)
                t.insert(op[1], toks, k, v)
                full[op[1]] = toks
            elif op[0] == "extend":
                toks = np.concatenate([full[op[1]], op[2]])
                k, v = prefix_keyed_kv(seed, toks, len(full[op[1]]), H, d, np.float64)
                t.extend(op[1], op[2], k, v)
                full[op[1]] = toks
            elif op[0] == "append":
                ks, vs = [], []
                for sid, tok in zip(op[1], op[2]):
                    toks = np.concatenate([full[sid], [tok]]).astype(np.int32)
                    k, v = prefix_keyed_kv(seed, toks, len(full[sid]), H, d, np.float64)
                    ks.append(k)
                    vs.append(v)
                    full[sid] = toks
                t.append_batch(op[1], op[2], np.concatenate(ks), np.concatenate(vs))
            else:
                t.remove(op[1])
                del full[op[1]]
            t.check_invariants()
        for sid, toks in full.items():
            k, v = prefix_keyed_kv(seed, toks, 0, H, d, np.float64)
            pk, pv = path_kv(t, sid)
            assert np.array_equal(pk, k) and np.array_equal(pv, v)


def test_b1_has_no_shared_chunks():
    wl = make_static(1)
    t = OracleTree(c=16)
    s = wl.seqs[0]
    k, v = s.kv(wl.segments)
    t.insert(0, s.tokens(wl.segments), k, v)
    tb = tables(t)
    assert tb.shr_node.shape[0] == 0 and tb.n_parts == 0
    assert list(tb.priv_node) == list(range(tb.n_nodes))


def test_plant_eqn2_swap_is_caught(monkeypatch):
    """A swapped rescale in Eqn 2 (x <-> y) must break the structured check."""
    import oracle.attention as A

    def bad_reduce(o_c, m_c, n_c, O, m, n):
        mx = max(m_c, m)
        x = np.exp(m_c - mx)
        y = np.exp(m - mx)
        return y * o_c + x * O, mx, y * n_c + x * n

    wl = make_static(1)
    t = OracleTree(c=16)
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        t.insert(s.seq_id, s.tokens(wl.segments), k, v)
    tb = tables(t)
    q = wl.q[tb.row_seq]
    good = A.structured_attention(t, tb.row_seq, q, wl.scale)
    monkeypatch.setattr(A, "attn_reduce", bad_reduce)
    bad = A.structured_attention(t, tb.row_seq, q, wl.scale)
    assert np.abs(bad - good).max() > 1e-3


# -- prefill with prefix reuse (Section 3.2, prefill paragraph) --------------

def _prefill_case(c, n_shared=40, n_new=23, H=2, d=16, seed=3):
    """A tree where a second sequence reuses the first one's prefix."""
    rng = np.random.default_rng(seed)
    shared = rng.integers(0, 100, n_shared).astype(np.int32)
    a = np.concatenate([shared, rng.integers(100, 200, 9).astype(np.int32)])
    b = np.concatenate([shared, rng.integers(200, 300, n_new).astype(np.int32)])
    t = OracleTree(c=c, with_kv=True)
    ka, va = prefix_keyed_kv(seed, a, 0, H, d, np.float64)
    kb, vb = prefix_keyed_kv(seed, b, 0, H, d, np.float64)
    t.insert(0, a, ka, va)
    t.insert(1, b, kb, vb)
    q = rng.standard_normal((n_new, H, d))
    return t, b, kb, vb, q


def _sdpa_masked(q, k, v, mask, scale):
    """torch SDPA in float64: q [n, H, d], k/v [L, H, d], mask [n, L] (True = attend)."""
    qq = torch.from_numpy(q.transpose(1, 0, 2).copy())
    kk = torch.from_numpy(k.transpose(1, 0, 2).copy())
    vv = torch.from_numpy(v.transpose(1, 0, 2).copy())
    o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, attn_mask=torch.from_numpy(mask),
                                                         scale=scale)
    return o.numpy().transpose(1, 0, 2)


def test_prefill_matches_masked_library_attention():
    """Suffix queries over prefix + suffix: torch SDPA with a position mask."""
    for c in (1, 4, 7, 64):
        t, toks, k, v, q = _prefill_case(c)
        L, n = len(toks), q.shape[0]
        mask = np.arange(L)[None, :] <= (L - n + np.arange(n))[:, None]
        ref = _sdpa_masked(q, k, v, mask, 0.25)
        o = prefill_attention(t, 1, q, 0.25)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def test_prefill_whole_prompt_is_causal_attention():
    """n_q = L (nothing matched): SDPA's own causal mode."""
    rng = np.random.default_rng(5)
    toks = rng.integers(0, 50, 37).astype(np.int32)
    k, v = prefix_keyed_kv(5, toks, 0, 3, 8, np.float64)
    t = OracleTree(c=5, with_kv=True)
    t.insert(0, toks, k, v)
    q = rng.standard_normal((37, 3, 8))
    qq = torch.from_numpy(q.transpose(1, 0, 2).copy())
    ref = torch.nn.functional.scaled_dot_product_attention(
        qq, torch.from_numpy(k.transpose(1, 0, 2).copy()), torch.from_numpy(v.transpose(1, 0, 2).copy()),
        is_causal=True).numpy().transpose(1, 0, 2)
    np.testing.assert_allclose(prefill_attention(t, 0, q, 1 / np.sqrt(8)), ref, rtol=0, atol=1e-12)


def test_prefill_last_query_is_decode_attention():
    """The last query sees the whole sequence: the decode result of that row."""
    t, toks, k, v, q = _prefill_case(4)
    tb = tables(t)
    r = int(np.nonzero(tb.row_seq == 1)[0][0])
    qrows = np.zeros((len(tb.row_seq),) + q.shape[1:])
    qrows[r] = q[-1]
    dec = dense_attention_rows(t, tb.row_seq, qrows, 0.3, rows=[r])
    pre = prefill_attention(t, 1, q, 0.3, queries=[q.shape[0] - 1])
    np.testing.assert_allclose(pre, dec, rtol=0, atol=1e-13)


def test_prefill_first_token_query_sees_only_itself():
    """Query at position 0 (n_q = L) attends to one token: o = v_0 exactly."""
    t, toks, k, v, q = _prefill_case(4)
    L = len(toks)
    qq = np.random.default_rng(1).standard_normal((L, 2, 16))
    o = prefill_attention(t, 1, qq, 0.5, queries=[0])
    np.testing.assert_allclose(o[0], v[0], rtol=0, atol=1e-15)


def test_plant_off_by_one_causal_mask_is_caught(monkeypatch):
    """A mask that also shows the next token must fail the SDPA pin."""
    import oracle.attention as A

    real = A._softmax_attend
    t, toks, k, v, q = _prefill_case(4)
    L, n = len(toks), q.shape[0]

    def leaky(qv, kk, vv, scale):
        # one extra row beyond the causal limit whenever one exists
        m = kk.shape[0]
        if m < L:
            kk, vv = k[: m + 1], v[: m + 1]
        return real(qv, kk, vv, scale)

    monkeypatch.setattr(A, "_softmax_attend", leaky)
    mask = np.arange(L)[None, :] <= (L - n + np.arange(n))[:, None]
    ref = _sdpa_masked(q, k, v, mask, 0.25)
    o = A.prefill_attention(t, 1, q, 0.25)
    assert np.abs(o - ref).max() > 1e-3
