"""GPU parity: the HIP library against the float64 oracle.

Tables and pool contents must match bit-exactly (they are copies); outputs
must be within max-abs 2e-3 and rel-L2 1e-3 for fp16 inputs (fp32
accumulation) and within 2e-5 / 1e-5 for fp32 inputs.
"""
import time

import numpy as np
import pytest
import torch

from parity_util import Pair, assert_close, host_threads, to_dev
from paper_2402_15220_amd import binding as B
from workloads import make_dynamic, make_static, prefix_keyed_kv, random_op_script

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.load()
    yield


def _static_pair(wl, slack=16, layout="interleaved"):
    nodes = sum(-(-len(s) // wl.c) for s in wl.segments)  # aligned configs: one chunk set per segment
    p = Pair(wl.c, wl.H, wl.d, wl.dtype, nodes + slack, layout=layout)
    seg_dev = [(to_dev(s.k), to_dev(s.v)) for s in wl.segments]
    for s in wl.seqs:
        toks = s.tokens(wl.segments)
        k, v = s.kv(wl.segments)
        dk = torch.cat([seg_dev[i][0] for i in s.segs])
        dv = torch.cat([seg_dev[i][1] for i in s.segs])
        p.insert(s.seq_id, toks, k, v, dev_k=dk, dev_v=dv)
    return p


@pytest.mark.parametrize("cfg,layout", [(1, "split"), (2, "split"), (3, "split"), (4, "split"),
                                        (1, "interleaved"), (2, "interleaved"), (3, "interleaved"),
                                        (4, "interleaved")])
def test_static_config(cfg, layout):
    """Full-size static trees; K/V pools split and interleaved (the default)."""
    wl = make_static(cfg)
    print(f"[case] {wl.name} layout={layout}", flush=True)
    p = _static_pair(wl, layout=layout)
    tb = p.check_tables()
    p.check_pool()
    o, q, row_seq = p.attention({s.seq_id: wl.q[s.seq_id] for s in wl.seqs})
    ref = p.reference(row_seq, q, 0.0)
    assert_close(o, ref, wl.dtype, f"{wl.name} (B={tb['row_seq'].shape[0]})")


@pytest.mark.parametrize("seg,split,sched", [(1, 0, 0), (16, 0, 0), (4, 3, 0), (2, 1, 0), (64, 5, 0),
                                             (1, 0, 1), (4, 0, 1), (16, 3, 1), (3, 1, 1),
                                             (1, 0, 2), (8, 0, 2), (16, 2, 2), (64, 1, 2), (4, 0, 3), (16, 3, 3),
                                             (-1, 0, 4), (1, 0, 4), (5, 3, 4)])
def test_config2_work_partitions(seg, split, sched):
    """Every schedule, segment size and split gives the same result, and
    repeated calls (counters reset by the kernels) stay correct."""
    print(f"[case] single-prompt tree seg={seg} split={split} schedule={sched}", flush=True)
    wl = make_static(2)
    p = _static_pair(wl)
    p.cache.set_tuning(seg_chunks=seg, split_chunks=split, schedule=sched)
    for rep in range(3):
        o, q, row_seq = p.attention({s.seq_id: wl.q[s.seq_id] for s in wl.seqs})
        ref = p.reference(row_seq, q, 0.0) if rep == 0 else ref
        assert_close(o, ref, wl.dtype, f"single-prompt tree seg={seg} split={split} schedule={sched} rep={rep}")


@pytest.mark.parametrize("cfg,seg", [(3, -1), (4, -1), (4, 1)])
def test_partial_free_multi_level(cfg, seg):
    """The partial-free schedule on trees with several levels of sharing:
    rows fold segments of different levels into one accumulator, one launch
    per position along the path."""
    wl = make_static(cfg)
    print(f"[case] {wl.name} schedule 4 seg={seg}", flush=True)
    p = _static_pair(wl)
    p.cache.set_tuning(seg_chunks=seg, schedule=4)
    for rep in range(2):
        o, q, row_seq = p.attention({s.seq_id: wl.q[s.seq_id] for s in wl.seqs})
        ref = p.reference(row_seq, q, 0.0) if rep == 0 else ref
        assert_close(o, ref, wl.dtype, f"{wl.name} schedule 4 seg={seg} rep={rep}")


@pytest.mark.timeout(900)
def test_config5_dynamic_decode():
    """64 decode steps over 128 rows with churn (13 rows leave and 13 join
    before steps 16, 32 and 48): tables bit-exact after every step, every
    row of every step against the oracle, and the pool rows of every live
    node at steps 0, 16, 17, 32, 48 and 63 (right after each churn event and
    the step after one)."""
    print("[case] 64-step decode with churn, 128 rows", flush=True)
    t_start = time.time()
    wl = make_dynamic()
    p = Pair(wl.c, wl.H, wl.d, wl.dtype, 2600)
    seg_dev = {}

    def dev_seg(i):
        if i not in seg_dev:
            seg_dev[i] = (to_dev(wl.segments[i].k), to_dev(wl.segments[i].v))
        return seg_dev[i]

    def insert(s):
        toks = s.tokens(wl.segments)
        k, v = s.kv(wl.segments)
        dk = torch.cat([dev_seg(i)[0] for i in s.segs])
        dv = torch.cat([dev_seg(i)[1] for i in s.segs])
        p.insert(s.seq_id, toks, k, v, dev_k=dk, dev_v=dv)

    for s in wl.seqs:
        insert(s)
    worst = (0.0, 0.0, -1)
    row_steps = 0
    pool_nodes = 0
    uploads_before = p.cache.stats()["uploads"]
    t_oracle = 0.0
    for st in wl.steps():
        if st.churn:
            for sid in st.churn.removed:
                p.remove(sid)
            for s in st.churn.added:
                insert(s)
        p.append(st.live, st.tokens, st.k, st.v)
        p.check_tables()
        qmap = {int(sid): st.q[i] for i, sid in enumerate(st.live)}
        o, q, row_seq = p.attention(qmap)
        t0 = time.time()
        ref = p.reference(row_seq, q, 0.0)
        t_oracle += time.time() - t0
        ma, rel = assert_close(o, ref, wl.dtype, f"decode step {st.step} (all {len(row_seq)} rows)")
        row_steps += len(row_seq)
        if ma > worst[0] or rel > worst[1]:
            worst = (max(worst[0], ma), max(worst[1], rel), st.step)
        if st.step in (0, 16, 17, 32, 48, 63):
            p.check_pool()
            pool_nodes += len(p.tree.nodes())
    print(f"[parity] 64-step decode: {row_steps} row-steps, worst max_abs={worst[0]:.3e} "
          f"rel_l2={worst[1]:.3e} (step {worst[2]}); pools of {pool_nodes} live nodes bit-exact; "
          f"uploads={p.cache.stats()['uploads'] - uploads_before}; oracle {t_oracle:.1f} s on "
          f"{host_threads()} threads; test {time.time() - t_start:.1f} s", flush=True)


@pytest.mark.parametrize("seed", range(16))
def test_random_trees(seed):
    """Small trees with collisions, splits, partial chunks, removals."""
    rng = np.random.default_rng(seed)
    c = [1, 2, 3, 4, 5, 16, 64, 7][seed % 8]
    d = [64, 128][seed % 2]
    dtype = [np.float16, np.float32][(seed // 2) % 2]
    H = 1 + seed % 3
    print(f"[case] random tree seed={seed} c={c} d={d} H={H} dtype={np.dtype(dtype).name}", flush=True)
    p = Pair(c, H, d, dtype, 4096, layout="interleaved" if seed % 5 == 2 else "split")
    if seed % 3 == 1:  # the partial-free schedule, one segment per chunk or per run
        p.cache.set_tuning(seg_chunks=1 if seed % 2 else -1, schedule=4)
    full = {}
    qrng = np.random.default_rng(1000 + seed)
    ops = random_op_script(seed, n_ops=50, alphabet=3, max_len=max(12, 2 * c + 3))
    for i, op in enumerate(ops):
        if op[0] == "insert":
            k, v = prefix_keyed_kv(seed, op[2], 0, H, d, dtype)
            p.insert(op[1], op[2], k, v)
            full[op[1]] = np.asarray(op[2], np.int32)
        elif op[0] == "extend":
            toks = np.concatenate([full[op[1]], op[2]]).astype(np.int32)
            k, v = prefix_keyed_kv(seed, toks, len(full[op[1]]), H, d, dtype)
            p.extend(op[1], op[2], k, v)
            full[op[1]] = toks
        elif op[0] == "append":
            ks, vs = [], []
            for sid, tok in zip(op[1], op[2]):
                toks = np.concatenate([full[sid], [tok]]).astype(np.int32)
                k, v = prefix_keyed_kv(seed, toks, len(full[sid]), H, d, dtype)
                ks.append(k)
                vs.append(v)
                full[sid] = toks
            p.append(op[1], op[2], np.concatenate(ks), np.concatenate(vs))
        else:
            p.remove(op[1])
            del full[op[1]]
        if full and (i % 5 == 4 or i == len(ops) - 1):
            p.check_tables()
            p.check_pool()
            qmap = {sid: qrng.standard_normal((H, d)).astype(np.float32).astype(dtype) for sid in full}
            o, q, row_seq = p.attention(qmap)
            ref = p.reference(row_seq, q, 0.0)
            assert_close(o, ref, dtype, f"random tree seed={seed} op={i}")


def _run_script(p, seed, ops, H, d, dtype, label, every=5):
    """Apply a random operation script to the pair; check tables and parity
    every `every` operations and after the last."""
    full = {}
    qrng = np.random.default_rng(2000 + seed)
    for i, op in enumerate(ops):
        if op[0] == "insert":
            k, v = prefix_keyed_kv(seed, op[2], 0, H, d, dtype)
            p.insert(op[1], op[2], k, v)
            full[op[1]] = np.asarray(op[2], np.int32)
        elif op[0] == "extend":
            toks = np.concatenate([full[op[1]], op[2]]).astype(np.int32)
            k, v = prefix_keyed_kv(seed, toks, len(full[op[1]]), H, d, dtype)
            p.extend(op[1], op[2], k, v)
            full[op[1]] = toks
        elif op[0] == "append":
            ks, vs = [], []
            for sid, tok in zip(op[1], op[2]):
                toks = np.concatenate([full[sid], [tok]]).astype(np.int32)
                k, v = prefix_keyed_kv(seed, toks, len(full[sid]), H, d, dtype)
                ks.append(k)
                vs.append(v)
                full[sid] = toks
            p.append(op[1], op[2], np.concatenate(ks), np.concatenate(vs))
        else:
            p.remove(op[1])
            del full[op[1]]
        if full and (i % every == every - 1 or i == len(ops) - 1):
            p.check_tables()
            qmap = {sid: qrng.standard_normal((H, d)).astype(np.float32).astype(dtype) for sid in full}
            o, q, row_seq = p.attention(qmap)
            ref = p.reference(row_seq, q, 0.0)
            assert_close(o, ref, dtype, f"{label} op={i}")


@pytest.mark.parametrize("c,dtype", [(128, np.float16), (100, np.float16), (65, np.float32),
                                     (200, np.float16)])
def test_random_trees_long_chunks(c, dtype):
    """Chunks longer than the kernels' 64-token blocks: every chunk spans
    several blocks, the last one ragged (c=100 under the partial-free
    schedule)."""
    seed = 40 + c
    d, H = 128 if c % 2 == 0 else 64, 2
    print(f"[case] long chunks c={c} dtype={np.dtype(dtype).name}", flush=True)
    p = Pair(c, H, d, dtype, 1024)
    if c == 100:  # the partial-free schedule, one segment per chunk
        p.cache.set_tuning(seg_chunks=1, schedule=4)
    ops = random_op_script(seed, n_ops=30, alphabet=3, max_len=2 * c + 40)
    _run_script(p, seed, ops, H, d, dtype, f"long chunks c={c}")


@pytest.mark.parametrize("case", range(4))
def test_random_trees_large(case):
    """Larger trees: up to 48 live sequences of up to a few hundred tokens over
    a 4-token alphabet (deep sharing, many splits and removals), 200
    operations, under the default schedule with automatic segments, split
    rows, and the partial-free schedule."""
    seed = 300 + case
    c = [8, 32, 16, 64][case]
    H, d = 4, 128
    tuning = [dict(), dict(split_chunks=2), dict(seg_chunks=2, schedule=4), dict(schedule=0)][case]
    print(f"[case] large random tree c={c} tuning={tuning}", flush=True)
    p = Pair(c, H, d, np.float16, 8192)
    if tuning:
        p.cache.set_tuning(**tuning)
    ops = random_op_script(seed, n_ops=200, alphabet=4, max_len=80, max_live=48,
                           p_insert=0.3, p_extend=0.25, p_append=0.3)
    _run_script(p, seed, ops, H, d, np.float16, f"large tree c={c}", every=20)


@pytest.mark.parametrize("sched", [0, 1, 2, 4])
def test_deep_tree_many_partials(sched):
    """A comb of 80 sequences, sequence k sharing its first k two-token chunks
    with every longer one: each chunk covers a different row range, so with
    one chunk per segment the longest rows fold 79 partials (more than one
    64-wide batch of the merge)."""
    print(f"[case] deep tree schedule={sched}", flush=True)
    c, H, d = 2, 2, 64
    rng = np.random.default_rng(77)
    base = rng.integers(0, 30, 2 * 80).astype(np.int32)
    p = Pair(c, H, d, np.float16, 4096)
    for k in range(1, 81):
        toks = np.concatenate([base[:2 * k], [1000 + k]]).astype(np.int32)
        kk, vv = prefix_keyed_kv(77, toks, 0, H, d, np.float16)
        p.insert(k, toks, kk, vv)
    p.cache.set_tuning(seg_chunks=1, split_chunks=0, schedule=sched)
    p.check_tables()
    qrng = np.random.default_rng(78)
    qmap = {k: qrng.standard_normal((H, d)).astype(np.float16) for k in range(1, 81)}
    for rep in range(2):
        o, q, row_seq = p.attention(qmap)
        ref = p.reference(row_seq, q, 0.0) if rep == 0 else ref
        assert_close(o, ref, np.float16, f"deep tree schedule={sched} rep={rep}")


def _small_pair(c=4, H=2, d=64, dtype=np.float16):
    return Pair(c, H, d, dtype, 256)


def _kv(rng, n, H, d, dtype):
    k = rng.standard_normal((n, H, d)).astype(np.float32).astype(dtype)
    v = rng.standard_normal((n, H, d)).astype(np.float32).astype(dtype)
    return k, v


@pytest.mark.parametrize("dtype", [np.float16, np.float32])
def test_edge_cases(dtype):
    print(f"[case] edge cases {np.dtype(dtype).name}", flush=True)
    rng = np.random.default_rng(11)
    H, d = 2, 128
    # B = 1: no shared chunks, plain decode attention
    p = _small_pair(c=16, H=H, d=d, dtype=dtype)
    k, v = _kv(rng, 37, H, d, dtype)
    p.insert(0, np.arange(37), k, v)
    q = {0: rng.standard_normal((H, d)).astype(dtype)}
    o, qq, rs = p.attention(q)
    assert_close(o, p.reference(rs, qq, 0.0), dtype, "B=1")
    # single-token sequences, all distinct (n_s = 0): o = v
    p = _small_pair(c=4, H=H, d=d, dtype=dtype)
    for sid in range(5):
        k, v = _kv(rng, 1, H, d, dtype)
        p.insert(sid, [100 + sid], k, v)
    o, qq, rs = p.attention({sid: rng.standard_normal((H, d)).astype(dtype) for sid in range(5)})
    for r, sid in enumerate(rs):
        np.testing.assert_allclose(o[r].astype(np.float64), p.tree.term[int(sid)].v[0].astype(np.float64),
                                   atol=1e-6)
    # identical sequences with identical q: identical outputs, every chunk shared
    p = _small_pair(c=4, H=H, d=d, dtype=dtype)
    k, v = _kv(rng, 13, H, d, dtype)
    for sid in range(4):
        p.insert(sid, np.arange(13), k, v)
    qv = rng.standard_normal((H, d)).astype(dtype)
    o, qq, rs = p.attention({sid: qv for sid in range(4)})
    assert_close(o, p.reference(rs, qq, 0.0), dtype, "identical")
    assert np.array_equal(o[0], o[1]) and np.array_equal(o[0], o[3])
    # q = 0 gives the mean of V; a spike key gives that key's V
    p = _small_pair(c=5, H=H, d=d, dtype=dtype)
    k, v = _kv(rng, 23, H, d, dtype)
    qv = rng.standard_normal((H, d)).astype(np.float32)
    k[9] = (qv * (60.0 * np.sqrt(d) / np.sum(qv ** 2, axis=1, keepdims=True))).astype(dtype)
    p.insert(0, np.arange(23), k, v)
    p.insert(1, np.concatenate([np.arange(11), [99, 98]]), *_kv(rng, 13, H, d, dtype))
    o, qq, rs = p.attention({0: np.zeros((H, d), dtype), 1: qv.astype(dtype)})
    assert_close(o, p.reference(rs, qq, 0.0), dtype, "q=0 / spike")
    r0 = int(np.where(rs == 0)[0][0])
    v0 = np.concatenate([n.v for n in p.tree.path(0)]).astype(np.float64)
    np.testing.assert_allclose(o[r0].astype(np.float64), v0.mean(axis=0),
                               atol=2e-3 if dtype == np.float16 else 1e-5)
    # a sequence that is a prefix of another ends inside a shared chunk
    p = _small_pair(c=8, H=H, d=d, dtype=dtype)
    toks = np.arange(20)
    kk, vv = prefix_keyed_kv(3, toks, 0, H, d, dtype)
    p.insert(0, toks, kk, vv)
    p.insert(1, toks[:11], kk[:11], vv[:11])
    p.insert(2, toks[:3], kk[:3], vv[:3])
    o, qq, rs = p.attention({sid: rng.standard_normal((H, d)).astype(dtype) for sid in range(3)})
    assert_close(o, p.reference(rs, qq, 0.0), dtype, "prefix sequences")
    # non-default scale
    o, qq, rs = p.attention({sid: rng.standard_normal((H, d)).astype(dtype) for sid in range(3)}, scale=0.37)
    assert_close(o, p.reference(rs, qq, 0.37), dtype, "scale 0.37")


@pytest.mark.parametrize("c,d", [(64, 128), (128, 128), (32, 64)])
def test_chunk_first_only_calls(c, d):
    """Identical prompts, so every chunk is shared and the call is chunk-first
    work alone (its own launch, several chains of chunks per block), with
    segments of 1, 2, 3 and 5 chunks and the automatic length (chains with
    no chunk, uneven chains), 20 rows (a second row block of 4 rows) and a
    partial last chunk."""
    print(f"[case] chunk-first-only calls c={c} d={d}", flush=True)
    rng = np.random.default_rng(31 + c + d)
    H, n, rows = 4, 700, 20
    p = Pair(c, H, d, np.float16, 64)
    k, v = _kv(rng, n, H, d, np.float16)
    for sid in range(rows):
        p.insert(sid, np.arange(n), k, v)
    qmap = {sid: rng.standard_normal((H, d)).astype(np.float16) for sid in range(rows)}
    ref = None
    for sched in (2, 1):
        for seg in (1, 2, 3, 5, -1):
            p.cache.set_tuning(seg_chunks=seg, schedule=sched)
            o, qq, rs = p.attention(qmap)
            if ref is None:
                ref = p.reference(rs, qq, 0.0)
            assert_close(o, ref, np.float16, f"chunk-first only c={c} d={d} schedule={sched} seg={seg}")


def test_workspace_is_checked():
    rng = np.random.default_rng(2)
    p = _small_pair()
    k, v = _kv(rng, 9, 2, 64, np.float16)
    p.insert(0, np.arange(9), k, v)
    p.insert(1, np.arange(9), k, v)
    need = B.ca_workspace_size(p.cache.h)
    assert need > 0
    q = to_dev(rng.standard_normal((2, 2, 64)).astype(np.float16))
    o = torch.empty_like(q)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.ChunkAttnError) as ei:
        B.ca_attention(p.cache.h, q.data_ptr(), o.data_ptr(), 0.0, ws.data_ptr(), need - 1,
                       torch.cuda.current_stream().cuda_stream)
    assert ei.value.status == B.CA_ERR_WORKSPACE
    B.ca_attention(p.cache.h, q.data_ptr(), o.data_ptr(), 0.0, ws.data_ptr(), need,
                   torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()


def test_lazy_context_upload():
    """Section 3.3: the context is re-uploaded only after structural changes."""
    rng = np.random.default_rng(4)
    H, d = 2, 64
    p = _small_pair(c=4, H=H, d=d)
    k, v = _kv(rng, 6, H, d, np.float16)
    p.insert(0, np.arange(6), k, v)
    p.insert(1, np.concatenate([np.arange(4), [50, 51]]), k, v)
    qmap = lambda: {s: rng.standard_normal((H, d)).astype(np.float16) for s in (0, 1)}  # noqa: E731
    p.attention(qmap())
    u0 = p.cache.stats()["uploads"]
    p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0          # nothing changed
    p.append([0, 1], [7, 7], *_kv(rng, 2, H, d, np.float16))   # fills private chunks
    o, qq, rs = p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0          # lengths live on the device
    assert_close(o, p.reference(rs, qq, 0.0), np.float16, "after in-place append")
    p.append([0, 1], [8, 8], *_kv(rng, 2, H, d, np.float16))   # fills the last free rows
    o, qq, rs = p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0
    p.append([0, 1], [9, 9], *_kv(rng, 2, H, d, np.float16))   # chunks full -> new chunks
    o, qq, rs = p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0 + 1
    assert_close(o, p.reference(rs, qq, 0.0), np.float16, "after chunk growth")


def test_prepare_moves_the_context_upload():
    """Section 3.3 (latency hiding): ca_prepare builds and uploads the context
    ahead of the attention call, which then uploads nothing; a second prepare
    with no tree change does nothing."""
    rng = np.random.default_rng(5)
    H, d = 2, 64
    p = _small_pair(c=4, H=H, d=d)
    k, v = _kv(rng, 6, H, d, np.float16)
    p.insert(0, np.arange(6), k, v)
    p.insert(1, np.concatenate([np.arange(4), [50, 51]]), k, v)
    qmap = lambda: {s: rng.standard_normal((H, d)).astype(np.float16) for s in (0, 1)}  # noqa: E731
    assert p.cache.prepare()
    u0 = p.cache.stats()["uploads"]
    assert not p.cache.prepare()
    o, qq, rs = p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0
    assert_close(o, p.reference(rs, qq, 0.0), np.float16, "after prepare")
    for tok in (7, 8, 9):                               # the third append grows new chunks
        p.append([0, 1], [tok, tok], *_kv(rng, 2, H, d, np.float16))
    assert p.cache.prepare()
    o, qq, rs = p.attention(qmap())
    assert p.cache.stats()["uploads"] == u0 + 1
    assert_close(o, p.reference(rs, qq, 0.0), np.float16, "after growth and prepare")


@pytest.mark.parametrize("sched", [2, 0, 4])
def test_attention_in_caller_order(sched):
    """ca_attention_ordered: q and o in an arbitrary order of the live
    sequences give the same rows as the tree-order call; the order may change
    between calls and the tree may change under a fixed order (joins, leaves,
    growth); bad orders are refused."""
    print(f"[case] caller order schedule={sched}", flush=True)
    rng = np.random.default_rng(11 + sched)
    H, d, c = 2, 64, 4
    p = Pair(c, H, d, np.float16, 1024)
    p.cache.set_tuning(schedule=sched)
    base = rng.integers(0, 20, 30).astype(np.int32)
    full = {}
    for sid in range(12):
        toks = np.concatenate([base[:int(rng.integers(1, 30))], rng.integers(20, 40, int(rng.integers(1, 20)))]).astype(np.int32)
        k, v = prefix_keyed_kv(11, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
        full[sid] = toks

    def check(order, label):
        qh = {s: rng.standard_normal((H, d)).astype(np.float16) for s in order}
        q = to_dev(np.stack([qh[s] for s in order]))
        o = p.cache.attention(q, seq_ids=np.asarray(order, np.int64))
        torch.cuda.synchronize()
        row_seq = p.cache.seq_order()
        qt = np.stack([qh[int(s)] for s in row_seq])
        ref = p.reference(row_seq, qt, 0.0)
        pos = {int(s): i for i, s in enumerate(row_seq)}
        assert_close(o.cpu().numpy(), ref[[pos[s] for s in order]], np.float16, label)

    live = list(full)
    for rep in range(3):
        order = [int(x) for x in rng.permutation(live)]
        check(order, f"order {rep}")
    # the tree changes under a fixed caller order: a leave, a join, growth
    p.remove(live[3])
    live.remove(live[3])
    toks = np.concatenate([base[:5], [99, 98, 97]]).astype(np.int32)
    k, v = prefix_keyed_kv(11, toks, 0, H, d, np.float16)
    p.insert(50, toks, k, v)
    full[50] = toks
    live.append(50)
    ks, vs = [], []
    for s in live:
        t2 = np.concatenate([full[s], [7]]).astype(np.int32)
        k, v = prefix_keyed_kv(11, t2, len(full[s]), H, d, np.float16)
        ks.append(k)
        vs.append(v)
        full[s] = t2
    p.append(live, [7] * len(live), np.concatenate(ks), np.concatenate(vs))
    order = sorted(live, reverse=True)
    check(order, "after tree changes")
    q = to_dev(np.zeros((len(live), H, d), np.float16))
    o = torch.empty_like(q)
    ws, _ = p.cache.workspace()
    for bad in (order[:-1], order[:-1] + [order[0]], order[:-1] + [12345]):
        with pytest.raises(B.ChunkAttnError) as ei:
            B.ca_attention_ordered(p.cache.h, q.data_ptr(), o.data_ptr(), np.asarray(bad, np.int64),
                                   0.0, ws.data_ptr(), ws.numel(), p.cache.stream())
        assert ei.value.status == B.CA_ERR_INVALID


def test_wrapper_rejects_bad_io_tensors():
    """The torch wrapper refuses q/o (and K/V) tensors whose shape, dtype,
    layout or device differ from what the kernels read and write, before any
    launch; a correct call afterwards still matches the oracle."""
    print("[case] wrapper argument checks", flush=True)
    H, d, c = 2, 64, 4
    p = Pair(c, H, d, np.float16, 256)
    rng = np.random.default_rng(5)
    for sid in range(3):
        toks = rng.integers(0, 9, 7).astype(np.int32)
        k, v = prefix_keyed_kv(5, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
    B_ = p.cache.num_seqs()
    q = to_dev(rng.standard_normal((B_, H, d)).astype(np.float16))
    bad_outs = [torch.empty((B_ - 1, H, d), dtype=torch.float16, device="cuda"),
                torch.empty((B_, H, d), dtype=torch.float32, device="cuda"),
                torch.empty((B_, d, H), dtype=torch.float16, device="cuda").transpose(1, 2),
                torch.empty((B_, H, d), dtype=torch.float16)]
    for bad in bad_outs:
        with pytest.raises(ValueError):
            p.cache.attention(q, out=bad)
        with pytest.raises(ValueError):
            p.cache.prefill(0, q[:1].contiguous(), out=bad)
    with pytest.raises(ValueError):
        p.cache.attention(q.cpu())
    with pytest.raises(ValueError):
        p.cache.attention(q[:, :, :32].contiguous())
    k_bad = torch.empty((1, H, d), dtype=torch.float16)
    with pytest.raises(ValueError):
        p.cache.append([0], [3], k_bad, k_bad)
    o = p.cache.attention(q)
    torch.cuda.synchronize()
    assert_close(o.cpu().numpy(), p.reference(p.cache.seq_order(), q.cpu().numpy(), 0.0), np.float16,
                 "after refused calls")


@pytest.mark.parametrize("sched", [2, 4])
def test_wide_batch_1024_rows(sched):
    """A wide batch: 1,024 live sequences on a three-level tree (a 48-token
    prompt, 32 branches of 20 tokens, unique suffixes of 1 to 40 tokens), so
    shared runs cover up to 1,024 rows (64 chunk-first row blocks per
    segment) and 4,096 (row, head) counters and partial slots are in use; a
    leave, a join and one decode step, then sampled rows against the oracle,
    tables bit-exact."""
    print(f"[case] 1024-row batch schedule={sched}", flush=True)
    rng = np.random.default_rng(1024 + sched)
    H, d, c = 4, 64, 16
    p = Pair(c, H, d, np.float16, 8192)
    p.cache.set_tuning(schedule=sched)
    prompt = rng.integers(0, 1000, 48).astype(np.int32)
    branches = [rng.integers(1000 + 100 * b, 1100 + 100 * b, 20).astype(np.int32) for b in range(32)]
    for sid in range(1024):
        suffix = rng.integers(5000, 30000, int(rng.integers(1, 41))).astype(np.int32)
        toks = np.concatenate([prompt, branches[sid % 32], suffix])
        k, v = prefix_keyed_kv(77, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
    p.remove(5)
    toks = np.concatenate([prompt, branches[7], [29999, 29998]]).astype(np.int32)
    k, v = prefix_keyed_kv(77, toks, 0, H, d, np.float16)
    p.insert(5000, toks, k, v)
    live = [int(s) for s in p.cache.seq_order()]
    step_tok = rng.integers(0, 30000, len(live)).astype(np.int32)
    kk = rng.standard_normal((len(live), H, d)).astype(np.float16)
    vv = rng.standard_normal((len(live), H, d)).astype(np.float16)
    p.append(live, step_tok, kk, vv)
    p.check_tables()
    qh = {s: rng.standard_normal((H, d)).astype(np.float16) for s in live}
    o, q, row_seq = p.attention(qh)
    rows = sorted(set([0, 1, len(row_seq) - 1] + [int(x) for x in rng.choice(len(row_seq), 40, replace=False)]))
    assert_close(o[rows], p.reference(row_seq, q, 0.0, rows=rows), np.float16, f"1024 rows sched={sched}")


@pytest.mark.parametrize("sched", [2, 4])
def test_long_context_32k(sched):
    """Long contexts: four rows of 32,768 tokens each (a 16,384-token shared
    prompt, 256 chunks, then 16,384 private tokens per row), d = 128, c = 64:
    the shared run is cut into many segments (each a partial per row, or a
    fold into the row's accumulator under the partial-free schedule) and
    every sequence-first row walks 256 private chunks. All rows against the
    oracle."""
    print(f"[case] 32k-token contexts schedule={sched}", flush=True)
    rng = np.random.default_rng(32768 + sched)
    H, d, c = 2, 128, 64
    p = Pair(c, H, d, np.float16, 1400)
    p.cache.set_tuning(schedule=sched)
    prompt = rng.integers(0, 1000, 16384).astype(np.int32)
    for sid in range(4):
        toks = np.concatenate([prompt, rng.integers(1000 + 2000 * sid, 3000 + 2000 * sid, 16384)]).astype(np.int32)
        k, v = prefix_keyed_kv(3, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
    p.check_tables()
    qh = {s: rng.standard_normal((H, d)).astype(np.float16) for s in range(4)}
    o, q, row_seq = p.attention(qh)
    assert_close(o, p.reference(row_seq, q, 0.0), np.float16, f"32k contexts sched={sched}")
