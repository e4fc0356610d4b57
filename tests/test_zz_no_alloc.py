"""ca_attention_noalloc (the entry point for callers that cannot allocate)
against ca_attention through the C ABI, on the single-shared-prompt tree
(32 rows, 1024 shared + 512 private tokens, H = 32, d = 128, fp16) under
several schedules, then a second call on a smaller batch; both calls also
against the float64 oracle. The refusals (stale kernel context, calls larger
than the device scratch) leave the output untouched."""
import numpy as np
import pytest
import torch

from parity_util import Pair, assert_close, to_dev
from paper_2402_15220_amd import binding as B
from workloads import make_static, prefix_keyed_kv

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.load()
    yield


def _both(p, qmap, label):
    """Tree-order q; o from ca_attention and from ca_attention_noalloc."""
    row_seq = p.cache.seq_order()
    q = to_dev(np.stack([qmap[int(s)] for s in row_seq]).astype(p.dtype))
    ws, _ = p.cache.workspace()
    o_ref = torch.empty_like(q)
    o_na = torch.full_like(q, float("nan"))
    s = p.cache.stream()
    B.ca_attention(p.cache.h, q.data_ptr(), o_ref.data_ptr(), 0.0, ws.data_ptr(), ws.numel(), s)
    B.ca_attention_noalloc(p.cache.h, q.data_ptr(), o_na.data_ptr(), 0.0, s)
    torch.cuda.synchronize()
    o_ref, o_na = o_ref.cpu().numpy(), o_na.cpu().numpy()
    assert np.isfinite(o_na).all(), label
    assert_close(o_na, o_ref.astype(np.float64), p.dtype, f"{label}: noalloc vs ca_attention")
    qh = q.cpu().numpy()
    assert_close(o_na, p.reference(row_seq, qh, 0.0), p.dtype, f"{label}: noalloc vs oracle")
    return row_seq


def test_noalloc_chunk_first_only_call():
    """Identical prompts: the call is chunk-first work alone (its own launch),
    here with its partials and counters in the device scratch."""
    print("[case] noalloc entry point, chunk-first work only", flush=True)
    rng = np.random.default_rng(23)
    H, d, n, rows = 4, 128, 700, 20
    p = Pair(64, H, d, np.float16, 64)
    k = rng.standard_normal((n, H, d)).astype(np.float16)
    v = rng.standard_normal((n, H, d)).astype(np.float16)
    for sid in range(rows):
        p.insert(sid, np.arange(n), k, v)
    qmap = {sid: rng.standard_normal((H, d)).astype(np.float16) for sid in range(rows)}
    for seg in (-1, 3):
        p.cache.set_tuning(seg_chunks=seg, schedule=2)
        p.cache.prepare()
        _both(p, qmap, f"chunk-first only seg={seg}")


def test_noalloc_matches_attention_two_calls_second_smaller():
    print("[case] noalloc entry point on the single-prompt tree", flush=True)
    wl = make_static(2)
    nodes = sum(-(-len(s) // wl.c) for s in wl.segments)
    p = Pair(wl.c, wl.H, wl.d, wl.dtype, nodes + 64)
    seg_dev = [(to_dev(s.k), to_dev(s.v)) for s in wl.segments]
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        p.insert(s.seq_id, s.tokens(wl.segments), k, v,
                 dev_k=torch.cat([seg_dev[i][0] for i in s.segs]),
                 dev_v=torch.cat([seg_dev[i][1] for i in s.segs]))
    qmap = {s.seq_id: wl.q[s.seq_id] for s in wl.seqs}
    for sched in (2, 0, 4, 1):
        p.cache.set_tuning(schedule=sched)
        p.cache.prepare()
        _both(p, qmap, f"B=32 schedule={sched}")
    # second call, smaller batch: 13 sequences leave, one decode step grows
    # new chunks (a structural change), the context is prepared again
    p.cache.set_tuning(schedule=2)
    for sid in range(3, 32, 2)[:13]:
        p.remove(sid)
    live = [int(s) for s in p.cache.seq_order()]
    rng = np.random.default_rng(19)
    kk = rng.standard_normal((len(live), wl.H, wl.d)).astype(np.float16)
    vv = rng.standard_normal((len(live), wl.H, wl.d)).astype(np.float16)
    p.append(live, rng.integers(0, 32000, len(live)).astype(np.int32), kk, vv)
    q_small = to_dev(rng.standard_normal((len(live), wl.H, wl.d)).astype(np.float16))
    o = torch.empty_like(q_small)
    with pytest.raises(B.ChunkAttnError) as ei:       # context not current yet
        B.ca_attention_noalloc(p.cache.h, q_small.data_ptr(), o.data_ptr(), 0.0, p.cache.stream())
    assert ei.value.status == B.CA_ERR_INVALID
    p.cache.prepare()
    qmap2 = {sid: rng.standard_normal((wl.H, wl.d)).astype(np.float16) for sid in live}
    rows = _both(p, qmap2, f"B={len(live)} after leaves and growth")
    assert len(rows) == 19


def test_noalloc_refuses_calls_larger_than_the_scratch():
    """More (row, head) counters, or more partial bytes, than the scratch
    holds: CA_ERR_WORKSPACE before any launch; ca_attention still works."""
    print("[case] noalloc limits", flush=True)
    H, d, c = 256, 128, 4
    # 257 rows x 256 heads = 65,792 counters (the scratch holds 65,536)
    p = Pair(c, H, d, np.float16, 600)
    for sid in range(257):
        toks = np.array([sid % 7, 1000 + sid], np.int32)
        k, v = prefix_keyed_kv(5, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
    p.cache.prepare()
    q = to_dev(np.zeros((257, H, d), np.float16))
    o = torch.zeros_like(q)
    with pytest.raises(B.ChunkAttnError) as ei:
        B.ca_attention_noalloc(p.cache.h, q.data_ptr(), o.data_ptr(), 0.0, p.cache.stream())
    assert ei.value.status == B.CA_ERR_WORKSPACE
    # 64 rows sharing two chunks: 128 partials x 256 heads x 520 bytes > 16 MiB
    p = Pair(c, H, d, np.float16, 600)
    for sid in range(64):
        toks = np.array([1, 2, 3, 4, 5, 6, 7, 8, 100 + sid], np.int32)
        k, v = prefix_keyed_kv(6, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
    p.cache.prepare()
    assert B.ca_workspace_size(p.cache.h) > (16 << 20) - (256 << 10)
    q = to_dev(np.random.default_rng(3).standard_normal((64, H, d)).astype(np.float16))
    o = torch.zeros_like(q)
    with pytest.raises(B.ChunkAttnError) as ei:
        B.ca_attention_noalloc(p.cache.h, q.data_ptr(), o.data_ptr(), 0.0, p.cache.stream())
    assert ei.value.status == B.CA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert float(o.abs().max()) == 0.0              # nothing was launched
    o2 = p.cache.attention(q)
    torch.cuda.synchronize()
    assert_close(o2.cpu().numpy(), p.reference(p.cache.seq_order(), q.cpu().numpy(), 0.0),
                 np.float16, "64 rows x 256 heads with a caller workspace")
