"""GPU parity of prefill with prefix reuse (ca_prefill_attention) against the
oracle's causal attention over the sequence's whole path."""
import numpy as np
import pytest
import torch

from oracle import prefill_attention
from paper_2402_15220_amd.binding import ChunkAttnError
from parity_util import Pair, assert_close, to_dev
from workloads import make_prefill_join, prefix_keyed_kv

pytestmark = pytest.mark.gpu


def test_join_single_prompt_tree_512_new_tokens():
    """The prefill workload: a 33rd sequence joins the single-shared-prompt tree
    (1024 shared + 512 unique per row) with the shared prompt plus 512 new
    tokens; its 512 new tokens attend over 1536 positions."""
    print("[case] prefill join of the single-prompt tree, 512 new tokens", flush=True)
    pj = make_prefill_join()
    wl = pj.static
    p = Pair(wl.c, wl.H, wl.d, wl.dtype, 400)
    seg_dev = [(to_dev(s.k), to_dev(s.v)) for s in wl.segments]
    for s in wl.seqs + [pj.seq]:
        k, v = s.kv(wl.segments)
        m = p.insert(s.seq_id, s.tokens(wl.segments), k, v,
                     dev_k=torch.cat([seg_dev[i][0] for i in s.segs]),
                     dev_v=torch.cat([seg_dev[i][1] for i in s.segs]))
    assert m == 1024  # the joining sequence reuses the whole shared prompt
    p.check_tables()
    o = p.cache.prefill(pj.seq.seq_id, to_dev(pj.q))
    torch.cuda.synchronize()
    ref = prefill_attention(p.tree, pj.seq.seq_id, pj.q, wl.scale)
    assert_close(o.cpu().numpy(), ref, wl.dtype, "prefill join 512")
    # the decode call still sees the joined tree correctly
    q_dec = {s.seq_id: wl.q[s.seq_id] for s in wl.seqs}
    q_dec[pj.seq.seq_id] = pj.q[-1]
    od, q, row_seq = p.attention(q_dec)
    rows = [int(np.nonzero(row_seq == pj.seq.seq_id)[0][0]), 0, len(row_seq) - 1]
    assert_close(od[rows], p.reference(row_seq, q, 0.0, rows=rows), wl.dtype, "decode after join")
    # the last prefill query equals the decode row of the joined sequence
    r = rows[0]
    assert np.abs(od[r].astype(np.float64) - o[-1].cpu().numpy().astype(np.float64)).max() < 2e-3


@pytest.mark.parametrize("case", range(13))
def test_prefill_random_trees(case):
    """Shared prefixes that split chunks mid-way, short chunks on the path,
    chunks longer than 64 tokens, n_q from 1 to the whole sequence, both head
    sizes and both pool layouts."""
    rng = np.random.default_rng(500 + case)
    c = [1, 3, 4, 7, 16, 64, 5, 64, 16, 2, 128, 100, 65][case]
    d = [64, 128][case % 2]
    H = 1 + case % 3
    layout = "interleaved" if case % 4 == 3 else "split"
    print(f"[case] prefill random c={c} d={d} H={H} layout={layout}", flush=True)
    p = Pair(c, H, d, np.float16, 4096, layout=layout)
    base = rng.integers(0, 20, int(rng.integers(5, 150))).astype(np.int32)
    seqs = {}
    for sid in range(4):
        cut = int(rng.integers(1, len(base) + 1))
        tail = rng.integers(20 + 40 * sid, 60 + 40 * sid, int(rng.integers(1, 200))).astype(np.int32)
        toks = np.concatenate([base[:cut], tail])
        k, v = prefix_keyed_kv(case, toks, 0, H, d, np.float16)
        p.insert(sid, toks, k, v)
        seqs[sid] = toks
    for sid, toks in seqs.items():
        L = len(toks)
        for n_q in sorted({1, min(L, 5), min(L, 63), min(L, 64), min(L, 65), L}):
            q = rng.standard_normal((n_q, H, d)).astype(np.float16)
            o = p.cache.prefill(sid, to_dev(q), scale=0.0 if n_q % 2 else 0.2)
            torch.cuda.synchronize()
            sc = 1.0 / np.sqrt(d) if n_q % 2 else 0.2
            ref = prefill_attention(p.tree, sid, q, sc)
            assert_close(o.cpu().numpy(), ref, np.float16, f"prefill c={c} seq={sid} L={L} n_q={n_q}")


def test_prefill_errors_and_noop():
    p = Pair(4, 2, 64, np.float16, 64)
    toks = np.arange(10, dtype=np.int32)
    k, v = prefix_keyed_kv(0, toks, 0, 2, 64, np.float16)
    p.insert(0, toks, k, v)
    q = to_dev(np.zeros((11, 2, 64), np.float16))
    with pytest.raises(ChunkAttnError):
        p.cache.prefill(0, q)           # more queries than tokens
    with pytest.raises(ChunkAttnError):
        p.cache.prefill(5, q[:3])       # unknown sequence
    o = torch.full((0, 2, 64), 7.0, dtype=torch.float16, device="cuda")
    p.cache.prefill(0, q[:0], out=o)    # n_q = 0: nothing to do
    p32 = Pair(4, 2, 64, np.float32, 64)
    k32, v32 = prefix_keyed_kv(0, toks, 0, 2, 64, np.float32)
    p32.insert(0, toks, k32, v32)
    with pytest.raises(ChunkAttnError):
        p32.cache.prefill(0, to_dev(np.zeros((3, 2, 64), np.float32)))


@pytest.mark.parametrize("c,L", [(16, 1024), (16, 1025), (3, 192), (1, 255), (1, 256), (2, 700)])
def test_prefill_long_paths(c, L):
    """Paths of up to 64 chunks keep their chunk table in register lanes, up
    to 255 travel in the kernel arguments, longer ones through a device
    upload: both sides of each limit (64 and 65, 255 and 256 chunks), and
    long paths of short chunks."""
    print(f"[case] prefill path of {-(-L // c)} chunks (c={c}, L={L})", flush=True)
    H, d = 2, 64
    rng = np.random.default_rng(900 + L)
    p = Pair(c, H, d, np.float16, 2048)
    toks = rng.integers(0, 50, L).astype(np.int32)
    k, v = prefix_keyed_kv(7, toks, 0, H, d, np.float16)
    p.insert(0, toks, k, v)
    for n_q in (1, 70, L):
        q = rng.standard_normal((n_q, H, d)).astype(np.float16)
        o = p.cache.prefill(0, to_dev(q))
        torch.cuda.synchronize()
        ref = prefill_attention(p.tree, 0, q, 1.0 / np.sqrt(d))
        assert_close(o.cpu().numpy(), ref, np.float16, f"prefill c={c} L={L} n_q={n_q}")


def test_prefill_long_context():
    """A long join: 2,048 new tokens after a 6,144-token cached prefix (an
    8,192-token path of 128 chunks), sampled queries against the oracle,
    including the first, the last and the 64-query tile boundaries."""
    print("[case] prefill of 2048 new tokens over 8192 positions", flush=True)
    rng = np.random.default_rng(8192)
    H, d, c = 2, 128, 64
    p = Pair(c, H, d, np.float16, 400)
    prefix = rng.integers(0, 500, 6144).astype(np.int32)
    k, v = prefix_keyed_kv(8, prefix, 0, H, d, np.float16)
    p.insert(0, prefix, k, v)
    toks = np.concatenate([prefix, rng.integers(500, 1000, 2048)]).astype(np.int32)
    k, v = prefix_keyed_kv(8, toks, 0, H, d, np.float16)
    assert p.insert(1, toks, k, v) == 6144
    q = rng.standard_normal((2048, H, d)).astype(np.float16)
    o = p.cache.prefill(1, to_dev(q)).cpu().numpy()
    rows = sorted({0, 1, 63, 64, 127, 128, 1023, 1024, 2046, 2047} |
                  {int(x) for x in rng.choice(2048, 20, replace=False)})
    ref = prefill_attention(p.tree, 1, q, 1.0 / np.sqrt(d), queries=rows)
    assert_close(o[rows], ref, np.float16, "prefill 2048 over 8192")


@pytest.mark.parametrize("split,layout", [(1, "split"), (2, "split"), (3, "split"), (5, "split"),
                                          (16, "split"), (3, "interleaved")])
def test_prefill_key_range_split(split, layout, monkeypatch):
    """The key-range split of a tile over several blocks (partials folded by
    the last part to arrive), forced to 1, 2, 3, 5 and 16 parts through
    CA_PREFILL_SPLIT: paths of 24 chunks of 64 (kernel-argument table in
    register lanes), 70 chunks of 16 and 300 chunks of 1 (device table),
    ragged and whole query tiles, more parts than units (empty parts), both
    head sizes."""
    import os
    monkeypatch.setenv("CA_PREFILL_SPLIT", str(split))
    print(f"[case] prefill split={split} layout={layout}", flush=True)
    rng = np.random.default_rng(4000 + split)
    for c, L, n_qs, d, H in [(64, 1536, (1, 64, 100, 512), 128, 2), (16, 1120, (7, 129), 64, 3),
                             (1, 300, (3, 300), 64, 1), (64, 300, (5,), 128, 1)]:
        p = Pair(c, H, d, np.float16, 2 * (L // c + 2), layout=layout)
        toks = rng.integers(0, 50, L).astype(np.int32)
        k, v = prefix_keyed_kv(split, toks, 0, H, d, np.float16)
        p.insert(0, toks, k, v)
        for n_q in n_qs:
            q = rng.standard_normal((n_q, H, d)).astype(np.float16)
            o = p.cache.prefill(0, to_dev(q)).cpu().numpy()
            rows = sorted({0, n_q - 1, n_q // 2} | {int(x) for x in rng.integers(0, n_q, 6)})
            ref = prefill_attention(p.tree, 0, q, 1.0 / np.sqrt(d), queries=rows)
            assert_close(o[rows], ref, np.float16, f"split={split} {layout} c={c} L={L} n_q={n_q} d={d}")
        p.cache.close()
    assert os.environ["CA_PREFILL_SPLIT"] == str(split)
