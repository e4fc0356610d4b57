"""GPU parity at the full sizes of the shapes the paper's sweeps time.

* Table 3's corners at b = 32 and n_p = 4096 tokens per sequence: nothing
  shared (n_s = 0: the call is sequence-first work only), half shared
  (n_s = 2048) and everything shared (n_s = 4096: identical sequences, the
  call is chunk-first work only).
* Figure 4's widest batch, b = 96 sequences on a 2048-token shared prompt,
  decoding 66 steps (a private chunk grows from 1 to 64 tokens, then the
  next chunk starts), with every row checked at several steps.

Every row against the float64 oracle, under the default schedule and the
partial-free schedule; tables and pool rows bit-exact.
"""
import time

import numpy as np
import pytest
import torch

from parity_util import Pair, assert_close, host_threads, to_dev
from paper_2402_15220_amd import binding as B
from workloads import make_decode_run, make_sweep

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.load()
    yield


@pytest.mark.timeout(600)
@pytest.mark.parametrize("n_s", [0, 2048, 4096])
def test_table3_corner_b32_np4096(n_s):
    print(f"[case] Table 3 cell b=32 n_p=4096 n_s={n_s}", flush=True)
    t_start = time.time()
    wl = make_sweep(32, 4096, n_s, seed=4096 + n_s)
    nodes = sum(-(-len(s) // wl.c) for s in wl.segments)
    p = Pair(wl.c, wl.H, wl.d, wl.dtype, nodes + 16)
    seg_dev = [(to_dev(s.k), to_dev(s.v)) for s in wl.segments]
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        p.insert(s.seq_id, s.tokens(wl.segments), k, v,
                 dev_k=torch.cat([seg_dev[i][0] for i in s.segs]),
                 dev_v=torch.cat([seg_dev[i][1] for i in s.segs]))
    del seg_dev
    tb = p.check_tables()
    assert tb["shr_node"].shape[0] == n_s // wl.c
    p.check_pool()
    qmap = {s.seq_id: wl.q[s.seq_id] for s in wl.seqs}
    ref = None
    for sched in (2, 4):
        p.cache.set_tuning(schedule=sched)
        for rep in range(2):
            o, q, row_seq = p.attention(qmap)
            if ref is None:
                ref = p.reference(row_seq, q, 0.0)
            assert_close(o, ref, wl.dtype, f"b=32 n_p=4096 n_s={n_s} schedule={sched} rep={rep}")
    print(f"[case] done in {time.time() - t_start:.1f} s ({host_threads()} oracle threads)", flush=True)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("sched", [2, 4])
def test_fig4_batch96_decode(sched):
    print(f"[case] Figure 4 batch b=96 n_s=2048, 66 decode steps, schedule={sched}", flush=True)
    t_start = time.time()
    run = make_decode_run(96, 2048, 66, seed=96)
    p = Pair(run.c, run.H, run.d, run.dtype, 2048 // run.c + 2 * 96 + 16)
    p.cache.set_tuning(schedule=sched)
    dk, dv = to_dev(run.prompt.k), to_dev(run.prompt.v)
    for sid in range(run.b):
        # every sequence starts as the same prompt (only the first stores K/V)
        assert p.insert(sid, run.prompt.tokens, run.prompt.k, run.prompt.v, dev_k=dk, dev_v=dv) == (
            0 if sid == 0 else 2048)
    check_at = {0, 1, 31, 62, 63, 64, 65}
    worst = (0.0, 0.0)
    for st in run.steps():
        p.append(st.live, st.tokens, st.k, st.v)
        qmap = {int(sid): st.q[i] for i, sid in enumerate(st.live)}
        o, q, row_seq = p.attention(qmap)
        if st.step in check_at:
            tb = p.check_tables()
            assert tb["row_seq"].shape[0] == 96 and tb["shr_node"].shape[0] == 2048 // run.c
            ma, rel = assert_close(o, p.reference(row_seq, q, 0.0), run.dtype,
                                   f"b=96 decode step {st.step} schedule={sched}")
            worst = (max(worst[0], ma), max(worst[1], rel))
            if st.step in (0, 64):
                p.check_pool()
    print(f"[parity] b=96 decode worst max_abs={worst[0]:.3e} rel_l2={worst[1]:.3e}; "
          f"{time.time() - t_start:.1f} s", flush=True)
