"""Decode-attention benchmark on one MI355X.

A step is one ca_attention call over the tree of the single-shared-prompt
workload: B=32 sequences sharing a 1024-token prompt plus 512 unique tokens
each, H=32, d=128, chunk 64, fp16 (synthetic, seeded; 285.7 MB of K/V, q and
o per call). By default the call is ONE launch: chunk-first items (dispatched
first) and sequence-first items in one grid, the last contributor to each
row merging its partials and writing o. The tree is built and its kernel
context uploaded before timing; inputs are resident in HBM.

Prints one JSON line: tokens/s (B per call) and µs per call from the timed
loop, the roofline of the dominant kernel (the fused two-phase kernel,
HBM-bound) from HIP events on the launch stream, per-phase figures measured
in isolation, and the CPU oracle timed on the host for the same workload.
Also, unless switched off:
  cold     calls timed after a clean 1 GiB read that evicts L2 and the
           256 MB Infinity Cache (the conservative figure: in a model, other
           layers' K/V pass between two calls of one layer);
  dynamic  the 64-step decode workload (2048-token prompt, 128 sequences of
           64..1024 unique tokens, 10% churn every 16 steps): per-step
           attention time and per-step library time (churn, append, context
           upload, attention).
  prefill  a 33rd sequence joins the bench tree with the shared prompt plus
           512 new tokens; causal attention of the new tokens over all 1536
           positions (prefill with prefix reuse), against the MFMA peak.
Profiler runs pass --no-cold --no-dynamic --no-prefill so that the
per-kernel averages cover the bench workload's warm launches only.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=2,
                    help="static workload: 2 = one 1024-token prompt shared by 32 rows with 512 "
                         "unique tokens each (default), 3 = the same with a 4096-token prompt, "
                         "4 = two-level tree of 64 rows")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=8.0,
                    help="target time of the oracle's all-cores sample of whole calls")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the warm and cold figures of the 4096-token-prompt and two-level trees")
    ap.add_argument("--no-cold", action="store_true", help="skip the cache-evicted timing")
    ap.add_argument("--no-dynamic", action="store_true", help="skip the 64-step decode workload")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill-with-prefix-reuse timing")
    ap.add_argument("--dynamic-only", action="store_true",
                    help="run only the 64-step decode workload and print its figures (for profiling it)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="run only the prefill join and print its figures (for profiling it)")
    ap.add_argument("--seg", type=int, default=0, help="chunk-first segment size (0: library default)")
    ap.add_argument("--split", type=int, default=-1, help="sequence-first split (-1: library default)")
    ap.add_argument("--schedule", type=int, default=-1,
                    help="0 sequential, 1 fused + merge launch, 2 fused with in-kernel merge, "
                         "3 two streams, 4 partial-free serial reduction (-1: library default)")
    return ap.parse_args()


def main():
    args = _parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(heads would shard across GPUs with no collective in attention).", file=sys.stderr)
        sys.exit(2)
    if args.dynamic_only:
        print(json.dumps({"dynamic": dynamic_run()}), flush=True)
        return
    if args.prefill_only:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps({"prefill": prefill_run()}), flush=True)
        return

    import numpy as np
    import torch

    from paper_2402_15220_amd.roofline import PEAK_HBM_GBPS, PEAK_MFMA_TFLOPS

    torch.cuda.set_device(0)
    wl, cache, q, o, rows, model = static_setup(args.config, args.seg, args.split, args.schedule)
    B = model["B"]
    stats = cache.stats()

    def call():
        cache.attention(q, out=o)

    for _ in range(args.warmup):      # also uploads the kernel context
        call()
    torch.cuda.synchronize()

    # timed region: exactly `steps` calls, synchronised on both sides
    t0 = time.perf_counter()
    for _ in range(args.steps):
        call()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps

    n_ev = max(args.steps, 50)
    call_us = back_to_back(call, n_ev)
    cache.set_tuning(phase_mask=3)        # the two-phase launch without a separate merge
    tpp_us = back_to_back(call, n_ev)
    cache.set_tuning(phase_mask=1)        # chunk-first items alone
    kcf_us = back_to_back(call, n_ev)
    cache.set_tuning(phase_mask=2)        # sequence-first items alone
    ksf_us = back_to_back(call, n_ev)
    cache.set_tuning(phase_mask=7)
    call()
    # a plain device copy of known size (context ceiling, and the reference
    # kernel for scaling hardware byte counters)
    src = torch.ones(1 << 28, dtype=torch.float16, device="cuda")   # 512 MiB
    dst = torch.empty_like(src)
    copy_us = back_to_back(lambda: dst.copy_(src), 10)
    copy_bytes = 2 * src.numel() * 2
    del src, dst
    torch.cuda.synchronize()

    tpp_bytes = model["shared_kv"] + model["private_kv"] + model["q"]
    traffic, traffic_source = counter_traffic(wl.name, cache.layout)
    tpp_gbps = tpp_bytes / (tpp_us * 1e-6) / 1e9
    ksf_gbps = model["ksf_bytes"] / (ksf_us * 1e-6) / 1e9
    kcf_tflops = model["kcf_flops"] / (kcf_us * 1e-6) / 1e12
    us = ms_per_step * 1e3
    out = {
        "metric": "decode attention µs/call + tokens/s; achieved HBM GB/s vs peak (B=32,H=32,d=128)",
        "value": B / (ms_per_step * 1e-3),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "H": wl.H, "d": wl.d, "c": wl.c,
                   "pool_layout": cache.layout,
                   "shared_tokens": int(model["shared_kv"] // (2 * wl.H * wl.d * 2)),
                   "private_tokens_per_row": int(model["private_kv"] // (2 * wl.H * wl.d * 2) // B)},
        "value_kind": "warm: back-to-back calls on one resident tree (its 285.7 MB partly stays in "
                      "the 256 MB Infinity Cache); see cold for calls after a cache flush",
        "us_per_call": us,
        "us_per_call_events": call_us,
        "algorithmic_bytes_per_call": model["total"],
        "achieved_GBps_per_call": model["total"] / (us * 1e-6) / 1e9,
        "dense_equivalent_bytes": model["dense_equivalent"],
        "schedule": stats["schedule"], "seg_chunks": stats["seg_chunks"],
        "roofline": {"bound": "hbm", "kernel": "tpp_kernel (fused chunk-first + sequence-first + merge)",
                     "achieved": tpp_gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                     "frac": tpp_gbps / PEAK_HBM_GBPS, "traffic": traffic,
                     "traffic_source": traffic_source,
                     "bytes_per_launch": tpp_bytes, "us_per_launch": tpp_us},
        "copy_512MiB": {"us": copy_us, "GBps": copy_bytes / (copy_us * 1e-6) / 1e9},
        "sequence_first_alone": {"kernel": "ksf_kernel", "us_per_launch": ksf_us,
                                 "bytes_per_launch": model["ksf_bytes"], "GBps": ksf_gbps,
                                 "frac": ksf_gbps / PEAK_HBM_GBPS},
        "chunk_first_alone": {"kernel": "kcf_kernel", "us_per_launch": kcf_us,
                              "flops_per_launch": model["kcf_flops"], "mfma_tflops": kcf_tflops,
                              "mfma_util": kcf_tflops / PEAK_MFMA_TFLOPS["f16"],
                              "GBps": (model["shared_kv"] + model["q"]) / (kcf_us * 1e-6) / 1e9},
    }
    if not args.no_cold:
        out["cold"] = cold_times(call, model["total"], model["B"])
        cache.set_tuning(phase_mask=2)    # the sequence-first kernel alone, same flush
        ksf_cold = cold_times(call, model["ksf_bytes"], model["B"])
        cache.set_tuning(phase_mask=7)
        out["sequence_first_alone"]["cold"] = {k: ksf_cold[k] for k in ("us_per_call", "GBps", "frac", "stream")}
    cache.close()
    del cache, q, o
    torch.cuda.empty_cache()
    if not args.no_other_configs and args.config == 2:
        out["other_configs"] = {str(c): other_config(c, args.steps, not args.no_cold) for c in (1, 3, 4)}
    if not args.no_dynamic:
        out["dynamic"] = dynamic_run()
    if not args.no_prefill:
        out["prefill"] = prefill_run()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, rows, args.cpu_seconds, with_dynamic=not args.no_dynamic)
    print(json.dumps(out), flush=True)


def static_setup(config, seg=0, split=-1, schedule=-1):
    """A static workload's tree in a fresh cache, its q in tree row order,
    an output buffer and the call's byte model; inputs resident on the GPU."""
    import numpy as np
    import torch

    from paper_2402_15220_amd.cache import Cache
    from paper_2402_15220_amd.roofline import call_model
    from workloads import make_static

    wl = make_static(config)
    nodes = sum(-(-len(s) // wl.c) for s in wl.segments)
    tdt = torch.float32 if np.dtype(wl.dtype) == np.float32 else torch.float16
    cache = Cache(wl.c, wl.H, wl.d, nodes + 16, dtype=tdt)
    seg_dev = [(torch.from_numpy(s.k).cuda(), torch.from_numpy(s.v).cuda()) for s in wl.segments]
    for s in wl.seqs:
        cache.insert(s.seq_id, s.tokens(wl.segments), torch.cat([seg_dev[i][0] for i in s.segs]),
                     torch.cat([seg_dev[i][1] for i in s.segs]))
    del seg_dev
    cache.set_tuning(seg_chunks=seg, split_chunks=split, schedule=schedule)
    rows = cache.seq_order()
    q = torch.from_numpy(np.ascontiguousarray(wl.q[rows])).cuda()
    o = torch.empty_like(q)
    model = call_model(cache.tables(), wl.H, wl.d, np.dtype(wl.dtype).itemsize)
    torch.cuda.synchronize()
    return wl, cache, q, o, rows, model


def back_to_back(fn, n):
    """Mean device time per fn() over n back-to-back launches, with events
    on the launch stream (no host synchronisation in between). A spin
    kernel holds the stream while the host enqueues, so a launch that is
    shorter than the host's per-call cost still runs back to back."""
    import torch

    fn()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    torch.cuda._sleep(40_000_000)
    a.record()
    for _ in range(n):
        fn()
    b.record()
    b.synchronize()
    return a.elapsed_time(b) * 1e3 / n


def other_config(config, n, cold):
    """Warm (back-to-back) and cold figures of another static workload: the
    4096-token prompt (3) or the two-level tree of 64 rows (4)."""
    import torch

    from paper_2402_15220_amd.roofline import PEAK_HBM_GBPS

    wl, cache, q, o, _, model = static_setup(config)

    def call():
        cache.attention(q, out=o)

    for _ in range(5):
        call()
    warm = back_to_back(call, max(n, 50))
    r = {"workload": wl.name, "B": model["B"], "algorithmic_bytes_per_call": model["total"],
         "warm": {"us_per_call": warm, "tok_per_s": model["B"] / (warm * 1e-6),
                  "GBps": model["total"] / (warm * 1e-6) / 1e9,
                  "frac": model["total"] / (warm * 1e-6) / 1e9 / PEAK_HBM_GBPS}}
    if cold:
        r["cold"] = cold_times(call, model["total"], model["B"])
    cache.close()
    del cache, q, o
    torch.cuda.empty_cache()
    return r


def decode_sources_hash(csrc):
    """Hash of the decode kernels' code (kernels.hip and device_common.hpp)
    with comments and blank space removed, so that only code changes make
    committed counter results stale."""
    import hashlib
    import re

    h = hashlib.sha256()
    for name in ("kernels.hip", "device_common.hpp"):
        with open(os.path.join(csrc, name)) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def counter_traffic(workload, layout):
    """HBM bytes per tpp_kernel launch, taken from the committed rocprofv3
    counter passes (FETCH_SIZE and WRITE_SIZE, each scaled by what it reads
    for a plain copy of known size); not measured in this run. Returns
    (bytes or None, source): None when the kernels' code changed since the
    counters were taken (hash mismatch), or the workload or pool layout
    differs."""
    rel = os.path.join("profiles", "tpp_kernel_single_prompt_b32_traffic.json")
    csrc = os.path.join(ROOT, "paper_2402_15220_amd", "csrc")
    sha = decode_sources_hash(csrc)
    src = {"taken_from": rel, "measured_in_this_run": False, "decode_sources_sha256_16": sha}
    try:
        with open(os.path.join(ROOT, rel)) as f:
            rec = json.load(f)
    except OSError:
        return None, dict(src, status="no counter record")
    if rec.get("decode_sources_sha256_16") != sha:
        return None, dict(src, status="stale: kernels changed since the counters were taken")
    if rec.get("workload") != workload or rec.get("pool_layout") != layout:
        return None, dict(src, status="counters are for another workload or pool layout")
    return rec["kernels"]["tpp_kernel"]["traffic_bytes"], dict(src, status="current")


def cold_times(call, nbytes, rows, n=30):
    """Median device time per call after a clean (read-only) 1 GiB pass that
    evicts L2 and the 256 MB Infinity Cache, events around the call only;
    rates for `nbytes` algorithmic bytes and `rows` tokens per call."""
    import numpy as np
    import torch

    flush = torch.ones(1 << 29, dtype=torch.float16, device="cuda")
    evs = []
    for _ in range(n):
        flush.sum()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        call()
        b.record()
        evs.append((a, b))
    torch.cuda.synchronize()
    us = float(np.median([a.elapsed_time(b) * 1e3 for a, b in evs]))
    # The same cold calls without a marker pair around each: n (flush, call)
    # pairs back to back, less n flushes alone, both between one event pair
    # (the device time a cold call adds to a stream, its launch gap included)
    def span(with_call):
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(n):
            flush.sum()
            if with_call:
                call()
        b.record()
        b.synchronize()
        return a.elapsed_time(b) * 1e3
    diffs = [(span(True) - span(False)) / n for _ in range(3)]
    us_diff = float(np.median(diffs))
    from paper_2402_15220_amd.roofline import PEAK_HBM_GBPS

    gbps = nbytes / (us * 1e-6) / 1e9
    return {"us_per_call": us, "tok_per_s": rows / (us * 1e-6), "GBps": gbps,
            "frac": gbps / PEAK_HBM_GBPS, "calls": n,
            "flush": "clean 1 GiB read between calls; median of per-call event pairs "
                     "(each pair adds ~2 us of marker overhead)",
            "stream": {"us_per_call": us_diff,
                       "frac": nbytes / (us_diff * 1e-6) / 1e9 / PEAK_HBM_GBPS,
                       "how": f"{n} (flush, call) pairs back to back less {n} flushes alone, "
                              "one event pair around each sequence; median of 3"}}


def prefill_run(n=100):
    """Prefill with prefix reuse: the joining sequence's 512 new tokens attend
    causally over its 1536 positions (1024 reused from the tree). Event-timed
    back-to-back calls on the launch stream, enqueued behind a spin kernel so
    the host's per-call cost stays out of the figure."""
    import numpy as np
    import torch

    from paper_2402_15220_amd.cache import Cache
    from paper_2402_15220_amd.roofline import PEAK_MFMA_TFLOPS
    from workloads import make_prefill_join

    pj = make_prefill_join()
    wl = pj.static
    cache = Cache(wl.c, wl.H, wl.d, 400, dtype=torch.float16)
    seg_dev = [(torch.from_numpy(s.k).cuda(), torch.from_numpy(s.v).cuda()) for s in wl.segments]
    matched = 0
    for s in wl.seqs + [pj.seq]:
        matched = cache.insert(s.seq_id, s.tokens(wl.segments), torch.cat([seg_dev[i][0] for i in s.segs]),
                               torch.cat([seg_dev[i][1] for i in s.segs]))
    sid = pj.seq.seq_id
    L = len(pj.seq.tokens(wl.segments))

    def timed(q):
        o = torch.empty_like(q)
        cache.prefill(sid, q, out=o)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(40_000_000)   # hold the stream while the calls are enqueued
        a.record()
        for _ in range(n):
            cache.prefill(sid, q, out=o)
        b.record()
        b.synchronize()
        us = a.elapsed_time(b) * 1e3 / n
        n_q = q.shape[0]
        ctx = sum(L - n_q + i + 1 for i in range(n_q))  # attended positions over all queries
        flops = 4 * wl.H * wl.d * ctx
        return us, flops, flops / (us * 1e-6) / 1e12

    q = torch.from_numpy(pj.q).cuda()
    n_q = pj.n_new
    us, flops, tflops = timed(q)
    # a short join: only the last 64 tokens are new (two query tiles' worth of
    # blocks per head at most, so the key range is split over blocks)
    us64, flops64, tflops64 = timed(q[-64:].contiguous())
    kv_bytes = 2 * L * wl.H * wl.d * 2
    cache.close()
    del cache, seg_dev
    torch.cuda.empty_cache()
    return {"workload": f"join_{wl.name}_plus_{n_q}_new_tokens", "n_q": n_q, "context": L,
            "matched": int(matched), "kernel": "kpf_kernel", "us_per_call": us,
            "tok_per_s": n_q / (us * 1e-6), "flops": flops, "tflops": tflops,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": PEAK_MFMA_TFLOPS["f16"],
                         "unit": "TFLOP/s", "frac": tflops / PEAK_MFMA_TFLOPS["f16"]},
            "kv_bytes": kv_bytes,
            "short_join": {"n_q": 64, "us_per_call": us64, "flops": flops64, "tflops": tflops64,
                           "kv_GBps": kv_bytes / (us64 * 1e-6) / 1e9}}


def dynamic_run():
    """The 64-step decode workload: every step appends one token to each live
    sequence (after churn on steps 16, 32, 48), then attends. Inputs of all
    steps are generated and copied to the GPU first; each step then times the
    library calls only: attention alone with events (q and o in the batch's
    own order through the row map of ca_attention_ordered), and the whole step
    (remove/insert, append, context preparation, attention) on the host clock
    up to a synchronisation. A first, pipelined pass runs the same
    steps with no synchronisation in between and reports wall time per step
    against the GPU's busy span (host work hidden under device work)."""
    import numpy as np
    import torch

    from paper_2402_15220_amd.cache import Cache
    from workloads import make_dynamic

    t_gen = time.perf_counter()
    wl = make_dynamic()
    steps = list(wl.steps())
    nodes = sum(-(-len(s) // wl.c) for s in wl.segments) + len(steps) * 128 // wl.c + 256
    cache = Cache(wl.c, wl.H, wl.d, nodes, dtype=torch.float16)
    seg_dev = {}

    def dev_seg(i):
        if i not in seg_dev:
            seg_dev[i] = (torch.from_numpy(wl.segments[i].k).cuda(), torch.from_numpy(wl.segments[i].v).cuda())
        return seg_dev[i]

    def full_kv(s):
        return (torch.cat([dev_seg(i)[0] for i in s.segs]), torch.cat([dev_seg(i)[1] for i in s.segs]))

    for s in wl.seqs:
        k, v = full_kv(s)
        cache.insert(s.seq_id, s.tokens(wl.segments), k, v)
        del k, v
    dev_steps = []
    for st in steps:
        added = []
        if st.churn:
            for s in st.churn.added:
                k, v = full_kv(s)
                added.append((s.seq_id, s.tokens(wl.segments), k, v))
        dev_steps.append((st, added, torch.from_numpy(st.k).cuda(), torch.from_numpy(st.v).cuda(),
                          torch.from_numpy(st.q).cuda()))
    q_rows = torch.empty((256, wl.H, wl.d), dtype=torch.float16, device="cuda")
    o = torch.empty_like(q_rows)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    st0 = cache.stats()
    up0, pa0 = st0["uploads"], st0["patches"]

    def one_step(i, st, added, k, v, q):
        if st.churn:
            for sid in st.churn.removed:
                cache.remove(sid)
            for sid, toks, kk, vv in added:
                cache.insert(sid, toks, kk, vv)
        cache.append(st.live, st.tokens, k, v)
        cache.prepare()                 # the step's context, ahead of the launches
        return len(st.live)

    # Pipelined pass: no synchronisation between steps, so the host work of a
    # step (tree update, context patch or rebuild and upload, launches) runs
    # while the GPU still executes earlier steps (latency hiding). Runs on a
    # copy of the starting tree and leaves it as the timed pass expects.
    pipe = {}
    if len(dev_steps) > 0:
        # one call on the starting tree first: one-time costs (the library's
        # device and pinned allocations) stay out of the pipelined span
        q_rows.zero_()
        n0 = cache.num_seqs()
        cache.attention(q_rows[:n0], out=o[:n0], seq_ids=cache.seq_order())
        torch.cuda.synchronize()
        ga = torch.cuda.Event(enable_timing=True)
        gb = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ga.record()
        for i, (st, added, k, v, q) in enumerate(dev_steps):
            n = one_step(i, st, added, k, v, q)
            cache.attention(q, out=o[:n], seq_ids=st.live)   # q and o in the batch's own order
        gb.record()
        host_done = time.perf_counter()
        gb.synchronize()
        wall = time.perf_counter() - t0
        pipe = {"step_us_pipelined": wall * 1e6 / len(dev_steps),
                "host_enqueue_us_per_step": (host_done - t0) * 1e6 / len(dev_steps),
                "gpu_us_per_step_pipelined": ga.elapsed_time(gb) * 1e3 / len(dev_steps)}
        # back to the starting tree for the per-step timed pass
        for sid in list(cache.seq_order()):
            cache.remove(int(sid))
        for s in wl.seqs:
            k, v = full_kv(s)
            cache.insert(s.seq_id, s.tokens(wl.segments), k, v)
            del k, v
        torch.cuda.synchronize()
        st0 = cache.stats()
        up0, pa0 = st0["uploads"], st0["patches"]

    att_us, step_us, rows = [], [], []
    for i, (st, added, k, v, q) in enumerate(dev_steps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        n = one_step(i, st, added, k, v, q)
        a.record()
        cache.attention(q, out=o[:n], seq_ids=st.live)
        b.record()
        b.synchronize()
        step_us.append((time.perf_counter() - t0) * 1e6)
        att_us.append(a.elapsed_time(b) * 1e3)
        rows.append(n)
    st1 = cache.stats()
    up, pa = st1["uploads"] - up0, st1["patches"] - pa0
    cache.close()
    del cache, seg_dev, dev_steps
    torch.cuda.empty_cache()
    return {"workload": wl.name, "steps": len(att_us), "rows_per_step": int(np.median(rows)),
            "attention_us_mean": float(np.mean(att_us)), "attention_us_median": float(np.median(att_us)),
            "step_us_mean": float(np.mean(step_us)), "step_us_median": float(np.median(step_us)),
            "tok_per_s": float(sum(rows) / (sum(att_us) * 1e-6)),
            "context_uploads": int(up), "context_patched_in_place": int(pa), "setup_s": t_gen,
            **pipe}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform

    return platform.processor() or platform.machine()


def _oracle_rows(tree, row_seq, q, scale, rows, pool, threads):
    """The oracle's dense_attention_rows over `rows`, split into groups that
    run on a thread pool (NumPy releases the GIL in its copies and
    reductions); the oracle itself is unchanged."""
    import numpy as np

    from oracle import dense_attention_rows

    rows = list(rows)
    if threads <= 1:
        return dense_attention_rows(tree, row_seq, q, scale, rows=rows)
    per = -(-len(rows) // threads)
    groups = [rows[i:i + per] for i in range(0, len(rows), per)]
    return np.concatenate(list(pool.map(
        lambda g: dense_attention_rows(tree, row_seq, q, scale, rows=g), groups)))


def cpu_baseline(wl, rows, seconds, with_dynamic=True):
    """The oracle (float64 NumPy, as written) timed on the host: whole calls
    of the bench workload (all B rows, all heads) with the rows split over
    one thread per host CPU (at most 16, the GPU's host share), repeated for
    about `seconds`; one single-threaded call; the oracle's tree operations
    (building the bench tree); and, on the 64-step decode workload, the
    oracle's per-step tree operations and attention for a sample of steps."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import OracleTree

    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    t = OracleTree(c=wl.c)
    t0 = time.perf_counter()
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        t.insert(s.seq_id, s.tokens(wl.segments), k, v)
    tree_build_s = time.perf_counter() - t0
    q = wl.q[rows]
    with ThreadPoolExecutor(threads) as pool:
        _oracle_rows(t, rows, q, wl.scale, range(len(rows)), pool, threads)   # warm-up
        n = 0
        t0 = time.perf_counter()
        while True:
            _oracle_rows(t, rows, q, wl.scale, range(len(rows)), pool, threads)
            n += 1
            if time.perf_counter() - t0 >= seconds:
                break
        el = time.perf_counter() - t0
        t0 = time.perf_counter()
        _oracle_rows(t, rows, q, wl.scale, range(len(rows)), pool, 1)
        single_s = time.perf_counter() - t0
        dyn = dynamic_oracle_sample(pool, threads) if with_dynamic else None
    c1 = config1_oracle()
    out = {"value": n * len(rows) / el, "unit": "tok/s", "cores": threads, "kind": "oracle",
           "sample": f"{n} full calls of the workload (B={len(rows)} rows x {wl.H} heads, float64 "
                     f"NumPy, rows split over {threads} threads), after one untimed call",
           "ms_per_call": el * 1e3 / n, "cpu": _cpu_model(),
           "host_cpus": len(os.sched_getaffinity(0)),
           "single_thread": {"ms_per_call": single_s * 1e3, "tok_per_s": len(rows) / single_s},
           "tree_ops": {"what": f"building the bench tree: {len(wl.seqs)} inserts with K/V rows",
                        "ms": tree_build_s * 1e3},
           "config1_single_thread": c1}
    if dyn is not None:
        out["dynamic"] = dyn
    return out


def config1_oracle(repeats=20):
    """The oracle on the tiny fp32 tree (4 rows of a 128-token prompt plus 32
    unique tokens, 2 heads, d=64), single-threaded: tree build and the call's
    attention (median of `repeats`)."""
    import numpy as np

    from oracle import OracleTree
    from workloads import make_static

    wl = make_static(1)
    t = OracleTree(c=wl.c)
    t0 = time.perf_counter()
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        t.insert(s.seq_id, s.tokens(wl.segments), k, v)
    build_ms = (time.perf_counter() - t0) * 1e3
    rows = [s.seq_id for s in wl.seqs]
    q = wl.q[rows]
    ts = []
    for _ in range(repeats):
        t0 = time.perf_counter()
        _oracle_rows(t, rows, q, wl.scale, range(len(rows)), None, 1)
        ts.append(time.perf_counter() - t0)
    ms = float(np.median(ts)) * 1e3
    return {"workload": wl.name, "tree_build_ms": build_ms, "ms_per_call": ms,
            "tok_per_s": len(rows) / (ms * 1e-3)}


def dynamic_oracle_sample(pool, threads, sample_steps=(0, 16)):
    """The oracle on the 64-step decode workload: its tree is built (timed
    as tree operations), then it runs the steps in order (churn, one append
    per row), timing each step's tree operations; at the sampled steps it
    also computes the step's attention for every row."""
    import numpy as np

    from oracle import OracleTree
    from workloads import make_dynamic

    wl = make_dynamic()
    t = OracleTree(c=wl.c)
    t0 = time.perf_counter()
    for s in wl.seqs:
        k, v = s.kv(wl.segments)
        t.insert(s.seq_id, s.tokens(wl.segments), k, v)
    build_s = time.perf_counter() - t0
    ops_s, att_s = [], []
    last = max(sample_steps)
    for st in wl.steps():
        t0 = time.perf_counter()
        if st.churn:
            for sid in st.churn.removed:
                t.remove(sid)
            for s in st.churn.added:
                k, v = s.kv(wl.segments)
                t.insert(s.seq_id, s.tokens(wl.segments), k, v)
        t.append_batch(st.live, st.tokens, st.k, st.v)
        ops_s.append(time.perf_counter() - t0)
        if st.step in sample_steps:
            # rows in the caller's (sorted id) order: the result does not depend on it
            t0 = time.perf_counter()
            _oracle_rows(t, st.live, st.q, wl.scale, range(len(st.live)), pool, threads)
            att_s.append(time.perf_counter() - t0)
        if st.step >= last:
            break
    return {"workload": wl.name, "initial_tree_build_ms": build_s * 1e3,
            "tree_ops_ms_per_step_mean": float(np.mean(ops_s)) * 1e3,
            "tree_ops_steps_timed": len(ops_s),
            "attention_ms_per_step": [a * 1e3 for a in att_s],
            "attention_steps": list(sample_steps), "threads": threads,
            "tok_per_s": len(st.live) * len(att_s) / sum(att_s)}


if __name__ == "__main__":
    main()
