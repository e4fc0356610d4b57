"""Host tree of the HIP library against the oracle, bit-exact, on the CPU.

The library runs in table-only mode (no pools, no GPU): every tree operation
goes through the C ABI and the canonical tables it exports must equal the
oracle's after every operation. Also: error paths and the exported symbols.
"""
import os
import re

import numpy as np
import pytest

from oracle import OracleTree, PoolExhausted, tables
from paper_2402_15220_amd import binding as B
from prefix_util import max_lcp, probes
from workloads import make_dynamic, make_static, random_op_script

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib_or_skip():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("library not built: run python -m paper_2402_15220_amd.build")
    return B.load()


def _same(lib_tab, ora_tab):
    o = ora_tab.as_dict()
    assert set(lib_tab) == set(o)
    for k in o:
        assert np.array_equal(np.asarray(lib_tab[k]), np.asarray(o[k])), k


def test_exports_every_declared_symbol():
    lib = _lib_or_skip()
    with open(os.path.join(ROOT, "include", "chunkattn.h")) as f:
        text = f.read()
    declared = set(re.findall(r"\b(ca_[a-z_]+)\s*\(", text))
    assert declared == set(B.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_fig2_through_abi():
    _lib_or_skip()
    h = B.ca_create(4, 1, 64, B.CA_FP16, 64)
    t = OracleTree(c=4, with_kv=False)
    shared = list(range(10, 22))
    for sid, suf in enumerate([range(30, 34), range(40, 48), range(50, 58)]):
        toks = np.array(shared + list(suf), np.int32)
        assert B.ca_insert(h, sid, toks) == t.insert(sid, toks)
    _same(B.ca_export_tables(h), tables(t))
    assert list(B.ca_seq_order(h)) == [0, 1, 2]
    B.ca_destroy(h)


def _apply(h, t, op):
    """Apply one op to both; return the oracle's exception type or None."""
    err = None
    try:
        if op[0] == "insert":
            r = t.insert(op[1], op[2])
        elif op[0] == "extend":
            r = t.extend(op[1], op[2])
        elif op[0] == "append":
            r = t.append_batch(op[1], op[2])
        else:
            r = t.remove(op[1])
    except PoolExhausted:
        err = B.CA_ERR_NOMEM
        r = None
    lib_err = None
    try:
        if op[0] == "insert":
            lr = B.ca_insert(h, op[1], op[2])
        elif op[0] == "extend":
            lr = B.ca_extend(h, op[1], op[2])
        elif op[0] == "append":
            lr = B.ca_append_batch(h, op[1], op[2])
        else:
            lr = B.ca_remove(h, op[1])
    except B.ChunkAttnError as e:
        lib_err = e.status
        lr = None
    assert lib_err == err, (op, lib_err, err)
    if err is None and op[0] in ("insert", "extend"):
        assert lr == r
    return err


@pytest.mark.parametrize("seed", range(40))
def test_random_scripts_bit_exact(seed):
    _lib_or_skip()
    c = 1 + seed % 5
    slots = None if seed % 3 else 6 + seed % 7   # some runs with a tight pool
    n_slots = slots if slots is not None else 1 << 20
    h = B.ca_create(c, 1, 64, B.CA_FP16, n_slots)
    t = OracleTree(c=c, num_slots=slots, with_kv=False)
    alphabet = 2 + seed % 3
    live = {}                      # sid -> tokens, kept by the test itself
    rng = np.random.default_rng(900 + seed)
    for op in random_op_script(seed, n_ops=80, alphabet=alphabet, max_len=3 * c + 4):
        # keep the script valid when a NOMEM insert was refused
        if op[0] in ("extend", "remove") and op[1] not in live:
            continue
        if op[0] == "append":
            ids = [s for s in op[1] if s in live]
            if not ids:
                continue
            op = ("append", ids, op[2][:len(ids)])
        err = _apply(h, t, op)
        if err is None:
            if op[0] == "insert":
                live[op[1]] = np.asarray(op[2], np.int32)
            elif op[0] == "extend":
                live[op[1]] = np.concatenate([live[op[1]], op[2]]).astype(np.int32)
            elif op[0] == "append":
                for sid, tok in zip(op[1], op[2]):
                    live[sid] = np.concatenate([live[sid], [tok]]).astype(np.int32)
            else:
                del live[op[1]]
        t.check_invariants()
        _same(B.ca_export_tables(h), tables(t))
        st = B.ca_stats(h)
        assert st["slots_used"] == t.slots_in_use()
        # prefix lookup through the ABI: oracle and brute force agree with it
        for p in probes(rng, list(live.values()), 6, alphabet):
            got = B.ca_match(h, p)
            assert got == t.match(p) == max_lcp(live.values(), p), (p, got)
    B.ca_destroy(h)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_static_configs_bit_exact(cfg):
    _lib_or_skip()
    wl = make_static(cfg)
    h = B.ca_create(wl.c, wl.H, wl.d, B.CA_FP16, 1 << 16)
    t = OracleTree(c=wl.c, with_kv=False)
    for s in wl.seqs:
        toks = s.tokens(wl.segments)
        assert B.ca_insert(h, s.seq_id, toks) == t.insert(s.seq_id, toks)
    _same(B.ca_export_tables(h), tables(t))
    B.ca_destroy(h)


def test_dynamic_config_replay_bit_exact():
    """64 decode steps with churn over 128 rows; tables equal after every step."""
    _lib_or_skip()
    wl = make_dynamic()
    h = B.ca_create(wl.c, wl.H, wl.d, B.CA_FP16, 1 << 16)
    t = OracleTree(c=wl.c, with_kv=False)
    for s in wl.seqs:
        toks = s.tokens(wl.segments)
        assert B.ca_insert(h, s.seq_id, toks) == t.insert(s.seq_id, toks)
    uploads_structural = 0
    live = {s.seq_id: s.tokens(wl.segments) for s in wl.seqs}
    rng = np.random.default_rng(55)
    for st in wl.steps():
        if st.churn:
            for sid in st.churn.removed:
                B.ca_remove(h, sid)
                t.remove(sid)
                del live[sid]
            for s in st.churn.added:
                toks = s.tokens(wl.segments)
                # the join's prefix lookup finds exactly the shared prompt
                assert B.ca_match(h, toks) == t.match(toks) == 2048
                assert B.ca_insert(h, s.seq_id, toks) == t.insert(s.seq_id, toks) == 2048
                live[s.seq_id] = toks
        B.ca_append_batch(h, st.live, st.tokens)
        t.append_batch(st.live, st.tokens)
        for sid, tok in zip(st.live, st.tokens):
            live[int(sid)] = np.concatenate([live[int(sid)], [tok]]).astype(np.int32)
        _same(B.ca_export_tables(h), tables(t))
        assert list(np.sort(B.ca_seq_order(h))) == list(st.live)
        for p in probes(rng, list(live.values()), 4, 32000):
            assert B.ca_match(h, p) == t.match(p) == max_lcp(live.values(), p)
        uploads_structural += 1
    t.check_invariants()
    B.ca_destroy(h)


def test_match_arguments_and_edge_cases():
    """ca_match: refused arguments change nothing; an empty tree matches
    nothing; a lookup may end inside a chunk (a split candidate) or run past
    every stored path; a lookup never changes the tree."""
    _lib_or_skip()
    h = B.ca_create(4, 1, 64, B.CA_FP16, 4096)
    assert B.ca_match(h, [1, 2, 3]) == 0
    B.ca_insert(h, 0, [1, 2, 3, 4, 5, 6])
    B.ca_insert(h, 1, [1, 2, 9])
    before = B.ca_export_tables(h)
    for bad in ([], [3, -1], [-5]):
        with pytest.raises(B.ChunkAttnError) as ei:
            B.ca_match(h, np.asarray(bad, np.int32))
        assert ei.value.status == B.CA_ERR_INVALID
    assert B.ca_match(h, [1, 2, 3]) == 3               # inside X' = [3, 4]
    assert B.ca_match(h, [1, 2, 3, 4, 5, 6] + [7] * 1000) == 6
    assert B.ca_match(h, [1, 2, 9, 9]) == 3
    assert B.ca_match(h, [2]) == 0
    long = np.arange(100000, dtype=np.int32)
    B.ca_insert(h, 2, long[:5000])
    assert B.ca_match(h, long) == 5000
    assert B.ca_match(h, long[:4321]) == 4321
    B.ca_remove(h, 2)
    after = B.ca_export_tables(h)
    for k in before:
        assert np.array_equal(before[k], after[k]), k
    B.ca_destroy(h)


def test_error_paths_leave_state_unchanged():
    _lib_or_skip()
    h = B.ca_create(2, 1, 64, B.CA_FP16, 3)
    B.ca_insert(h, 0, [1, 2, 3, 4])
    before = B.ca_export_tables(h)

    def unchanged():
        after = B.ca_export_tables(h)
        for k in before:
            assert np.array_equal(before[k], after[k]), k

    cases = [
        (lambda: B.ca_insert(h, 1, [1, 9, 9, 9]), B.CA_ERR_NOMEM),
        (lambda: B.ca_insert(h, 0, [5]), B.CA_ERR_EXISTS),
        (lambda: B.ca_extend(h, 7, [5]), B.CA_ERR_NOT_FOUND),
        (lambda: B.ca_remove(h, 7), B.CA_ERR_NOT_FOUND),
        (lambda: B.ca_insert(h, 1, np.zeros(0, np.int32)), B.CA_ERR_INVALID),
        (lambda: B.ca_insert(h, 1, [3, -1]), B.CA_ERR_INVALID),
        (lambda: B.ca_extend(h, 0, [5, 6, 7]), B.CA_ERR_NOMEM),
        (lambda: B.ca_append_batch(h, [0, 0], [1, 1]), B.CA_ERR_INVALID),
        (lambda: B.ca_append_batch(h, [0, 5], [1, 1]), B.CA_ERR_NOT_FOUND),
        (lambda: B.ca_attention(h, None, None, 0.0, None, 0), B.CA_ERR_INVALID),
    ]
    for fn, status in cases:
        with pytest.raises(B.ChunkAttnError) as ei:
            fn()
        assert ei.value.status == status, ei.value
        assert B.ca_last_error()
        unchanged()
    # NOMEM of a batch that needs two slots with one left: all or nothing
    B.ca_insert(h, 1, [5])           # takes the last slot; both terminals full
    before = B.ca_export_tables(h)
    with pytest.raises(B.ChunkAttnError) as ei:
        B.ca_append_batch(h, [1, 0], [6, 7])
    assert ei.value.status == B.CA_ERR_NOMEM
    unchanged()
    B.ca_destroy(h)


@pytest.mark.parametrize("bad", [
    dict(chunk_size=0), dict(num_heads=0), dict(head_dim=96), dict(dtype=7), dict(num_slots=0),
    dict(head_stride=4 * 64 - 8),                                  # a tile is c*d = 256 elements
    dict(num_heads=4, head_stride=4 * 64, slot_stride=3 * 4 * 64),  # slots would overlap
    dict(head_stride=4 * 64 + 4)])                                 # not a multiple of 16 bytes
def test_create_rejects_bad_config(bad):
    _lib_or_skip()
    cfg = dict(chunk_size=4, num_heads=1, head_dim=64, dtype=B.CA_FP16, num_slots=8)
    cfg.update(bad)
    with pytest.raises(B.ChunkAttnError) as ei:
        B.ca_create(**cfg)
    assert ei.value.status == B.CA_ERR_INVALID


def test_work_lists_follow_lazy_context_rule():
    """Section 3.3: the context is rebuilt only on structural change.

    In table-only mode nothing is uploaded, but the workspace size tracks the
    structure: appends that only fill a private chunk leave it unchanged.
    """
    _lib_or_skip()
    h = B.ca_create(4, 2, 64, B.CA_FP16, 64)
    B.ca_insert(h, 0, [1, 2, 3, 4, 5])
    B.ca_insert(h, 1, [1, 2, 3, 4, 6])
    ws0 = B.ca_workspace_size(h)
    B.ca_append_batch(h, [0, 1], [7, 7])   # fills the private chunks [5], [6]
    assert B.ca_workspace_size(h) == ws0
    B.ca_destroy(h)


def _checked_cache(*args):
    """A table-only cache that compares every in-place context update with a
    full rebuild (a difference makes ca_stats raise)."""
    old = os.environ.get("CA_CHECK_PATCH")
    os.environ["CA_CHECK_PATCH"] = "1"
    try:
        return B.ca_create(*args)
    finally:
        if old is None:
            del os.environ["CA_CHECK_PATCH"]
        else:
            os.environ["CA_CHECK_PATCH"] = old


def test_decode_growth_updates_context_in_place():
    """Section 3.3 (lazy context): decode growth that only adds private chunks
    patches the per-row lists; each patch equals a full rebuild, through 64
    decode steps with churn (where the context is rebuilt)."""
    _lib_or_skip()
    wl = make_dynamic()
    h = _checked_cache(wl.c, wl.H, wl.d, B.CA_FP16, 1 << 16)
    for s in wl.seqs:
        B.ca_insert(h, s.seq_id, s.tokens(wl.segments))
    B.ca_seq_order(h)
    for st in wl.steps():
        if st.churn:
            for sid in st.churn.removed:
                B.ca_remove(h, sid)
            for s in st.churn.added:
                B.ca_insert(h, s.seq_id, s.tokens(wl.segments))
        B.ca_append_batch(h, st.live, st.tokens)
        B.ca_seq_order(h)          # brings the context up to date
        B.ca_stats(h)              # raises if a patch differed from a rebuild
    assert B.ca_stats(h)["patches"] >= 40
    B.ca_destroy(h)


@pytest.mark.parametrize("seed", range(12))
def test_random_growth_patches_match_rebuild(seed):
    """Small trees, small chunks: appends and extends that grow private chains,
    mixed with inserts, splits and removals (which rebuild). Every third seed
    runs the partial-free schedule's work lists."""
    _lib_or_skip()
    c = 1 + seed % 4
    h = _checked_cache(c, 1, 64, B.CA_FP16, 1 << 20)
    if seed % 3 == 2:
        B.ca_set_tuning(h, schedule=4)
    live = set()
    for op in random_op_script(seed, n_ops=120, alphabet=3, max_len=2 * c + 3):
        if op[0] in ("extend", "remove") and op[1] not in live:
            continue
        if op[0] == "insert":
            B.ca_insert(h, op[1], op[2])
            live.add(op[1])
        elif op[0] == "extend":
            B.ca_extend(h, op[1], op[2])
        elif op[0] == "append":
            ids = [s for s in op[1] if s in live]
            if not ids:
                continue
            B.ca_append_batch(h, ids, op[2][:len(ids)])
        elif op[0] == "remove":
            B.ca_remove(h, op[1])
            live.discard(op[1])
        B.ca_seq_order(h)
        B.ca_stats(h)
    B.ca_destroy(h)


def _align(x, a=256):
    return (x + a - 1) // a * a


def test_partial_free_workspace_is_one_accumulator_per_row():
    """Section 3.3 (further optimizations): the partial-free schedule keeps one
    (O, m, n) per (sequence, head), however many shared segments and tree
    levels a row's path crosses; the partial-writing schedules keep one per
    (segment, row, head) plus one per split or partial-writing item."""
    _lib_or_skip()
    H, d = 2, 64
    h = B.ca_create(2, H, d, B.CA_FP16, 256)
    # three levels of sharing: [1..8] by all, [9, 10] by 0-2, [11, 12] by 0-1
    for sid, tail in enumerate([[9, 10, 11, 12, 20], [9, 10, 11, 12, 21], [9, 10, 22], [23]]):
        B.ca_insert(h, sid, list(range(1, 9)) + tail)
    Bn = 4
    B.ca_set_tuning(h, seg_chunks=1, schedule=2)
    ws2 = B.ca_workspace_size(h)
    B.ca_set_tuning(h, schedule=4)
    ws4 = B.ca_workspace_size(h)
    assert ws4 == _align(Bn * H * d * 4) + _align(Bn * H * 2 * 4)
    # 4 + 1 + 1 single-chunk segments over 4, 3, 2 rows, plus 4 own items
    n2 = 4 * 4 + 1 * 3 + 1 * 2 + 4
    assert ws2 == _align(n2 * H * d * 4) + _align(n2 * H * 2 * 4)
    B.ca_set_tuning(h, seg_chunks=-1)   # automatic: one segment per run
    assert B.ca_stats(h)["seg_chunks"] == 64
    assert B.ca_workspace_size(h) == ws4
    B.ca_destroy(h)


def _auto_segment(c, H, seqs):
    h = B.ca_create(c, H, 128, B.CA_FP16, 1 << 14)
    for sid, toks in enumerate(seqs):
        B.ca_insert(h, sid, toks)
    B.ca_workspace_size(h)  # builds the work lists
    seg = B.ca_stats(h)["seg_chunks"]
    B.ca_destroy(h)
    return seg


def _prompt_plus_one(rows, n_shared):
    return [list(range(n_shared)) + [1_000_000 + r] for r in range(rows)]


@pytest.mark.parametrize("case,want", [
    ("config2", 4),          # quota 16 chunks x 2 row blocks x 32 heads / 256 CUs = 4
    ("config3", 16),         # quota 16
    ("config4", 8),          # quota 16, capped at twice the 4 private chunks (2,048 blocks)
    ("b32_p4096_u1", 16),    # quota 16; one round of blocks: no private cap
    ("b96_p2048_u1", 16),    # quota 24 -> 32, base cap 16; one private chunk: no private cap
    ("b48_p2048_u1", 16),    # quota 12 -> 16
    ("b48_p1024_u1", 8),     # quota 6 -> 8
])
def test_automatic_segment_length(case, want):
    """The automatic chunk-first segment length: about one block per compute
    unit (256 on MI355X), rounded up to a power of two, at most 16 chunks
    unless the private stream is long enough to hide longer chains, and at
    most twice the longest private chunk list when the sequence-first blocks
    take more than one round of resident slots and stream at least 4 chunks
    each."""
    _lib_or_skip()
    if case.startswith("config"):
        wl = make_static(int(case[-1]))
        seqs = [s.tokens(wl.segments) for s in wl.seqs]
        c, H = wl.c, wl.H
    else:
        rows, n_shared = {"b32_p4096_u1": (32, 4096), "b96_p2048_u1": (96, 2048),
                          "b48_p2048_u1": (48, 2048), "b48_p1024_u1": (48, 1024)}[case]
        seqs, c, H = _prompt_plus_one(rows, n_shared), 64, 32
    assert _auto_segment(c, H, seqs) == want


def test_prepare_on_a_table_only_cache():
    """ca_prepare builds the host context only (nothing to upload)."""
    _lib_or_skip()
    h = B.ca_create(4, 2, 64, B.CA_FP16, 64)
    assert B.ca_prepare(h) is False                 # empty tree
    B.ca_insert(h, 0, [1, 2, 3, 4, 5])
    B.ca_insert(h, 1, [1, 2, 3, 4, 6])
    assert B.ca_prepare(h) is False
    assert B.ca_workspace_size(h) > 0
    B.ca_destroy(h)


def test_host_allocation_failure_is_a_status():
    """A host allocation failure inside the library comes back as CA_ERR_HOST
    with a message instead of an exception crossing the C ABI: a child
    process caps its address space 128 MiB above what it uses, then inserts
    a 10^8-token sequence into a table-only cache (the tree's chunks need
    ~400 MB)."""
    import subprocess
    import sys
    _lib_or_skip()
    script = (
        "import resource, sys\n"
        "import numpy as np\n"
        f"sys.path.insert(0, {ROOT!r})\n"
        "from paper_2402_15220_amd import binding as B\n"
        "h = B.ca_create(1024, 2, 64, B.CA_FP16, 1 << 20)\n"
        "toks = (np.arange(100_000_000, dtype=np.int64) % 50000).astype(np.int32)\n"
        "vm = int(open('/proc/self/statm').read().split()[0]) * resource.getpagesize()\n"
        "resource.setrlimit(resource.RLIMIT_AS, (vm + (128 << 20), resource.getrlimit(resource.RLIMIT_AS)[1]))\n"
        "try:\n"
        "    B.ca_insert(h, 1, toks)\n"
        "    print('inserted')\n"
        "except B.ChunkAttnError as e:\n"
        "    print('status', e.status, str(e))\n")
    r = subprocess.run([sys.executable, "-c", script], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    assert f"status {B.CA_ERR_HOST}" in r.stdout, r.stdout + r.stderr[-2000:]
    assert "out of host memory" in r.stdout


@pytest.mark.parametrize("seed", range(12))
def test_random_calls_with_invalid_arguments(seed):
    """Valid and invalid calls mixed at random through the C ABI: every call
    returns the status the oracle (or the documented argument rules) gives,
    a refused call changes nothing observable, and an accepted one leaves the
    tables equal to the oracle's. Invalid kinds: duplicate and unknown ids,
    empty and negative tokens, repeated ids in a batch, null arrays with a
    positive count, a seq_order buffer that is too small, and pool
    exhaustion."""
    import ctypes
    lib = _lib_or_skip()
    rng = np.random.default_rng(7000 + seed)
    c = 1 + seed % 4
    slots = 8 + seed % 5
    h = B.ca_create(c, 1, 64, B.CA_FP16, slots)
    t = OracleTree(c=c, num_slots=slots, with_kv=False)
    live = set()
    next_sid = 0
    ora_err = {KeyError: None, ValueError: B.CA_ERR_INVALID, PoolExhausted: B.CA_ERR_NOMEM}

    def toks(n):
        return rng.integers(0, 3, n).astype(np.int32)

    def lib_status(fn):
        try:
            fn()
            return B.CA_OK
        except B.ChunkAttnError as e:
            return e.status

    def ora_status(fn, key_status):
        try:
            fn()
            return B.CA_OK
        except PoolExhausted:
            return B.CA_ERR_NOMEM
        except KeyError:
            return key_status
        except ValueError:
            return ora_err[ValueError]

    m = ctypes.c_int64()
    for _ in range(70):
        before = B.ca_export_tables(h)
        used = B.ca_stats(h)["slots_used"]
        kind = int(rng.integers(0, 12))
        ids = sorted(live)
        if kind == 0 or (kind in (1, 4, 6, 8) and not ids):
            sid, tk = next_sid, toks(int(rng.integers(1, 3 * c + 4)))
            want = ora_status(lambda: t.insert(sid, tk), B.CA_ERR_EXISTS)
            got = lib_status(lambda: B.ca_insert(h, sid, tk))
            if want == B.CA_OK:
                live.add(sid)
                next_sid += 1
        elif kind == 1:                                     # duplicate id
            sid = int(rng.choice(ids))
            want, got = B.CA_ERR_EXISTS, lib_status(lambda: B.ca_insert(h, sid, toks(2)))
        elif kind == 2:                                     # empty or negative tokens
            bad = np.zeros(0, np.int32) if rng.integers(0, 2) else np.array([1, -3], np.int32)
            want, got = B.CA_ERR_INVALID, lib_status(lambda: B.ca_insert(h, next_sid, bad))
        elif kind == 3:                                     # null array with n > 0
            fn = [lambda: lib.ca_insert(h, next_sid, None, 3, None, None, None, None),
                  lambda: lib.ca_extend(h, next_sid, None, 1, None, None, None, None),
                  lambda: lib.ca_match(h, None, 2, ctypes.byref(m)),
                  lambda: lib.ca_append_batch(h, 1, None, None, None, None, None)][int(rng.integers(0, 4))]
            want, got = B.CA_ERR_INVALID, fn()
        elif kind == 4:                                     # extend a live sequence
            sid, tk = int(rng.choice(ids)), toks(int(rng.integers(1, 2 * c + 2)))
            want = ora_status(lambda: t.extend(sid, tk), B.CA_ERR_NOT_FOUND)
            got = lib_status(lambda: B.ca_extend(h, sid, tk))
        elif kind == 5:                                     # unknown id
            fn = [lambda: B.ca_extend(h, 10_000, toks(1)), lambda: B.ca_remove(h, 10_000),
                  lambda: B.ca_append_batch(h, ids[:1] + [10_000], toks(len(ids[:1]) + 1))]
            want, got = B.CA_ERR_NOT_FOUND, lib_status(fn[int(rng.integers(0, 3))])
        elif kind == 6:                                     # batch append
            sel = [int(s) for s in rng.permutation(ids)[:int(rng.integers(1, len(ids) + 1))]]
            tk = toks(len(sel))
            want = ora_status(lambda: t.append_batch(sel, tk), B.CA_ERR_NOT_FOUND)
            got = lib_status(lambda: B.ca_append_batch(h, sel, tk))
        elif kind == 7:                                     # an id twice in a batch
            if not ids:
                continue
            sid = int(rng.choice(ids))
            want, got = B.CA_ERR_INVALID, lib_status(lambda: B.ca_append_batch(h, [sid, sid], toks(2)))
        elif kind == 8:                                     # remove a live sequence
            sid = int(rng.choice(ids))
            want = ora_status(lambda: t.remove(sid), B.CA_ERR_NOT_FOUND)
            got = lib_status(lambda: B.ca_remove(h, sid))
            if want == B.CA_OK:
                live.discard(sid)
        elif kind == 9:                                     # seq_order buffer too small
            n = B.ca_num_seqs(h)
            if n == 0:
                continue
            buf = np.zeros(n, np.int64)
            want = B.CA_ERR_INVALID
            got = lib.ca_seq_order(h, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), n - 1)
        elif kind == 10:                                    # prefix lookup, valid or empty
            tk = toks(int(rng.integers(0, 2 * c + 3)))
            got = lib.ca_match(h, tk.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), tk.shape[0],
                               ctypes.byref(m))
            want = B.CA_OK if tk.shape[0] > 0 else B.CA_ERR_INVALID
            if got == B.CA_OK:
                assert m.value == t.match(tk)
        else:                                               # null output pointers
            fn = [lambda: lib.ca_num_seqs(h, None), lambda: lib.ca_workspace_size(h, None),
                  lambda: lib.ca_export_tables(h, None)][int(rng.integers(0, 3))]
            want, got = B.CA_ERR_INVALID, fn()
        assert got == want, (kind, got, want)
        if got != B.CA_OK:
            after = B.ca_export_tables(h)
            for k in before:
                assert np.array_equal(before[k], after[k]), (kind, k)
            assert B.ca_stats(h)["slots_used"] == used
        t.check_invariants()
        _same(B.ca_export_tables(h), tables(t))
    B.ca_destroy(h)
