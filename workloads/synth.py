"""Seeded synthetic workloads shaped like the paper's decode experiments.

The paper's kernel workload (Experiments, microkernel evaluation) is batch
decoding with h=32 heads, head dim d=128, chunk size c=64 and FP16 tensors,
where every sequence starts with n_s shared prompt tokens. Real shared prompts
(the system prompts of Table 2 and Appendix A) are not available here; random
token ids of the same lengths stand in for them, and K/V/q are N(0,1) draws.

Recipe (identical for every consumer):
  * generator ``numpy.random.Generator(PCG64(1000 + config))``;
  * draw order: prompt/branch tokens, per-sequence unique tokens, then K and V
    once per segment (each shared prompt or branch once, each unique suffix
    once), then q;
  * values are drawn as float32 N(0,1) and rounded to the config dtype
    (round-to-nearest-even); the rounded values are the ground truth;
  * token ids are uniform in [0, 32000); the first token of a segment that
    starts a new branch is redrawn until it differs from the first tokens of
    its siblings, so the designed tree shape holds (``redraws`` counts them).

Nothing here builds a tree or computes attention.
"""
from __future__ import annotations

import dataclasses
import os
from typing import Iterator

import numpy as np

VOCAB = 32000

CONFIG_NAMES = {
    1: "tiny_p128_u32_b4_h2_d64_c16_fp32",
    2: "single_prompt_p1024_u512_b32_h32_d128_c64_fp16",
    3: "long_prompt_p4096_u512_b32_h32_d128_c64_fp16",
    4: "multi_prompt_2level_b64_h32_d128_c64_fp16",
    5: "dynamic_p2048_u64to1024_b128_h32_d128_c64_fp16_64steps",
}


@dataclasses.dataclass
class Segment:
    """A run of tokens with their K/V rows, [L], [L, H, d], [L, H, d]."""

    tokens: np.ndarray
    k: np.ndarray
    v: np.ndarray

    def __len__(self) -> int:
        return int(self.tokens.shape[0])


@dataclasses.dataclass
class Sequence:
    seq_id: int
    segs: list  # indices into the workload's segment list, root first

    def tokens(self, segments) -> np.ndarray:
        return np.concatenate([segments[s].tokens for s in self.segs])

    def kv(self, segments):
        k = np.concatenate([segments[s].k for s in self.segs], axis=0)
        v = np.concatenate([segments[s].v for s in self.segs], axis=0)
        return k, v

    def length(self, segments) -> int:
        return sum(len(segments[s]) for s in self.segs)


@dataclasses.dataclass
class StaticWorkload:
    config: int
    name: str
    H: int
    d: int
    c: int
    dtype: np.dtype
    scale: float
    segments: list
    seqs: list          # insert order; seq_id = position
    q: np.ndarray       # [B, H, d], indexed by seq_id
    redraws: int = 0

    @property
    def B(self) -> int:
        return len(self.seqs)


@dataclasses.dataclass
class ChurnEvent:
    removed: list       # seq ids removed (before the step's append)
    added: list         # Sequence objects inserted afterwards
    new_segments: dict  # segment index -> Segment for the added suffixes


@dataclasses.dataclass
class DecodeStep:
    step: int
    churn: ChurnEvent | None
    live: np.ndarray    # sorted live seq ids after churn, int64 [n]
    tokens: np.ndarray  # appended token per live seq, int32 [n]
    k: np.ndarray       # appended K rows [n, H, d]
    v: np.ndarray       # appended V rows [n, H, d]
    q: np.ndarray       # queries [n, H, d] in live (sorted id) order


@dataclasses.dataclass
class DynamicWorkload:
    """The 64-step decode workload: initial tree plus a generator of decode steps."""

    config: int
    name: str
    H: int
    d: int
    c: int
    dtype: np.dtype
    scale: float
    segments: list          # grows as churn adds suffixes
    seqs: list              # initial sequences, insert order
    n_steps: int
    churn_steps: tuple
    churn_count: int
    rng: np.random.Generator
    redraws: int = 0

    def steps(self) -> Iterator[DecodeStep]:
        """Yield the decode steps in order; each draw follows the previous."""
        rng = self.rng
        live = {s.seq_id: s for s in self.seqs}
        # first token of each live sequence's unique suffix (branch siblings)
        first = {s.seq_id: int(self.segments[s.segs[-1]].tokens[0]) for s in self.seqs}
        next_id = max(live) + 1
        prompt_seg = self.seqs[0].segs[0]
        for step in range(self.n_steps):
            churn = None
            if step in self.churn_steps:
                ids = np.array(sorted(live), dtype=np.int64)
                removed = sorted(int(x) for x in rng.choice(ids, size=self.churn_count, replace=False))
                for r in removed:
                    del live[r]
                    del first[r]
                lens = rng.integers(64, 1025, size=self.churn_count)
                added, new_segments = [], {}
                toks = []
                for L in lens:
                    t, nr = _draw_tokens(rng, int(L), set(first.values()))
                    self.redraws += nr
                    first[next_id] = int(t[0])
                    toks.append((next_id, t))
                    next_id += 1
                for sid, t in toks:
                    k = _draw_values(rng, (len(t), self.H, self.d), self.dtype)
                    v = _draw_values(rng, (len(t), self.H, self.d), self.dtype)
                    idx = len(self.segments)
                    seg = Segment(t, k, v)
                    self.segments.append(seg)
                    new_segments[idx] = seg
                    s = Sequence(sid, [prompt_seg, idx])
                    added.append(s)
                    live[sid] = s
                churn = ChurnEvent(removed, added, new_segments)
            ids = np.array(sorted(live), dtype=np.int64)
            n = ids.shape[0]
            tokens = rng.integers(0, VOCAB, size=n).astype(np.int32)
            k = _draw_values(rng, (n, self.H, self.d), self.dtype)
            v = _draw_values(rng, (n, self.H, self.d), self.dtype)
            q = _draw_values(rng, (n, self.H, self.d), self.dtype)
            yield DecodeStep(step, churn, ids, tokens, k, v, q)


def _draw_tokens(rng, n, forbidden_first):
    t = rng.integers(0, VOCAB, size=n).astype(np.int32)
    redraws = 0
    while int(t[0]) in forbidden_first:
        t[0] = np.int32(rng.integers(0, VOCAB))
        redraws += 1
    return t, redraws


def _draw_values(rng, shape, dtype):
    return rng.standard_normal(size=shape, dtype=np.float32).astype(dtype)


def _spec(config):
    if config == 1:
        return dict(H=2, d=64, c=16, dtype=np.dtype(np.float32))
    if config in (2, 3, 4, 5):
        return dict(H=32, d=128, c=64, dtype=np.dtype(np.float16))
    raise ValueError(f"unknown config {config}")


def make_static(config: int) -> StaticWorkload:
    """Configs 1-4: a tree built once and one decode step of queries."""
    sp = _spec(config)
    H, d, c, dt = sp["H"], sp["d"], sp["c"], sp["dtype"]
    rng = np.random.Generator(np.random.PCG64(1000 + config))
    redraws = 0
    seg_tokens = []   # token arrays in segment order
    seqs = []
    if config in (1, 2, 3):
        P, U, B = {1: (128, 32, 4), 2: (1024, 512, 32), 3: (4096, 512, 32)}[config]
        prompt, nr = _draw_tokens(rng, P, set())
        redraws += nr
        seg_tokens.append(prompt)
        firsts = set()
        for i in range(B):
            t, nr = _draw_tokens(rng, U, firsts)
            redraws += nr
            firsts.add(int(t[0]))
            seg_tokens.append(t)
            seqs.append(Sequence(i, [0, 1 + i]))
    else:  # two roots, two branches under each, 16 suffixes per branch
        roots = []
        rf = set()
        for _ in range(2):
            t, nr = _draw_tokens(rng, 1024, rf)
            redraws += nr
            rf.add(int(t[0]))
            roots.append(len(seg_tokens))
            seg_tokens.append(t)
        branches = []
        for r in roots:
            bf = set()
            for _ in range(2):
                t, nr = _draw_tokens(rng, 1024, bf)
                redraws += nr
                bf.add(int(t[0]))
                branches.append((r, len(seg_tokens)))
                seg_tokens.append(t)
        sid = 0
        for r, b in branches:
            sf = set()
            for _ in range(16):
                t, nr = _draw_tokens(rng, 256, sf)
                redraws += nr
                sf.add(int(t[0]))
                seqs.append(Sequence(sid, [r, b, len(seg_tokens)]))
                seg_tokens.append(t)
                sid += 1
    segments = []
    for t in seg_tokens:
        k = _draw_values(rng, (len(t), H, d), dt)
        v = _draw_values(rng, (len(t), H, d), dt)
        segments.append(Segment(t, k, v))
    q = _draw_values(rng, (len(seqs), H, d), dt)
    return StaticWorkload(config, CONFIG_NAMES[config], H, d, c, dt, 1.0 / np.sqrt(d),
                          segments, seqs, q, redraws)


def make_dynamic(config: int = 5, n_steps: int = 64, B: int = 128,
                 prompt_len: int = 2048, H: int | None = None, d: int | None = None) -> DynamicWorkload:
    """Shared prompt plus suffixes of U[64,1024] tokens, then decode.

    Churn: before steps 16, 32 and 48, round(0.1*B) live sequences chosen
    uniformly without replacement leave, and as many new ones (the same prompt
    plus a fresh suffix) join with ids counting up from B.
    ``H``/``d``/``B``/``prompt_len`` may be shrunk for fast tests; the draw
    order is unchanged.
    """
    sp = _spec(config)
    H = sp["H"] if H is None else H
    d = sp["d"] if d is None else d
    c, dt = sp["c"], sp["dtype"]
    rng = np.random.Generator(np.random.PCG64(1000 + config))
    redraws = 0
    prompt, nr = _draw_tokens(rng, prompt_len, set())
    redraws += nr
    lens = rng.integers(64, 1025, size=B)
    seg_tokens = [prompt]
    firsts = set()
    seqs = []
    for i in range(B):
        t, nr = _draw_tokens(rng, int(lens[i]), firsts)
        redraws += nr
        firsts.add(int(t[0]))
        seg_tokens.append(t)
        seqs.append(Sequence(i, [0, 1 + i]))
    segments = []
    for t in seg_tokens:
        k = _draw_values(rng, (len(t), H, d), dt)
        v = _draw_values(rng, (len(t), H, d), dt)
        segments.append(Segment(t, k, v))
    churn_steps = tuple(s for s in (16, 32, 48) if s < n_steps)
    return DynamicWorkload(config, CONFIG_NAMES[config], H, d, c, dt, 1.0 / np.sqrt(d),
                           segments, seqs, n_steps, churn_steps, int(round(0.1 * B)), rng, redraws)


@dataclasses.dataclass
class PrefillJoin:
    """A sequence joining a built tree: its prompt repeats an existing shared
    prompt and adds new tokens, whose K/V and queries are drawn here."""

    static: StaticWorkload   # the tree it joins (its segments grow by one)
    seq: Sequence            # the joining sequence (shared prompt + new segment)
    n_new: int
    q: np.ndarray            # [n_new, H, d] queries of the new tokens


def make_prefill_join(n_new: int = 512, config: int = 2) -> PrefillJoin:
    """The prefill-with-prefix-reuse workload: one more sequence joins the
    single-shared-prompt tree (32 rows, 1024 shared + 512 unique tokens, by
    default) with the 1024-token
    shared prompt plus ``n_new`` new tokens. Seeded with PCG64(1100 + config)
    after the static workload's own draws: new tokens (first token distinct
    from the existing branches), then K and V of the new tokens, then q."""
    wl = make_static(config)
    rng = np.random.Generator(np.random.PCG64(1100 + config))
    prompt = wl.seqs[0].segs[0]
    firsts = {int(wl.segments[s.segs[-1]].tokens[0]) for s in wl.seqs}
    t, nr = _draw_tokens(rng, n_new, firsts)
    wl.redraws += nr
    k = _draw_values(rng, (n_new, wl.H, wl.d), wl.dtype)
    v = _draw_values(rng, (n_new, wl.H, wl.d), wl.dtype)
    q = _draw_values(rng, (n_new, wl.H, wl.d), wl.dtype)
    wl.segments.append(Segment(t, k, v))
    seq = Sequence(max(s.seq_id for s in wl.seqs) + 1, [prompt, len(wl.segments) - 1])
    return PrefillJoin(wl, seq, n_new, q)


def sweep_tokens(b: int, n_p: int, n_s: int, seed: int):
    """Token ids of a batch of b prompts of n_p tokens whose first n_s tokens
    are one shared prefix (the paper's microkernel workload). The first
    unique token of each prompt is redrawn until it differs from the other
    prompts' (so the shared part is exactly n_s tokens); with n_s = n_p all
    prompts are the same. Returns (shared [n_s], list of b unique arrays)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shared = rng.integers(0, VOCAB, size=n_s).astype(np.int32)
    firsts, uniq = set(), []
    for _ in range(b):
        if n_p > n_s:
            t, _ = _draw_tokens(rng, n_p - n_s, firsts)
            firsts.add(int(t[0]))
        else:
            t = np.zeros(0, np.int32)
        uniq.append(t)
    return shared, uniq


def make_sweep(b: int, n_p: int, n_s: int, seed: int, H: int = 32, d: int = 128,
               c: int = 64) -> StaticWorkload:
    """One cell of the microkernel grid (Table 3): b prompts of n_p tokens
    whose first n_s tokens are one shared prefix, fp16. Token ids from
    ``sweep_tokens(b, n_p, n_s, seed)``; then, from PCG64(seed + 1), K and V
    once per segment (the shared prefix, then each unique part) and q.
    Segment i's K then V come from its own generator PCG64([seed, 1, i]), so
    segments are drawn on several threads (NumPy releases the GIL while it
    fills) with results independent of the thread count; q comes from
    PCG64([seed, 2]). With n_s = n_p every sequence is the same prompt; with
    n_s = 0 nothing is shared."""
    from concurrent.futures import ThreadPoolExecutor

    dt = np.dtype(np.float16)
    shared, uniq = sweep_tokens(b, n_p, n_s, seed)
    seg_tokens = ([shared] if n_s > 0 else []) + [u for u in uniq if len(u) > 0]

    def draw(i):
        rng = np.random.Generator(np.random.PCG64([seed, 1, i]))
        t = seg_tokens[i]
        k = _draw_values(rng, (len(t), H, d), dt)
        v = _draw_values(rng, (len(t), H, d), dt)
        return Segment(t, k, v)

    with ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        segments = list(ex.map(draw, range(len(seg_tokens))))
    rng = np.random.Generator(np.random.PCG64([seed, 2]))
    base = 1 if n_s > 0 else 0
    seqs = []
    for i in range(b):
        segs = ([0] if n_s > 0 else []) + ([base + i] if n_p > n_s else [])
        seqs.append(Sequence(i, segs))
    q = _draw_values(rng, (b, H, d), dt)
    return StaticWorkload(0, f"sweep_b{b}_np{n_p}_ns{n_s}_h{H}_d{d}_c{c}_fp16", H, d, c, dt,
                          1.0 / np.sqrt(d), segments, seqs, q, 0)


@dataclasses.dataclass
class DecodeRun:
    """A batch decode run (Figure 3 / Figure 4): b sequences start as the
    same n_s-token prompt and each step appends one token per sequence."""

    name: str
    H: int
    d: int
    c: int
    dtype: np.dtype
    scale: float
    prompt: Segment
    b: int
    n_c: int
    seed: int

    def steps(self) -> Iterator[DecodeStep]:
        """Step i: every sequence (ids 0..b-1) appends token [i, id] of
        ``decode_tokens``, whose first step is redrawn where two sequences
        would start with the same token (so each grows its own chunk); K, V
        and q of the step from PCG64(seed + 1), in that order."""
        toks = decode_tokens(self.b, self.n_c, self.seed)
        if self.n_c > 0:
            fix = np.random.Generator(np.random.PCG64(self.seed + 2))
            seen = set()
            for j in range(self.b):
                while int(toks[0, j]) in seen:
                    toks[0, j] = np.int32(fix.integers(0, VOCAB))
                seen.add(int(toks[0, j]))
        rng = np.random.Generator(np.random.PCG64(self.seed + 1))
        ids = np.arange(self.b, dtype=np.int64)
        for i in range(self.n_c):
            k = _draw_values(rng, (self.b, self.H, self.d), self.dtype)
            v = _draw_values(rng, (self.b, self.H, self.d), self.dtype)
            q = _draw_values(rng, (self.b, self.H, self.d), self.dtype)
            yield DecodeStep(i, None, ids, toks[i].copy(), k, v, q)


def make_decode_run(b: int, n_s: int, n_c: int, seed: int, H: int = 32, d: int = 128,
                    c: int = 64) -> DecodeRun:
    """The batch-sweep workload (Figure 4: n_s shared prompt tokens, n_c
    decode steps): prompt tokens from PCG64(seed), its K and V from
    PCG64(seed + 3); the steps draw their own values."""
    dt = np.dtype(np.float16)
    rng = np.random.Generator(np.random.PCG64(seed))
    prompt = rng.integers(0, VOCAB, size=n_s).astype(np.int32)
    vr = np.random.Generator(np.random.PCG64(seed + 3))
    k = _draw_values(vr, (n_s, H, d), dt)
    v = _draw_values(vr, (n_s, H, d), dt)
    return DecodeRun(f"decode_b{b}_ns{n_s}_nc{n_c}_h{H}_d{d}_c{c}_fp16", H, d, c, dt,
                     1.0 / np.sqrt(d), Segment(prompt, k, v), b, n_c, seed)


def decode_tokens(b: int, n_c: int, seed: int) -> np.ndarray:
    """Completion token ids [n_c, b] for a decode run (one per sequence per step)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, VOCAB, size=(n_c, b)).astype(np.int32)


# ---------------------------------------------------------------------------
# Random operation scripts for tree tests (small alphabets force sharing,
# splits, sibling collisions and prefix sequences).

def random_op_script(seed: int, n_ops: int = 40, alphabet: int = 3, max_len: int = 12,
                     max_live: int = 8, p_insert: float = 0.35, p_extend: float = 0.2,
                     p_append: float = 0.25):
    """Return a list of operations (tuples) over live sequence ids.

    ("insert", sid, tokens) | ("extend", sid, tokens) |
    ("append", [sids], tokens[n]) | ("remove", sid)
    Only ids are tracked here; the tree semantics live elsewhere.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    ops = []
    live = []
    next_id = 0
    for _ in range(n_ops):
        u = rng.random()
        if not live or (u < p_insert and len(live) < max_live):
            n = int(rng.integers(1, max_len + 1))
            t = rng.integers(0, alphabet, size=n).astype(np.int32)
            ops.append(("insert", next_id, t))
            live.append(next_id)
            next_id += 1
        elif u < p_insert + p_extend:
            sid = int(live[int(rng.integers(0, len(live)))])
            n = int(rng.integers(1, max_len // 2 + 2))
            t = rng.integers(0, alphabet, size=n).astype(np.int32)
            ops.append(("extend", sid, t))
        elif u < p_insert + p_extend + p_append:
            k = int(rng.integers(1, len(live) + 1))
            sids = sorted(int(x) for x in rng.choice(np.array(live), size=k, replace=False))
            t = rng.integers(0, alphabet, size=k).astype(np.int32)
            ops.append(("append", sids, t))
        else:
            sid = int(live[int(rng.integers(0, len(live)))])
            ops.append(("remove", sid))
            live.remove(sid)
    return ops


def prefix_keyed_kv(seed: int, tokens: np.ndarray, start: int, H: int, d: int, dtype):
    """K/V rows [start, n) where row i depends only on (seed, tokens[:i+1]).

    Two sequences with a common token prefix then carry identical K/V for it,
    which is what a prefix-shared cache assumes.
    """
    n = int(tokens.shape[0])
    k = np.empty((n - start, H, d), dtype=dtype)
    v = np.empty((n - start, H, d), dtype=dtype)
    h = np.uint64(1469598103934665603)
    prime = np.uint64(1099511628211)
    with np.errstate(over="ignore"):
        for i in range(n):
            h = np.uint64((h ^ np.uint64(int(tokens[i]) & 0xFFFFFFFF)) * prime)
            if i >= start:
                g = np.random.Generator(np.random.PCG64([seed, int(h), i]))
                x = g.standard_normal(size=(2, H, d), dtype=np.float32).astype(dtype)
                k[i - start] = x[0]
                v[i - start] = x[1]
    return k, v
