"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This package draws token ids, key/value rows and queries. It computes none of
the attention method's arithmetic and builds no tree: it only says which
sequences exist, which tokens and K/V rows they hold, and in which order
operations happen. Both the HIP path and the CPU oracle consume its output.
"""
from .synth import (  # noqa: F401
    Segment,
    Sequence,
    StaticWorkload,
    DynamicWorkload,
    ChurnEvent,
    DecodeStep,
    CONFIG_NAMES,
    make_static,
    make_dynamic,
    random_op_script,
    prefix_keyed_kv,
    sweep_tokens,
    make_prefill_join,
    PrefillJoin,
    decode_tokens,
    make_sweep,
    make_decode_run,
    DecodeRun,
)
