"""ctypes binding of ``include/chunkattn.h``: argument marshalling only.

Functions keep the C names. Device buffers are passed as integer addresses
(``tensor.data_ptr()``), streams as the integer ``hipStream_t`` handle; host
arrays are converted to contiguous numpy arrays. Every failure raises
``ChunkAttnError`` carrying the C status and message. There is no fallback:
if the library is not built, loading raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

# The library built in-tree; CA_LIBRARY names another build of the same
# sources (for example one with host-side sanitizers).
LIB_PATH = os.environ.get("CA_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "_lib", "libchunkattn.so")

CA_OK = 0
CA_ERR_INVALID = -1
CA_ERR_NOMEM = -2
CA_ERR_NOT_FOUND = -3
CA_ERR_EXISTS = -4
CA_ERR_DEVICE = -5
CA_ERR_WORKSPACE = -6
CA_ERR_HOST = -7
STATUS_NAMES = {0: "OK", -1: "INVALID", -2: "NOMEM", -3: "NOT_FOUND", -4: "EXISTS",
                -5: "DEVICE", -6: "WORKSPACE", -7: "HOST"}

CA_FP16 = 0
CA_FP32 = 1

EXPORTED = ["ca_create", "ca_destroy", "ca_match", "ca_insert", "ca_extend", "ca_append_batch",
            "ca_remove", "ca_num_seqs", "ca_seq_order", "ca_workspace_size", "ca_attention",
            "ca_attention_ordered", "ca_attention_noalloc", "ca_prefill_attention", "ca_prepare", "ca_export_tables", "ca_stats", "ca_set_tuning", "ca_last_error"]


class ChunkAttnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status
        self.message = message


class CaConfig(ctypes.Structure):
    _fields_ = [("chunk_size", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("num_slots", ctypes.c_int64), ("k_pool", ctypes.c_void_p),
                ("v_pool", ctypes.c_void_p), ("slot_stride", ctypes.c_int64),
                ("head_stride", ctypes.c_int64)]


_P32 = ctypes.POINTER(ctypes.c_int32)
_P64 = ctypes.POINTER(ctypes.c_int64)


class CaTables(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int64), ("n_nodes", ctypes.c_int64), ("n_shared", ctypes.c_int64),
                ("row_seq", _P64),
                ("node_slot", _P32), ("node_len", _P32), ("node_row_begin", _P32),
                ("node_row_end", _P32), ("node_parent", _P32), ("node_start_pos", _P32),
                ("shr_node", _P32), ("shr_part_base", _P32),
                ("priv_ptr", _P32), ("priv_node", _P32), ("shr_ptr", _P32), ("shr_part", _P32)]


_lib = None


def load():
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2402_15220_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    sig = {
        "ca_create": [ctypes.POINTER(CaConfig), ctypes.POINTER(vp)],
        "ca_destroy": [vp],
        "ca_match": [vp, _P32, i64, _P64],
        "ca_insert": [vp, i64, _P32, i64, vp, vp, vp, _P64],
        "ca_extend": [vp, i64, _P32, i64, vp, vp, vp, _P64],
        "ca_append_batch": [vp, i64, _P64, _P32, vp, vp, vp],
        "ca_remove": [vp, i64],
        "ca_num_seqs": [vp, _P64],
        "ca_seq_order": [vp, _P64, i64],
        "ca_workspace_size": [vp, ctypes.POINTER(ctypes.c_size_t)],
        "ca_attention": [vp, vp, vp, ctypes.c_float, vp, ctypes.c_size_t, vp],
        "ca_prefill_attention": [vp, i64, vp, vp, i64, ctypes.c_float, vp],
        "ca_prepare": [vp, vp, ctypes.POINTER(i32)],
        "ca_attention_ordered": [vp, vp, vp, _P64, i64, ctypes.c_float, vp, ctypes.c_size_t, vp],
        "ca_attention_noalloc": [vp, vp, vp, ctypes.c_float, vp],
        "ca_export_tables": [vp, ctypes.POINTER(CaTables)],
        "ca_stats": [vp, _P64, _P64, _P64, ctypes.POINTER(i32), ctypes.POINTER(i32), _P64],
        "ca_set_tuning": [vp, i32, i32, i32, i32],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = i32
    lib.ca_last_error.argtypes = []
    lib.ca_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status):
    if status != CA_OK:
        msg = load().ca_last_error().decode()
        raise ChunkAttnError(status, msg)


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(_P32)


def _i64(a):
    a = np.ascontiguousarray(a, dtype=np.int64)
    return a, a.ctypes.data_as(_P64)


def ca_last_error() -> str:
    return load().ca_last_error().decode()


def ca_create(chunk_size, num_heads, head_dim, dtype, num_slots, k_pool=None, v_pool=None,
              slot_stride=0, head_stride=0):
    cfg = CaConfig(chunk_size, num_heads, head_dim, dtype, num_slots, k_pool, v_pool, slot_stride,
                   head_stride)
    h = ctypes.c_void_p()
    _check(load().ca_create(ctypes.byref(cfg), ctypes.byref(h)))
    return h


def ca_destroy(h):
    _check(load().ca_destroy(h))


def ca_match(h, tokens) -> int:
    t, tp = _i32(tokens)
    m = ctypes.c_int64()
    _check(load().ca_match(h, tp, t.shape[0], ctypes.byref(m)))
    return m.value


def ca_insert(h, seq_id, tokens, k=None, v=None, stream=None) -> int:
    t, tp = _i32(tokens)
    m = ctypes.c_int64()
    _check(load().ca_insert(h, seq_id, tp, t.shape[0], k, v, stream, ctypes.byref(m)))
    return m.value


def ca_extend(h, seq_id, tokens, k=None, v=None, stream=None) -> int:
    t, tp = _i32(tokens)
    m = ctypes.c_int64()
    _check(load().ca_extend(h, seq_id, tp, t.shape[0], k, v, stream, ctypes.byref(m)))
    return m.value


def ca_append_batch(h, seq_ids, tokens, k=None, v=None, stream=None):
    s, sp = _i64(seq_ids)
    t, tp = _i32(tokens)
    if s.shape[0] != t.shape[0]:
        raise ValueError("seq_ids and tokens differ in length")
    _check(load().ca_append_batch(h, s.shape[0], sp, tp, k, v, stream))


def ca_remove(h, seq_id):
    _check(load().ca_remove(h, seq_id))


def ca_num_seqs(h) -> int:
    b = ctypes.c_int64()
    _check(load().ca_num_seqs(h, ctypes.byref(b)))
    return b.value


def ca_seq_order(h) -> np.ndarray:
    B = ca_num_seqs(h)
    out = np.empty(max(B, 1), np.int64)
    _check(load().ca_seq_order(h, out.ctypes.data_as(_P64), out.shape[0]))
    return out[:B]


def ca_workspace_size(h) -> int:
    n = ctypes.c_size_t()
    _check(load().ca_workspace_size(h, ctypes.byref(n)))
    return n.value


def ca_attention(h, q, o, scale, ws, ws_bytes, stream=None):
    _check(load().ca_attention(h, q, o, ctypes.c_float(scale), ws, ws_bytes, stream))


def ca_attention_ordered(h, q, o, seq_ids, scale, ws, ws_bytes, stream=None):
    ids = np.ascontiguousarray(seq_ids, dtype=np.int64)
    _check(load().ca_attention_ordered(h, q, o, ids.ctypes.data_as(_P64), ids.shape[0],
                                       ctypes.c_float(scale), ws, ws_bytes, stream))


def ca_attention_noalloc(h, q, o, scale, stream=None):
    _check(load().ca_attention_noalloc(h, q, o, ctypes.c_float(scale), stream))


def ca_prepare(h, stream=None) -> bool:
    """True if an upload of the kernel context was enqueued."""
    up = ctypes.c_int32()
    _check(load().ca_prepare(h, stream, ctypes.byref(up)))
    return bool(up.value)


def ca_prefill_attention(h, seq_id, q, o, n_q, scale, stream=None):
    _check(load().ca_prefill_attention(h, seq_id, q, o, n_q, ctypes.c_float(scale), stream))


def ca_export_tables(h) -> dict:
    t = CaTables()
    _check(load().ca_export_tables(h, ctypes.byref(t)))
    B, nn, ns = t.B, t.n_nodes, t.n_shared

    def arr(p, n, dt):
        if n == 0:
            return np.zeros(0, dt)
        return np.ctypeslib.as_array(p, shape=(n,)).astype(dt, copy=True)

    priv_ptr = arr(t.priv_ptr, B + 1, np.int32)
    shr_ptr = arr(t.shr_ptr, B + 1, np.int32)
    return dict(
        row_seq=arr(t.row_seq, B, np.int64),
        node_slot=arr(t.node_slot, nn, np.int32), node_len=arr(t.node_len, nn, np.int32),
        node_row_begin=arr(t.node_row_begin, nn, np.int32),
        node_row_end=arr(t.node_row_end, nn, np.int32),
        node_parent=arr(t.node_parent, nn, np.int32),
        node_start_pos=arr(t.node_start_pos, nn, np.int32),
        shr_node=arr(t.shr_node, ns, np.int32), shr_part_base=arr(t.shr_part_base, ns, np.int32),
        priv_ptr=priv_ptr, priv_node=arr(t.priv_node, int(priv_ptr[-1]), np.int32),
        shr_ptr=shr_ptr, shr_part=arr(t.shr_part, int(shr_ptr[-1]), np.int32),
    )


def ca_stats(h):
    u, s, t, p = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    sc, sg = ctypes.c_int32(), ctypes.c_int32()
    _check(load().ca_stats(h, ctypes.byref(u), ctypes.byref(s), ctypes.byref(t), ctypes.byref(sc),
                           ctypes.byref(sg), ctypes.byref(p)))
    return dict(uploads=u.value, slots_used=s.value, slots_total=t.value, schedule=sc.value,
                seg_chunks=sg.value, patches=p.value)


def ca_set_tuning(h, seg_chunks=0, split_chunks=-1, phase_mask=0, schedule=-1):
    _check(load().ca_set_tuning(h, seg_chunks, split_chunks, phase_mask, schedule))
