"""Python binding of libpask.so: the C ABI declared in include/pask.h, one
function per entry point with the same name.  Argument marshalling only:
pointers may be given as torch tensors (their data_ptr) or integers; every
step of the hot path runs in the library's HIP kernels.

Importing this module loads libpask.so and fails loudly when it is missing;
there is no fallback.
"""

from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# The in-tree build; PASK_LIB names another build of the same sources to load.
LIB_PATH = os.environ.get("PASK_LIB") or os.path.join(_HERE, "libpask.so")

PASK_OK = 0
PASK_E_ARG = -1
PASK_E_POLICY = -2
PASK_E_SHAPE = -3
PASK_E_CAPACITY = -4
PASK_E_HIP = -5
PASK_E_DEVICE_FLAG = -6
PASK_E_UNSUPPORTED = -7

PASK_DROP, PASK_RETAIN_LOW, PASK_RETAIN_HIGH = 0, 1, 2
PASK_FLAG_BAD_TAG = 1 << 0
PASK_FLAG_HI_POOL_EXHAUSTED = 1 << 1
PASK_FLAG_LO_POOL_EXHAUSTED = 1 << 2
PASK_FLAG_SEQ_CAPACITY = 1 << 3
PASK_FLAG_BAD_COUNT = 1 << 4
PASK_FLAG_BAD_STATE = 1 << 5
PASK_FLAG_NO_BUDGET = 1 << 6
PASK_FLAG_WORKSPACE = 1 << 7
PASK_APPEND_KEEP_ALL = 1 << 0

PASK_MAX_TAGS, PASK_MAX_GROUPS, PASK_MAX_LAYERS, PASK_MAX_STATES = 64, 16, 128, 64
EXPORTS = ("pask_policy_load", "pask_cache_layout_query", "pask_cache_bytes", "pask_cache_init",
           "pask_cache_reset", "pask_kv_append", "pask_budget_init", "pask_workspace_bytes",
           "pask_decode_attn", "pask_decode_attn_noalloc", "pask_attn_distortion", "pask_cache_stats",
           "pask_status_string")
PASK_NOALLOC_SCRATCH_BYTES = 32 << 20


class PaskError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {pask_status_string(status)} ({status})")


class pask_geom(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("max_batch", "n_layers", "n_q_heads", "n_kv_heads", "head_dim",
                                         "page_tokens", "max_tokens_per_seq", "hi_pages", "lo_pages",
                                         "recent_window")]


class pask_policy(C.Structure):
    _fields_ = [("n_tags", C.c_uint32), ("n_groups", C.c_uint32), ("n_layers", C.c_uint32),
                ("n_sink", C.c_uint32), ("recent_window", C.c_uint32),
                ("group_of_layer", C.c_uint8 * PASK_MAX_LAYERS),
                ("action", (C.c_uint8 * PASK_MAX_GROUPS) * PASK_MAX_TAGS),
                ("floor_", (C.c_uint8 * PASK_MAX_GROUPS) * PASK_MAX_TAGS),
                ("rho_up", ((C.c_float * 2) * PASK_MAX_GROUPS) * PASK_MAX_TAGS),
                ("entry_bytes", C.c_uint64 * 3),
                ("n_states", C.c_uint32), ("beta_q", C.c_uint32),
                ("reserve_q", C.c_uint32 * PASK_MAX_STATES), ("crit", C.c_uint8 * PASK_MAX_STATES)]


class pask_cache(C.Structure):
    _fields_ = [("geom", pask_geom), ("base", C.c_void_p), ("bytes", C.c_uint64)]


class pask_cache_layout(C.Structure):
    _fields_ = [(n, C.c_uint64) for n in ("status_off", "counters_off", "block_table_off", "index_list_off",
                                          "staging_off", "budget_off", "ring_act_off", "hi_pool_off", "lo_pool_off",
                                          "total_bytes", "hi_page_bytes", "lo_page_bytes")] + \
               [("max_pages", C.c_int32), ("counter_stride", C.c_int32), ("ring_pages", C.c_int32),
                ("staging_stride", C.c_int32)]


class pask_stats(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("n_entries", "n_high", "n_low", "n_drop", "n_lost", "n_forced_high",
                                         "bytes_high", "bytes_low", "hi_pages_used", "lo_pages_used")] + \
               [("c_kv_governed", C.c_double), ("c_kv_all", C.c_double), ("device_flags", C.c_uint32),
                ("reserved", C.c_uint32), ("n_window", C.c_int64)]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"libpask.so not built at {LIB_PATH}; run `python -m paper_2608_28276_amd.build`")
_lib = C.CDLL(LIB_PATH)

_P = C.c_void_p
_lib.pask_status_string.restype = C.c_char_p
_lib.pask_status_string.argtypes = [C.c_int]
_lib.pask_policy_load.argtypes = [_P, C.c_size_t, C.POINTER(pask_geom), C.POINTER(pask_policy)]
_lib.pask_cache_layout_query.argtypes = [C.POINTER(pask_geom), C.POINTER(pask_cache_layout)]
_lib.pask_cache_bytes.restype = C.c_size_t
_lib.pask_cache_bytes.argtypes = [C.POINTER(pask_geom)]
_lib.pask_cache_init.argtypes = [C.POINTER(pask_cache), C.POINTER(pask_geom), _P, C.c_size_t, _P]
_lib.pask_cache_reset.argtypes = [C.POINTER(pask_cache), _P]
_lib.pask_kv_append.argtypes = [C.POINTER(pask_policy), C.POINTER(pask_cache), C.c_int32, C.c_int32, _P,
                                C.c_int32, _P, _P, _P, _P, C.c_uint32, _P]
_lib.pask_budget_init.argtypes = [C.POINTER(pask_policy), C.POINTER(pask_cache), C.c_int32, C.c_int32, _P]
_lib.pask_workspace_bytes.restype = C.c_size_t
_lib.pask_workspace_bytes.argtypes = [C.POINTER(pask_geom), C.c_int32, C.c_int32]
_lib.pask_decode_attn.argtypes = [C.POINTER(pask_policy), C.POINTER(pask_cache), C.c_int32, C.c_int32, _P, _P,
                                  _P, _P, _P, _P, _P, C.c_float, C.c_int32, _P, C.c_size_t, _P]
_lib.pask_decode_attn_noalloc.argtypes = [C.POINTER(pask_policy), C.POINTER(pask_cache), C.c_int32, C.c_int32, _P,
                                          _P, _P, _P, _P, _P, _P, C.c_float, C.c_int32, _P]
_lib.pask_attn_distortion.argtypes = [C.POINTER(pask_cache), C.POINTER(pask_cache), C.c_int32, C.c_int32, _P, _P,
                                      C.c_float, C.c_int32, _P, C.c_size_t, _P, _P]
_lib.pask_cache_stats.argtypes = [C.POINTER(pask_policy), C.POINTER(pask_cache), C.c_int32,
                                  C.POINTER(pask_stats), _P, _P]


def _ptr(x):
    """Tensor -> data_ptr, int -> itself, None -> NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x or None
    return x.data_ptr()


def _check(status: int, where: str):
    if status != PASK_OK:
        raise PaskError(status, where)


def library() -> C.CDLL:
    return _lib


def pask_status_string(status: int) -> str:
    return _lib.pask_status_string(int(status)).decode()


def make_geom(**kw) -> pask_geom:
    g = pask_geom()
    g.page_tokens = 16
    for k, v in kw.items():
        setattr(g, k, int(v))
    return g


def pask_policy_load(blob: bytes, geom: pask_geom | None) -> pask_policy:
    out = pask_policy()
    buf = C.create_string_buffer(bytes(blob), len(blob))
    st = _lib.pask_policy_load(C.cast(buf, _P), len(blob), C.byref(geom) if geom is not None else None,
                               C.byref(out))
    _check(st, "pask_policy_load")
    return out


def pask_cache_layout_query(geom: pask_geom) -> pask_cache_layout:
    out = pask_cache_layout()
    _check(_lib.pask_cache_layout_query(C.byref(geom), C.byref(out)), "pask_cache_layout_query")
    return out


def pask_cache_bytes(geom: pask_geom) -> int:
    return int(_lib.pask_cache_bytes(C.byref(geom)))


def pask_cache_init(cache: pask_cache, geom: pask_geom, base, nbytes: int, stream=0) -> None:
    _check(_lib.pask_cache_init(C.byref(cache), C.byref(geom), _ptr(base), int(nbytes), _ptr(stream)),
           "pask_cache_init")


def pask_cache_reset(cache: pask_cache, stream=0) -> None:
    _check(_lib.pask_cache_reset(C.byref(cache), _ptr(stream)), "pask_cache_reset")


def pask_kv_append(policy: pask_policy, cache: pask_cache, layer: int, batch: int, n_new, max_new: int,
                   tags, k, v, flags: int = 0, stream=0, states=None) -> None:
    """states (keyword here, after tags in the C signature): parser states
    [batch][max_new] uint8 for the online controller, or None."""
    _check(_lib.pask_kv_append(C.byref(policy), C.byref(cache), int(layer), int(batch), _ptr(n_new),
                               int(max_new), _ptr(tags), _ptr(states), _ptr(k), _ptr(v), int(flags),
                               _ptr(stream)),
           "pask_kv_append")


def pask_budget_init(policy: pask_policy, cache: pask_cache, batch: int, t_max: int, stream=0) -> None:
    _check(_lib.pask_budget_init(C.byref(policy), C.byref(cache), int(batch), int(t_max), _ptr(stream)),
           "pask_budget_init")


def pask_workspace_bytes(geom: pask_geom, batch: int, max_ctx_hint: int) -> int:
    return int(_lib.pask_workspace_bytes(C.byref(geom), int(batch), int(max_ctx_hint)))


def pask_decode_attn(policy: pask_policy, cache: pask_cache, layer: int, batch: int, q, out, lse=None,
                     tags_new=None, k_new=None, v_new=None, softmax_scale: float = 1.0,
                     max_ctx_hint: int = 0, ws=None, ws_bytes: int = 0, stream=0, states_new=None) -> None:
    """states_new (keyword here, after tags_new in the C signature): parser
    states [batch] uint8 of the fused append, or None."""
    _check(_lib.pask_decode_attn(C.byref(policy), C.byref(cache), int(layer), int(batch), _ptr(q), _ptr(out),
                                 _ptr(lse), _ptr(tags_new), _ptr(states_new), _ptr(k_new), _ptr(v_new),
                                 float(softmax_scale),
                                 int(max_ctx_hint), _ptr(ws), int(ws_bytes), _ptr(stream)),
           "pask_decode_attn")


def pask_decode_attn_noalloc(policy: pask_policy, cache: pask_cache, layer: int, batch: int, q, out, lse=None,
                             tags_new=None, k_new=None, v_new=None, softmax_scale: float = 1.0,
                             max_ctx_hint: int = 0, stream=0, states_new=None) -> None:
    """pask_decode_attn with the library's own device scratch in place of a
    caller workspace (no allocation in the call)."""
    _check(_lib.pask_decode_attn_noalloc(C.byref(policy), C.byref(cache), int(layer), int(batch), _ptr(q), _ptr(out),
                                         _ptr(lse), _ptr(tags_new), _ptr(states_new), _ptr(k_new), _ptr(v_new),
                                         float(softmax_scale), int(max_ctx_hint), _ptr(stream)),
           "pask_decode_attn_noalloc")


def pask_attn_distortion(ref: pask_cache, intervened: pask_cache, layer: int, batch: int, q, in_s, softmax_scale: float,
                         max_ctx_hint: int, ws, ws_bytes: int, dist, stream=0) -> None:
    """dist[b] += max_h ||o_ref[b][h] - o_int[b][h]||^2 for the flagged sequences (Eq. 4)."""
    _check(_lib.pask_attn_distortion(C.byref(ref), C.byref(intervened), int(layer), int(batch), _ptr(q), _ptr(in_s),
                                     float(softmax_scale), int(max_ctx_hint), _ptr(ws), int(ws_bytes), _ptr(dist),
                                     _ptr(stream)),
           "pask_attn_distortion")


def pask_cache_stats(policy: pask_policy, cache: pask_cache, batch: int, per_seq_group_head=None, stream=0):
    """Returns (stats, status); status is PASK_OK or PASK_E_DEVICE_FLAG.
    per_seq_group_head: optional host int64 buffer (numpy array) of
    batch * n_groups * n_kv_heads * 3 entries."""
    out = pask_stats()
    p = None
    if per_seq_group_head is not None:
        p = per_seq_group_head.ctypes.data
    st = _lib.pask_cache_stats(C.byref(policy), C.byref(cache), int(batch), C.byref(out), p, _ptr(stream))
    if st not in (PASK_OK, PASK_E_DEVICE_FLAG):
        raise PaskError(st, "pask_cache_stats")
    return out, st
