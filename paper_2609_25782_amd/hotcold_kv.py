"""ctypes binding of ``libhotcold_kv.so`` (the C ABI in ``include/hotcold_kv.h``).

Argument marshalling only: every function keeps its C name, takes device
pointers as integers (``tensor.data_ptr()``) and streams as integers
(``torch.cuda.current_stream().cuda_stream``), and raises ``KVError`` when the
library returns a non-zero status.  All work happens in the library's HIP
kernels; there is no fallback: if the library is not built, importing this
module fails.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhotcold_kv.so")

KV_PAGE_TOKENS = 16
KV_OK, KV_ERR_INVALID, KV_ERR_STATE = 0, -1, -2
KV_ERR_NO_HOT_PAGES, KV_ERR_NO_COLD_PAGES, KV_ERR_HIP, KV_ERR_OOM = -3, -4, -5, -6
KV_DTYPE_BF16, KV_DTYPE_F32 = 0, 1
KV_COLD_DEVICE, KV_COLD_PINNED_HOST = 0, 1
KV_SESSION_FREE, KV_SESSION_ACTIVE, KV_SESSION_PAUSED = 0, 1, 2
KV_POOL_METADATA_ONLY = 1
KV_KERNEL_DECODE_SPLIT, KV_KERNEL_DECODE_COMBINE, KV_KERNEL_PAGE_COPY, KV_KERNEL_EVICT_COPY = 0, 1, 2, 3
KV_KERNEL_PREFETCH_COPY, KV_KERNEL_COUNT = 4, 5
KV_PAGE_COLD, KV_PAGE_STAGED = 1 << 30, 1 << 29
KV_COMBINE_SEPARATE, KV_COMBINE_FUSED = 0, 1
KV_DECODE_MATRIX, KV_DECODE_VECTOR = 0, 1
KV_HOST_COPY_DMA, KV_HOST_COPY_KERNEL = 0, 1


class KVError(RuntimeError):
    def __init__(self, status: int, func: str, message: str):
        super().__init__("%s failed: %s (%d): %s" % (func, _strerror(status), status, message))
        self.status = status


class kv_pool_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_layers", "num_kv_heads", "head_dim", "page_size", "dtype", "num_hot_pages",
        "num_cold_pages", "cold_location", "max_sessions", "max_pages_per_session", "device",
        "flags")]


class kv_pool_stats_t(ctypes.Structure):
    _fields_ = [("free_hot_pages", ctypes.c_int32), ("free_cold_pages", ctypes.c_int32),
                ("active_sessions", ctypes.c_int32), ("paused_sessions", ctypes.c_int32),
                ("pages_to_cold", ctypes.c_int64), ("pages_to_hot", ctypes.c_int64),
                ("bytes_to_cold", ctypes.c_int64), ("bytes_to_hot", ctypes.c_int64),
                ("resumes", ctypes.c_int64), ("evicts", ctypes.c_int64),
                ("resume_pages_resident", ctypes.c_int64), ("resume_pages_total", ctypes.c_int64),
                ("lru_evicted_pages", ctypes.c_int64), ("spilled_pages", ctypes.c_int64),
                ("promoted_pages", ctypes.c_int64), ("cold_active_pages", ctypes.c_int64)]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


if not os.path.exists(LIB_PATH):
    raise ImportError("%s is not built: run `python -m paper_2609_25782_amd.build`" % LIB_PATH)

_lib = ctypes.CDLL(LIB_PATH)

_P = ctypes.c_void_p
_I32, _I64, _U64, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t
_PI32 = ctypes.POINTER(ctypes.c_int32)

_SIGS = {
    "kv_page_bytes": (_SZ, [ctypes.POINTER(kv_pool_desc)]),
    "kv_pool_create": (ctypes.c_int, [ctypes.POINTER(kv_pool_desc), _P, _SZ, _P, _SZ, _P, _P,
                                      ctypes.POINTER(_P)]),
    "kv_pool_destroy": (None, [_P]),
    "kv_pool_stats": (ctypes.c_int, [_P, ctypes.POINTER(kv_pool_stats_t)]),
    "kv_session_create": (ctypes.c_int, [_P, _I32, _PI32, _P, _PI32]),
    "kv_session_import_cold": (ctypes.c_int, [_P, _I32, _PI32, _PI32]),
    "kv_session_extend": (ctypes.c_int, [_P, _I32, _I32, _P]),
    "kv_session_pause": (ctypes.c_int, [_P, _I32]),
    "kv_evict_pages": (ctypes.c_int, [_P, _I32, _P, _PI32]),
    "kv_session_destroy": (ctypes.c_int, [_P, _I32, _P]),
    "kv_session_info": (ctypes.c_int, [_P, _I32, _PI32, _PI32, _PI32, _PI32, _I32]),
    "kv_write_tokens": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _P, _P, _P]),
    "kv_append_tokens": (ctypes.c_int, [_P, _I32, _P, _P, _I32, _P, _P, _P]),
    "kv_write_tokens_layers": (ctypes.c_int, [_P, _I32, _I32, _I32, _I32, _I32, _P, _P, _P]),
    "kv_append_tokens_table": (ctypes.c_int, [_P, _I32, _I32, _P, _I64, _I32, _P, _P, _I32, _P, _P, _P]),
    "kv_fill_synthetic": (ctypes.c_int, [_P, _I32, _I32, _U64, ctypes.c_float, _P]),
    "kv_fill_synthetic_pages": (ctypes.c_int, [_P, _I32, _I32, _U64, ctypes.c_float, _I32, _I32, _P]),
    "kv_evict_session": (ctypes.c_int, [_P, _I32, _P]),
    "kv_pool_set_spill": (ctypes.c_int, [_P, _I32]),
    "kv_promote_pages": (ctypes.c_int, [_P, _I32, _P, _PI32]),
    "kv_resume_sessions_lazy": (ctypes.c_int, [_P, _PI32, _I32, _P]),
    "kv_pool_set_staging": (ctypes.c_int, [_P, _P, _SZ, _PI32]),
    "paged_decode_stage": (ctypes.c_int, [_P, _PI32, _I32, _P, _P, _PI32]),
    "paged_decode_prefetch": (ctypes.c_int, [_P, _I32, _P]),
    "kv_evict_sessions": (ctypes.c_int, [_P, _PI32, _I32, _P]),
    "kv_resume_session": (ctypes.c_int, [_P, _I32, _P]),
    "kv_resume_sessions": (ctypes.c_int, [_P, _PI32, _I32, _P]),
    "kv_pool_set_copy_blocks": (ctypes.c_int, [_P, _I32]),
    "paged_decode_waves": (_I32, [_P]),
    "kv_pool_set_decode_waves": (ctypes.c_int, [_P, _I32]),
    "kv_pool_set_decode_combine": (ctypes.c_int, [_P, _I32]),
    "kv_pool_set_decode_compute": (ctypes.c_int, [_P, _I32]),
    "kv_pool_set_host_copy": (ctypes.c_int, [_P, _I32]),
    "kv_read_probe": (ctypes.c_int, [_P, ctypes.c_size_t, _P, _I32, _P]),
    "kv_device_cu_slots": (ctypes.c_int, [_I32, _PI32, _PI32]),
    "kv_stream_create_cu_slots": (ctypes.c_int, [_I32, _I32, _I32, ctypes.POINTER(_P)]),
    "kv_stream_destroy": (ctypes.c_int, [_P]),
    "paged_decode_workspace_bytes": (_SZ, [_P, _I32, _I32]),
    "paged_decode_attention": (ctypes.c_int, [_P, _I32, _P, _P, _I64, _P, _I32, _I32,
                                              ctypes.c_float, _P, _P, _SZ, _P]),
    "paged_decode_attention_append": (ctypes.c_int, [_P, _I32, _P, _P, _P, _P, _I64, _P, _I32, _I32,
                                                     ctypes.c_float, _P, _P, _SZ, _P]),
    "paged_decode_attention_noalloc": (ctypes.c_int, [_P, _I32, _P, _P, _I64, _P, _I32, _I32,
                                                      ctypes.c_float, _P, _P]),
    "paged_decode_partition": (ctypes.c_int, [_P, _P, _I32, _I32, _P, _P]),
    "paged_decode_gather_table": (ctypes.c_int, [_P, _P, _I32, _P, _P]),
    "kv_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "kv_last_error": (ctypes.c_char_p, []),
    "kv_pool_set_profiling": (ctypes.c_int, [_P, ctypes.c_int]),
    "kv_pool_profile_read": (ctypes.c_int, [_P, _I32, _PI32, ctypes.POINTER(ctypes.c_double)]),
}

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def exported_names():
    return sorted(_SIGS)


def _strerror(status: int) -> str:
    return _lib.kv_strerror(status).decode()


def _check(status: int, func: str) -> None:
    if status != KV_OK:
        raise KVError(status, func, _lib.kv_last_error().decode())


def _i32_array(values: Optional[Sequence[int]]):
    if values is None:
        return None
    return (ctypes.c_int32 * len(values))(*[int(v) for v in values])


# -- pool ---------------------------------------------------------------------

def kv_page_bytes(desc: kv_pool_desc) -> int:
    return int(_lib.kv_page_bytes(ctypes.byref(desc)))


def kv_pool_create(desc: kv_pool_desc, hot_ptr: int, hot_bytes: int, cold_ptr: int,
                   cold_bytes: int, page_table_ptr: int, stream: int = 0) -> int:
    out = _P()
    _check(_lib.kv_pool_create(ctypes.byref(desc), hot_ptr or None, hot_bytes, cold_ptr or None,
                               cold_bytes, page_table_ptr or None, stream or None,
                               ctypes.byref(out)), "kv_pool_create")
    return out.value


def kv_pool_destroy(pool: int) -> None:
    _lib.kv_pool_destroy(pool)


def kv_pool_stats(pool: int) -> dict:
    st = kv_pool_stats_t()
    _check(_lib.kv_pool_stats(pool, ctypes.byref(st)), "kv_pool_stats")
    return st.as_dict()


# -- sessions -----------------------------------------------------------------

def kv_session_create(pool: int, seq_len: int, hot_pages: Optional[Sequence[int]] = None,
                      stream: int = 0) -> int:
    sid = ctypes.c_int32()
    _check(_lib.kv_session_create(pool, seq_len, _i32_array(hot_pages), stream or None,
                                  ctypes.byref(sid)), "kv_session_create")
    return sid.value


def kv_session_import_cold(pool: int, seq_len: int, cold_pages: Sequence[int]) -> int:
    sid = ctypes.c_int32()
    _check(_lib.kv_session_import_cold(pool, seq_len, _i32_array(cold_pages), ctypes.byref(sid)),
           "kv_session_import_cold")
    return sid.value


def kv_session_extend(pool: int, sid: int, new_seq_len: int, stream: int = 0) -> None:
    _check(_lib.kv_session_extend(pool, sid, new_seq_len, stream or None), "kv_session_extend")


def kv_session_pause(pool: int, sid: int) -> None:
    _check(_lib.kv_session_pause(pool, sid), "kv_session_pause")


def kv_evict_pages(pool: int, n: int, stream: int = 0) -> int:
    got = ctypes.c_int32()
    _check(_lib.kv_evict_pages(pool, n, stream or None, ctypes.byref(got)), "kv_evict_pages")
    return got.value


def kv_session_destroy(pool: int, sid: int, stream: int = 0) -> None:
    _check(_lib.kv_session_destroy(pool, sid, stream or None), "kv_session_destroy")


def kv_session_info(pool: int, sid: int, cap: int = 0):
    """Returns (state, seq_len, hot_pages, cold_pages) with lists of up to `cap` ids
    (cap 0 = the session's page count)."""
    state, seq_len = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.kv_session_info(pool, sid, ctypes.byref(state), ctypes.byref(seq_len), None, None, 0),
           "kv_session_info")
    n = cap or (seq_len.value + KV_PAGE_TOKENS - 1) // KV_PAGE_TOKENS
    hot, cold = (ctypes.c_int32 * max(n, 1))(), (ctypes.c_int32 * max(n, 1))()
    _check(_lib.kv_session_info(pool, sid, None, None, hot, cold, n), "kv_session_info")
    n = n if state.value != KV_SESSION_FREE else 0
    return state.value, seq_len.value, list(hot[:n]), list(cold[:n])


def kv_write_tokens(pool: int, sid: int, layer: int, tok_begin: int, n_tok: int, k_ptr: int,
                    v_ptr: int, stream: int = 0) -> None:
    _check(_lib.kv_write_tokens(pool, sid, layer, tok_begin, n_tok, k_ptr or None, v_ptr or None,
                                stream or None), "kv_write_tokens")


def kv_append_tokens(pool: int, layer: int, sids, positions, k: int, v: int, stream: int = 0) -> None:
    sids = [int(x) for x in sids]
    positions = [int(x) for x in positions]
    if len(sids) != len(positions):
        raise ValueError("sids and positions differ in length")
    n = len(sids)
    sa = (ctypes.c_int32 * max(n, 1))(*sids)
    pa = (ctypes.c_int32 * max(n, 1))(*positions)
    _check(_lib.kv_append_tokens(pool, layer, sa, pa, n, k or None, v or None, stream or None),
           "kv_append_tokens")


def kv_write_tokens_layers(pool: int, sid: int, layer_begin: int, num_layers: int, tok_begin: int, n_tok: int,
                           k_ptr: int, v_ptr: int, stream: int = 0) -> None:
    _check(_lib.kv_write_tokens_layers(pool, sid, layer_begin, num_layers, tok_begin, n_tok, k_ptr or None,
                                       v_ptr or None, stream or None), "kv_write_tokens_layers")


def kv_append_tokens_table(pool: int, layer_begin: int, num_layers: int, table_ptr: int, pt_stride: int,
                           table_rows: int, rows_ptr: int, positions_ptr: int, n: int, k_ptr: int, v_ptr: int,
                           stream: int = 0) -> None:
    _check(_lib.kv_append_tokens_table(pool, layer_begin, num_layers, table_ptr or None, pt_stride, table_rows,
                                       rows_ptr or None, positions_ptr or None, n, k_ptr or None, v_ptr or None,
                                       stream or None), "kv_append_tokens_table")


def kv_fill_synthetic(pool: int, sid: int, gen_sid: int, seed: int, value_mult: float,
                      stream: int = 0) -> None:
    _check(_lib.kv_fill_synthetic(pool, sid, gen_sid, seed, value_mult, stream or None),
           "kv_fill_synthetic")


def kv_fill_synthetic_pages(pool: int, sid: int, gen_sid: int, seed: int, value_mult: float,
                            first_page: int, num_pages: int, stream: int = 0) -> None:
    _check(_lib.kv_fill_synthetic_pages(pool, sid, gen_sid, seed, value_mult, first_page, num_pages,
                                        stream or None), "kv_fill_synthetic_pages")


def kv_pool_set_spill(pool: int, enable: bool) -> None:
    _check(_lib.kv_pool_set_spill(pool, 1 if enable else 0), "kv_pool_set_spill")


def kv_promote_pages(pool: int, n: int, stream: int = 0) -> int:
    got = ctypes.c_int32()
    _check(_lib.kv_promote_pages(pool, n, stream or None, ctypes.byref(got)), "kv_promote_pages")
    return got.value


def kv_resume_sessions_lazy(pool: int, sids: Sequence[int], stream: int = 0) -> None:
    _check(_lib.kv_resume_sessions_lazy(pool, _i32_array(sids), len(sids), stream or None),
           "kv_resume_sessions_lazy")


def kv_pool_set_staging(pool: int, staging_ptr: int, nbytes: int) -> int:
    slots = ctypes.c_int32()
    _check(_lib.kv_pool_set_staging(pool, staging_ptr or None, nbytes, ctypes.byref(slots)),
           "kv_pool_set_staging")
    return slots.value


def paged_decode_stage(pool: int, sids: Sequence[int], table_ptr: int, stream: int = 0) -> int:
    staged = ctypes.c_int32()
    _check(_lib.paged_decode_stage(pool, _i32_array(sids), len(sids), table_ptr or None, stream or None,
                                   ctypes.byref(staged)), "paged_decode_stage")
    return staged.value


def paged_decode_prefetch(pool: int, layer: int, copy_stream: int = 0) -> None:
    _check(_lib.paged_decode_prefetch(pool, layer, copy_stream or None), "paged_decode_prefetch")


def kv_evict_session(pool: int, sid: int, stream: int = 0) -> None:
    _check(_lib.kv_evict_session(pool, sid, stream or None), "kv_evict_session")


def kv_evict_sessions(pool: int, sids: Sequence[int], stream: int = 0) -> None:
    _check(_lib.kv_evict_sessions(pool, _i32_array(sids), len(sids), stream or None),
           "kv_evict_sessions")


def kv_resume_session(pool: int, sid: int, stream: int = 0) -> None:
    _check(_lib.kv_resume_session(pool, sid, stream or None), "kv_resume_session")


def kv_resume_sessions(pool: int, sids: Sequence[int], stream: int = 0) -> None:
    _check(_lib.kv_resume_sessions(pool, _i32_array(sids), len(sids), stream or None),
           "kv_resume_sessions")


def kv_pool_set_copy_blocks(pool: int, blocks: int) -> None:
    _check(_lib.kv_pool_set_copy_blocks(pool, blocks), "kv_pool_set_copy_blocks")


# -- decode -------------------------------------------------------------------

def paged_decode_waves(pool: int) -> int:
    return int(_lib.paged_decode_waves(pool))


def kv_pool_set_decode_waves(pool: int, waves: int) -> None:
    _check(_lib.kv_pool_set_decode_waves(pool, waves), "kv_pool_set_decode_waves")


def kv_pool_set_decode_combine(pool: int, mode: int) -> None:
    _check(_lib.kv_pool_set_decode_combine(pool, mode), "kv_pool_set_decode_combine")


def kv_pool_set_decode_compute(pool: int, mode: int) -> None:
    _check(_lib.kv_pool_set_decode_compute(pool, mode), "kv_pool_set_decode_compute")


def kv_pool_set_host_copy(pool: int, mode: int) -> None:
    _check(_lib.kv_pool_set_host_copy(pool, mode), "kv_pool_set_host_copy")


def kv_read_probe(buf: int, nbytes: int, out: int, blocks: int, stream: int = 0) -> None:
    _check(_lib.kv_read_probe(buf, nbytes, out, blocks, stream), "kv_read_probe")


def kv_device_cu_slots(device: int = 0):
    """(XCDs, CUs per XCD) of the device."""
    x, n = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.kv_device_cu_slots(device, ctypes.byref(x), ctypes.byref(n)), "kv_device_cu_slots")
    return x.value, n.value


def kv_stream_create_cu_slots(device: int, slot_begin: int, slot_end: int) -> int:
    """A new stream whose kernels run on CU slots [slot_begin, slot_end) of every XCD."""
    s = _P()
    _check(_lib.kv_stream_create_cu_slots(device, slot_begin, slot_end, ctypes.byref(s)),
           "kv_stream_create_cu_slots")
    return s.value


def kv_stream_destroy(stream: int) -> None:
    _check(_lib.kv_stream_destroy(stream), "kv_stream_destroy")


def paged_decode_workspace_bytes(pool: int, batch: int, num_q_heads: int) -> int:
    return int(_lib.paged_decode_workspace_bytes(pool, batch, num_q_heads))


def paged_decode_attention(pool: int, layer: int, q_ptr: int, page_table_ptr: int, pt_stride: int,
                           seq_lens_ptr: int, batch: int, num_q_heads: int, scale: float,
                           out_ptr: int, workspace_ptr: int, ws_bytes: int, stream: int = 0) -> None:
    _check(_lib.paged_decode_attention(pool, layer, q_ptr or None, page_table_ptr or None, pt_stride,
                                       seq_lens_ptr or None, batch, num_q_heads, scale,
                                       out_ptr or None, workspace_ptr or None, ws_bytes,
                                       stream or None), "paged_decode_attention")


def paged_decode_attention_append(pool: int, layer: int, q_ptr: int, k_new_ptr: int, v_new_ptr: int,
                                  page_table_ptr: int, pt_stride: int, seq_lens_ptr: int, batch: int,
                                  num_q_heads: int, scale: float, out_ptr: int, workspace_ptr: int, ws_bytes: int,
                                  stream: int = 0) -> None:
    _check(_lib.paged_decode_attention_append(pool, layer, q_ptr or None, k_new_ptr or None, v_new_ptr or None,
                                              page_table_ptr or None, pt_stride, seq_lens_ptr or None, batch,
                                              num_q_heads, scale, out_ptr or None, workspace_ptr or None,
                                              ws_bytes, stream or None), "paged_decode_attention_append")


KV_DECODE_SCRATCH_BYTES = 32 << 20


def paged_decode_attention_noalloc(pool: int, layer: int, q_ptr: int, page_table_ptr: int, pt_stride: int,
                                   seq_lens_ptr: int, batch: int, num_q_heads: int, scale: float,
                                   out_ptr: int, stream: int = 0) -> None:
    _check(_lib.paged_decode_attention_noalloc(pool, layer, q_ptr or None, page_table_ptr or None, pt_stride,
                                               seq_lens_ptr or None, batch, num_q_heads, scale,
                                               out_ptr or None, stream or None),
           "paged_decode_attention_noalloc")


def paged_decode_gather_table(pool: int, sids_ptr: int, n: int, table_ptr: int, stream: int = 0) -> None:
    _check(_lib.paged_decode_gather_table(pool, sids_ptr or None, n, table_ptr or None, stream or None),
           "paged_decode_gather_table")


def paged_decode_partition(pool: int, seq_lens_ptr: int, batch: int, waves: int, slots_ptr: int,
                           stream: int = 0) -> None:
    _check(_lib.paged_decode_partition(pool, seq_lens_ptr or None, batch, waves, slots_ptr or None,
                                       stream or None), "paged_decode_partition")


# -- diagnostics --------------------------------------------------------------

def kv_strerror(status: int) -> str:
    return _strerror(status)


def kv_last_error() -> str:
    return _lib.kv_last_error().decode()


def kv_pool_set_profiling(pool: int, enable: bool) -> None:
    _check(_lib.kv_pool_set_profiling(pool, 1 if enable else 0), "kv_pool_set_profiling")


def kv_pool_profile_read(pool: int, kernel_id: int):
    """Returns (launches, total_ms) of the recorded launches of one kernel and forgets them."""
    n, ms = ctypes.c_int32(), ctypes.c_double()
    _check(_lib.kv_pool_profile_read(pool, kernel_id, ctypes.byref(n), ctypes.byref(ms)),
           "kv_pool_profile_read")
    return n.value, ms.value
