"""Oracle for the hot-cold KV hot path — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import or call anything in this package.  The GPU library neither
imports nor links it, and the two share no code: the pool layout, the page
allocation policy and the attention arithmetic are each written here a second
time, from their definitions.

Contents
--------
* ``paged_attention``: fp64 paged grouped-query decode attention, the plain
  definition (C, ``paged_attention_ref.c``).  Decoding attends to past KV held in
  fixed-size blocks (Sec. II, "Large Language Models").
* ``pack_pool``: writes logical per-session K/V into a host pool buffer with the
  documented page layout (its own implementation of that layout).
* ``PoolModel`` (``pool_model.py``): the allocator and session-state model that
  predicts page tables, copies and cold-write counts (Sec. III, write-on-evict;
  resume before the session runs).
* ``partition`` (``partition.py``): the reference split of decode work over
  waves, by brute-force enumeration.

Pins (what fixes each function independently of itself) live in
``tests/test_oracle_pins.py``, ``tests/test_pool_model.py`` and
``tests/test_partition_oracle.py``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

from .pool_model import PoolModel, ModelError  # noqa: F401
from . import partition  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "paged_attention_ref.c")
_LIB_PATH = os.path.join(_HERE, "liboracle_ref.so")
_lock = threading.Lock()
_lib = None

BF16, F32 = 0, 1
PAGE_SIZE = 16


class _Layout(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int), ("num_kv_heads", ctypes.c_int),
                ("head_dim", ctypes.c_int), ("page_size", ctypes.c_int), ("dtype", ctypes.c_int)]


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (fp64, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load_library(path: str):
    """A ctypes handle on a compiled copy of the C oracle, its functions typed."""
    lib = ctypes.CDLL(path)
    lib.oracle_paged_attention.restype = ctypes.c_int
    lib.oracle_paged_attention.argtypes = [
        ctypes.c_void_p, ctypes.c_long, ctypes.POINTER(_Layout), ctypes.c_int,
        ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_long,
        ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_long, ctypes.c_int]
    lib.oracle_page_bytes.restype = ctypes.c_long
    lib.oracle_page_bytes.argtypes = [ctypes.POINTER(_Layout)]
    lib.oracle_pack_session.restype = ctypes.c_int
    lib.oracle_pack_session.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Layout), ctypes.c_int,
                                        ctypes.c_void_p, ctypes.c_long, ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_elem_offset.restype = ctypes.c_long
    lib.oracle_elem_offset.argtypes = [ctypes.POINTER(_Layout), ctypes.c_long, ctypes.c_int,
                                       ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int]
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            _lib = load_library(_LIB_PATH)
    return _lib


def _layout(num_layers, num_kv_heads, head_dim, dtype):
    return _Layout(num_layers, num_kv_heads, head_dim, PAGE_SIZE, dtype)


def elt_bytes(dtype: int) -> int:
    return 2 if dtype == BF16 else 4


def page_bytes(num_layers: int, num_kv_heads: int, head_dim: int, dtype: int) -> int:
    """Bytes of one page: K and V of PAGE_SIZE tokens for every layer and KV head."""
    return int(_load().oracle_page_bytes(ctypes.byref(_layout(num_layers, num_kv_heads, head_dim, dtype))))


def kv_bytes_per_token(num_layers: int, num_kv_heads: int, head_dim: int, dtype: int) -> int:
    return 2 * num_layers * num_kv_heads * head_dim * elt_bytes(dtype)


def pack_pool(pool: np.ndarray, num_layers: int, num_kv_heads: int, head_dim: int, dtype: int,
              layer: int, pages: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
    """Write one session's logical K/V ``[L, Hkv, D]`` of one layer into a host pool.

    ``pool`` is a flat uint8 array; ``pages[i]`` is the pool page holding tokens
    ``16 i .. 16 i + 15``.  ``k``/``v`` are uint16 bf16 bit patterns or float32.
    Element offsets follow the documented layout (see ``paged_attention_ref.c``).
    """
    e = elt_bytes(dtype)
    store = np.uint16 if dtype == BF16 else np.float32
    P, D, H = PAGE_SIZE, head_dim, num_kv_heads
    L = k.shape[0]
    pb = PAGE_SIZE * D * e * 2 * H * num_layers
    tile = P * D * e
    x = 16 // e
    t = np.arange(L)[:, None, None]
    g = np.arange(H)[None, :, None]
    d = np.arange(D)[None, None, :]
    page = np.asarray(pages, dtype=np.int64)[t // P]
    base = page * pb + ((layer * H + g) * 2) * tile
    k_off = base + (((d // x) * P + (t % P)) * x + (d % x)) * e
    v_off = base + tile + (d * P + (t % P)) * e
    typed = pool.view(store)
    typed[(k_off // e).ravel()] = np.asarray(k, dtype=store).ravel()
    typed[(v_off // e).ravel()] = np.asarray(v, dtype=store).ravel()


def pack_session(pool: np.ndarray, num_layers: int, num_kv_heads: int, head_dim: int, dtype: int,
                 layer: int, pages: np.ndarray, k: np.ndarray, v: np.ndarray) -> None:
    """``pack_pool`` done by the C oracle's packer (same arguments, same bytes;
    for the full-size workloads, where the numpy scatter takes minutes)."""
    store = np.uint16 if dtype == BF16 else np.float32
    k = np.ascontiguousarray(k, dtype=store)
    v = np.ascontiguousarray(v, dtype=store)
    pages = np.ascontiguousarray(pages, dtype=np.int32)
    L = int(k.shape[0])
    assert k.shape == v.shape == (L, num_kv_heads, head_dim) and pages.shape[0] * PAGE_SIZE >= L
    pb = page_bytes(num_layers, num_kv_heads, head_dim, dtype)
    assert pool.dtype == np.uint8 and pool.flags.c_contiguous
    assert L == 0 or (int(pages[:(L + PAGE_SIZE - 1) // PAGE_SIZE].max()) + 1) * pb <= pool.size
    lay = _layout(num_layers, num_kv_heads, head_dim, dtype)
    rc = _load().oracle_pack_session(pool.ctypes.data, ctypes.byref(lay), int(layer), pages.ctypes.data, L,
                                     k.ctypes.data, v.ctypes.data)
    if rc != 0:
        raise ValueError("oracle_pack_session failed with status %d" % rc)


def paged_attention(pool: np.ndarray, num_pages: int, num_layers: int, num_kv_heads: int,
                    head_dim: int, dtype: int, layer: int, q: np.ndarray, page_table: np.ndarray,
                    seq_lens: np.ndarray, scale: float, return_weights: bool = False,
                    num_threads: int = 0):
    """fp64 paged GQA decode attention (the plain definition).

    q: ``[B, Hq, D]`` (uint16 bf16 bits or float32); page_table: int32 ``[B, stride]``;
    seq_lens: int32 ``[B]``.  Returns ``out [B, Hq, D]`` float64, and when asked the
    normalised weights ``[B, Hq, max L]`` (zero past each row's length).
    """
    lib = _load()
    q = np.ascontiguousarray(q)
    pt = np.ascontiguousarray(page_table, dtype=np.int32)
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    B, Hq, D = q.shape
    assert D == head_dim and pt.shape[0] >= B and sl.shape[0] >= B
    out = np.zeros((B, Hq, D), dtype=np.float64)
    wmax = int(sl.max()) if (return_weights and B) else 0
    w = np.zeros((B, Hq, max(wmax, 1)), dtype=np.float64) if return_weights else None
    lay = _layout(num_layers, num_kv_heads, head_dim, dtype)
    rc = lib.oracle_paged_attention(pool.ctypes.data, int(num_pages), ctypes.byref(lay), int(layer),
                                    int(B), int(Hq), q.ctypes.data, pt.ctypes.data, int(pt.shape[1]),
                                    sl.ctypes.data, float(scale), out.ctypes.data,
                                    w.ctypes.data if w is not None else None,
                                    int(w.shape[2]) if w is not None else 0, int(num_threads))
    if rc != 0:
        raise ValueError("oracle_paged_attention failed with status %d" % rc)
    return (out, w) if return_weights else out


def elem_offset(num_layers, num_kv_heads, head_dim, dtype, page, layer, head, kind, t, d) -> int:
    """Byte offset of one K (kind 0) or V (kind 1) element, from the C oracle's accessor."""
    lay = _layout(num_layers, num_kv_heads, head_dim, dtype)
    return int(_load().oracle_elem_offset(ctypes.byref(lay), page, layer, head, kind, t, d))
