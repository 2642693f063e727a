"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle's callers.

This module only draws numbers.  It holds no attention arithmetic, no page
layout and no allocation policy: callers turn what it returns into pools,
page tables and reference outputs with their own code.

Two kinds of randomness are used:

* ``numpy.random.Generator(PCG64(seed))`` for workload structure: context
  lengths and the random placement of pages in the hot pool.
* A counter-based generator for tensor values, so that any single element of a
  48-layer, hundreds-of-GB KV pool can be regenerated on the CPU from its
  logical coordinate alone.  The GPU library carries its own implementation of
  the same published definition (SplitMix64, Steele, Lea and Flood, OOPSLA
  2014) for filling pools in device memory; the two agree bit for bit because
  every step below is integer arithmetic plus one IEEE-754 float32 multiply.

Value recipe for coordinate ``c`` (a packed 64-bit integer, see ``coord``):

1. ``h = mix(mix(seed) ^ c)`` where ``mix`` is the SplitMix64 finaliser applied
   to ``x + 0x9E3779B97F4A7C15``.
2. Split ``h`` into four 16-bit fields ``a0..a3`` and form the integer
   ``s = a0 + a1 + a2 + a3 - 131070`` (an Irwin-Hall sum, mean 0, standard
   deviation ``IH_STD``; it approximates a normal distribution and is bounded
   by about 3.46 standard deviations).
3. ``value = float32(s) * k`` with ``k = float32(scale / IH_STD)``, one correctly
   rounded float32 multiply.
4. For bf16 storage, round ``value`` to bf16 with round-to-nearest-even on the
   float32 bit pattern.
"""

from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth_gen.c")
_LIB_PATH = os.path.join(_HERE, "libsynth_gen.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile the C form of the value generator (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-o", tmp, _SRC])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            lib = ctypes.CDLL(_LIB_PATH)
            lib.synth_session_kv.restype = None
            lib.synth_session_kv.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                             ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_int32,
                                             ctypes.c_void_p, ctypes.c_void_p]
            _lib = lib
    return _lib

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# Standard deviation of a sum of four independent uniform integers on [0, 65535].
IH_STD = math.sqrt(4.0 * (65536.0 ** 2 - 1.0) / 12.0)

KIND_K, KIND_V, KIND_Q = 0, 1, 2

DTYPE_BF16 = "bf16"
DTYPE_F32 = "f32"


def _mix(x: np.ndarray) -> np.ndarray:
    """SplitMix64 output function applied to ``x + golden`` (uint64, wraps)."""
    with np.errstate(over="ignore"):
        z = (x + GOLDEN).astype(np.uint64)
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        return z ^ (z >> np.uint64(31))


def coord(kind, sid, layer, head, token, dim) -> np.ndarray:
    """Pack a logical element coordinate into 64 bits.

    Bit fields, most significant first: kind (2), session (20), layer (6),
    head (5), token (23), dim (8).
    """
    u = np.uint64
    return ((u(kind) << u(62)) | (np.asarray(sid, dtype=np.uint64) << u(42))
            | (np.asarray(layer, dtype=np.uint64) << u(36))
            | (np.asarray(head, dtype=np.uint64) << u(32))
            | (np.asarray(token, dtype=np.uint64) << u(8))
            | np.asarray(dim, dtype=np.uint64))


def value_multiplier(scale: float) -> np.float32:
    """The float32 constant ``k`` of step 3; the GPU fill takes the same value."""
    return np.float32(scale / IH_STD)


def values_f32(seed: int, c: np.ndarray, scale: float) -> np.ndarray:
    """Counter-based pseudo-normal float32 values for packed coordinates ``c``."""
    key = _mix(np.asarray([seed], dtype=np.uint64))[0]
    h = _mix(key ^ np.asarray(c, dtype=np.uint64))
    m = np.uint64(0xFFFF)
    s = ((h & m).astype(np.int64) + ((h >> np.uint64(16)) & m).astype(np.int64)
         + ((h >> np.uint64(32)) & m).astype(np.int64) + (h >> np.uint64(48)).astype(np.int64)
         - 131070)
    return s.astype(np.float32) * value_multiplier(scale)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def session_kv(seed: int, sid: int, seq_len: int, layer: int, num_kv_heads: int,
               head_dim: int, scale: float, dtype: str):
    """Logical K and V of one session and layer, shape ``[seq_len, num_kv_heads, head_dim]``.

    bf16 is returned as uint16 bit patterns, f32 as float32.  Computed by the C
    form of the generator (``synth_gen.c``, the same definition step for step;
    ``session_kv_numpy`` is the numpy form, and tests hold the two equal bit for
    bit).
    """
    store = np.uint16 if dtype == DTYPE_BF16 else np.float32
    shape = (int(seq_len), int(num_kv_heads), int(head_dim))
    k = np.empty(shape, store)
    v = np.empty(shape, store)
    if k.size:
        _load().synth_session_kv(int(seed), int(sid), int(seq_len), int(layer), int(num_kv_heads),
                                 int(head_dim), float(value_multiplier(scale)),
                                 1 if dtype == DTYPE_BF16 else 0, k.ctypes.data, v.ctypes.data)
    return k, v


def session_kv_numpy(seed: int, sid: int, seq_len: int, layer: int, num_kv_heads: int,
                     head_dim: int, scale: float, dtype: str):
    """``session_kv`` computed with numpy from ``values_f32`` (the reference form)."""
    t = np.arange(seq_len, dtype=np.uint64)[:, None, None]
    g = np.arange(num_kv_heads, dtype=np.uint64)[None, :, None]
    d = np.arange(head_dim, dtype=np.uint64)[None, None, :]
    out = []
    for kind in (KIND_K, KIND_V):
        v = values_f32(seed, coord(kind, sid, layer, g, t, d), scale)
        out.append(f32_to_bf16_bits(v) if dtype == DTYPE_BF16 else v)
    return out[0], out[1]


def queries(seed: int, batch: int, num_q_heads: int, head_dim: int, scale: float,
            dtype: str, layer: int = 0) -> np.ndarray:
    """Decode queries ``[batch, num_q_heads, head_dim]`` (bf16 bits or float32)."""
    b = np.arange(batch, dtype=np.uint64)[:, None, None]
    h = np.arange(num_q_heads, dtype=np.uint64)[None, :, None]
    d = np.arange(head_dim, dtype=np.uint64)[None, None, :]
    v = values_f32(seed, coord(KIND_Q, b, layer, h, 0, d), scale)
    return f32_to_bf16_bits(v) if dtype == DTYPE_BF16 else v


# ---------------------------------------------------------------------------
# Workload recipes (structure only: lengths, placement, sizes).
# ---------------------------------------------------------------------------

PAGE_TOKENS = 16


def pages_for(seq_len: int) -> int:
    return (int(seq_len) + PAGE_TOKENS - 1) // PAGE_TOKENS


@dataclass
class Workload:
    name: str
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str
    seq_lens: np.ndarray                 # int32 [batch]
    value_scale: float                   # data scale of Q/K/V
    seed: int
    hot_pages: int                       # size of the hot pool in pages
    placement: List[np.ndarray]          # hot page ids per active session
    cold_pages: int = 0
    paused_lens: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    notes: str = ""

    @property
    def batch(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def elt_bytes(self) -> int:
        return 2 if self.dtype == DTYPE_BF16 else 4


def _place(rng: np.random.Generator, seq_lens: np.ndarray, slack: float, min_pages: int = 0):
    need = sum(pages_for(L) for L in seq_lens)
    hot = max(int(math.ceil(need * slack)), need, min_pages)
    perm = rng.permutation(hot).astype(np.int32)
    placement, off = [], 0
    for L in seq_lens:
        n = pages_for(L)
        placement.append(perm[off:off + n].copy())
        off += n
    return hot, placement


def config_tiny(seed: int = 0) -> Workload:
    """1 layer, 4 Q heads / 1 KV head, d=64, fp32, 4 sessions with L ~ U{100..500};
    plus 2 paused sessions of 256 tokens resumed from a 64-page cold pool."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(100, 500, size=4, endpoint=True).astype(np.int32)
    hot, placement = _place(rng, lens, 2.0)
    return Workload("tiny", 1, 4, 1, 64, DTYPE_F32, lens, 1.0, seed, hot + 2 * pages_for(256),
                    placement, cold_pages=64, paused_lens=np.array([256, 256], np.int32))


def config_layer(seed: int = 0, batch: int = 32) -> Workload:
    """One Qwen3-Coder-30B-A3B-shaped layer: 32 Q / 4 KV heads, d=128, bf16,
    B=32 sessions with L ~ U{8192..32768}, values N(0,1)/sqrt(128), pages randomly
    scattered over a hot pool 1.25x the pages needed."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(8192, 32768, size=batch, endpoint=True).astype(np.int32)
    hot, placement = _place(rng, lens, 1.25)
    return Workload("layer_b32_8k_32k", 1, 32, 4, 128, DTYPE_BF16, lens, 1.0 / math.sqrt(128.0),
                    seed, hot, placement)


def config_step48(seed: int = 0, batch: int = 64, sigma: float = 0.5) -> Workload:
    """48 layers of the same attention shape, B=64, lognormal L (median 24K, sigma 0.5,
    capped at 64K), hot pool 1.1x the pages needed, fully permuted."""
    rng = np.random.Generator(np.random.PCG64(seed))
    z = rng.standard_normal(batch)
    lens = np.minimum(65536, np.maximum(1, np.rint(24576.0 * np.exp(sigma * z)))).astype(np.int32)
    hot, placement = _place(rng, lens, 1.1)
    return Workload("step48_b64_lognormal24k", 48, 32, 4, 128, DTYPE_BF16, lens,
                    1.0 / math.sqrt(128.0), seed, hot, placement)


def config_skewed(seed: int = 0, batch: int = 128, s: float = 1.1) -> Workload:
    """B=128, context lengths from a bounded power law p(L) ~ L^-s on [1024, 262144]
    drawn by inverse CDF, one layer, fully permuted pages."""
    rng = np.random.Generator(np.random.PCG64(seed))
    u = rng.random(batch)
    a, b, e = 1024.0, 262144.0, 1.0 - s
    lens = np.floor((a ** e - u * (a ** e - b ** e)) ** (1.0 / e)).astype(np.int64)
    lens = np.clip(lens, 1024, 262144).astype(np.int32)
    hot, placement = _place(rng, lens, 1.05)
    return Workload("skewed_b128_zipf1.1_1k_256k", 1, 32, 4, 128, DTYPE_BF16, lens,
                    1.0 / math.sqrt(128.0), seed, hot, placement)


def config_resume_mix(seed: int = 0, active: int = 32, paused: int = 1024,
                      physical_cold_pages: int = 49152, resume_per_step: int = 8) -> Workload:
    """Resume-heavy agentic mix: 32 active sessions U{8K..32K}, 48 layers, plus a
    logical cold pool of paused sessions U{32K..128K} backed by a physical pool of
    ``physical_cold_pages`` pages (paused sessions draw their cold pages from it)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    lens = rng.integers(8192, 32768, size=active, endpoint=True).astype(np.int32)
    plens = rng.integers(32768, 131072, size=paused, endpoint=True).astype(np.int32)
    headroom = resume_per_step * pages_for(131072)
    need = sum(pages_for(L) for L in lens)
    hot, placement = _place(rng, lens, 1.0, min_pages=need + headroom)
    w = Workload("resume_mix_48l", 48, 32, 4, 128, DTYPE_BF16, lens, 1.0 / math.sqrt(128.0),
                 seed, hot, placement, cold_pages=physical_cold_pages, paused_lens=plens)
    return w


def cold_page_draw(seed: int, sid: int, n: int, physical_pages: int) -> np.ndarray:
    """Cold page ids of a paused session in a virtualised cold pool: n distinct ids
    drawn without replacement from the physical pool (sessions may alias)."""
    rng = np.random.Generator(np.random.PCG64([seed, sid]))
    return rng.choice(physical_pages, size=n, replace=False).astype(np.int32)
