"""Shared helpers for the GPU parity tests.

The GPU side gets its pool contents through the library (``kv_write_tokens`` or
``kv_fill_synthetic``); the oracle side gets the same logical K/V from the
seeded generator, packed into a host pool by the oracle's own packer.  Nothing
the oracle reads comes from the GPU.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import oracle
import synth

ORACLE_DTYPE = {"bf16": oracle.BF16, "f32": oracle.F32}


def tolerance_check(got: np.ndarray, ref: np.ndarray, max_abs: float = 1e-2, max_norm: float = 1e-2):
    """The parity bar for attention outputs: max-abs error <= 1e-2 (the stated
    contract) and max error normalised by the largest reference magnitude <= 1e-2
    (bf16 output rounding alone is 2^-9 relative).  Returns (abs, normalised)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), "non-finite output"
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    norm = err / scale if scale > 0 else err
    assert err <= max_abs, "max abs error %g > %g" % (err, max_abs)
    assert norm <= max_norm, "normalised error %g > %g (max|ref| %g)" % (norm, max_norm, scale)
    return err, norm


@dataclass
class Case:
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                     # "bf16" | "f32"
    seq_lens: List[int]
    seed: int = 0
    value_scale: float = 1.0
    layer: int = 0
    slack: float = 1.5
    extra_stride: int = 2
    placement: Optional[List[np.ndarray]] = None
    hot_pages: int = 0
    kv: list = field(default_factory=list)  # per session (k, v) logical arrays of `layer`

    def __post_init__(self):
        rng = np.random.Generator(np.random.PCG64(self.seed))
        need = sum(synth.pages_for(L) for L in self.seq_lens)
        if self.placement is None:
            self.hot_pages = max(int(math.ceil(need * self.slack)), need, 1)
            perm = rng.permutation(self.hot_pages).astype(np.int32)
            self.placement, off = [], 0
            for L in self.seq_lens:
                n = synth.pages_for(L)
                self.placement.append(perm[off:off + n])
                off += n
        elif not self.hot_pages:
            self.hot_pages = max([int(p.max()) + 1 for p in self.placement if len(p)] + [1])
        self.stride = max([synth.pages_for(L) for L in self.seq_lens] + [1]) + self.extra_stride
        self.kv = [synth.session_kv(self.seed, b, L, self.layer, self.num_kv_heads, self.head_dim,
                                    self.value_scale, self.dtype)
                   for b, L in enumerate(self.seq_lens)]
        self.q = synth.queries(self.seed + 1, len(self.seq_lens), self.num_q_heads, self.head_dim,
                               self.value_scale, self.dtype, self.layer)

    @property
    def batch(self):
        return len(self.seq_lens)

    def page_table(self) -> np.ndarray:
        pt = np.full((self.batch, self.stride), -1, np.int32)
        for b, pages in enumerate(self.placement):
            pt[b, :len(pages)] = pages
        return pt

    def oracle_out(self, scale: Optional[float] = None, rows=None) -> np.ndarray:
        """fp64 reference for all (or the listed) batch rows."""
        rows = list(range(self.batch)) if rows is None else list(rows)
        od = ORACLE_DTYPE[self.dtype]
        # a compact host pool: only the pages these rows use, renumbered
        pages_needed = sum(len(self.placement[b]) for b in rows)
        pb = oracle.page_bytes(self.num_layers, self.num_kv_heads, self.head_dim, od)
        pool = np.zeros(max(pages_needed, 1) * pb, np.uint8)
        pt = np.full((len(rows), self.stride), -1, np.int32)
        off = 0
        for j, b in enumerate(rows):
            n = len(self.placement[b])
            local = np.arange(off, off + n, dtype=np.int32)
            off += n
            pt[j, :n] = local
            k, v = self.kv[b]
            oracle.pack_session(pool, self.num_layers, self.num_kv_heads, self.head_dim, od,
                                self.layer, local, k, v)
        sl = np.array([self.seq_lens[b] for b in rows], np.int32)
        s = self.head_dim ** -0.5 if scale is None else scale
        return oracle.paged_attention(pool, max(pages_needed, 1), self.num_layers, self.num_kv_heads,
                                      self.head_dim, od, self.layer, self.q[rows], pt, sl, s)


def oracle_rows(seed: int, gen_sids, seq_lens, layer: int, q: np.ndarray, num_kv_heads: int, head_dim: int,
                dtype: str, value_scale: float, scale: Optional[float] = None, kv_override=None,
                chunk_tokens: int = 1 << 20) -> np.ndarray:
    """fp64 oracle outputs ``[rows, Hq, D]`` for rows whose K/V are the generator's
    values of logical session ``gen_sids[i]`` at ``layer`` (``kv_override[i]``, a
    (k, v) pair, replaces row i's).  Each chunk of about ``chunk_tokens`` tokens
    is packed by the oracle into a one-layer host pool of its own (pages numbered
    in row order) and decoded there; attention of one layer depends only on that
    layer's K/V, so this is the same definition at a fraction of the memory."""
    od = ORACLE_DTYPE[dtype]
    kv_override = kv_override or {}
    lens = [int(L) for L in seq_lens]
    rows = len(lens)
    out = np.zeros((rows, q.shape[1], head_dim), np.float64)
    s = head_dim ** -0.5 if scale is None else scale
    pb = oracle.page_bytes(1, num_kv_heads, head_dim, od)
    i = 0
    while i < rows:
        j, tok = i, 0
        while j < rows and (j == i or tok + lens[j] <= chunk_tokens):
            tok += lens[j]
            j += 1
        n_pages = sum(synth.pages_for(L) for L in lens[i:j])
        stride = max([synth.pages_for(L) for L in lens[i:j]] + [1])
        pool = np.zeros(max(n_pages, 1) * pb, np.uint8)
        pt = np.full((j - i, stride), -1, np.int32)
        off = 0
        for r in range(i, j):
            n = synth.pages_for(lens[r])
            local = np.arange(off, off + n, dtype=np.int32)
            pt[r - i, :n] = local
            off += n
            if lens[r] == 0:
                continue
            k, v = kv_override[r] if r in kv_override else synth.session_kv(
                seed, int(gen_sids[r]), lens[r], layer, num_kv_heads, head_dim, value_scale, dtype)
            oracle.pack_session(pool, 1, num_kv_heads, head_dim, od, 0, local, k, v)
        out[i:j] = oracle.paged_attention(pool, max(n_pages, 1), 1, num_kv_heads, head_dim, od, 0, q[i:j], pt,
                                          np.array(lens[i:j], np.int32), s)
        i = j
    return out


def rowwise_check(got: np.ndarray, ref: np.ndarray, max_abs: float = 1e-2, max_norm: float = 1e-2):
    """tolerance_check on every batch row separately (each row normalised by its
    own largest reference magnitude); returns the worst (abs, normalised)."""
    worst = (0.0, 0.0)
    for b in range(got.shape[0]):
        err, norm = tolerance_check(got[b], ref[b], max_abs, max_norm)
        worst = (max(worst[0], err), max(worst[1], norm))
    return worst


def torch_dtype(dtype: str):
    import torch
    return torch.bfloat16 if dtype == "bf16" else torch.float32


def to_device(arr: np.ndarray, dtype: str, device):
    """Upload bf16 bit patterns (uint16) or float32 as a torch tensor of the pool dtype."""
    import torch
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


def to_host(t) -> np.ndarray:
    """Device tensor of the pool dtype -> float64 numpy."""
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def build_gpu(case: Case, device, num_cold_pages: int = 0, poison: bool = False, pool_kwargs=None):
    """A HotColdPool holding the case's sessions (session b = row b), written with
    kv_write_tokens at the case's placement."""
    import torch
    from paper_2609_25782_amd.pool import HotColdPool

    kw = dict(pool_kwargs or {})
    pool = HotColdPool(case.num_layers, case.num_kv_heads, case.head_dim, case.dtype,
                       case.hot_pages, num_cold_pages, max(case.batch, kw.pop("max_sessions", 1)),
                       case.stride, device=device.index or 0, **kw)
    if poison:
        if case.dtype == "bf16":
            pool.hot.view(torch.int16).fill_(0x7FC0)
        else:
            pool.hot.view(torch.float32).fill_(float("nan"))
    for b, L in enumerate(case.seq_lens):
        sid = pool.create_session(L, [int(p) for p in case.placement[b]])
        assert sid == b
        if L > 0:
            k, v = case.kv[b]
            kt = to_device(k, case.dtype, device)
            vt = to_device(v, case.dtype, device)
            pool.write_tokens(sid, case.layer, 0, kt, vt)
    return pool
