"""A pool object over the C ABI: torch supplies device memory and streams,
every operation is a call into the HIP library."""

from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import hotcold_kv as kv

_DTYPES = {"bf16": (kv.KV_DTYPE_BF16, torch.bfloat16), "f32": (kv.KV_DTYPE_F32, torch.float32)}


def _stream(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class HotColdPool:
    """Hot and cold page pools plus the pool's page table, all caller-owned torch
    tensors, bound to one library pool handle."""

    def __init__(self, num_layers: int, num_kv_heads: int, head_dim: int, dtype: str,
                 num_hot_pages: int, num_cold_pages: int, max_sessions: int,
                 max_pages_per_session: int, device: int = 0, cold_location: str = "device",
                 stream: Optional[torch.cuda.Stream] = None):
        kdtype, self.torch_dtype = _DTYPES[dtype]
        self.dtype = dtype
        self.device = torch.device("cuda", device)
        self.desc = kv.kv_pool_desc(num_layers, num_kv_heads, head_dim, kv.KV_PAGE_TOKENS, kdtype,
                                    num_hot_pages, num_cold_pages,
                                    kv.KV_COLD_PINNED_HOST if cold_location == "host" else kv.KV_COLD_DEVICE,
                                    max_sessions, max_pages_per_session, device, 0)
        self.page_bytes = kv.kv_page_bytes(self.desc)
        if self.page_bytes == 0:
            raise ValueError("invalid pool shape")
        self.num_layers, self.num_kv_heads, self.head_dim = num_layers, num_kv_heads, head_dim
        self.num_hot_pages, self.num_cold_pages = num_hot_pages, num_cold_pages
        self.max_sessions, self.stride = max_sessions, max_pages_per_session
        self.hot = torch.empty(max(num_hot_pages, 1) * self.page_bytes, dtype=torch.uint8,
                               device=self.device)
        if cold_location == "host":
            self.cold = torch.empty(max(num_cold_pages, 1) * self.page_bytes, dtype=torch.uint8,
                                    pin_memory=True)
        else:
            self.cold = torch.empty(max(num_cold_pages, 1) * self.page_bytes, dtype=torch.uint8,
                                    device=self.device)
        self.page_table = torch.empty((max_sessions, max_pages_per_session), dtype=torch.int32,
                                      device=self.device)
        self.handle = kv.kv_pool_create(self.desc, self.hot.data_ptr(), self.hot.numel(),
                                        self.cold.data_ptr(), self.cold.numel(),
                                        self.page_table.data_ptr(), _stream(stream))
        self._ws = {}   # decode workspace per stream: decodes on different streams may overlap

    # -- layout ------------------------------------------------------------
    @property
    def slice_bytes(self) -> int:
        """Bytes of one layer of one page: [kv_head][K tile, V tile]."""
        return self.page_bytes // self.num_layers

    def hot_pages(self) -> torch.Tensor:
        """The hot pool as [num_hot_pages][num_layers][slice_bytes], a view in page
        order.  The hot pool is layer-major: the slice of page p for layer l sits at
        byte (l * num_hot_pages + p) * slice_bytes."""
        return self.hot.view(self.num_layers, max(self.num_hot_pages, 1), self.slice_bytes).transpose(0, 1)

    def hot_page_bytes(self, ids=None) -> torch.Tensor:
        """Hot pages (all, or the ids given) as [n][page_bytes] in the cold pool's
        page-major order (a copy): what the same pages hold, byte for byte, once
        copied to the cold tier."""
        v = self.hot_pages()
        if ids is not None:
            v = v[torch.as_tensor(ids, dtype=torch.long, device=self.device).reshape(-1)]
        return v.reshape(v.shape[0], self.page_bytes)

    # -- lifetime ----------------------------------------------------------
    def close(self) -> None:
        if getattr(self, "handle", None):
            torch.cuda.synchronize(self.device)
            kv.kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- sessions ----------------------------------------------------------
    def create_session(self, seq_len: int, hot_pages: Optional[Sequence[int]] = None, stream=None) -> int:
        return kv.kv_session_create(self.handle, int(seq_len), hot_pages, _stream(stream))

    def import_cold(self, seq_len: int, cold_pages: Sequence[int]) -> int:
        return kv.kv_session_import_cold(self.handle, int(seq_len), cold_pages)

    def extend(self, sid: int, new_seq_len: int, stream=None) -> None:
        kv.kv_session_extend(self.handle, sid, int(new_seq_len), _stream(stream))

    def pause(self, sid: int) -> None:
        kv.kv_session_pause(self.handle, sid)

    def evict_pages(self, n: int, stream=None) -> int:
        return kv.kv_evict_pages(self.handle, int(n), _stream(stream))

    def destroy_session(self, sid: int, stream=None) -> None:
        kv.kv_session_destroy(self.handle, sid, _stream(stream))

    def info(self, sid: int):
        return kv.kv_session_info(self.handle, sid)

    def write_tokens(self, sid: int, layer: int, tok_begin: int, k: torch.Tensor, v: torch.Tensor,
                     stream=None) -> None:
        assert k.is_contiguous() and v.is_contiguous() and k.shape == v.shape
        assert k.dtype == self.torch_dtype and k.device == self.device
        kv.kv_write_tokens(self.handle, sid, layer, tok_begin, k.shape[0], k.data_ptr(), v.data_ptr(),
                           _stream(stream))

    def append_tokens(self, layer: int, sids, positions, k: torch.Tensor, v: torch.Tensor, stream=None) -> None:
        """One token per row: row i of k and v is token positions[i] of session sids[i]."""
        assert k.is_contiguous() and v.is_contiguous() and k.shape == v.shape and k.shape[0] == len(sids)
        assert k.dtype == self.torch_dtype and k.device == self.device
        kv.kv_append_tokens(self.handle, layer, sids, positions, k.data_ptr(), v.data_ptr(), _stream(stream))

    def write_tokens_layers(self, sid: int, layer_begin: int, tok_begin: int, k: torch.Tensor, v: torch.Tensor,
                            stream=None) -> None:
        """k and v [num_layers][n_tok][kv_heads][head_dim]: tokens of layers layer_begin.. in one launch."""
        assert k.is_contiguous() and v.is_contiguous() and k.shape == v.shape and k.dim() == 4
        assert k.dtype == self.torch_dtype and k.device == self.device
        kv.kv_write_tokens_layers(self.handle, sid, layer_begin, k.shape[0], tok_begin, k.shape[1], k.data_ptr(),
                                  v.data_ptr(), _stream(stream))

    def append_tokens_table(self, layer_begin: int, table: torch.Tensor, rows: torch.Tensor, positions: torch.Tensor,
                            k: torch.Tensor, v: torch.Tensor, stream=None) -> None:
        """Device-resolved append: entry i is token positions[i] of table row rows[i]; k and v
        [num_layers][n][kv_heads][head_dim].  Capturable in a HIP graph."""
        assert table.dtype == torch.int32 and table.is_contiguous() and table.dim() == 2
        assert rows.dtype == positions.dtype == torch.int32 and rows.shape == positions.shape
        assert k.is_contiguous() and v.is_contiguous() and k.shape == v.shape and k.dim() == 4
        assert k.shape[1] == rows.shape[0] and k.dtype == self.torch_dtype
        kv.kv_append_tokens_table(self.handle, layer_begin, k.shape[0], table.data_ptr(), table.shape[1],
                                  table.shape[0], rows.data_ptr(), positions.data_ptr(), rows.shape[0],
                                  k.data_ptr(), v.data_ptr(), _stream(stream))

    def fill_synthetic(self, sid: int, gen_sid: int, seed: int, value_mult: float, stream=None) -> None:
        kv.kv_fill_synthetic(self.handle, sid, gen_sid, seed, float(value_mult), _stream(stream))

    def fill_synthetic_pages(self, sid: int, gen_sid: int, seed: int, value_mult: float,
                             first_page: int, num_pages: int, stream=None) -> None:
        kv.kv_fill_synthetic_pages(self.handle, sid, gen_sid, seed, float(value_mult), int(first_page),
                                   int(num_pages), _stream(stream))

    def evict(self, sids, stream=None) -> None:
        if isinstance(sids, int):
            kv.kv_evict_session(self.handle, sids, _stream(stream))
        else:
            kv.kv_evict_sessions(self.handle, list(sids), _stream(stream))

    def resume(self, sids, stream=None) -> None:
        if isinstance(sids, int):
            kv.kv_resume_session(self.handle, sids, _stream(stream))
        else:
            kv.kv_resume_sessions(self.handle, list(sids), _stream(stream))

    def resume_lazy(self, sids, stream=None) -> None:
        kv.kv_resume_sessions_lazy(self.handle, [sids] if isinstance(sids, int) else list(sids),
                                   _stream(stream))

    def set_spill(self, enable: bool) -> None:
        kv.kv_pool_set_spill(self.handle, enable)

    def promote(self, n: int, stream=None) -> int:
        return kv.kv_promote_pages(self.handle, int(n), _stream(stream))

    def set_copy_blocks(self, blocks: int) -> None:
        kv.kv_pool_set_copy_blocks(self.handle, int(blocks))

    def stats(self) -> dict:
        return kv.kv_pool_stats(self.handle)

    # -- decode ------------------------------------------------------------
    def workspace(self, batch: int, num_q_heads: int, stream=None) -> torch.Tensor:
        """The decode workspace of `stream` (one per stream: separate-merge decodes
        on different streams run concurrently and must not share partials)."""
        key = _stream(stream)
        need = kv.paged_decode_workspace_bytes(self.handle, batch, num_q_heads)
        ws = self._ws.get(key)
        if ws is None or ws.numel() < need:
            # allocated on that stream, so torch reuses a dropped buffer only in its order
            with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
                ws = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
            self._ws[key] = ws
        return ws

    def decode(self, layer: int, q: torch.Tensor, seq_lens: torch.Tensor,
               page_table: Optional[torch.Tensor] = None, scale: Optional[float] = None,
               out: Optional[torch.Tensor] = None, stream=None, k_new: Optional[torch.Tensor] = None,
               v_new: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Decode attention of one layer; with k_new / v_new ([B][kv_heads][head_dim]) each
        row's token seq_lens[b] - 1 is appended first, in the same launch."""
        pt = self.page_table if page_table is None else page_table
        assert q.is_contiguous() and q.dtype == self.torch_dtype and q.dim() == 3
        assert pt.dtype == torch.int32 and pt.is_contiguous() and seq_lens.dtype == torch.int32
        B, Hq, D = q.shape
        if out is None:
            out = torch.empty_like(q)
        ws = self.workspace(B, Hq, stream)
        s = float(scale if scale is not None else D ** -0.5)
        if k_new is None:
            kv.paged_decode_attention(self.handle, layer, q.data_ptr(), pt.data_ptr(), pt.shape[1],
                                      seq_lens.data_ptr(), B, Hq, s, out.data_ptr(), ws.data_ptr(), ws.numel(),
                                      _stream(stream))
        else:
            assert k_new.is_contiguous() and v_new.is_contiguous() and k_new.shape == v_new.shape
            assert k_new.shape == (B, self.num_kv_heads, D) and k_new.dtype == self.torch_dtype
            kv.paged_decode_attention_append(self.handle, layer, q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
                                             pt.data_ptr(), pt.shape[1], seq_lens.data_ptr(), B, Hq, s,
                                             out.data_ptr(), ws.data_ptr(), ws.numel(), _stream(stream))
        return out

    def gather_table(self, sids: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
        """Page-table rows of the given sessions (device int32 ids), for decoding them as a batch."""
        assert sids.dtype == torch.int32 and sids.is_contiguous() and sids.device == self.device
        n = sids.shape[0]
        if out is None:
            out = torch.empty((n, self.stride), dtype=torch.int32, device=self.device)
        assert out.shape[0] >= n and out.shape[1] == self.stride and out.is_contiguous()
        kv.paged_decode_gather_table(self.handle, sids.data_ptr(), n, out.data_ptr(), _stream(stream))
        return out

    def partition(self, seq_lens: torch.Tensor, waves: int, stream=None) -> torch.Tensor:
        B = seq_lens.shape[0]
        slots = torch.empty((waves + B * self.num_kv_heads, 4), dtype=torch.int32, device=self.device)
        kv.paged_decode_partition(self.handle, seq_lens.data_ptr(), B, waves, slots.data_ptr(),
                                  _stream(stream))
        return slots

    def waves(self) -> int:
        return kv.paged_decode_waves(self.handle)

    def set_waves(self, waves: int) -> None:
        kv.kv_pool_set_decode_waves(self.handle, waves)

    def set_combine(self, fused: bool) -> None:
        kv.kv_pool_set_decode_combine(self.handle, kv.KV_COMBINE_FUSED if fused else kv.KV_COMBINE_SEPARATE)

    def set_host_copy(self, kernel: bool) -> None:
        kv.kv_pool_set_host_copy(self.handle, kv.KV_HOST_COPY_KERNEL if kernel else kv.KV_HOST_COPY_DMA)

    def set_compute(self, vector: bool) -> None:
        kv.kv_pool_set_decode_compute(self.handle, kv.KV_DECODE_VECTOR if vector else kv.KV_DECODE_MATRIX)


class CUStream:
    """A torch stream whose kernels run only on CU slots [begin, end) of every
    XCD (one slot = one CU per XCD).  The library creates the HIP stream; close()
    waits for the device and destroys it."""

    def __init__(self, begin: int, end: int, device: int = 0):
        xcds, _ = kv.kv_device_cu_slots(device)
        self.device = torch.device("cuda", device)
        self.handle = kv.kv_stream_create_cu_slots(device, begin, end)
        self.stream = torch.cuda.ExternalStream(self.handle, device=self.device)
        self.cus = xcds * (end - begin)

    def close(self) -> None:
        if getattr(self, "handle", None):
            torch.cuda.synchronize(self.device)
            kv.kv_stream_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def split_streams(copy_slots: int, device: int = 0):
    """A decode stream and a copy stream on disjoint CUs: the copy stream gets
    `copy_slots` CUs of every XCD, the decode stream the rest."""
    _, slots = kv.kv_device_cu_slots(device)
    if not 0 < copy_slots < slots:
        raise ValueError("copy_slots must be in [1, %d)" % slots)
    return CUStream(copy_slots, slots, device), CUStream(0, copy_slots, device)
