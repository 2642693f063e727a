"""Parity at the workloads' full sizes, in the launch configuration the benchmark
uses (automatic wave count, default merge).  Pools are filled on the GPU with the
counter-based generator; the oracle recomputes sampled rows from the same values
regenerated on the CPU, packed by its own code.  Resume copies are checked byte
for byte against the cold pages and the page tables against the pool model."""

import gc
import math
import sys

import numpy as np
import pytest
import torch

import synth
from helpers import Case, tolerance_check, to_host
from oracle.pool_model import PoolModel

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _free():
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _filled_pool(w, dev, extra_hot=0, num_cold=0, max_sessions=None, stride=None):
    from paper_2609_25782_amd.pool import HotColdPool
    stride = stride or max(synth.pages_for(int(w.seq_lens.max())), 1)
    pool = HotColdPool(w.num_layers, w.num_kv_heads, w.head_dim, w.dtype, w.hot_pages + extra_hot,
                       num_cold, max_sessions or w.batch, stride)
    mult = float(synth.value_multiplier(w.value_scale))
    for b in range(w.batch):
        sid = pool.create_session(int(w.seq_lens[b]), [int(p) for p in w.placement[b]])
        assert sid == b
        pool.fill_synthetic(sid, b, w.seed, mult)
    return pool


def _check_rows(w, pool, dev, layer, rows, q_np):
    q = torch.from_numpy(q_np.view(np.int16)).to(dev).view(torch.bfloat16)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    got = to_host(pool.decode(layer, q, sl, page_table=pool.page_table[:w.batch]))
    torch.cuda.synchronize()
    for b in rows:
        L = int(w.seq_lens[b])
        case = Case(w.num_layers, w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype, [L],
                    seed=w.seed, value_scale=w.value_scale, layer=layer,
                    placement=[np.arange(synth.pages_for(L), dtype=np.int32)])
        case.kv = [synth.session_kv(w.seed, b, L, layer, w.num_kv_heads, w.head_dim, w.value_scale,
                                    w.dtype)]
        case.q = q_np[b:b + 1]
        err, norm = tolerance_check(got[b:b + 1], case.oracle_out())
        _say("  layer %d row %d (L=%d): max abs %.3g normalised %.3g" % (layer, b, L, err, norm))
    return got


def test_layer_config_full_size(dev):
    """One Qwen3-Coder-30B-A3B-shaped layer, B=32, L ~ U[8192, 32768]: sampled rows."""
    w = synth.config_layer(0)
    _say("layer config: %d tokens, %d hot pages" % (int(w.seq_lens.sum()), w.hot_pages))
    pool = _filled_pool(w, dev)
    q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")
    rows = [int(np.argmax(w.seq_lens)), int(np.argmin(w.seq_lens)), 7]
    _check_rows(w, pool, dev, 0, rows, q_np)
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(400)
def test_step48_config_full_size(dev):
    """48 layers, B=64, lognormal lengths (median 24K, cap 64K), ~170 GB hot pool:
    every layer decodes; sampled rows of three layers against the oracle."""
    w = synth.config_step48(0)
    gb = w.hot_pages * 1.5 / 1024
    _say("step48 config: %d tokens, %d hot pages (%.0f GiB)" % (int(w.seq_lens.sum()), w.hot_pages, gb))
    pool = _filled_pool(w, dev)
    q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")
    q = torch.from_numpy(q_np.view(np.int16)).to(dev).view(torch.bfloat16)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    out = torch.empty_like(q)
    for layer in range(48):
        pool.decode(layer, q, sl, page_table=pool.page_table[:w.batch], out=out)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all()
    capped = int(np.argmax(w.seq_lens))
    for layer, rows in ((0, [capped, 5]), (23, [int(np.argmin(w.seq_lens))]), (47, [40])):
        _check_rows(w, pool, dev, layer, rows, q_np)
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(300)
def test_skewed_config_full_size(dev):
    """B=128, lengths from a bounded power law on [1K, 256K], one layer."""
    w = synth.config_skewed(0)
    _say("skewed config: %d tokens, longest %d, %d hot pages" % (
        int(w.seq_lens.sum()), int(w.seq_lens.max()), w.hot_pages))
    pool = _filled_pool(w, dev)
    q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")
    rows = [int(np.argmax(w.seq_lens)), int(np.argmin(w.seq_lens)), 64]
    _check_rows(w, pool, dev, 0, rows, q_np)
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(400)
def test_resume_mix_config_full_size(dev):
    """Resume-heavy mix: 1,024 paused sessions of 32K-128K tokens at 48 layers over a
    physical cold pool of 49,152 pages (72 GiB), 32 active sessions; resume 8
    sessions in one call: page tables equal the model's, every resumed page equals
    its cold page byte for byte, and an active session still decodes to the
    oracle's answer."""
    from paper_2609_25782_amd.pool import HotColdPool
    w = synth.config_resume_mix(0)
    n_cold = w.cold_pages
    stride = synth.pages_for(131072)
    paused = len(w.paused_lens)
    ms = w.batch + paused
    _say("resume mix: %d hot pages, %d cold pages, %d paused sessions" % (w.hot_pages, n_cold, paused))
    pool = HotColdPool(48, 4, 128, "bf16", w.hot_pages, n_cold, ms, stride)
    model = PoolModel(w.hot_pages, n_cold, ms, stride)
    mult = float(synth.value_multiplier(w.value_scale))
    for b in range(w.batch):
        pages = [int(p) for p in w.placement[b]]
        assert pool.create_session(int(w.seq_lens[b]), pages) == model.create(int(w.seq_lens[b]), pages) == b
        pool.fill_synthetic(b, b, w.seed, mult)
    # the physical cold pool: random bytes (the copies must move them unchanged)
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    view = pool.cold.view(n_cold, -1)
    for i in range(0, n_cold, 4096):
        view[i:i + 4096].copy_(torch.randint(0, 256, view[i:i + 4096].shape, dtype=torch.uint8,
                                             device=dev, generator=g))
    sids = []
    for j, L in enumerate(w.paused_lens):
        cold = synth.cold_page_draw(w.seed, j, synth.pages_for(int(L)), n_cold)
        sid = pool.import_cold(int(L), cold)
        assert sid == model.import_cold(int(L), cold)
        sids.append(sid)
    rng = np.random.default_rng(3)
    chosen = [int(sids[i]) for i in rng.choice(paused, size=8, replace=False)]
    pool.resume(chosen)
    copies = model.resume(chosen)
    torch.cuda.synchronize()
    got_rows = pool.page_table[chosen].cpu().numpy()
    want_rows = np.array([model.row(s) for s in chosen], dtype=np.int32)
    assert np.array_equal(got_rows, want_rows)
    pb = pool.page_bytes
    hot = pool.hot.view(-1, pb)
    total = 0
    for per in copies:
        src = torch.tensor([c for c, _ in per], dtype=torch.long, device=dev)
        dst = torch.tensor([h for _, h in per], dtype=torch.long, device=dev)
        for i in range(0, len(per), 512):
            assert torch.equal(hot.index_select(0, dst[i:i + 512]), view.index_select(0, src[i:i + 512]))
        total += len(per)
    _say("resumed %d pages (%.1f GiB), all bit-exact" % (total, total * pb / 2 ** 30))
    # the active sessions were not touched: decode one of them at layer 10 against the oracle
    q_np = synth.queries(w.seed + 1, w.batch, 32, 128, w.value_scale, "bf16")
    q = torch.from_numpy(q_np.view(np.int16)).to(dev).view(torch.bfloat16)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    got = to_host(pool.decode(10, q, sl, page_table=pool.page_table[:w.batch].contiguous()))
    torch.cuda.synchronize()
    b = 3
    L = int(w.seq_lens[b])
    case = Case(48, 32, 4, 128, "bf16", [L], seed=w.seed, value_scale=w.value_scale, layer=10,
                placement=[np.arange(synth.pages_for(L), dtype=np.int32)])
    case.kv = [synth.session_kv(w.seed, b, L, 10, 4, 128, w.value_scale, "bf16")]
    case.q = q_np[b:b + 1]
    tolerance_check(got[b:b + 1], case.oracle_out())
    pool.close()
    del pool
    _free()
