"""Parity at the workloads' full sizes, in the launch configuration the benchmark
uses (automatic wave count, default merge).  Pools are filled on the GPU with the
counter-based generator; the oracle recomputes sampled rows from the same values
regenerated on the CPU, packed by its own code.  Resume copies are checked byte
for byte against the cold pages and the page tables against the pool model."""

import gc
import math
import sys
import time

import numpy as np
import pytest
import torch

import synth
from helpers import Case, oracle_rows, rowwise_check, to_device, to_host, tolerance_check
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


def _all_rows(w, got, layer, q_np, kv_override=None):
    """Every row of `got` (the GPU output of the whole batch at `layer`) against
    the oracle, row by row; returns the worst (abs, normalised) error."""
    t0 = time.time()
    ref = oracle_rows(w.seed, range(w.batch), w.seq_lens, layer, q_np, w.num_kv_heads, w.head_dim, w.dtype,
                      w.value_scale, kv_override=kv_override)
    err, norm = rowwise_check(got, ref)
    _say("  layer %d: all %d rows (%d tokens) vs oracle in %.1f s: worst max abs %.3g, normalised %.3g"
         % (layer, w.batch, int(w.seq_lens.sum()), time.time() - t0, err, norm))
    return ref


def _q(q_np, dev):
    return torch.from_numpy(np.ascontiguousarray(q_np).view(np.int16)).to(dev).view(torch.bfloat16)


@pytest.mark.timeout(600)
def test_layer_config_full_size(dev):
    """One Qwen3-Coder-30B-A3B-shaped layer, B=32, L ~ U[8192, 32768], in the
    benchmark's launch configuration (hot pool with the resume headroom, row
    stride 2,048, automatic wave count, separate merge).  Every row against the
    oracle; then poison of every tail slot past each row's length and of every
    free hot page (bitwise equal to the clean run); then needles at the last token
    of the longest row and at a mid-row page start of another (O(1) outputs that
    catch any page-table or offset slip), every row against the oracle again;
    then the same call with the fused merge and with the vector-ALU split."""
    from paper_2609_25782_amd.pool import HotColdPool
    w = synth.config_layer(0)
    headroom = 8 * synth.pages_for(32768)
    num_hot = w.hot_pages + headroom
    _say("layer config: %d tokens, %d hot pages" % (int(w.seq_lens.sum()), num_hot))
    pool = HotColdPool(1, 4, 128, "bf16", num_hot, 0, w.batch + 8, synth.pages_for(32768))
    mult = float(synth.value_multiplier(w.value_scale))
    padded = [16 * synth.pages_for(int(L)) for L in w.seq_lens]
    for b in range(w.batch):
        # sessions span whole pages, so the slots past L can be written (poisoned) below
        assert pool.create_session(padded[b], [int(p) for p in w.placement[b]]) == b
        pool.fill_synthetic(b, b, w.seed, mult)
    q_np = synth.queries(w.seed + 1, w.batch, 32, 128, w.value_scale, "bf16")
    q = _q(q_np, dev)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    pt = pool.page_table[:w.batch]
    assert pool.waves() == 3 * torch.cuda.get_device_properties(0).multi_processor_count
    clean = pool.decode(0, q, sl, page_table=pt).clone()
    torch.cuda.synchronize()
    _all_rows(w, to_host(clean), 0, q_np)
    # poison: NaN in every slot past each row's length, and in every free hot page
    nan_tok = torch.full((16, 4, 128), float("nan"), dtype=torch.bfloat16, device=dev)
    for b in range(w.batch):
        L = int(w.seq_lens[b])
        if padded[b] > L:
            pool.write_tokens(b, 0, L, nan_tok[:padded[b] - L].contiguous(), nan_tok[:padded[b] - L].contiguous())
    used = np.zeros(num_hot, bool)
    used[np.concatenate(w.placement)] = True
    free = torch.from_numpy(np.flatnonzero(~used)).to(dev)
    pool.hot_pages().view(torch.int16).index_fill_(0, free, 0x7FC0)
    dirty = pool.decode(0, q, sl, page_table=pt).clone()
    torch.cuda.synchronize()
    assert torch.equal(dirty, clean)
    _say("  poison of %d tail slots and %d free pages: bitwise equal to the clean run"
         % (sum(padded) - int(w.seq_lens.sum()), int(free.numel())))
    # needles
    b1 = int(np.argmax(w.seq_lens))
    b2 = int(np.argsort(w.seq_lens)[w.batch // 2])
    t1 = int(w.seq_lens[b1]) - 1
    t2 = 16 * (synth.pages_for(int(w.seq_lens[b2])) // 2)
    override = {}
    for b, t, g in ((b1, t1, 1), (b2, t2, 3)):
        k, v = synth.session_kv(w.seed, b, int(w.seq_lens[b]), 0, 4, 128, w.value_scale, "bf16")
        q_np[b, 8 * g:8 * (g + 1)] = q_np[b, 8 * g]
        qv = synth.bf16_bits_to_f32(q_np[b, 8 * g]).astype(np.float64)
        k[t, g] = synth.f32_to_bf16_bits((60.0 * math.sqrt(128) * qv / np.dot(qv, qv)).astype(np.float32))
        v[t, g] = synth.f32_to_bf16_bits(np.linspace(-1, 1, 128).astype(np.float32))
        pool.write_tokens(b, 0, t, to_device(k[t:t + 1], "bf16", dev), to_device(v[t:t + 1], "bf16", dev))
        override[b] = (k, v)
    q = _q(q_np, dev)
    got = to_host(pool.decode(0, q, sl, page_table=pt))
    torch.cuda.synchronize()
    for b, t, g in ((b1, t1, 1), (b2, t2, 3)):
        want = synth.bf16_bits_to_f32(override[b][1][t, g]).astype(np.float64)
        for h in range(8 * g, 8 * (g + 1)):
            assert np.max(np.abs(got[b, h] - want)) <= 2 ** -8
        _say("  needle at row %d (L=%d) token %d, KV head %d: output = its value" % (b, w.seq_lens[b], t, g))
    _all_rows(w, got, 0, q_np, kv_override=override)
    same = [b for b in range(w.batch) if b not in override]
    assert np.array_equal(got[same], to_host(clean)[same])
    # the fused merge and the vector-ALU products, at the same full size
    for name, fused, vector in (("fused merge", True, False), ("vector-ALU split", False, True)):
        pool.set_combine(fused)
        pool.set_compute(vector)
        other = to_host(pool.decode(0, q, sl, page_table=pt))
        torch.cuda.synchronize()
        _say("  %s:" % name)
        _all_rows(w, other, 0, q_np, kv_override=override)
    pool.set_combine(False)
    pool.set_compute(False)
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(600)
def test_layer_config_round_trip_relocates_bitwise(dev):
    """The headline layer workload (B=32, L ~ U[8192, 32768], pages scattered at
    random) in the benchmark's launch configuration: evict 8 sessions to the cold
    tier and resume them, which puts them on the lowest free hot pages, not their
    old ones.  Every resumed page holds the bytes its session's page held before
    the eviction, and the whole batch decodes bit for bit as before."""
    from paper_2609_25782_amd.pool import HotColdPool
    w = synth.config_layer(0)
    headroom = 8 * synth.pages_for(32768)
    num_hot = w.hot_pages + headroom
    movers = [int(b) for b in np.argsort(w.seq_lens)[-8:]]  # the 8 longest rows
    n_cold = sum(synth.pages_for(int(w.seq_lens[b])) for b in movers)
    pool = HotColdPool(1, 4, 128, "bf16", num_hot, n_cold, w.batch, synth.pages_for(32768))
    mult = float(synth.value_multiplier(w.value_scale))
    for b in range(w.batch):
        assert pool.create_session(int(w.seq_lens[b]), [int(p) for p in w.placement[b]]) == b
        pool.fill_synthetic(b, b, w.seed, mult)
    q = _q(synth.queries(w.seed + 1, w.batch, 32, 128, w.value_scale, "bf16"), dev)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    before_rows = pool.page_table[movers].clone()
    lens = [synth.pages_for(int(w.seq_lens[b])) for b in movers]
    saved = [pool.hot_page_bytes(before_rows[j, :n].long()).clone() for j, n in enumerate(lens)]
    before = pool.decode(0, q, sl, page_table=pool.page_table[:w.batch]).clone()
    pool.evict(movers)
    pool.resume(movers)
    torch.cuda.synchronize()
    after_rows = pool.page_table[movers]
    moved = int((after_rows != before_rows).sum())
    assert moved > 0
    after = pool.decode(0, q, sl, page_table=pool.page_table[:w.batch])
    torch.cuda.synchronize()
    assert torch.equal(after, before)
    for j, n in enumerate(lens):
        assert torch.equal(pool.hot_page_bytes(after_rows[j, :n].long()), saved[j])
    _say("round trip of %d sessions: %d page-table entries changed; decode bitwise equal" % (len(movers), moved))
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(900)
def test_step48_config_full_size(dev):
    """48 layers, B=64, lognormal lengths (median 24K, cap 64K), ~170 GB hot pool:
    every layer decodes finite; all 64 rows of layers 0 and 47 against the oracle."""
    w = synth.config_step48(0)
    gb = w.hot_pages * 1.5 / 1024
    _say("step48 config: %d tokens, %d hot pages (%.0f GiB)" % (int(w.seq_lens.sum()), w.hot_pages, gb))
    pool = _filled_pool(w, dev)
    q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")
    q = _q(q_np, dev)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    outs = torch.empty((48,) + tuple(q.shape), dtype=q.dtype, device=dev)
    for layer in range(48):
        pool.decode(layer, q, sl, page_table=pool.page_table[:w.batch], out=outs[layer])
    torch.cuda.synchronize()
    assert torch.isfinite(outs.float()).all()
    for layer in (0, 47):
        _all_rows(w, to_host(outs[layer]), layer, q_np)
    pool.close()
    del pool
    _free()


@pytest.mark.timeout(900)
def test_skewed_config_full_size(dev):
    """B=128, lengths from a bounded power law on [1K, 256K], one layer: all 128
    rows against the oracle."""
    w = synth.config_skewed(0)
    _say("skewed config: %d tokens, longest %d, %d hot pages" % (
        int(w.seq_lens.sum()), int(w.seq_lens.max()), w.hot_pages))
    pool = _filled_pool(w, dev)
    q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")
    got = to_host(pool.decode(0, _q(q_np, dev), torch.from_numpy(w.seq_lens.copy()).to(dev),
                              page_table=pool.page_table[:w.batch]))
    torch.cuda.synchronize()
    _all_rows(w, got, 0, q_np)
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
    total = 0
    for per in copies:
        src = torch.tensor([c for c, _ in per], dtype=torch.long, device=dev)
        dst = torch.tensor([h for _, h in per], dtype=torch.long, device=dev)
        for i in range(0, len(per), 512):
            assert torch.equal(pool.hot_page_bytes(dst[i:i + 512]), view.index_select(0, src[i:i + 512]))
        total += len(per)
    _say("resumed %d pages (%.1f GiB), all bit-exact" % (total, total * pb / 2 ** 30))
    # the active sessions were not touched: all 32 decode at layer 10 as the oracle says
    q_np = synth.queries(w.seed + 1, w.batch, 32, 128, w.value_scale, "bf16")
    q = torch.from_numpy(q_np.view(np.int16)).to(dev).view(torch.bfloat16)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    got = to_host(pool.decode(10, q, sl, page_table=pool.page_table[:w.batch].contiguous()))
    torch.cuda.synchronize()
    _all_rows(w, got, 10, q_np)
    pool.close()
    del pool
    _free()
