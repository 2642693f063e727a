#!/usr/bin/env python3
"""Benchmark of the hot-cold KV hot path on one MI355X.

One step is one pass of the whole hot path over one batch:
  1. resume R paused sessions (batched cold -> hot gather + page-table rewrite),
  2. paged GQA decode attention over the B active sessions (split + combine),
  3. evict the R sessions again in one batched call (write-on-evict: their
     cold copies are still valid, so no page is rewritten; rows are cleared and
     pages freed).

Default workload: one Qwen3-Coder-30B-A3B-shaped attention layer (32 query /
4 KV heads, head_dim 128, bf16, 16-token pages), 32 active sessions with
context lengths uniform in [8192, 32768], values N(0,1)/sqrt(128), pages
randomly scattered over a hot pool 1.25x the pages needed; plus 8 paused
sessions of the same length distribution in the cold pool.

Prints one JSON line (kept under 12 KB: the sweeps of the other workloads go
to stderr as one summary line each, and in full to --full-json).  `value` is
decode-attention throughput in GB/s: algorithmic bytes (K and V of every valid
token, Q, out, page-table entries, lengths) per decode call divided by the
median time of one decode call in the timed pass (HIP events on the launch
stream just before and after the call: both kernels, the gap between them and
the event packets).  Inputs are resident in HBM.  The split kernel's own rate
(events the dispatch records at its start and end) is under `roofline`.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "decode-attention HBM GB/s (% of peak) + resume latency ms/session, 1 GPU"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def decode_bytes(seq_lens, hq, hkv, d, elt):
    """Algorithmic bytes of one decode call: K+V of each valid token for every KV
    head, Q and out rows, one page-table entry per used page, one length per row."""
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    B = len(seq_lens)
    kv = int(seq_lens.sum()) * hkv * d * 2 * elt
    qo = B * hq * d * elt * 2
    pt = 4 * int(((seq_lens + 15) // 16).sum()) + 4 * B
    return kv, qo, pt


def split_kernel_bytes(seq_lens, hq, hkv, d, elt):
    kv, qo, pt = decode_bytes(seq_lens, hq, hkv, d, elt)
    return kv + qo // 2 + pt  # K/V, Q, page table, lengths (the output is the combine's)


PMC_SUMMARY = os.path.join(ROOT, "profiles", "decode_split_layer_b32_pmc.md")
SPLIT_SOURCES = ("paper_2609_25782_amd/csrc/decode_attention.hip",
                 "paper_2609_25782_amd/csrc/device_common.h",
                 "paper_2609_25782_amd/csrc/kernels.h")


def measured_traffic():
    """HBM bytes per split-kernel launch from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE, calibrated against a copy of known size),
    or None when the kernel sources changed since the counters were taken."""
    import hashlib
    try:
        text = open(PMC_SUMMARY).read()
    except OSError:
        return None
    fields = dict(l.split(": ", 1) for l in text.splitlines()
                  if l.startswith(("traffic_bytes_per_launch: ", "kernel_source_sha256: ")))
    h = hashlib.sha256()
    for f in SPLIT_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    if fields.get("kernel_source_sha256") != h.hexdigest():
        return None
    return int(fields["traffic_bytes_per_launch"])


def cpu_baseline(w, budget_s: float):
    """Time the fp64 oracle on whole sessions of the same workload, cycling over
    the sessions (each packed once) until about `budget_s` seconds of oracle
    time have been spent (at least one session)."""
    import oracle
    import synth
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
    d, hkv, hq = w.head_dim, w.num_kv_heads, w.num_q_heads
    spent, nbytes, calls, tokens = 0.0, 0, 0, 0
    q_all = synth.queries(w.seed + 1, w.batch, hq, d, w.value_scale, w.dtype)
    packed = {}
    while True:
        b = calls % w.batch
        L = int(w.seq_lens[b])
        if b not in packed:
            k, v = synth.session_kv(w.seed, b, L, 0, hkv, d, w.value_scale, w.dtype)
            n = synth.pages_for(L)
            pool = np.zeros(n * oracle.page_bytes(1, hkv, d, oracle.BF16), np.uint8)
            pages = np.arange(n, dtype=np.int32)
            oracle.pack_pool(pool, 1, hkv, d, oracle.BF16, 0, pages, k, v)
            packed[b] = (pool, n, pages[None, :].copy())
        pool, n, pt = packed[b]
        t0 = time.perf_counter()
        oracle.paged_attention(pool, n, 1, hkv, d, oracle.BF16, 0, q_all[b:b + 1], pt,
                               np.array([L], np.int32), 1.0 / math.sqrt(d), num_threads=threads)
        spent += time.perf_counter() - t0
        kvb, qo, ptb = decode_bytes([L], hq, hkv, d, 2)
        nbytes += kvb + qo + ptb
        calls += 1
        tokens += L
        if calls % w.batch == 0 or spent >= budget_s:
            log("cpu baseline: %d session decodes, %.1f s of oracle time" % (calls, spent))
        if spent >= budget_s:
            break
    # the same oracle on one thread, over the first two sessions
    t1_s, t1_bytes = 0.0, 0
    for b in range(min(2, w.batch)):
        pool, n, pt = packed[b]
        L = int(w.seq_lens[b])
        t0 = time.perf_counter()
        oracle.paged_attention(pool, n, 1, hkv, d, oracle.BF16, 0, q_all[b:b + 1], pt,
                               np.array([L], np.int32), 1.0 / math.sqrt(d), num_threads=1)
        t1_s += time.perf_counter() - t0
        t1_bytes += sum(decode_bytes([L], hq, hkv, d, 2))
    log("cpu baseline: one thread, 2 sessions, %.1f s" % t1_s)
    return {"value": round(nbytes / spent / 1e9, 4), "unit": "GB/s", "cores": threads,
            "value_1_thread": round(t1_bytes / t1_s / 1e9, 4),
            "kind": "oracle",
            "sample": "fp64 C oracle (OpenMP over query heads): %d whole-session decodes cycling over "
                      "the workload's %d sessions (%.2f passes, %d tokens, all 32 query heads), %.1f s" % (
                          calls, w.batch, calls / w.batch, tokens, spent)}


def measure_resume_mix(seed: int, steps: int, warmup: int):
    """Resume-heavy mix at 48 layers: 32 active sessions (8K-32K tokens), 1,024 paused
    sessions of 32K-128K tokens over a physical cold pool of 49,152 pages, 8 resumes
    per step.  Times the batched resume alone, the 48-layer decode of the active
    sessions alone, and both together on two streams (TBT impact)."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool

    w = synth.config_resume_mix(seed)
    dev = torch.device("cuda", 0)
    stride = synth.pages_for(131072)
    n_paused = len(w.paused_lens)
    pool = HotColdPool(48, 4, 128, "bf16", w.hot_pages, w.cold_pages, w.batch + n_paused, stride)
    mult = float(synth.value_multiplier(w.value_scale))
    for b in range(w.batch):
        pool.create_session(int(w.seq_lens[b]), [int(p) for p in w.placement[b]])
        pool.fill_synthetic(b, b, w.seed, mult)
    paused = [pool.import_cold(int(L), synth.cold_page_draw(w.seed, j, synth.pages_for(int(L)), w.cold_pages))
              for j, L in enumerate(w.paused_lens)]
    log("resume mix: %d hot pages, %d cold pages, %d paused sessions imported" % (
        w.hot_pages, w.cold_pages, n_paused))
    q = torch.from_numpy(synth.queries(w.seed + 1, w.batch, 32, 128, w.value_scale, "bf16")
                         .view(np.int16)).to(dev).view(torch.bfloat16)
    sl = torch.from_numpy(w.seq_lens.copy()).to(dev)
    pt = pool.page_table[:w.batch]
    out = torch.empty_like(q)
    rng = np.random.Generator(np.random.PCG64([seed, 11]))
    picks = [[paused[i] for i in rng.choice(n_paused, size=8, replace=False)]
             for _ in range(warmup + 3 * steps)]
    side = torch.cuda.Stream()
    main_s = torch.cuda.current_stream()

    def decode48(stream):
        for layer in range(48):
            pool.decode(layer, q, sl, page_table=pt, out=out, stream=stream)

    def resume_batch(sids, stream):
        pool.resume(sids, stream=stream)
        pool.evict(sids, stream=stream)

    def timed(fn, stream, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(n):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    k = 0
    for _ in range(warmup):
        resume_batch(picks[k], main_s)
        k += 1
        decode48(main_s)
    torch.cuda.synchronize()
    decode_ms = timed(lambda i: decode48(main_s), main_s, steps)
    # resume alone: kernel time from the profiling hook, host time of the call
    kv.kv_pool_set_profiling(pool.handle, True)
    kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
    payload, host_s = 0, 0.0
    for i in range(steps):
        sids = picks[k]
        k += 1
        for sid in sids:
            payload += synth.pages_for(pool.info(sid)[1]) * pool.page_bytes
        torch.cuda.synchronize()  # the call's own host cost, not a wait for a staging slot
        t0 = time.perf_counter()
        pool.resume(sids, stream=main_s)
        host_s += time.perf_counter() - t0
        pool.evict(sids, stream=main_s)
    torch.cuda.synchronize()
    n_copy, copy_ms = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
    kv.kv_pool_set_profiling(pool.handle, False)
    # one session resumed alone: events around the call
    single = []
    for j in range(3):
        sid = picks[k][j]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(main_s)
        pool.resume([sid], stream=main_s)
        e1.record(main_s)
        torch.cuda.synchronize()
        single.append({"bytes": synth.pages_for(pool.info(sid)[1]) * pool.page_bytes,
                       "ms": round(e0.elapsed_time(e1), 3)})
        pool.evict([sid], stream=main_s)
    k += 1
    # both at once: resumes on a second stream while the 48 layers decode
    e = [torch.cuda.Event(enable_timing=True) for _ in range(2 * steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        side.wait_stream(main_s)
        resume_batch(picks[k], side)
        k += 1
        e[2 * i].record(main_s)
        decode48(main_s)
        e[2 * i + 1].record(main_s)
        main_s.wait_stream(side)
    torch.cuda.synchronize()
    both_ms = sum(e[2 * i].elapsed_time(e[2 * i + 1]) for i in range(steps)) / steps
    # resume bandwidth budget: a capped copy grid leaves decode more of the GPU
    budget = []
    for blocks in (1024, 256, 64):
        pool.set_copy_blocks(blocks)
        kv.kv_pool_set_profiling(pool.handle, True)
        kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        sids = picks[k % len(picks)]
        k += 1
        side.wait_stream(main_s)
        resume_batch(sids, side)
        ev[0].record(main_s)
        decode48(main_s)
        ev[1].record(main_s)
        main_s.wait_stream(side)
        torch.cuda.synchronize()
        n_b, ms_b = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
        kv.kv_pool_set_profiling(pool.handle, False)
        budget.append({"copy_blocks": blocks, "resume_ms_per_session": round(ms_b / len(sids), 3),
                       "decode48_ms_with_concurrent_resume": round(ev[0].elapsed_time(ev[1]), 3)})
    pool.set_copy_blocks(0)
    # the same pair on streams confined to disjoint CUs: the copy stream gets
    # `copy_slots` CUs of every XCD, the decode stream the others
    from paper_2609_25782_amd.pool import split_streams
    cu_split = []
    for copy_slots in (8, 4, 2):
        dec_s, cpy_s = split_streams(copy_slots)
        torch.cuda.synchronize()
        decode48(dec_s.stream)
        torch.cuda.synchronize()
        dec_alone = timed(lambda i: decode48(dec_s.stream), dec_s.stream, 2)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        sids = picks[k % len(picks)]
        k += 1
        ev[0].record(cpy_s.stream)
        resume_batch(sids, cpy_s.stream)
        ev[1].record(cpy_s.stream)
        torch.cuda.synchronize()
        sids = picks[k % len(picks)]
        k += 1
        ev[2].record(cpy_s.stream)
        resume_batch(sids, cpy_s.stream)
        ev[3].record(cpy_s.stream)
        ev[4].record(dec_s.stream)
        decode48(dec_s.stream)
        ev[5].record(dec_s.stream)
        torch.cuda.synchronize()
        both_split = ev[4].elapsed_time(ev[5])
        cu_split.append({"copy_cus": cpy_s.cus, "decode_cus": dec_s.cus,
                         "decode48_ms_alone": round(dec_alone, 3),
                         "resume_evict_ms_per_session_alone": round(ev[0].elapsed_time(ev[1]) / len(sids), 3),
                         "decode48_ms_with_concurrent_resume": round(both_split, 3),
                         "resume_evict_ms_per_session_beside": round(ev[2].elapsed_time(ev[3]) / len(sids), 3),
                         "tbt_impact": round(both_split / decode_ms, 3)})
        log("CU-split streams: %s" % json.dumps(cu_split[-1]))
        dec_s.close()
        cpy_s.close()
    # lazy resume: no copy when the sessions resume (their pages are read in
    # place from the cold tier), then promotion under a per-step page budget on a
    # second stream while the 48 layers decode; versus the eager resume above
    pool.set_spill(True)
    lazy = {"budgets": []}
    for per_step in (256, 1024, 4096):
        sids = picks[k % len(picks)]
        k += 1
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pool.resume_lazy(sids, stream=main_s)
        lazy["host_ms_per_call"] = round(1e3 * (time.perf_counter() - t0), 3)
        steps_needed, dec_ms, moved = 0, [], 0
        while True:
            side.wait_stream(main_s)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            n = pool.promote(per_step, stream=side)
            ev[0].record(main_s)
            decode48(main_s)
            ev[1].record(main_s)
            main_s.wait_stream(side)
            torch.cuda.synchronize()
            moved += n
            if n == 0:
                break
            steps_needed += 1
            dec_ms.append(ev[0].elapsed_time(ev[1]))
        lazy["budgets"].append({"pages_per_step": per_step,
                                "gb_per_step": round(per_step * pool.page_bytes / 1e9, 2),
                                "decode48_ms_while_promoting": round(float(np.mean(dec_ms)), 3),
                                "steps_to_promote": steps_needed, "pages_promoted": moved})
        log("lazy resume: %s" % json.dumps(lazy["budgets"][-1]))
        pool.evict(sids, stream=main_s)
    # the largest budget again with the promotion confined to 16 CUs and the
    # decode on the other 240 (disjoint CU sets, as for the eager resume)
    dec_s, cpy_s = split_streams(2)
    sids = picks[k % len(picks)]
    k += 1
    torch.cuda.synchronize()
    pool.resume_lazy(sids, stream=dec_s.stream)
    steps_needed, dec_ms, moved = 0, [], 0
    while True:
        cpy_s.stream.wait_stream(dec_s.stream)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        n = pool.promote(4096, stream=cpy_s.stream)
        ev[0].record(dec_s.stream)
        decode48(dec_s.stream)
        ev[1].record(dec_s.stream)
        dec_s.stream.wait_stream(cpy_s.stream)
        torch.cuda.synchronize()
        moved += n
        if n == 0:
            break
        steps_needed += 1
        dec_ms.append(ev[0].elapsed_time(ev[1]))
    lazy["cu_split_16_copy_cus"] = {"pages_per_step": 4096, "decode48_ms_while_promoting": round(float(np.mean(dec_ms)), 3),
                                    "steps_to_promote": steps_needed, "pages_promoted": moved}
    log("lazy resume, promotion on 16 CUs: %s" % json.dumps(lazy["cu_split_16_copy_cus"]))
    pool.evict(sids, stream=dec_s.stream)
    torch.cuda.synchronize()
    dec_s.close()
    cpy_s.close()
    pool.set_spill(False)
    torch.cuda.synchronize()
    # partial residency: sessions paused with all pages resident, a fraction of
    # their pages evicted page by page (LRU; clean, so no cold writes), resumed
    partial = []
    for j, frac in enumerate((0.25, 0.5, 0.75)):
        sids = picks[k % len(picks)]
        k += 1
        pool.resume(sids, stream=main_s)
        for sid in sids:
            pool.pause(sid)
        n_pages = sum(synth.pages_for(pool.info(sid)[1]) for sid in sids)
        pool.evict_pages(int(frac * n_pages), stream=main_s)
        torch.cuda.synchronize()
        st0 = pool.stats()
        kv.kv_pool_set_profiling(pool.handle, True)
        kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
        pool.resume(sids, stream=main_s)
        n_k, ms_k = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
        kv.kv_pool_set_profiling(pool.handle, False)
        st1 = pool.stats()
        hit = (st1["resume_pages_resident"] - st0["resume_pages_resident"]) / \
            (st1["resume_pages_total"] - st0["resume_pages_total"])
        partial.append({"evicted_fraction": frac, "hit_rate": round(hit, 4),
                        "ms_per_session": round(ms_k / len(sids), 4)})
        pool.evict(sids, stream=main_s)
    torch.cuda.synchronize()
    pool.close()
    del pool
    torch.cuda.empty_cache()
    per_session_ms = copy_ms / (8 * steps)
    gbs = 2 * payload / (copy_ms / 1e3) / 1e9
    return {
        "workload": "48 layers, 32q/4kv heads, d=128, bf16, 1.5 MiB pages; 1024 paused sessions "
                    "U[32768,131072] over %d physical cold pages; 8 resumed per step" % w.cold_pages,
        "ms_per_session": round(per_session_ms, 4),
        "mean_session_bytes": int(payload / (8 * steps)),
        "copy_GBps": round(gbs, 1),
        "frac_of_copy_roofline": round(gbs / HBM_PEAK_GBS, 4),
        "host_ms_per_call": round(1e3 * host_s / steps, 3),
        "single_session": single,
        "decode48_ms": round(decode_ms, 3),
        "decode48_ms_with_concurrent_resume": round(both_ms, 3),
        "tbt_impact": round(both_ms / decode_ms, 3),
        "decode48_GBps": round(48 * sum(decode_bytes(w.seq_lens, 32, 4, 128, 2)) / (decode_ms / 1e3) / 1e9, 1),
        "partial_residency": partial,
        "copy_budget": budget,
        "cu_split_streams": cu_split,
        "lazy_resume": lazy,
    }


def measure_host_tier(seed: int):
    """Resume from a cold tier in pinned host memory (read over PCIe by the copy
    kernel): 8 one-layer sessions of the benchmark's shape, and one 48-layer
    session of 32K tokens."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    out = {}
    rng = np.random.Generator(np.random.PCG64([seed, 13]))
    for name, layers, lens in (("layer_8_sessions", 1, rng.integers(8192, 32768, size=8, endpoint=True)),
                               ("step48_1_session", 48, np.array([32768]))):
        n_pages = int(sum(synth.pages_for(int(L)) for L in lens))
        pool = HotColdPool(layers, 4, 128, "bf16", n_pages, n_pages, len(lens), synth.pages_for(32768),
                           cold_location="host")
        sids = [pool.create_session(int(L)) for L in lens]
        pool.evict(sids)                       # first write of every page to the host tier
        torch.cuda.synchronize()
        times = []
        for rep in range(3):
            kv.kv_pool_set_profiling(pool.handle, True)
            kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
            pool.resume(sids)
            n, ms = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
            times.append(ms)
            pool.evict(sids)                   # clean: frees the hot pages, writes nothing
            torch.cuda.synchronize()
        kv.kv_pool_set_profiling(pool.handle, False)
        ms = min(times)
        payload = n_pages * pool.page_bytes
        out[name] = {"payload_bytes": payload, "resume_ms": round(ms, 3),
                     "ms_per_session": round(ms / len(lens), 3),
                     "pcie_GBps": round(payload / (ms / 1e3) / 1e9, 2)}
        pool.close()
        del pool
        torch.cuda.empty_cache()
    out["beside_decode"] = measure_host_overlap(seed)
    return out


def measure_host_overlap(seed: int):
    """A 48-layer session of 32K tokens (3.2 GB) resumed from the pinned-host
    tier on one stream while another stream decodes 32 active sessions of 8K
    tokens (48 layers, three steps), with the host-tier copies on the DMA
    engines (the default) and in the copy kernel."""
    import torch
    from paper_2609_25782_amd.pool import HotColdPool
    B, L, LR = 32, 8192, 32768
    pool = HotColdPool(48, 4, 128, "bf16", B * (L // 16) + LR // 16 + 64, LR // 16 + 8, B + 1, LR // 16,
                       cold_location="host")
    dev = pool.device
    for b in range(B):
        pool.create_session(L)
        pool.fill_synthetic(b, b, seed, 0.01)
    r = pool.create_session(LR)
    pool.evict([r])
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    q = torch.randn((B, 32, 128), generator=g, device=dev).to(torch.bfloat16)
    sl = torch.full((B,), L, dtype=torch.int32, device=dev)
    pt = pool.page_table[:B]
    out_t = torch.empty_like(q)
    dec_s, res_s = torch.cuda.Stream(), torch.cuda.Stream()

    def ev():
        return torch.cuda.Event(enable_timing=True)

    def decode_steps(n):
        for _ in range(n):
            for layer in range(48):
                pool.decode(layer, q, sl, page_table=pt, out=out_t, stream=dec_s)

    decode_steps(2)
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record(dec_s)
    decode_steps(3)
    e1.record(dec_s)
    torch.cuda.synchronize()
    res = {"decode48_ms_alone": round(e0.elapsed_time(e1) / 3, 3), "resume_bytes": (LR // 16) * pool.page_bytes}
    for name, kernel in (("dma", False), ("kernel", True)):
        pool.set_host_copy(kernel)
        r0, r1 = ev(), ev()
        r0.record(res_s)
        pool.resume([r], stream=res_s)
        r1.record(res_s)
        torch.cuda.synchronize()
        alone = r0.elapsed_time(r1)
        pool.evict([r], stream=res_s)
        torch.cuda.synchronize()
        r0, r1, d0, d1 = ev(), ev(), ev(), ev()
        r0.record(res_s)
        pool.resume([r], stream=res_s)
        r1.record(res_s)
        d0.record(dec_s)
        decode_steps(3)
        d1.record(dec_s)
        torch.cuda.synchronize()
        res[name] = {"resume_ms_alone": round(alone, 2), "resume_ms_beside": round(r0.elapsed_time(r1), 2),
                     "decode48_ms_beside": round(d0.elapsed_time(d1) / 3, 3)}
        pool.evict([r], stream=res_s)
        torch.cuda.synchronize()
    pool.set_host_copy(False)
    pool.close()
    torch.cuda.empty_cache()
    return res


def measure_agentic_replay(seed: int, plateau_s: float = 20.0, paper_node: bool = False):
    """The replay driver over a device pool of the paper's shape (48 layers, 4 KV
    heads, 128, bf16, 1.5 MiB pages; 32 query heads), so LRU eviction,
    write-back and partial resumes run on real pages.  Default: N_a = 32
    sessions decoding over 40 GiB of hot pages and 160 GiB of device-memory cold
    pages (heavy LRU pressure).  paper_node: the paper's node, N_a = 48 over 192
    GiB of HBM less 56.8 GiB of weights (135 GiB of hot pages), with 90 GiB of
    device-memory cold pages.  The warm-up only moves pages; the plateau also
    decodes all 48 layers of the running sessions every step.  Times, per step
    on the GPU: the decode, and the whole step (its admissions, resumes,
    evictions and page fills plus the decode)."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd import replay as rp
    from paper_2609_25782_amd.pool import HotColdPool

    n_active = 48 if paper_node else 32
    cfg = rp.ReplayConfig(n_active=n_active, weight_bytes=0.0, warmup_s=420.0, plateau_s=plateau_s,
                          sample_s=0.5, max_sessions=512 if paper_node else 320, seed=seed)
    page = cfg.page_bytes
    if paper_node:
        # the cold tier must take every page evicted during the warm-up (about
        # 115 GiB at this load); it gets what HBM has left, up to 125 GiB
        cfg.hbm_bytes, cfg.weight_bytes = 192.0 * 2 ** 30, 56.8 * 2 ** 30
        import gc
        gc.collect()
        torch.cuda.empty_cache()
        free = torch.cuda.mem_get_info()[0]
        cold = min(125 * 2 ** 30, free - cfg.num_hot_pages * page - 6 * 2 ** 30)
        if cold < 115 * 2 ** 30:
            return {"skipped": "needs %.0f GiB of free HBM for 135 GiB of hot and 115 GiB of cold pages, "
                               "%.0f GiB free" % ((cfg.num_hot_pages * page + 121 * 2 ** 30) / 2 ** 30,
                                                  free / 2 ** 30)}
        cfg.cold_bytes = float(cold // page * page)
    else:
        cfg.hbm_bytes = float(40 * 2 ** 30 // page * page)
        cfg.cold_bytes = float(160 * 2 ** 30 // page * page)
    hp = HotColdPool(48, 4, 128, "bf16", cfg.num_hot_pages, cfg.num_cold_pages, cfg.max_sessions,
                     cfg.stride)
    dp = rp.DevicePool(cfg, hp, seed, float(synth.value_multiplier(1.0)))
    q = torch.randn(cfg.n_active, 32, 128, generator=torch.Generator().manual_seed(seed))
    dec = rp.DeviceDecode(hp, q.to(torch.bfloat16).to(hp.device))
    r = rp.Replay(cfg, dp)
    prof = [kv.KV_KERNEL_DECODE_SPLIT, kv.KV_KERNEL_DECODE_COMBINE, kv.KV_KERNEL_PAGE_COPY,
            kv.KV_KERNEL_EVICT_COPY]

    profiled = 300              # the library's per-kernel profiling runs over these steps only
    kernels = {}

    class Decode:
        """The decode hook; the library's profiling brackets every launch with
        events, so it is on for the first plateau steps and off for the rest."""
        def step_begin(self):
            if len(dec.marks) in (0, profiled):
                torch.cuda.synchronize()
                kv.kv_pool_set_profiling(hp.handle, not dec.marks)
                for k, name in zip(prof, ("decode_split", "decode_combine", "resume_copy", "evict_copy")):
                    n, ms = kv.kv_pool_profile_read(hp.handle, k)
                    if dec.marks:
                        kernels[name] = {"launches": n, "ms_per_step": round(ms / profiled, 4)}
            dec.step_begin()

        def __call__(self, lengths):
            dec(lengths)

    t0 = time.perf_counter()
    summary = r.run(Decode())
    wall = time.perf_counter() - t0
    t = {k: v[profiled:] for k, v in dec.timings().items()}
    token_bytes = cfg.token_bytes
    kv_bytes = t["tokens"].astype(np.float64) * token_bytes
    out = {
        "config": ("48 layers x 4 KV heads x 128 bf16 (1.5 MiB pages), 32 query heads, N_a=48, the paper's "
                   "node: 192 GiB HBM less 56.8 GiB weights = %.1f GiB hot, cold %.0f GiB device memory, "
                   "synthetic trajectories, TBT model %.1f ms" % (cfg.num_hot_pages * page / 2 ** 30,
                                                                   cfg.num_cold_pages * page / 2 ** 30,
                                                                   1e3 * cfg.step_s))
        if paper_node else
                  "48 layers x 4 KV heads x 128 bf16 (1.5 MiB pages), 32 query heads, N_a=32, "
                  "hot 40 GiB, cold 160 GiB device memory, synthetic trajectories",
        "plateau_steps": int(len(t["step_ms"]) + profiled),
        "timed_steps": int(len(t["step_ms"])),
        "mean_batch": round(float(t["batch"].mean()), 2),
        "kv_read_per_step_gib": round(float(kv_bytes.mean()) / 2 ** 30, 2),
        "decode_ms": {"mean": round(float(t["decode_ms"].mean()), 3),
                      "p50": round(float(np.percentile(t["decode_ms"], 50)), 3),
                      "p99": round(float(np.percentile(t["decode_ms"], 99)), 3)},
        "step_ms": {"mean": round(float(t["step_ms"].mean()), 3),
                    "p50": round(float(np.percentile(t["step_ms"], 50)), 3),
                    "p99": round(float(np.percentile(t["step_ms"], 99)), 3)},
        "decode_GBps": round(float(kv_bytes.sum()) / (float(t["decode_ms"].sum()) / 1e3) / 1e9, 1),
        "kernels_first_%d_steps" % profiled: kernels,
        "replay": {k: summary[k] for k in ("resume_hit_rate", "resumes_per_s", "resume_miss_mib",
                                           "sessions_resident", "kv_per_resident_session_gib",
                                           "preemptions", "refused_admissions", "plateau_counts")},
        "wall_s": round(wall, 1),
    }
    r.close()
    hp.close()
    del r, hp, dp, dec, Decode             # the replay holds the device pool's buffers
    torch.cuda.empty_cache()
    return out


def _pct(xs):
    xs = np.asarray(xs, dtype=np.float64)
    return {"median": round(float(np.median(xs)), 3), "p10": round(float(np.percentile(xs, 10)), 3),
            "p90": round(float(np.percentile(xs, 90)), 3)}


def measure_configs(seed: int, steps: int = 10, warmup: int = 3, only=None):
    """Decode throughput on the other workloads: the tiny one (launch-bound), the
    48-layer step (B=64, lognormal lengths, all 48 layers per step, ~170 GB) and
    the skewed one (B=128, power-law lengths up to 256K, one layer timed, also
    scaled to 48).  HIP events around each decode call (or each 48-layer step);
    median, p10, p90.  Also the same run's device-to-device copy bandwidth, as
    context for the 8 TB/s peak."""
    import torch
    import synth
    from paper_2609_25782_amd.pool import HotColdPool
    out = {}
    dev = torch.device("cuda", 0)
    for name, make in (("tiny", synth.config_tiny), ("step48", synth.config_step48),
                       ("skewed", synth.config_skewed)):
        if only and name not in only:
            continue
        w = make(seed)
        pool = HotColdPool(w.num_layers, w.num_kv_heads, w.head_dim, w.dtype, w.hot_pages, 0, w.batch,
                           max(synth.pages_for(int(w.seq_lens.max())), 1))
        mult = float(synth.value_multiplier(w.value_scale))
        for b in range(w.batch):
            pool.create_session(int(w.seq_lens[b]), [int(p) for p in w.placement[b]])
            pool.fill_synthetic(b, b, w.seed, mult)
        q_np = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, w.dtype)
        if w.dtype == "bf16":
            q = torch.from_numpy(q_np.view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            q = torch.from_numpy(np.ascontiguousarray(q_np, dtype=np.float32)).to(dev)
        seq = torch.from_numpy(w.seq_lens.copy()).to(dev)
        pt = pool.page_table[:w.batch]
        o = torch.empty_like(q)
        layers = list(range(w.num_layers))
        times = []
        for it in range(warmup + steps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for layer in layers:
                pool.decode(layer, q, seq, page_table=pt, out=o)
            e1.record()
            torch.cuda.synchronize()
            if it >= warmup:
                times.append(1e3 * e0.elapsed_time(e1))
        elt = 2 if w.dtype == "bf16" else 4
        nbytes = len(layers) * sum(decode_bytes(w.seq_lens, w.num_q_heads, w.num_kv_heads, w.head_dim, elt))
        med = float(np.median(times))
        out[name] = {"workload": w.name, "batch": w.batch, "layers": len(layers),
                     "tokens": int(w.seq_lens.sum()), "bytes_per_call": nbytes,
                     "us_per_call": _pct(times), "GBps": round(nbytes / (med * 1e-6) / 1e9, 1),
                     "pct_of_peak": round(100.0 * nbytes / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 2)}
        if name == "skewed":
            out[name]["scaled_to_48_layers_ms"] = round(48 * med / 1e3, 3)
        log("configs: %s %s" % (name, json.dumps(out[name])))
        pool.close()
        del pool
        torch.cuda.empty_cache()
    if only:
        return out
    out["combine_scaling"] = measure_combine_scaling(seed)
    out["graph_step48"] = measure_graph(seed)
    out["append"] = measure_append(seed)
    log("append: %s" % json.dumps(out["append"]))
    a = torch.empty(2 ** 31, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    times = []
    for it in range(8):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        if it >= 2:
            times.append(e0.elapsed_time(e1))
    dtod = 2 * a.numel() / (float(np.median(times)) / 1e3) / 1e9
    del b
    x = a.view(torch.bfloat16)
    times = []
    for it in range(8):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.sum(x, dtype=torch.float32)
        e1.record()
        torch.cuda.synchronize()
        if it >= 2:
            times.append(e0.elapsed_time(e1))
    out["context"] = {"dtod_copy_GBps": round(dtod, 1),
                      "torch_sum_read_GBps": round(a.numel() / (float(np.median(times)) / 1e3) / 1e9, 1),
                      "note": "2 GiB device-to-device copy (torch; read + write bytes) and a torch sum "
                              "over the same 2 GiB (read bytes), same run; the library's own streaming-read "
                              "ceiling is roofline.measured_read_ceiling"}
    del a, x
    torch.cuda.empty_cache()
    return out


def measure_combine_scaling(seed: int, steps: int = 10, warmup: int = 3):
    """Split and combine kernel times (the library's profiling hook) for one
    layer at batches of 128, 1,024 and 8,192 short sessions (512 tokens each):
    the combine reads each row's page prefix from the split kernel instead of
    every block rescanning all lengths, so its cost follows the partials it
    merges, not the batch squared."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    rows = []
    L = 512
    for B in (128, 1024, 8192):
        pool = HotColdPool(1, 4, 128, "bf16", B * synth.pages_for(L), 0, B, synth.pages_for(L))
        mult = float(synth.value_multiplier(1.0 / math.sqrt(128)))
        for b in range(B):
            pool.create_session(L)
        for b in range(B):
            pool.fill_synthetic(b, b, seed, mult)
        q = torch.randn(B, 32, 128, generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16).cuda()
        sl = torch.full((B,), L, dtype=torch.int32, device="cuda")
        pt = pool.page_table[:B]
        out_t = torch.empty_like(q)
        for _ in range(warmup):
            pool.decode(0, q, sl, page_table=pt, out=out_t)
        torch.cuda.synchronize()
        kv.kv_pool_set_profiling(pool.handle, True)
        for k in range(kv.KV_KERNEL_COUNT):
            kv.kv_pool_profile_read(pool.handle, k)
        for _ in range(steps):
            pool.decode(0, q, sl, page_table=pt, out=out_t)
        torch.cuda.synchronize()
        n1, ms1 = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_DECODE_SPLIT)
        n2, ms2 = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_DECODE_COMBINE)
        kv.kv_pool_set_profiling(pool.handle, False)
        nbytes = sum(decode_bytes([L] * B, 32, 4, 128, 2))
        rows.append({"batch": B, "seq_len": L, "split_us": round(1e3 * ms1 / n1, 2),
                     "combine_us": round(1e3 * ms2 / n2, 2),
                     "GBps_kernels": round(nbytes / ((ms1 / n1 + ms2 / n2) / 1e3) / 1e9, 1)})
        log("combine scaling: %s" % json.dumps(rows[-1]))
        pool.close()
        del pool
        torch.cuda.empty_cache()
    return rows


def measure_evict(seed: int, reps: int = 3):
    """Write-on-evict at 48 layers (data path 4): 8 sessions of 8K-32K tokens
    whose pages have no cold copy are evicted in one call (every page copied hot
    -> cold), resumed, refilled (which drops the cold copies again), and so on.
    Also the eviction of the same sessions right after a resume, when every
    page still has its cold copy: no page is written."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    rng = np.random.Generator(np.random.PCG64([seed, 13]))
    lens = [int(x) for x in rng.integers(8192, 32768, size=8, endpoint=True)]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = HotColdPool(48, 4, 128, "bf16", n_pages + 8, n_pages + 8, 8, synth.pages_for(32768))
    mult = float(synth.value_multiplier(1.0 / math.sqrt(128)))
    sids = [pool.create_session(L) for L in lens]
    payload = n_pages * pool.page_bytes
    dirty, clean = [], []
    for r in range(reps + 1):
        for j, sid in enumerate(sids):
            pool.fill_synthetic(sid, j, seed, mult)
        torch.cuda.synchronize()
        kv.kv_pool_set_profiling(pool.handle, True)
        kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_EVICT_COPY)
        pool.evict(sids)
        n, ms = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_EVICT_COPY)
        pool.resume(sids)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        pool.evict(sids)                    # clean: the cold copies are still valid
        e1.record()
        torch.cuda.synchronize()
        kv.kv_pool_set_profiling(pool.handle, False)
        pool.resume(sids)
        if r > 0:                           # the first round warms up
            dirty.append(ms)
            clean.append(e0.elapsed_time(e1))
    st = pool.stats()
    pool.close()
    torch.cuda.empty_cache()
    d = float(np.median(dirty))
    return {"sessions": 8, "layers": 48, "payload_bytes": payload,
            "dirty_evict_ms": round(d, 3), "dirty_ms_per_session": round(d / 8, 4),
            "copy_GBps": round(2 * payload / (d / 1e3) / 1e9, 1),
            "frac_of_copy_roofline": round(2 * payload / (d / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
            "clean_evict_ms": round(float(np.median(clean)), 4),
            "cold_writes_total": st["pages_to_cold"]}


def measure_append(seed: int, steps: int = 20, warmup: int = 3):
    """Data path 3 at the paper's shape (48 layers, 4 KV heads, 128, bf16): a
    decode step appends one token to each of 32 sessions in every layer.  Times
    the batched append (kv_append_tokens, one call per layer) against one
    kv_write_tokens call per session and layer, and an 8,192-token prompt
    written into one session (kv_write_tokens, one call per layer)."""
    import torch
    from paper_2609_25782_amd.pool import HotColdPool
    B, NL, L0 = 32, 48, 1024
    prompt = 8192
    pages = B * ((L0 + steps + warmup + 16) // 16 + 1) + (prompt // 16 + 2)
    pool = HotColdPool(NL, 4, 128, "bf16", pages, 0, B + 1, (L0 + steps + warmup + prompt) // 16 + 4)
    dev = pool.device
    sids = [pool.create_session(L0) for _ in range(B)]
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    k = torch.randn((B, 4, 128), generator=g, device=dev).to(torch.bfloat16)
    v = torch.randn((B, 4, 128), generator=g, device=dev).to(torch.bfloat16)
    lens = [L0] * B

    def step(batched):
        for i, sid in enumerate(sids):
            lens[i] += 1
            pool.extend(sid, lens[i])
        for layer in range(NL):
            if batched:
                pool.append_tokens(layer, sids, [n - 1 for n in lens], k, v)
            else:
                for i, sid in enumerate(sids):
                    pool.write_tokens(sid, layer, lens[i] - 1, k[i:i + 1], v[i:i + 1])

    out = {"sessions": B, "layers": NL}
    for batched in (True, False):
        for _ in range(warmup):
            step(batched)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record()
        for _ in range(steps):
            step(batched)
        e1.record()
        host = time.perf_counter() - t0
        torch.cuda.synchronize()
        name = "batched_append" if batched else "per_session_write"
        out[name] = {"ms_per_step": round(e0.elapsed_time(e1) / steps, 4),
                     "host_ms_per_step": round(1e3 * host / steps, 4),
                     "calls_per_step": NL if batched else NL * B}
    pool.close()
    torch.cuda.empty_cache()
    out.update(measure_prompt_write(seed))
    out["graph_step"] = measure_graph_append(seed)
    return out


def measure_prompt_write(seed: int, reps: int = 7):
    """Fresh KV of a whole prompt (data path 3): 8,192 tokens into one session
    at the paper's shape (48 layers, 4 KV heads, 128, bf16), one
    kv_write_tokens call per layer, and one kv_write_tokens_layers call for all
    48.  Algorithmic bytes: the K and V written, and the same again read."""
    import torch
    from paper_2609_25782_amd.pool import HotColdPool
    NL, prompt = 48, 8192
    pool = HotColdPool(NL, 4, 128, "bf16", prompt // 16 + 2, 0, 1, prompt // 16 + 1)
    dev = pool.device
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    out = {}
    sid = pool.create_session(prompt)
    kp = torch.randn((NL, prompt, 4, 128), generator=g, device=dev).to(torch.bfloat16)
    vp = torch.randn((NL, prompt, 4, 128), generator=g, device=dev).to(torch.bfloat16)
    nbytes = 2 * prompt * 4 * 128 * 2 * NL          # K and V written (the same again read)

    def per_layer():
        for layer in range(NL):
            pool.write_tokens(sid, layer, 0, kp[layer], vp[layer])

    def all_layers():
        pool.write_tokens_layers(sid, 0, 0, kp, vp)

    for name, fn in (("prompt_write", per_layer), ("prompt_write_one_call", all_layers)):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        times = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        ms = float(np.median(times))
        out[name] = {"tokens": prompt, "layers": NL, "calls": NL if fn is per_layer else 1, "ms": round(ms, 4),
                     "bytes_written": nbytes, "GBps_written": round(nbytes / (ms / 1e3) / 1e9, 1),
                     "GBps_read_write": round(2 * nbytes / (ms / 1e3) / 1e9, 1),
                     "frac_of_hbm_peak": round(2 * nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
        log("append: %s %s" % (name, json.dumps(out[name])))
    pool.close()
    del kp, vp
    torch.cuda.empty_cache()
    return out


def measure_graph_append(seed: int, steps: int = 20, warmup: int = 3):
    """A serving step captured in one HIP graph at the paper's shape (48 layers,
    32 sessions of 8K tokens): the batch-table gather, then for every layer the
    step's token appended and the decode, with the append fused into the decode
    launch (paged_decode_attention_append) or as a launch of its own through the
    table (kv_append_tokens_table).  Against the same graph without appends this
    gives the append's cost inside a captured step.  The host extends every
    session by one token before each replay."""
    import torch
    import synth
    from paper_2609_25782_amd.pool import HotColdPool
    B, NL, L0 = 32, 48, 8192
    total = 4 * (warmup + steps) + 2          # tokens appended over all graphs' replays
    pool = HotColdPool(NL, 4, 128, "bf16", B * (synth.pages_for(L0 + total) + 1), 0, B,
                       synth.pages_for(L0 + total) + 1)
    dev = pool.device
    mult = float(synth.value_multiplier(1.0 / math.sqrt(128)))
    for b in range(B):
        pool.create_session(L0)
        pool.fill_synthetic(b, b, seed, mult)
    q = torch.randn(B, 32, 128, generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16).to(dev)
    k_new = (0.05 * torch.randn(NL, B, 4, 128, generator=torch.Generator().manual_seed(seed + 1))).to(
        torch.bfloat16).to(dev)
    v_new = k_new.flip(0).contiguous()
    sid_t = torch.arange(B, dtype=torch.int32, device=dev)
    rows_t = torch.arange(B, dtype=torch.int32, device=dev)
    pos_t = torch.zeros(B, dtype=torch.int32, device=dev)
    sl_t = torch.zeros(B, dtype=torch.int32, device=dev)
    table = torch.empty((B, pool.stride), dtype=torch.int32, device=dev)
    outs = [torch.empty_like(q) for _ in range(NL)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    lens = [L0] * B

    def body(append, decode):
        pool.gather_table(sid_t, out=table, stream=s)
        for l in range(NL):
            if append == "table":
                pool.append_tokens_table(l, table, rows_t, pos_t, k_new[l:l + 1], v_new[l:l + 1], stream=s)
            if decode:
                pool.decode(l, q, sl_t, page_table=table, out=outs[l], stream=s,
                            k_new=k_new[l] if append == "fused" else None,
                            v_new=v_new[l] if append == "fused" else None)

    def advance():
        for b in range(B):
            lens[b] += 1
            pool.extend(b, lens[b], stream=s)
        pos_t.copy_(torch.tensor([n - 1 for n in lens], dtype=torch.int32), non_blocking=False)
        sl_t.copy_(torch.tensor(lens, dtype=torch.int32), non_blocking=False)

    graphs = {}
    with torch.cuda.stream(s):
        advance()
        body("table", True)                     # eager once: the workspace exists before capture
        torch.cuda.synchronize()
        for name, a, d in (("table_append_and_decode", "table", True), ("fused_append_decode", "fused", True),
                           ("decode_only", None, True), ("table_append_only", "table", False)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                body(a, d)
            graphs[name] = g
        res = {}
        for name, g in graphs.items():
            times = []
            for it in range(warmup + steps):
                if name != "decode_only":
                    advance()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                g.replay()
                e1.record(s)
                torch.cuda.synchronize()
                if it >= warmup:
                    times.append(e0.elapsed_time(e1))
            res[name] = float(np.median(times))
    out = {"sessions": B, "layers": NL, "context": L0,
           "step_ms": {k: round(v, 4) for k, v in res.items()},
           "append_ms_per_step_in_graph": round(res["fused_append_decode"] - res["decode_only"], 4),
           "table_append_ms_per_step_in_graph": round(res["table_append_and_decode"] - res["decode_only"], 4)}
    log("append: graph step %s" % json.dumps(out))
    del graphs
    pool.close()
    torch.cuda.empty_cache()
    return out


def measure_read_ceiling(nbytes: int = 16 * 2 ** 30):
    """The streaming-read rate this GPU reaches: the library's read probe
    (kv_read_probe, the decode kernel's 16-byte nontemporal loads, 8 in flight
    per thread, 32 KiB contiguous per block and step) over a 16 GiB buffer,
    best median over a few grid sizes."""
    import torch
    from paper_2609_25782_amd import hotcold_kv as kv
    dev = torch.device("cuda", 0)
    buf = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    out = torch.empty(1 << 16, dtype=torch.int32, device=dev)
    best = None
    for blocks in (2048, 4096, 8192, 16384, 65536):
        times = []
        for it in range(7):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            kv.kv_read_probe(buf.data_ptr(), nbytes, out.data_ptr(), blocks,
                             torch.cuda.current_stream().cuda_stream)
            e1.record()
            torch.cuda.synchronize()
            if it >= 2:
                times.append(e0.elapsed_time(e1))
        gbps = nbytes / (float(np.median(times)) / 1e3) / 1e9
        if best is None or gbps > best["GBps"]:
            best = {"GBps": round(gbps, 1), "blocks": blocks}
    del buf, out
    torch.cuda.empty_cache()
    best.update({"bytes": nbytes, "method": "kv_read_probe: 16-byte nontemporal loads, contiguous 32 KiB "
                                            "chunks per block, events around one launch, best median over "
                                            "grid sizes"})
    return best


def measure_graph(seed: int, steps: int = 10, warmup: int = 3):
    """A 48-layer decode step launched eagerly (96 launches from the host) and as
    a captured HIP graph replayed, for a small batch (launch-bound) and a large
    one (bandwidth-bound).  HIP events around each step; medians."""
    import torch
    import synth
    from paper_2609_25782_amd.pool import HotColdPool
    rows = []
    for B, L in ((8, 2048), (8, 8192), (32, 8192)):
        pages = B * synth.pages_for(L)
        pool = HotColdPool(48, 4, 128, "bf16", pages, 0, B, synth.pages_for(L))
        for b in range(B):
            pool.create_session(L)
            pool.fill_synthetic(b, b, seed, float(synth.value_multiplier(1.0 / math.sqrt(128))))
        q = torch.randn(B, 32, 128, generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16).cuda()
        sl = torch.full((B,), L, dtype=torch.int32, device="cuda")
        pt = pool.page_table[:B]
        outs = [torch.empty_like(q) for _ in range(48)]
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())

        def step():
            for layer in range(48):
                pool.decode(layer, q, sl, page_table=pt, out=outs[layer], stream=s)

        with torch.cuda.stream(s):
            step()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            step()
        res = {}
        for mode, fn in (("eager", step), ("graph", g.replay)):
            times = []
            for it in range(warmup + steps):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                with torch.cuda.stream(s):
                    e0.record(s)
                    fn()
                    e1.record(s)
                torch.cuda.synchronize()
                if it >= warmup:
                    times.append(e0.elapsed_time(e1))
            res[mode] = float(np.median(times))
        nbytes = 48 * sum(decode_bytes([L] * B, 32, 4, 128, 2))
        rows.append({"batch": B, "seq_len": L, "eager_ms": round(res["eager"], 3),
                     "graph_ms": round(res["graph"], 3),
                     "graph_GBps": round(nbytes / (res["graph"] / 1e3) / 1e9, 1),
                     "speedup": round(res["eager"] / res["graph"], 3)})
        log("graph: %s" % json.dumps(rows[-1]))
        del g
        pool.close()
        del pool
        torch.cuda.empty_cache()
    return rows


def measure_spill(seed: int, steps: int = 6, warmup: int = 2):
    """Decode from the cold tier: 32 active sessions of 4,096 tokens at the
    paper's shape (48 layers, 4 KV heads, 128, bf16; 32 query heads), 12 GiB of
    KV, with a fraction of their pages spilled to the cold tier (device memory or
    pinned host memory over PCIe).  Each step decodes all 48 layers, reading the
    spilled pages in place ("direct") or through the staging buffer that a
    second stream fills one layer ahead ("prefetch").  Spilling everything to
    the host tier is the paper's configuration without tiering: the hot set
    read over PCIe every step."""
    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool

    n_s, L, hq = 32, 4096, 32
    pages = n_s * synth.pages_for(L)
    mult = float(synth.value_multiplier(1.0 / math.sqrt(128)))
    q = torch.randn(n_s, hq, 128, generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16).cuda()
    sl = torch.full((n_s,), L, dtype=torch.int32, device="cuda")
    kv_bytes = 48 * sum(decode_bytes([L] * n_s, hq, 4, 128, 2))
    rows = []
    copy_stream = torch.cuda.Stream()
    # the gather on 8 CUs (one per XCD) and the decode on the other 248, so the
    # gather's waves, which wait on PCIe, never share a CU with the decode
    from paper_2609_25782_amd.pool import split_streams
    dec_cu, copy_cu = split_streams(1)
    # The host tier's small fractions look for the prefetch crossover: one
    # layer's gather of f x 269 MB over PCIe (about f x 4.8 ms) fits under one
    # layer's decode (about 55 us) only for f below about 1%.
    for tier in ("device", "host"):
        for frac in ((0.0, 0.25, 1.0) if tier == "device" else (0.0025, 0.005, 0.01, 0.02, 0.04, 0.25, 1.0)):
            hot = pages - int(round(frac * pages))
            pool = HotColdPool(48, 4, 128, "bf16", max(hot, 1), pages + 16, n_s, synth.pages_for(L) + 1,
                               cold_location=tier)
            kv.kv_pool_set_spill(pool.handle, True)
            for b in range(n_s):
                pool.create_session(L)
                pool.fill_synthetic(b, b, seed, mult)
            spilled = pool.stats()["spilled_pages"]
            sids = torch.arange(n_s, dtype=torch.int32, device="cuda")
            direct = pool.gather_table(sids)
            out = torch.empty_like(q)
            staging = table = None
            if spilled:
                staging = torch.empty(2 * spilled * pool.page_bytes // 48, dtype=torch.uint8, device="cuda")
                kv.kv_pool_set_staging(pool.handle, staging.data_ptr(), staging.numel())
                table = torch.empty((n_s, pool.stride), dtype=torch.int32, device="cuda")
                kv.paged_decode_stage(pool.handle, list(range(n_s)), table.data_ptr())
            torch.cuda.synchronize()
            for mode in (("direct", "prefetch", "prefetch_cu8") if spilled else ("hot", "hot_tiered_kernel")):
                # all pages hot: the plain kernel, then the tier-aware one (spill on)
                kv.kv_pool_set_spill(pool.handle, mode != "hot")
                pre = mode.startswith("prefetch")
                dec_stream = dec_cu.stream if mode == "prefetch_cu8" else torch.cuda.current_stream()
                cpy = copy_cu.stream if mode == "prefetch_cu8" else copy_stream
                times = []
                for it in range(warmup + steps):
                    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    t0.record(dec_stream)
                    if pre:
                        cpy.wait_event(t0)
                        kv.paged_decode_prefetch(pool.handle, 0, cpy.cuda_stream)
                    for layer in range(48):
                        if pre and layer + 1 < 48:
                            kv.paged_decode_prefetch(pool.handle, layer + 1, cpy.cuda_stream)
                        pool.decode(layer, q, sl, page_table=table if pre else direct, out=out,
                                    stream=dec_stream if mode == "prefetch_cu8" else None)
                    t1.record(dec_stream)
                    torch.cuda.synchronize()
                    if it >= warmup:
                        times.append(t0.elapsed_time(t1))
                ms = float(np.median(times))
                rows.append({"cold_tier": tier, "spilled_frac": round(spilled / pages, 3), "mode": mode,
                             "step_ms": round(ms, 3), "GBps": round(kv_bytes / (ms / 1e3) / 1e9, 1)})
                log("spill: %s" % json.dumps(rows[-1]))
            if spilled:
                kv.kv_pool_set_staging(pool.handle, 0, 0)
            pool.close()
            del pool, staging, table, direct
            torch.cuda.empty_cache()
    dec_cu.close()
    copy_cu.close()
    return {"config": "32 sessions x 4,096 tokens, 48 layers x 4 KV heads x 128 bf16, 32 query heads "
                      "(12 GiB of KV per step)", "kv_bytes_per_step": kv_bytes, "rows": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--resume-per-step", type=int, default=8)
    ap.add_argument("--batch", type=int, default=32, help="active sessions (the workload has 32)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--waves", type=int, default=0, help="override the decode wave count")
    ap.add_argument("--copy-blocks", type=int, default=0,
                    help="cap on the resume copy's persistent grid (0 = the library default)")
    ap.add_argument("--combine", choices=["fused", "separate"], default="separate",
                    help="merge split partials in the split kernel's last wave or in a second kernel")
    ap.add_argument("--compute", choices=["matrix", "vector"], default="matrix",
                    help="units the decode split kernel computes on: matrix cores, or bf16 dot2 on "
                         "the vector ALU")
    ap.add_argument("--cpu-budget", type=float, default=12.0,
                    help="seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--no-check", action="store_true", help="skip the sampled oracle check")
    ap.add_argument("--sections", default="resume48,host,replay,spill,configs",
                    help="measurements after the hot-path step, comma separated: resume48 (48-layer "
                         "resume mix, ~235 GB of HBM), host (pinned-host cold tier), replay (agentic "
                         "replay on a device pool), spill (decode from the cold tier), configs (the "
                         "tiny, 48-layer and skewed workloads); 'none' for none")
    ap.add_argument("--no-resume-mix", action="store_true", help="same as --sections none")
    ap.add_argument("--flush-mb", type=int, default=0,
                    help="write a scratch buffer of this many MiB before every timed step, so the "
                         "decode starts with the 256 MB Infinity Cache and the L2s holding other data")
    ap.add_argument("--full-json", default="", help="also write the full result (every sweep row) here")
    ap.add_argument("--only-config", default="", choices=["", "tiny", "step48", "skewed", "prompt_write", "evict48"],
                    help="profiling aid: time only this workload's decode (no hot-path step) and print "
                         "its figures")
    args = ap.parse_args()
    sections = set() if args.no_resume_mix else {x for x in args.sections.split(",") if x and x != "none"}
    unknown = sections - {"resume48", "host", "replay", "spill", "configs"}
    if unknown:
        ap.error("unknown sections: %s" % ", ".join(sorted(unknown)))

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(sharded by session, each GPU would own its own sessions and page tables).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    if args.only_config == "prompt_write":
        print(json.dumps(measure_prompt_write(args.seed, reps=args.steps)), flush=True)
        return
    if args.only_config == "evict48":
        print(json.dumps(measure_evict(args.seed, reps=args.steps)), flush=True)
        return
    if args.only_config:
        print(json.dumps(measure_configs(args.seed, steps=args.steps, warmup=args.warmup,
                                         only=[args.only_config])), flush=True)
        return
    w = synth.config_layer(args.seed, batch=args.batch)
    R = args.resume_per_step
    rng = np.random.Generator(np.random.PCG64([args.seed, 7]))
    paused_lens = rng.integers(8192, 32768, size=R, endpoint=True).astype(np.int32)
    paused_pages = int(sum(synth.pages_for(L) for L in paused_lens))
    active_pages = int(sum(synth.pages_for(L) for L in w.seq_lens))
    num_hot = w.hot_pages + paused_pages
    stride = max(synth.pages_for(32768), 1)
    log("workload %s: B=%d, %d tokens, %d active pages, %d resumed pages/step, hot pool %d pages"
        % (w.name, w.batch, int(w.seq_lens.sum()), active_pages, paused_pages, num_hot))

    pool = HotColdPool(1, w.num_kv_heads, w.head_dim, "bf16", num_hot, paused_pages,
                       w.batch + R, stride)
    mult = float(synth.value_multiplier(w.value_scale))
    # active sessions 0..B-1 at the workload's scattered pages
    for b in range(w.batch):
        sid = pool.create_session(int(w.seq_lens[b]), [int(p) for p in w.placement[b]])
        assert sid == b
        pool.fill_synthetic(sid, b, w.seed, mult)
    # paused sessions: written once, evicted (the one cold write each page gets)
    paused = []
    for j, L in enumerate(paused_lens):
        sid = pool.create_session(int(L))
        pool.fill_synthetic(sid, w.batch + j, w.seed, mult)
        paused.append(sid)
    pool.evict(paused)
    torch.cuda.synchronize()
    if args.waves:
        pool.set_waves(args.waves)
    pool.set_combine(args.combine == "fused")
    pool.set_compute(args.compute == "vector")
    if args.copy_blocks:
        kv.kv_pool_set_copy_blocks(pool.handle, args.copy_blocks)

    q = torch.from_numpy(synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim,
                                       w.value_scale, "bf16").view(np.int16)).to(dev).view(torch.bfloat16)
    seq = torch.from_numpy(w.seq_lens.copy()).to(dev)
    pt = pool.page_table[:w.batch]
    out = torch.empty_like(q)
    scale = 1.0 / math.sqrt(w.head_dim)

    def step():
        pool.resume(paused)
        pool.decode(0, q, seq, page_table=pt, scale=scale, out=out)
        pool.evict(paused)

    for i in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)

    # sampled parity check of this exact launch configuration
    check = None
    if not args.no_check:
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from helpers import Case, tolerance_check
        b = int(np.argmax(w.seq_lens))
        case = Case(1, w.num_q_heads, w.num_kv_heads, w.head_dim, "bf16", [int(w.seq_lens[b])],
                    seed=w.seed, value_scale=w.value_scale,
                    placement=[np.arange(synth.pages_for(int(w.seq_lens[b])), dtype=np.int32)])
        case.kv = [synth.session_kv(w.seed, b, int(w.seq_lens[b]), 0, w.num_kv_heads, w.head_dim,
                                    w.value_scale, "bf16")]
        case.q = synth.queries(w.seed + 1, w.batch, w.num_q_heads, w.head_dim, w.value_scale, "bf16")[b:b + 1]
        ref = case.oracle_out()
        got = out[b:b + 1].float().cpu().numpy().astype(np.float64)
        err, norm = tolerance_check(got, ref)
        check = {"session": b, "seq_len": int(w.seq_lens[b]), "max_abs_err": err, "normalised_err": norm}
        log("sampled oracle check: session %d max abs %.3g normalised %.3g" % (b, err, norm))

    # Timed region: K steps with the library's profiling off; HIP events on the
    # launch stream bracket the K steps and each decode call (split + combine,
    # the gap between them and the event packets: decode_call_us).
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]

    flush = torch.empty(args.flush_mb << 20, dtype=torch.uint8, device=dev) if args.flush_mb else None

    def timed_step(i):
        if flush is not None:
            flush.fill_(i & 0xFF)
        pool.resume(paused)
        ev[i][0].record()
        pool.decode(0, q, seq, page_table=pt, scale=scale, out=out)
        ev[i][1].record()
        pool.evict(paused)

    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(args.steps):
        timed_step(i)
    stop.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    call_ms = [a.elapsed_time(b) for a, b in ev]
    decode_ms = float(np.median(call_ms))
    # Per-kernel times (roofline, resume): K more steps with the profiling hook,
    # whose events bracket every launch on its stream.
    kv.kv_pool_set_profiling(pool.handle, True)
    for k in range(kv.KV_KERNEL_COUNT):
        kv.kv_pool_profile_read(pool.handle, k)
    torch.cuda.synchronize()
    for i in range(args.steps):
        step()
    torch.cuda.synchronize()
    n1, ms1 = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_DECODE_SPLIT)
    n2, ms2 = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_DECODE_COMBINE)
    n3, ms3 = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_PAGE_COPY)
    kv.kv_pool_set_profiling(pool.handle, False)
    assert n1 == args.steps and n3 == args.steps and n2 == (0 if args.combine == "fused" else args.steps), (n1, n2, n3)
    log("timed %d steps: %.3f ms/step, decode call %.1f us; profiled: split %.1f us, combine %.1f us, "
        "resume copy %.1f us" % (args.steps, total_ms / args.steps, 1e3 * decode_ms, 1e3 * ms1 / n1,
                                 1e3 * ms2 / max(n2, 1), 1e3 * ms3 / n3))

    # The same steps with the split's two products on the vector ALU instead of
    # the matrix cores (same work split, loads and merge): the measured case for
    # matrix cores.  Split-kernel time on the default grid and on 8 waves per CU
    # (two per SIMD, which the vector form's registers allow and which suits it
    # best); each output is compared with the matrix-core result of the same step.
    other = None
    if args.compute == "matrix" and args.combine == "separate" and not args.waves:
        ref_out = out.float().clone()
        cus = torch.cuda.get_device_properties(dev).multi_processor_count
        pool.set_compute(True)
        other = {"matrix_split_us": round(1e3 * ms1 / n1, 2), "matrix_waves": pool.waves()}
        for tag, nw in (("same_grid", 0), ("two_waves_per_simd", 8 * cus)):
            pool.set_waves(nw)
            for i in range(args.warmup):
                step()
            kv.kv_pool_set_profiling(pool.handle, True)
            for k in range(kv.KV_KERNEL_COUNT):
                kv.kv_pool_profile_read(pool.handle, k)
            for i in range(args.steps):
                step()
            torch.cuda.synchronize()
            nv, msv = kv.kv_pool_profile_read(pool.handle, kv.KV_KERNEL_DECODE_SPLIT)
            kv.kv_pool_set_profiling(pool.handle, False)
            diff = float((out.float() - ref_out).abs().max() / ref_out.abs().max())
            other[tag] = {"waves": pool.waves(), "split_us": round(1e3 * msv / nv, 2),
                          "time_vs_matrix": round((msv / nv) / (ms1 / n1), 4),
                          "max_normalised_diff_vs_matrix": diff}
            log("vector-ALU split, %d waves: %.1f us (matrix cores %.1f us), normalised difference %.3g"
                % (pool.waves(), 1e3 * msv / nv, 1e3 * ms1 / n1, diff))
        pool.set_compute(False)
        pool.set_waves(0)

    kvb, qo, ptb = decode_bytes(w.seq_lens, w.num_q_heads, w.num_kv_heads, w.head_dim, 2)
    dec_bytes = kvb + qo + ptb
    dec_s = (ms1 + ms2) / 1e3 / args.steps     # device time of the two decode kernels
    value = dec_bytes / (decode_ms / 1e3) / 1e9  # the median timed decode call
    # the split kernel's algorithmic bytes: with the fused merge it also writes the output
    k1_bytes = dec_bytes if args.combine == "fused" else split_kernel_bytes(
        w.seq_lens, w.num_q_heads, w.num_kv_heads, w.head_dim, 2)
    k1_s = ms1 / 1e3 / n1
    k1_gbs = k1_bytes / k1_s / 1e9
    payload = paused_pages * pool.page_bytes
    res_s = ms3 / 1e3 / n3
    res_gbs = 2 * payload / res_s / 1e9

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "qwen3-coder-30b-a3b attention layer: 32 active sessions, context U[8192,32768], "
                        "32q/4kv heads, d=128, bf16, 16-token pages scattered over the hot pool; "
                        "%d paused sessions resumed and evicted per step" % R,
            "batch": w.batch, "total_tokens": int(w.seq_lens.sum()), "num_q_heads": w.num_q_heads,
            "num_kv_heads": w.num_kv_heads, "head_dim": w.head_dim, "layers": 1, "page_tokens": 16,
            "hot_pages": num_hot, "decode_waves": pool.waves(), "combine": args.combine,
            "copy_blocks": args.copy_blocks,
            "compute": args.compute,
            "seed": args.seed,
        },
        "pct_of_peak": round(100.0 * value / HBM_PEAK_GBS, 2),
        "value_basis": "algorithmic bytes / median decode call of the timed pass (events around the call)",
        "decode_call_us": round(1e3 * decode_ms, 2),
        "decode_call_us_dist": _pct([1e3 * x for x in call_ms]),
        "decode_kernels_us": round(1e6 * dec_s, 2),
        "decode_kernels_GBps": round(dec_bytes / dec_s / 1e9, 2),
        "flush_mb_between_steps": args.flush_mb,
        "decode_bytes": dec_bytes,
        "resume": {
            "ms_per_session": round(1e3 * res_s / R, 5),
            "ms_per_batch": round(1e3 * res_s, 5),
            "sessions_per_batch": R,
            "payload_bytes": payload,
            "copy_GBps": round(res_gbs, 2),
            "frac_of_copy_roofline": round(res_gbs / HBM_PEAK_GBS, 4),
            "note": "copy roofline counts each payload byte read once and written once",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "decode_split_kernel",
            "achieved": round(k1_gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(k1_gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic() if args.combine == "separate" and args.compute == "matrix" else None,
            "bytes_per_launch": k1_bytes,
            "us_per_launch": round(1e6 * k1_s, 2),
        },
        "check": check,
        "split_on_vector_alu": other,
    }
    pool.close()
    del pool
    torch.cuda.empty_cache()
    ceiling = measure_read_ceiling()
    log("streaming-read ceiling (library read probe): %.0f GB/s" % ceiling["GBps"])
    result["roofline"]["measured_read_ceiling"] = ceiling
    result["roofline"]["frac_of_measured_read_ceiling"] = round(k1_gbs / ceiling["GBps"], 4)
    if "resume48" in sections:
        result["resume48"] = measure_resume_mix(args.seed, max(3, args.steps // 4), 1)
        log("resume mix: %s" % json.dumps(result["resume48"]))
        result["evict48"] = measure_evict(args.seed)
        log("write-on-evict: %s" % json.dumps(result["evict48"]))
    if "host" in sections:
        result["resume_host_tier"] = measure_host_tier(args.seed)
        log("host tier: %s" % json.dumps(result["resume_host_tier"]))
    if "replay" in sections:
        result["agentic_replay"] = measure_agentic_replay(args.seed)
        log("agentic replay: %s" % json.dumps(result["agentic_replay"]))
        result["agentic_replay_paper_node"] = measure_agentic_replay(args.seed, paper_node=True)
        log("agentic replay, paper's node: %s" % json.dumps(result["agentic_replay_paper_node"]))
    if "spill" in sections:
        result["spill_decode"] = measure_spill(args.seed)
    if "configs" in sections:
        result["configs"] = measure_configs(args.seed)
    if args.cpu_budget > 0:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_budget)
    if args.full_json:
        with open(args.full_json, "w") as f:
            json.dump(result, f, indent=1)
    line = json.dumps(compact(result))
    log("result line: %d bytes" % len(line))
    print(line, flush=True)


# Fields kept in the stdout line for the sections measured after the hot-path
# step (the rest is logged to stderr and written to --full-json).
_KEEP = {
    "resume48": ("ms_per_session", "mean_session_bytes", "copy_GBps", "frac_of_copy_roofline",
                 "host_ms_per_call", "decode48_ms", "decode48_ms_with_concurrent_resume", "tbt_impact",
                 "decode48_GBps"),
    "evict48": ("dirty_ms_per_session", "copy_GBps", "frac_of_copy_roofline", "clean_evict_ms"),
    "agentic_replay": ("kv_read_per_step_gib", "decode_GBps"),
    "agentic_replay_paper_node": ("kv_read_per_step_gib", "decode_GBps"),
}


def compact(result: dict) -> dict:
    """The stdout line: the hot-path fields in full, and for the other sections
    their headline numbers (the driver keeps only the tail of stdout)."""
    out = {k: v for k, v in result.items() if k not in (
        "resume48", "evict48", "resume_host_tier", "agentic_replay", "agentic_replay_paper_node",
        "spill_decode", "configs")}
    for sec, keys in _KEEP.items():
        if sec in result:
            out[sec] = {k: result[sec][k] for k in keys if k in result[sec]}
    if "resume48" in result:
        r = result["resume48"]
        out["resume48"]["single_session_ms"] = [x["ms"] for x in r.get("single_session", [])]
        out["resume48"]["cu_split_tbt_impact"] = {str(x["copy_cus"]): x["tbt_impact"]
                                                  for x in r.get("cu_split_streams", [])}
    for sec in ("agentic_replay", "agentic_replay_paper_node"):
        if sec in result:
            r = result[sec]
            out[sec].update({"decode_ms_p50": r["decode_ms"]["p50"], "decode_ms_p99": r["decode_ms"]["p99"],
                             "step_ms_p99": r["step_ms"]["p99"], "hit_rate": r["replay"]["resume_hit_rate"]})
    if "resume_host_tier" in result:
        r = result["resume_host_tier"]
        out["resume_host_tier"] = {"pcie_GBps": r["step48_1_session"]["pcie_GBps"],
                                   "decode48_ms_beside_dma_resume": r["beside_decode"]["dma"]["decode48_ms_beside"],
                                   "decode48_ms_alone": r["beside_decode"]["decode48_ms_alone"]}
    if "spill_decode" in result:
        out["spill_decode_step_ms"] = {"%s_%g_%s" % (x["cold_tier"], x["spilled_frac"], x["mode"]): x["step_ms"]
                                       for x in result["spill_decode"]["rows"]}
    if "configs" in result:
        c = result["configs"]
        out["configs"] = {}
        for name in ("tiny", "step48", "skewed"):
            if name in c:
                out["configs"][name] = {"us_per_call_median": c[name]["us_per_call"]["median"],
                                        "GBps": c[name]["GBps"], "pct_of_peak": c[name]["pct_of_peak"]}
        a = c.get("append")
        if isinstance(a, dict):
            keep = {}
            if "batched_append" in a:
                keep["host_resolved_ms_per_step"] = a["batched_append"]["ms_per_step"]
            for name in ("prompt_write", "prompt_write_one_call"):
                if name in a:
                    keep[name + "_GBps_read_write"] = a[name]["GBps_read_write"]
                    keep[name + "_ms"] = a[name]["ms"]
            if "graph_step" in a:
                keep["graph_append_ms_per_step"] = a["graph_step"]["append_ms_per_step_in_graph"]
                keep["graph_step_ms"] = a["graph_step"]["step_ms"]
            out["configs"]["append"] = keep
        for name, x in c.items():
            if name not in ("tiny", "step48", "skewed", "context", "append") and isinstance(x, dict):
                out["configs"][name] = {k: v for k, v in x.items() if not isinstance(v, (list, dict))}
    return out


if __name__ == "__main__":
    main()
