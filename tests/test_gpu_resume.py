"""GPU parity of resume (cold -> hot gather + page-table rewrite) and eviction
(write-on-evict scatter): page tables must equal the oracle pool model's
prediction and page bytes must match bit for bit."""

import sys

import numpy as np
import pytest
import torch

from helpers import Case, build_gpu, to_device, to_host
from oracle.pool_model import PoolModel
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _pages(t: torch.Tensor, page_bytes: int, ids) -> np.ndarray:
    """Host copy of the given pages of a pool tensor (uint8 rows)."""
    idx = torch.tensor([int(i) for i in ids], dtype=torch.long, device=t.device)
    return t.view(-1, page_bytes).index_select(0, idx).cpu().numpy() if len(ids) else \
        np.zeros((0, page_bytes), np.uint8)


def _hot_pages(pool, ids) -> np.ndarray:
    """Host copy of the given hot pages in page order (the hot pool is layer-major)."""
    return pool.hot_page_bytes([int(i) for i in ids]).cpu().numpy() if len(ids) else \
        np.zeros((0, pool.page_bytes), np.uint8)


def _random_fill(pool, seed):
    g = torch.Generator(device=pool.device)
    g.manual_seed(seed)
    pool.hot.copy_(torch.randint(0, 256, pool.hot.shape, dtype=torch.uint8, device=pool.device, generator=g))
    # the cold pool may be pinned host memory: generate on the device, then copy
    pool.cold.copy_(torch.randint(0, 256, pool.cold.shape, dtype=torch.uint8, device=pool.device, generator=g))


COLD_TIERS = ["device", "host"]


def _check_table(pool, model: PoolModel):
    got = pool.page_table.cpu().numpy()
    want = np.array(model.table(), dtype=np.int32)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("cold", COLD_TIERS)
def test_tiny_resume_config(dev, cold):
    """Two paused sessions of 256 tokens resumed from a 64-page cold pool (fp32,
    d=64, one layer): exact page table and bytes, cold pool in device memory or
    in pinned host memory read over PCIe."""
    from paper_2609_25782_amd.pool import HotColdPool
    _say("tiny resume config, cold tier in %s memory" % cold)
    pool = HotColdPool(1, 1, 64, "f32", 80, 64, 8, 32, cold_location=cold)
    model = PoolModel(80, 64, 8, 32)
    _random_fill(pool, 1)
    torch.cuda.synchronize()
    cold_before = pool.cold.clone()
    # the paused sessions' KV already sits in the cold tier at known pages
    rng = np.random.default_rng(0)
    cold_lists = [rng.choice(64, 16, replace=False), rng.choice(64, 16, replace=False)]
    sids = [pool.import_cold(256, c) for c in cold_lists]
    assert sids == [model.import_cold(256, c) for c in cold_lists]
    # some active sessions first so the resumed pages are not simply 0..31
    for L in (100, 37):
        assert pool.create_session(L) == model.create(L)
    pool.resume(sids)
    copies = model.resume(sids)
    torch.cuda.synchronize()
    _check_table(pool, model)
    pb = pool.page_bytes
    for per in copies:
        src = [c for c, _ in per]
        dst = [h for _, h in per]
        assert np.array_equal(_hot_pages(pool, dst), _pages(cold_before, pb, src))
    assert torch.equal(pool.cold, cold_before)  # resume never writes the cold tier
    st = pool.stats()
    assert st["pages_to_hot"] == 32 and st["resumes"] == 2
    pool.close()


@pytest.mark.parametrize("cold", COLD_TIERS)
def test_evict_resume_round_trip_decode_bitwise(dev, cold):
    """Decode before eviction equals decode after resume into other pages (P8)."""
    case = Case(1, 32, 4, 128, "bf16", [3000, 700, 16, 4099], seed=21, slack=1.3)
    pool = build_gpu(case, dev, num_cold_pages=sum(synth.pages_for(L) for L in case.seq_lens),
                     pool_kwargs={"max_sessions": 8, "cold_location": cold})
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    before = to_host(pool.decode(0, q, sl))
    rows_before = pool.page_table[:4].clone()
    for sid in (0, 2):
        pool.evict(sid)
    # occupy the freed pages so the resume must land elsewhere
    blocker = pool.create_session(16 * 40)
    pool.resume([2, 0])
    torch.cuda.synchronize()
    assert not torch.equal(pool.page_table[:4], rows_before)
    after = to_host(pool.decode(0, q, sl, page_table=pool.page_table[:4].contiguous()))
    torch.cuda.synchronize()
    assert np.array_equal(before, after)
    pool.destroy_session(blocker)
    pool.close()


def test_write_on_evict_writes_each_page_once(dev):
    """Sec. III: an unmodified page reaches the cold tier at most once; a page
    written to after its cold copy was made is written again."""
    case = Case(1, 8, 2, 64, "bf16", [16 * 9 + 5], seed=22)
    pool = build_gpu(case, dev, num_cold_pages=64, pool_kwargs={"max_sessions": 2})
    model = PoolModel(case.hot_pages, 64, 2, case.stride)
    model.create(case.seq_lens[0], case.placement[0])
    for _ in range(3):
        pool.evict(0), model.evict(0)
        pool.resume(0), model.resume([0])
    st = pool.stats()
    assert st["pages_to_cold"] == 10 == model.cold_writes
    # rewrite token 40 (page 2) -> only that page is written on the next eviction
    k, v = case.kv[0]
    pool.write_tokens(0, 0, 40, to_device(k[40:41], "bf16", dev), to_device(v[40:41], "bf16", dev))
    model.write_tokens(0, 40, 1)
    copies = model.evict(0)
    pool.evict(0)
    assert len(copies) == 1 and pool.stats()["pages_to_cold"] == 11
    pool.resume(0), model.resume([0])
    torch.cuda.synchronize()
    _check_table(pool, model)
    pool.close()


def test_resume_exhaustion_changes_nothing(dev):
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    pool = HotColdPool(2, 2, 64, "bf16", 10, 20, 4, 8)
    a = pool.create_session(16 * 6)
    pool.evict(a)
    b = pool.create_session(16 * 6)  # 6 of 10 hot pages used: a (6 pages) cannot come back
    torch.cuda.synchronize()
    table = pool.page_table.clone()
    st = pool.stats()
    with pytest.raises(kv.KVError) as e:
        pool.resume(a)
    assert e.value.status == kv.KV_ERR_NO_HOT_PAGES
    with pytest.raises(kv.KVError) as e:
        pool.resume([a, b])
    assert e.value.status == kv.KV_ERR_STATE
    torch.cuda.synchronize()
    assert torch.equal(pool.page_table, table) and pool.stats() == st
    pool.close()


def test_aliased_cold_pages_resume(dev):
    """Paused sessions sharing cold pages (virtualised cold pool) resume correctly."""
    from paper_2609_25782_amd.pool import HotColdPool
    pool = HotColdPool(1, 4, 128, "bf16", 64, 16, 4, 16)
    _random_fill(pool, 2)
    torch.cuda.synchronize()
    cold_before = pool.cold.clone()
    a = pool.import_cold(16 * 10, list(range(10)))
    b = pool.import_cold(16 * 8 + 3, [9, 8, 7, 15, 14, 13, 0, 1, 2])
    model = PoolModel(64, 16, 4, 16)
    model.import_cold(16 * 10, list(range(10)))
    model.import_cold(16 * 8 + 3, [9, 8, 7, 15, 14, 13, 0, 1, 2])
    copies = model.resume([b, a])
    pool.resume([b, a])
    torch.cuda.synchronize()
    _check_table(pool, model)
    pb = pool.page_bytes
    for per in copies:
        assert np.array_equal(_hot_pages(pool, [h for _, h in per]),
                              _pages(cold_before, pb, [c for c, _ in per]))
    pool.close()


@pytest.mark.parametrize("cold,host_kernel", [("device", False), ("host", False), ("host", True)])
def test_random_sequences_match_model(dev, cold, host_kernel):
    """Random create / write / evict / pause / LRU-evict / extend / resume /
    destroy sequences: page tables, statistics and the bytes of every resident
    page and every valid cold copy follow the model exactly.  The pinned-host
    tier runs with its copies on the DMA engines (default) and in the copy
    kernel."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    nh, nc, ms, stride = 48, 40, 6, 8
    pool = HotColdPool(2, 2, 64, "bf16", nh, nc, ms, stride, cold_location=cold)
    pool.set_host_copy(host_kernel)
    model = PoolModel(nh, nc, ms, stride)
    _random_fill(pool, 3)
    torch.cuda.synchronize()
    # expected content of every hot and cold page, tracked through the copies
    hot_img = pool.hot_page_bytes().cpu().numpy().copy()
    cold_img = pool.cold.view(nc, -1).cpu().numpy().copy()
    rng = np.random.default_rng(4)

    def apply(copies, src_img, dst_img):
        for a_, b_ in copies:
            dst_img[b_] = src_img[a_]

    for step in range(400):
        op = int(rng.integers(0, 8))
        sid = int(rng.integers(0, ms))
        try:
            if op == 0:
                L = int(rng.integers(0, 16 * stride + 1))
                try:
                    model_sid = model.create(L)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.create_session(L)
                    raise e
                assert pool.create_session(L) == model_sid
                apply(model.last_victim_copies, hot_img, cold_img)
            elif op == 5:
                try:
                    model.pause(sid)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.pause(sid)
                    raise e
                pool.pause(sid)
            elif op == 6:
                n = int(rng.integers(0, 10))
                try:
                    got, copies = model.evict_pages(n)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.evict_pages(n)
                    raise e
                assert pool.evict_pages(n) == got
                apply(copies, hot_img, cold_img)
            elif op == 7:
                new_len = int(rng.integers(0, 16 * stride + 1))
                try:
                    model.extend(sid, new_len)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.extend(sid, new_len)
                    raise e
                pool.extend(sid, new_len)
                apply(model.last_victim_copies, hot_img, cold_img)
            elif op == 1:
                sids = [int(x) for x in rng.choice(ms, size=int(rng.integers(1, 3)), replace=False)]
                try:
                    copies = model.evict_many(sids)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.evict(sids)
                    raise e
                pool.evict(sids)
                for h, c in copies:
                    cold_img[c] = hot_img[h]
            elif op == 2:
                sids = [int(x) for x in rng.choice(ms, size=int(rng.integers(1, 3)), replace=False)]
                try:
                    res = model.resume(sids)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.resume(sids)
                    raise e
                pool.resume(sids)
                apply(model.last_victim_copies, hot_img, cold_img)  # victims first
                for per in res:
                    for c, h in per:
                        hot_img[h] = cold_img[c]
            elif op == 3:
                try:
                    model.destroy(sid)
                except Exception as e:
                    with pytest.raises(kv.KVError):
                        pool.destroy_session(sid)
                    raise e
                pool.destroy_session(sid)
            else:
                s = model.sessions[sid]
                if s.state == 1 and s.seq_len > 0:
                    t0 = int(rng.integers(0, s.seq_len))
                    n = int(rng.integers(1, min(20, s.seq_len - t0) + 1))
                    layer = int(rng.integers(0, 2))
                    kk = rng.integers(0, 65535, size=(n, 2, 64), dtype=np.uint16)
                    vv = rng.integers(0, 65535, size=(n, 2, 64), dtype=np.uint16)
                    pool.write_tokens(sid, layer, t0, to_device(kk, "bf16", dev), to_device(vv, "bf16", dev))
                    model.write_tokens(sid, t0, n)
                    # mirror the writes on the host image with the oracle's packer
                    import oracle
                    flat = hot_img.reshape(-1)
                    pages = np.array(model.sessions[sid].hot, dtype=np.int64)
                    full_k = np.zeros((t0 + n, 2, 64), np.uint16)
                    full_v = np.zeros((t0 + n, 2, 64), np.uint16)
                    full_k[t0:] = kk
                    full_v[t0:] = vv
                    tmp = flat.copy()
                    oracle.pack_pool(tmp, 2, 2, 64, oracle.BF16, layer, pages, full_k, full_v)
                    # only tokens t0.. are written: copy those elements back
                    for t in range(t0, t0 + n):
                        for g in range(2):
                            for d in range(64):
                                for kind in (0, 1):
                                    off = oracle.elem_offset(2, 2, 64, oracle.BF16, int(pages[t // 16]),
                                                             layer, g, kind, t % 16, d)
                                    flat[off:off + 2] = tmp[off:off + 2]
        except Exception as e:  # the model refused: the library refused as well
            if not hasattr(e, "code"):
                raise
        if step % 25 == 24:
            torch.cuda.synchronize()
            _check_table(pool, model)
            st = pool.stats()
            assert st["free_hot_pages"] == model.free_hot() and st["free_cold_pages"] == model.free_cold()
            assert st["pages_to_cold"] == model.cold_writes
            assert st["lru_evicted_pages"] == model.lru_evicted
            assert (st["resume_pages_resident"], st["resume_pages_total"]) == (model.resume_resident,
                                                                               model.resume_total)
            gpu_hot = pool.hot_page_bytes().cpu().numpy()
            gpu_cold = pool.cold.view(nc, -1).cpu().numpy()
            for s in model.sessions:
                for p in s.hot:
                    if p >= 0:
                        assert np.array_equal(gpu_hot[p], hot_img[p])
                for c in s.cold:
                    if c >= 0:
                        assert np.array_equal(gpu_cold[c], cold_img[c])
    pool.close()


def test_resume_48_layer_pages(dev):
    """1.5 MiB pages (48 layers x 4 KV heads x 128 x bf16): a resumed session's
    pages are bit-exact copies and its decode matches the oracle on a sampled layer."""
    from paper_2609_25782_amd.pool import HotColdPool
    lens = [16 * 300 + 7, 16 * 120]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = HotColdPool(48, 4, 128, "bf16", n_pages + 50, n_pages, 4, 320)
    assert pool.page_bytes == 1536 * 1024
    for b, L in enumerate(lens):
        sid = pool.create_session(L)
        pool.fill_synthetic(sid, b, 77, float(synth.value_multiplier(1.0)))
    for sid in range(2):
        pool.evict(sid)
    blocker = pool.create_session(16 * 40)
    pool.resume([1, 0])
    torch.cuda.synchronize()
    st0, L0, hot0, cold0 = pool.info(0)
    pb = pool.page_bytes
    for i in (0, 1, len(hot0) - 1, 150):
        assert torch.equal(pool.hot_page_bytes([hot0[i]])[0], pool.cold.view(-1, pb)[cold0[i]])
    # decode layer 31 of both sessions against the oracle on regenerated KV
    from helpers import Case
    case = Case(48, 32, 4, 128, "bf16", lens, seed=77, layer=31,
                placement=[np.array(pool.info(s)[2], np.int32) for s in range(2)],
                hot_pages=n_pages + 50)
    case.kv = [synth.session_kv(77, b, L, 31, 4, 128, 1.0, "bf16") for b, L in enumerate(lens)]
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    got = to_host(pool.decode(31, q, sl, page_table=pool.page_table[:2].contiguous()))
    torch.cuda.synchronize()
    from helpers import tolerance_check
    tolerance_check(got, case.oracle_out())
    pool.destroy_session(blocker)
    pool.close()


@pytest.mark.parametrize("cold", COLD_TIERS)
def test_partial_residency_round_trip(dev, cold):
    """Pause, evict part of a session page by page (LRU), resume: only the missing
    pages are fetched (the statistics show the hit rate) and decode is bitwise
    the same as before the pause."""
    case = Case(1, 32, 4, 128, "bf16", [4000, 1500, 3000], seed=41, slack=1.5)
    n_pages = sum(synth.pages_for(L) for L in case.seq_lens)
    pool = build_gpu(case, dev, num_cold_pages=n_pages,
                     pool_kwargs={"max_sessions": 6, "cold_location": cold})
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    before = to_host(pool.decode(0, q, sl))
    pool.pause(0)
    pool.pause(2)
    assert pool.evict_pages(100) == 100          # 100 of session 0's 250 pages (oldest pause)
    st0 = pool.stats()
    filler = pool.create_session(16 * 60)        # takes free pages, may evict more LRU pages
    pool.resume([2, 0])
    torch.cuda.synchronize()
    st = pool.stats()
    fetched = st["pages_to_hot"] - st0["pages_to_hot"]
    resident = st["resume_pages_resident"] - st0["resume_pages_resident"]
    assert fetched + resident == synth.pages_for(4000) + synth.pages_for(3000)
    assert fetched >= 100 and resident > 0
    after = to_host(pool.decode(0, q, sl, page_table=pool.page_table[:3].contiguous()))
    torch.cuda.synchronize()
    assert np.array_equal(before, after)
    pool.destroy_session(filler)
    pool.close()


def test_copy_lists_larger_than_one_staging_slot(dev):
    """One eviction and one resume of 80,000 pages (two sessions of 40,000): the
    copy list spans two staging slots and two launches.  Page tables follow the
    model; every resumed page equals its cold copy."""
    from paper_2609_25782_amd.pool import HotColdPool
    n = 40000
    pool = HotColdPool(1, 1, 64, "bf16", 2 * n + 100, 2 * n + 10, 3, n)
    model = PoolModel(2 * n + 100, 2 * n + 10, 3, n)
    for b in range(2):
        assert pool.create_session(16 * n) == model.create(16 * n) == b
        pool.fill_synthetic(b, b, 3, 1.0)
    pool.evict([0, 1])
    model.evict_many([0, 1])
    blocker = pool.create_session(16 * 90)        # the resume lands on other hot pages
    assert blocker == model.create(16 * 90)
    pool.resume([1, 0])
    model.resume([1, 0])
    torch.cuda.synchronize()
    _check_table(pool, model)
    pb = pool.page_bytes
    for sid in (0, 1):
        st, L, hot, cold = pool.info(sid)
        h = torch.tensor(hot, dtype=torch.long, device=dev)
        c = torch.tensor(cold, dtype=torch.long, device=dev)
        assert torch.equal(pool.hot_page_bytes(h), pool.cold.view(-1, pb).index_select(0, c))
    pool.close()


def test_copy_launch_shapes_and_budget(dev):
    """The page copy takes one of two launch shapes by size: up to 16 GiB of
    4 KiB rows (10,922 pages of 1.5 MiB) one row per block on a large grid,
    above it (10,923 pages) 32 KiB chunks on the persistent grid; a caller's
    copy-block budget takes the persistent shape with the budget as the grid.
    Each resume: page table as the model predicts, sampled pages bit-exact."""
    from paper_2609_25782_amd.pool import HotColdPool
    fine, coarse = 10922, 10923
    assert fine * 384 <= 4 << 20 < coarse * 384
    n_hot, n_cold, stride = coarse + 8, fine + coarse + 8, coarse
    _say("copy launch shapes: %d and %d pages of 1.5 MiB" % (fine, coarse))
    pool = HotColdPool(48, 4, 128, "bf16", n_hot, n_cold, 2, stride)
    model = PoolModel(n_hot, n_cold, 2, stride)
    g = torch.Generator(device=dev)
    g.manual_seed(8)
    view = pool.cold.view(n_cold, -1)
    for i in range(0, n_cold, 1024):
        view[i:i + 1024].copy_(torch.randint(0, 256, view[i:i + 1024].shape, dtype=torch.uint8,
                                             device=dev, generator=g))
    rng = np.random.default_rng(8)
    perm = rng.permutation(n_cold)
    lists = [[int(p) for p in perm[:fine]], [int(p) for p in perm[fine:fine + coarse]]]
    for n, cold in zip((fine, coarse), lists):
        assert pool.import_cold(16 * n, cold) == model.import_cold(16 * n, cold)
    pb = pool.page_bytes

    def resume_and_check(sid, what):
        pool.resume([sid])
        copied = sum(len(per) for per in model.resume([sid]))
        torch.cuda.synchronize()
        _check_table(pool, model)
        _, _, h, c = pool.info(sid)
        idx = sorted(set([0, len(h) - 1] + [int(x) for x in rng.choice(len(h), size=300, replace=False)]))
        hh = torch.tensor([h[i] for i in idx], dtype=torch.long, device=dev)
        cc = torch.tensor([c[i] for i in idx], dtype=torch.long, device=dev)
        assert torch.equal(pool.hot_page_bytes(hh), view.index_select(0, cc))
        _say("%s: %d pages resumed, %d copied, %d sampled pages bit-exact" % (what, len(h), copied, len(idx)))
        return copied

    n1 = resume_and_check(0, "fine shape")
    pool.evict([0])
    model.evict_many([0])
    n2 = resume_and_check(1, "persistent shape")  # takes session 0's former hot pages
    pool.evict([1])
    model.evict_many([1])
    pool.set_copy_blocks(64)
    n3 = resume_and_check(0, "budget of 64 blocks")
    assert (n1, n2) == (fine, coarse) and n3 > fine - 16
    assert pool.stats()["pages_to_hot"] == n1 + n2 + n3
    pool.close()


def test_frees_on_alternating_streams_are_all_waited_for(dev):
    """A 1 GiB eviction on stream A frees hot pages, a destroy on stream B frees
    one more, and a session created on stream C takes A's freed pages and is
    filled at once.  C must wait for A's copy as well as B's work: the evicted
    session's cold copy equals its hot pages before the eviction."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL = 8
    n = 4096
    pool = HotColdPool(NL, 4, 128, "bf16", n + 64, n + 64, 8, n)
    pb = pool.page_bytes
    big = pool.create_session(16 * n)
    small = pool.create_session(16)
    pool.fill_synthetic(big, 0, 5, 1.0)
    pool.fill_synthetic(small, 1, 5, 1.0)
    hot_big = pool.info(big)[2]
    torch.cuda.synchronize()
    idx = torch.tensor(hot_big, dtype=torch.long, device=dev)
    before = pool.hot_page_bytes(idx)
    sa, sb, sc = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    _say("evict %d pages of %d KiB on stream A, destroy on B, refill on C" % (n, pb // 1024))
    pool.evict(big, stream=sa)
    pool.destroy_session(small, stream=sb)
    other = pool.create_session(16 * n, stream=sc)
    assert sorted(pool.info(other)[2])[:n] == sorted(hot_big)  # the evicted session's pages
    pool.fill_synthetic(other, 2, 6, 1.0, stream=sc)
    torch.cuda.synchronize()
    cold_big = pool.info(big)[3]
    cidx = torch.tensor(cold_big, dtype=torch.long, device=dev)
    assert torch.equal(pool.cold.view(-1, pb).index_select(0, cidx), before)
    pool.close()
