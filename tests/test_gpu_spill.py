"""Spill and decode from the cold tier (GPU).

With spill on, pages that find no hot page live in the cold tier and the page
table names them with KV_PAGE_COLD.  Checked here against the oracle: the
device page table and every page's bytes follow the pool model through random
spill / promote / resume / evict sequences; decode reads spilled pages directly
(device memory or pinned host memory over PCIe) or through the staging buffer
that the one-layer-ahead prefetch fills, and matches the fp64 oracle; writes
into spilled pages land in the cold tier; promotion copies them back bit for
bit.  A layer decoded without its prefetch reads no staged data (NaN rows).
"""

import sys

import numpy as np
import pytest
import torch

import synth
from helpers import Case, to_device, to_host, tolerance_check
from oracle.pool_model import COLD_BIT, PoolModel

pytestmark = pytest.mark.gpu

COLD_TIERS = ["device", "host"]
SEED = 23


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _random_fill(pool, seed):
    g = torch.Generator(device=pool.device)
    g.manual_seed(seed)
    pool.hot.copy_(torch.randint(0, 256, pool.hot.shape, dtype=torch.uint8, device=pool.device, generator=g))
    pool.cold.copy_(torch.randint(0, 256, pool.cold.shape, dtype=torch.uint8, device=pool.device, generator=g))


@pytest.mark.parametrize("cold,host_kernel", [("device", False), ("host", False), ("host", True)])
def test_spill_sequences_match_model(dev, cold, host_kernel):
    """Random create / extend / pause / resume / promote / evict / LRU-evict /
    destroy in spill mode: the device page table (cold-tagged entries
    included), the statistics and the bytes of every resident page and valid
    cold copy follow the model."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    _say("spill sequences, cold tier in %s memory" % cold)
    nh, nc, ms, stride = 14, 70, 6, 8
    pool = HotColdPool(2, 2, 64, "bf16", nh, nc, ms, stride, cold_location=cold)
    pool.set_host_copy(host_kernel)
    kv.kv_pool_set_spill(pool.handle, True)
    model = PoolModel(nh, nc, ms, stride, spill=True)
    _random_fill(pool, 5)
    torch.cuda.synchronize()
    hot_img = pool.hot_page_bytes().cpu().numpy().copy()
    cold_img = pool.cold.view(nc, -1).cpu().numpy().copy()
    rng = np.random.default_rng(6)

    def both(model_call, lib_call):
        try:
            r = model_call()
        except Exception:
            with pytest.raises(kv.KVError):
                lib_call()
            return None
        got = lib_call()
        return r, got

    for step in range(300):
        op, sid = int(rng.integers(0, 8)), int(rng.integers(0, ms))
        if op == 0:
            L = int(rng.integers(0, 16 * stride + 1))
            r = both(lambda: model.create(L), lambda: pool.create_session(L))
            if r:
                assert r[0] == r[1]
                for h, c in model.last_victim_copies:
                    cold_img[c] = hot_img[h]
        elif op == 1:
            both(lambda: model.pause(sid), lambda: pool.pause(sid))
        elif op == 2:
            r = both(lambda: model.resume([sid]), lambda: pool.resume([sid]))
            if r:
                for h, c in model.last_victim_copies:
                    cold_img[c] = hot_img[h]
                for c, h in r[0][0]:
                    hot_img[h] = cold_img[c]
        elif op == 3:
            L = int(rng.integers(0, 16 * stride + 1))
            r = both(lambda: model.extend(sid, L), lambda: pool.extend(sid, L))
            if r:
                for h, c in model.last_victim_copies:
                    cold_img[c] = hot_img[h]
        elif op == 4:
            n = int(rng.integers(0, 6))
            r = both(lambda: model.promote(n), lambda: kv.kv_promote_pages(pool.handle, n))
            if r:
                assert len(r[0]) == r[1]
                for h, c in model.last_victim_copies:
                    cold_img[c] = hot_img[h]
                for c, h in r[0]:
                    hot_img[h] = cold_img[c]
        elif op == 5:
            r = both(lambda: model.evict(sid), lambda: pool.evict(sid))
            if r:
                for h, c in r[0]:
                    cold_img[c] = hot_img[h]
        elif op == 6:
            n = int(rng.integers(0, 5))
            r = both(lambda: model.evict_pages(n), lambda: pool.evict_pages(n))
            if r:
                assert r[0][0] == r[1]
                for h, c in r[0][1]:
                    cold_img[c] = hot_img[h]
        else:
            both(lambda: model.destroy(sid), lambda: pool.destroy_session(sid))
        torch.cuda.synchronize()
        got = pool.page_table.cpu().numpy()
        assert np.array_equal(got, np.array(model.table(), np.int32)), "step %d op %d" % (step, op)
    st = pool.stats()
    assert st["spilled_pages"] == model.spilled_pages > 10
    assert st["promoted_pages"] == model.promoted_pages > 3
    assert np.any((got >= 0) & ((got & COLD_BIT) != 0))
    hot_now = pool.hot_page_bytes().cpu().numpy()
    cold_now = pool.cold.view(nc, -1).cpu().numpy()
    for s in model.sessions:
        for h, c in zip(s.hot, s.cold):
            if h >= 0:
                assert np.array_equal(hot_now[h], hot_img[h])
            if c >= 0:
                assert np.array_equal(cold_now[c], cold_img[c])
    pool.close()


def _spilled_pool(dev, cold, lens, hot_pages, layers=2, fill=True, dtype="bf16", d=128):
    """Sessions b = 0.. of the given lengths created in spill mode with fewer hot
    pages than they need, filled with generator id b (so the oracle's Case
    regenerates them)."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    n_pages = sum(synth.pages_for(L) for L in lens)
    stride = max(synth.pages_for(L) for L in lens) + 1
    pool = HotColdPool(layers, 2, d, dtype, hot_pages, n_pages + 8, len(lens) + 2, stride,
                       cold_location=cold)
    kv.kv_pool_set_spill(pool.handle, True)
    for b, L in enumerate(lens):
        assert pool.create_session(L) == b
        if fill:
            pool.fill_synthetic(b, b, SEED, float(synth.value_multiplier(1.0)))
    return pool


def _oracle(lens, layer, num_layers=2, dtype="bf16", d=128):
    return Case(num_layers, 8, 2, d, dtype, lens, seed=SEED, layer=layer)


LENS = [200, 333, 64, 517, 1]


@pytest.mark.parametrize("cold,dtype,d", [("device", "bf16", 128), ("host", "bf16", 128),
                                         ("device", "f32", 64), ("host", "f32", 128),
                                         ("device", "bf16", 64)])
def test_decode_reads_spilled_pages(dev, cold, dtype, d):
    """Direct reads: the pool's rows name spilled pages with KV_PAGE_COLD and
    the tiered decode reads them from the cold tier (every shape's kernel)."""
    from paper_2609_25782_amd import hotcold_kv as kv
    _say("decode of spilled pages read in place, cold tier in %s memory, %s d=%d" % (cold, dtype, d))
    pool = _spilled_pool(dev, cold, LENS, hot_pages=30, dtype=dtype, d=d)
    st = pool.stats()
    assert st["spilled_pages"] == sum(synth.pages_for(L) for L in LENS) - 30
    sids = torch.arange(len(LENS), dtype=torch.int32, device=dev)
    table = pool.gather_table(sids)
    t = table.cpu().numpy()
    assert np.any((t >= 0) & ((t & COLD_BIT) != 0))
    sl = torch.tensor(LENS, dtype=torch.int32, device=dev)
    tol = {} if dtype == "bf16" else {"max_norm": 1e-5}
    for layer in (0, 1):
        case = _oracle(LENS, layer, dtype=dtype, d=d)
        got = to_host(pool.decode(layer, to_device(case.q, dtype, dev), sl, page_table=table))
        torch.cuda.synchronize()
        tolerance_check(got, case.oracle_out(), **tol)
    pool.close()


@pytest.mark.parametrize("cold,slots,dtype,d", [("device", 64, "bf16", 128), ("host", 64, "bf16", 128),
                                               ("device", 11, "bf16", 128), ("device", 20, "f32", 64)])
def test_decode_through_prefetched_staging(dev, cold, slots, dtype, d):
    """Staged reads: paged_decode_stage puts spilled pages in staging slots
    (the rest, when slots run out, stay direct cold reads); each layer's slices
    are gathered on a second stream one layer ahead of its decode."""
    from paper_2609_25782_amd import hotcold_kv as kv
    _say("decode through staging, cold tier in %s memory, %d slots, %s d=%d" % (cold, slots, dtype, d))
    pool = _spilled_pool(dev, cold, LENS, hot_pages=30, dtype=dtype, d=d)
    spilled = pool.stats()["spilled_pages"]
    slice_bytes = 2 * 2 * 16 * d * (2 if dtype == "bf16" else 4)
    staging = torch.empty(2 * slots * slice_bytes, dtype=torch.uint8, device=dev)
    assert kv.kv_pool_set_staging(pool.handle, staging.data_ptr(), staging.numel()) == slots
    table = torch.empty((len(LENS), pool.stride), dtype=torch.int32, device=dev)
    staged = kv.paged_decode_stage(pool.handle, list(range(len(LENS))), table.data_ptr())
    assert staged == min(slots, spilled)
    t = table.cpu().numpy()
    assert np.sum((t >= 0) & ((t & kv.KV_PAGE_STAGED) != 0) & ((t & COLD_BIT) == 0)) == staged
    assert np.sum((t >= 0) & ((t & COLD_BIT) != 0)) == spilled - staged
    sl = torch.tensor(LENS, dtype=torch.int32, device=dev)
    copy_stream = torch.cuda.Stream()
    cases = [_oracle(LENS, layer, dtype=dtype, d=d) for layer in (0, 1)]
    qs = [to_device(c.q, dtype, dev) for c in cases]
    tol = {} if dtype == "bf16" else {"max_norm": 1e-5}
    kv.paged_decode_prefetch(pool.handle, 0, copy_stream.cuda_stream)
    outs = []
    for layer in (0, 1):
        if layer + 1 < 2:
            kv.paged_decode_prefetch(pool.handle, layer + 1, copy_stream.cuda_stream)
        outs.append(pool.decode(layer, qs[layer], sl, page_table=table))
    torch.cuda.synchronize()
    for layer in (0, 1):
        tolerance_check(to_host(outs[layer]), cases[layer].oracle_out(), **tol)
    # the next step reuses the plan: prefetch again, decode again, same result
    for layer in (0, 1):
        kv.paged_decode_prefetch(pool.handle, layer, copy_stream.cuda_stream)
        got = to_host(pool.decode(layer, qs[layer], sl, page_table=table))
        tolerance_check(got, cases[layer].oracle_out(), **tol)
    # a layer decoded without its gather reads no staged data: rows with staged
    # pages are NaN, rows without them are still right
    kv.paged_decode_stage(pool.handle, list(range(len(LENS))), table.data_ptr())
    got = to_host(pool.decode(1, qs[1], sl, page_table=table))
    torch.cuda.synchronize()
    has_staged = [bool(np.any((r >= 0) & ((r & kv.KV_PAGE_STAGED) != 0))) for r in table.cpu().numpy()]
    assert any(has_staged)
    ref = cases[1].oracle_out()
    for b, flag in enumerate(has_staged):
        if flag:
            assert np.all(np.isnan(got[b]))
        else:
            tolerance_check(got[b], ref[b], **tol)
    kv.kv_pool_set_staging(pool.handle, 0, 0)
    pool.close()


@pytest.mark.parametrize("cold", ["host", "device"])
def test_prefetch_on_cu_confined_streams(dev, cold):
    """The measured arrangement for a PCIe tier: the gather on a stream with one
    CU per XCD, the decode on a stream over the other CUs; results match the
    oracle, layer after layer, for two steps."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import split_streams
    _say("prefetch on CU-confined streams, cold tier in %s memory" % cold)
    pool = _spilled_pool(dev, cold, LENS, hot_pages=30)
    slice_bytes = 2 * 2 * 16 * 128 * 2
    staging = torch.empty(2 * 64 * slice_bytes, dtype=torch.uint8, device=dev)
    kv.kv_pool_set_staging(pool.handle, staging.data_ptr(), staging.numel())
    table = torch.empty((len(LENS), pool.stride), dtype=torch.int32, device=dev)
    assert kv.paged_decode_stage(pool.handle, list(range(len(LENS))), table.data_ptr()) > 0
    sl = torch.tensor(LENS, dtype=torch.int32, device=dev)
    dec, cpy = split_streams(1)
    cases = [_oracle(LENS, layer) for layer in (0, 1)]
    qs = [to_device(c.q, "bf16", dev) for c in cases]
    torch.cuda.synchronize()
    for step in range(2):
        kv.paged_decode_prefetch(pool.handle, 0, cpy.handle)
        outs = []
        for layer in (0, 1):
            if layer + 1 < 2:
                kv.paged_decode_prefetch(pool.handle, layer + 1, cpy.handle)
            outs.append(pool.decode(layer, qs[layer], sl, page_table=table, stream=dec.stream))
        torch.cuda.synchronize()
        for layer in (0, 1):
            tolerance_check(to_host(outs[layer]), cases[layer].oracle_out())
    kv.kv_pool_set_staging(pool.handle, 0, 0)
    pool.close()
    dec.close()
    cpy.close()


def test_promote_and_write_into_spilled_pages(dev):
    """Tokens written into spilled pages land in the cold tier; after the other
    session is evicted, promotion copies spilled pages into the freed hot pages
    bit for bit; resuming the evicted session with no hot page left leaves it
    entirely in the cold tier.  Decode matches the oracle throughout."""
    from paper_2609_25782_amd import hotcold_kv as kv
    lens = [150, 260]                     # 10 and 17 pages; 12 hot pages
    pool = _spilled_pool(dev, "device", lens, hot_pages=12, fill=False)
    assert pool.stats()["spilled_pages"] == 15
    for layer in (0, 1):                  # every token of both layers through kv_write_tokens
        for b, L in enumerate(lens):
            k, v = synth.session_kv(SEED, b, L, layer, 2, 128, 1.0, "bf16")
            pool.write_tokens(b, layer, 0, to_device(k, "bf16", dev), to_device(v, "bf16", dev))
    sids = torch.arange(2, dtype=torch.int32, device=dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)

    def check():
        table = pool.gather_table(sids)
        for layer in (0, 1):
            case = _oracle(lens, layer)
            got = to_host(pool.decode(layer, to_device(case.q, "bf16", dev), sl, page_table=table))
            tolerance_check(got, case.oracle_out())

    check()
    pool.evict(0)                         # 10 dirty pages written, 10 hot pages free
    assert kv.kv_promote_pages(pool.handle, 100) == 10
    torch.cuda.synchronize()
    st, L1, hot1, cold1 = pool.info(1)
    assert sum(h < 0 for h in hot1) == 5
    pb = pool.page_bytes
    for h, c in zip(hot1, cold1):
        if h >= 0 and c >= 0:
            assert torch.equal(pool.hot_page_bytes([h])[0], pool.cold.view(-1, pb)[c])
    pool.resume(0)                        # nothing free or evictable: stays in the cold tier
    assert all(h < 0 for h in pool.info(0)[2])
    check()
    assert pool.stats()["promoted_pages"] == 10
    pool.close()


@pytest.mark.parametrize("cold", COLD_TIERS)
def test_lazy_resume_decodes_in_place_then_promotes(dev, cold):
    """Lazy resume: no copy at resume, the rows name the cold pages and decode
    reads them in place; promotion in budgeted chunks then moves them into HBM.
    The page table follows the model after every call, decode matches the
    oracle throughout, promoted pages equal their cold copies bit for bit."""
    from paper_2609_25782_amd import hotcold_kv as kv
    _say("lazy resume, cold tier in %s memory" % cold)
    lens = [300, 170, 45]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = _spilled_pool(dev, cold, lens, hot_pages=n_pages + 4)
    model = PoolModel(n_pages + 4, n_pages + 8, len(lens) + 2, pool.stride, spill=True)
    for L in lens:
        model.create(L)
    pool.evict([0, 1, 2])
    model.evict_many([0, 1, 2])
    st0 = pool.stats()
    pool.resume_lazy([0, 1, 2])
    model.resume_lazy([0, 1, 2])
    assert pool.stats()["pages_to_hot"] == st0["pages_to_hot"]      # nothing copied
    sids = torch.arange(3, dtype=torch.int32, device=dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)

    def check():
        torch.cuda.synchronize()
        assert np.array_equal(pool.page_table.cpu().numpy(), np.array(model.table(), np.int32))
        table = pool.gather_table(sids)
        for layer in (0, 1):
            case = _oracle(lens, layer)
            got = to_host(pool.decode(layer, to_device(case.q, "bf16", dev), sl, page_table=table))
            tolerance_check(got, case.oracle_out())

    check()
    # spill cannot be turned off while rows name cold pages (decode without
    # spill would read them as invalid ids); the refused call changes nothing
    from paper_2609_25782_amd import hotcold_kv as kv
    with pytest.raises(kv.KVError) as e:
        pool.set_spill(False)
    assert e.value.status == kv.KV_ERR_STATE
    check()
    moved = 0
    while True:
        n = pool.promote(7)
        assert len(model.promote(7)) == n
        moved += n
        check()
        if n == 0:
            break
    assert moved == n_pages and pool.stats()["cold_active_pages"] == 0
    pool.set_spill(False)                      # nothing spilled any more: accepted
    check()
    pb = pool.page_bytes
    for sid in range(3):
        _, _, hot, cold_ids = pool.info(sid)
        for h, c in zip(hot, cold_ids):
            assert torch.equal(pool.hot_page_bytes([h])[0].cpu(), pool.cold.view(-1, pb)[c].cpu())
    pool.close()


def test_staging_error_paths(dev):
    """Misuse of the staging calls fails with an error and leaves decode intact:
    prefetch without a staging buffer, a misaligned buffer, a paused session in
    the batch, a bad layer."""
    from paper_2609_25782_amd import hotcold_kv as kv
    pool = _spilled_pool(dev, "device", [100, 40], hot_pages=5)
    for call, code in ((lambda: kv.paged_decode_prefetch(pool.handle, 0), kv.KV_ERR_INVALID),):
        with pytest.raises(kv.KVError) as e:
            call()
        assert e.value.status == code
    staging = torch.empty(2 * 8 * 16384 + 512, dtype=torch.uint8, device=dev)
    with pytest.raises(kv.KVError) as e:
        kv.kv_pool_set_staging(pool.handle, staging.data_ptr() + 16, 2 * 8 * 16384)
    assert e.value.status == kv.KV_ERR_INVALID
    assert kv.kv_pool_set_staging(pool.handle, staging.data_ptr(), 2 * 8 * 16384) == 8
    table = torch.empty((2, pool.stride), dtype=torch.int32, device=dev)
    pool.pause(1)
    with pytest.raises(kv.KVError) as e:
        kv.paged_decode_stage(pool.handle, [0, 1], table.data_ptr())
    assert e.value.status == kv.KV_ERR_STATE
    with pytest.raises(kv.KVError) as e:
        kv.paged_decode_prefetch(pool.handle, 2)
    assert e.value.status == kv.KV_ERR_INVALID
    assert kv.paged_decode_stage(pool.handle, [0], table.data_ptr()) == 2   # 7 pages, 5 hot
    kv.paged_decode_prefetch(pool.handle, 1)
    case = _oracle([100], 1)
    got = to_host(pool.decode(1, to_device(case.q, "bf16", dev), torch.tensor([100], dtype=torch.int32, device=dev),
                              page_table=table[:1]))
    tolerance_check(got, case.oracle_out())
    kv.kv_pool_set_staging(pool.handle, 0, 0)
    pool.close()


def test_promotion_concurrent_with_decode(dev):
    """Promotion on a second stream while the same sessions decode on the first:
    rows are rewritten only after the copies, so every decode reads each page
    either from its cold copy or from a finished hot copy, and its output is
    bit-identical to the decode with every page cold (decode does not depend on
    where a page lives)."""
    from paper_2609_25782_amd import hotcold_kv as kv
    lens = [400, 260, 333, 515]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = _spilled_pool(dev, "device", lens, hot_pages=n_pages + 4)
    sids = list(range(len(lens)))
    pool.evict(sids)
    pool.resume_lazy(sids)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    sid_t = torch.tensor(sids, dtype=torch.int32, device=dev)
    case = _oracle(lens, 1)
    q = to_device(case.q, "bf16", dev)
    ref = pool.decode(1, q, sl, page_table=pool.gather_table(sid_t)).clone()
    torch.cuda.synchronize()
    tolerance_check(to_host(ref), case.oracle_out())
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    outs, moved = [], 0
    for it in range(40):
        side.wait_stream(main)
        n = pool.promote(3, stream=side)          # copies, then row entries, on `side`
        table = pool.gather_table(sid_t)          # on `main`, concurrently
        outs.append(pool.decode(1, q, sl, page_table=table).clone())
        main.wait_stream(side)
        moved += n
    torch.cuda.synchronize()
    assert moved == n_pages and pool.stats()["cold_active_pages"] == 0
    for o in outs:
        assert torch.equal(o, ref)
    pool.close()
