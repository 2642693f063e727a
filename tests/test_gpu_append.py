"""Batched append (kv_append_tokens): decode-step appends, one token per
session per call, produce the documented page layout byte for byte (the
oracle's packer fed with the seeded generator's values), on hot pages and on
spilled pages in either cold tier; the pool's decode then matches the oracle."""

import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import ORACLE_DTYPE, Case, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu

SEED = 29


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _page_images(NL, hkv, D, dtype, layer, k, v, n_pages):
    """The packer's bytes of one session's pages, local page ids 0 .. n - 1."""
    pb = oracle.page_bytes(NL, hkv, D, ORACLE_DTYPE[dtype])
    buf = np.zeros(n_pages * pb, np.uint8)
    oracle.pack_pool(buf, NL, hkv, D, ORACLE_DTYPE[dtype], layer, np.arange(n_pages, dtype=np.int32), k, v)
    return buf.reshape(n_pages, pb)


def _append_all(pool, dev, dtype, layer, sids, lens, kv_rows):
    """Decode-step order: step t appends token t of every session longer than t."""
    for t in range(max(lens)):
        rows = [i for i, L in enumerate(lens) if L > t]
        k = np.stack([kv_rows[i][0][t] for i in rows])
        v = np.stack([kv_rows[i][1][t] for i in rows])
        pool.append_tokens(layer, [sids[i] for i in rows], [t] * len(rows),
                           to_device(k, dtype, dev), to_device(v, dtype, dev))


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("bf16", 64), ("f32", 64)])
def test_decode_step_appends_match_packer(dev, dtype, D):
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, layer = 2, 2, 1
    lens = [37, 16, 1, 50, 17]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = HotColdPool(NL, hkv, D, dtype, n_pages + 3, 0, len(lens), 4)
    pool.hot.zero_()
    perm = np.random.default_rng(SEED).permutation(n_pages + 3)
    sids, off = [], 0
    for L in lens:
        n = synth.pages_for(L)
        sids.append(pool.create_session(L, [int(p) for p in perm[off:off + n]]))
        off += n
    kv_rows = [synth.session_kv(SEED, b, L, layer, hkv, D, 1.0, dtype) for b, L in enumerate(lens)]
    _append_all(pool, dev, dtype, layer, sids, lens, kv_rows)
    torch.cuda.synchronize()
    want = np.zeros(pool.hot.numel(), np.uint8)
    for b, L in enumerate(lens):
        pages = np.array(pool.info(sids[b])[2], np.int32)
        oracle.pack_pool(want, NL, hkv, D, ORACLE_DTYPE[dtype], layer, pages, *kv_rows[b])
    assert np.array_equal(pool.hot_page_bytes().cpu().numpy().reshape(-1), want)
    pool.close()


@pytest.mark.parametrize("cold", ["device", "host"])
def test_appends_into_spilled_pages(dev, cold):
    """Spill on, fewer hot pages than the sessions need: tokens of spilled
    pages land in the cold tier.  Every page, wherever it lives, equals the
    packer's; decode over the batch table matches the oracle."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, dtype, layer = 2, 2, 128, "bf16", 0
    lens = [200, 333, 64, 517, 1]
    n_pages = sum(synth.pages_for(L) for L in lens)
    pool = HotColdPool(NL, hkv, D, dtype, 30, n_pages + 8, len(lens) + 1, max(synth.pages_for(L) for L in lens) + 1,
                       cold_location=cold)
    pool.set_spill(True)
    pool.hot.zero_()                      # whole pages are compared, the other layer included
    pool.cold.zero_()
    sids = [pool.create_session(L) for L in lens]
    assert pool.stats()["spilled_pages"] == n_pages - 30
    kv_rows = [synth.session_kv(SEED, b, L, layer, hkv, D, 1.0, dtype) for b, L in enumerate(lens)]
    print("appending %d tokens into %d sessions, cold tier in %s memory" % (sum(lens), len(lens), cold), flush=True)
    _append_all(pool, dev, dtype, layer, sids, lens, kv_rows)
    torch.cuda.synchronize()
    pb = pool.page_bytes
    hot = pool.hot_page_bytes().cpu().numpy()
    cold_img = pool.cold.view(-1, pb).cpu().numpy()
    spilled = 0
    for b, L in enumerate(lens):
        want = _page_images(NL, hkv, D, dtype, layer, *kv_rows[b], synth.pages_for(L))
        _, _, h, c = pool.info(sids[b])
        for i in range(synth.pages_for(L)):
            got = hot[h[i]] if h[i] >= 0 else cold_img[c[i]]
            spilled += h[i] < 0
            assert np.array_equal(got, want[i]), (b, i)
    assert spilled == n_pages - 30
    table = pool.gather_table(torch.tensor(sids, dtype=torch.int32, device=dev))
    case = Case(NL, 8, hkv, D, dtype, lens, seed=SEED, layer=layer)
    got = to_host(pool.decode(layer, to_device(case.q, dtype, dev),
                              torch.tensor(lens, dtype=torch.int32, device=dev), page_table=table))
    torch.cuda.synchronize()
    tolerance_check(got, case.oracle_out())
    pool.close()


def test_long_lists_through_a_staging_slot(dev):
    """Calls of more than 256 rows send their write list through a staging
    slot instead of the kernel arguments: 2 calls of 300 rows, and 1 of 256."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, dtype, layer = 1, 2, 128, "bf16", 0
    L = 856
    n = synth.pages_for(L)
    pool = HotColdPool(NL, hkv, D, dtype, n + 2, 0, 1, n + 1)
    pool.hot.zero_()
    sid = pool.create_session(L)
    k, v = synth.session_kv(SEED, 0, L, layer, hkv, D, 1.0, dtype)
    for a, b in ((0, 300), (300, 600), (600, 856)):
        pool.append_tokens(layer, [sid] * (b - a), list(range(a, b)), to_device(k[a:b], dtype, dev),
                           to_device(v[a:b], dtype, dev))
    torch.cuda.synchronize()
    want = np.zeros(pool.hot.numel(), np.uint8)
    oracle.pack_pool(want, NL, hkv, D, ORACLE_DTYPE[dtype], layer, np.array(pool.info(sid)[2], np.int32), k, v)
    assert np.array_equal(pool.hot_page_bytes().cpu().numpy().reshape(-1), want)
    pool.close()


def test_append_refuses_bad_rows_and_writes_nothing(dev):
    """A call with one bad row launches nothing: the pool's bytes are unchanged."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    pool = HotColdPool(1, 2, 64, "bf16", 8, 0, 2, 4)
    pool.hot.zero_()
    a = pool.create_session(20)
    k = torch.ones((2, 2, 64), dtype=torch.bfloat16, device=dev)
    for sids, pos in (([a, a], [3, 3]), ([a, a], [3, 20]), ([a, 1], [3, 0])):
        with pytest.raises(kv.KVError):
            pool.append_tokens(0, sids, pos, k, k)
    torch.cuda.synchronize()
    assert int(pool.hot.count_nonzero()) == 0
    pool.append_tokens(0, [a, a], [3, 19], k, k)
    torch.cuda.synchronize()
    assert int(pool.hot.count_nonzero()) == 2 * 2 * 2 * 64 * 2
    pool.close()
