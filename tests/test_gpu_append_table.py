"""Fresh-KV writes without host-side page resolution (data path 3):

* kv_write_tokens_layers: a token range of several layers in one launch writes
  the bytes the oracle's packer gives, the same as one kv_write_tokens per layer.
* kv_append_tokens_table: a decode step's append resolved on the device through
  a batch page table writes the packer's bytes on hot and spilled pages, skips
  entries that name no page, and keeps write-on-evict exact through the
  extension's cold-copy drop.
* A whole serving step (batch-table gather, then append and decode for every
  layer) captured into one HIP graph: every replay equals the same step done
  eagerly with host-resolved appends, bit for bit, and the last step matches
  the oracle.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import ORACLE_DTYPE, Case, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu

SEED = 41


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _token_mask(NL, hkv, D, pb, n_tok):
    """Bytes of one bf16 page that hold slots 0 .. n_tok - 1 (every layer, head, K and V),
    found by packing a marker with the oracle's packer."""
    img = np.zeros(pb, np.uint8)
    marker = np.full((n_tok, hkv, D), 0xFFFF, np.uint16)
    for l in range(NL):
        oracle.pack_pool(img, NL, hkv, D, oracle.BF16, l, np.array([0], np.int32), marker, marker)
    return img != 0


def _stack_layers(seed, b, L, layers, hkv, D, dtype):
    """K and V of session b for the given layers: [len(layers)][L][hkv][D]."""
    kv = [synth.session_kv(seed, b, L, l, hkv, D, 1.0, dtype) for l in layers]
    return np.stack([k for k, _ in kv]), np.stack([v for _, v in kv])


@pytest.mark.parametrize("dtype,D", [("bf16", 128), ("f32", 64)])
def test_write_tokens_layers_matches_packer_and_per_layer_writes(dev, dtype, D):
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, L = 5, 2, 70
    pools = [HotColdPool(NL, hkv, D, dtype, 12, 0, 1, 6) for _ in range(2)]
    pages = [int(p) for p in np.random.default_rng(SEED).permutation(12)[:synth.pages_for(L)]]
    for p in pools:
        p.hot.zero_()
        assert p.create_session(L, pages) == 0
    k, v = _stack_layers(SEED, 0, L, range(NL), hkv, D, dtype)
    t0, t1, l0, nl = 5, 61, 1, 3                    # partial first and last pages; layers 1..3
    pools[0].write_tokens_layers(0, l0, t0, to_device(np.ascontiguousarray(k[l0:l0 + nl, t0:t1]), dtype, dev),
                                 to_device(np.ascontiguousarray(v[l0:l0 + nl, t0:t1]), dtype, dev))
    for l in range(l0, l0 + nl):
        pools[1].write_tokens(0, l, t0, to_device(np.ascontiguousarray(k[l, t0:t1]), dtype, dev),
                              to_device(np.ascontiguousarray(v[l, t0:t1]), dtype, dev))
    torch.cuda.synchronize()
    want = np.zeros(pools[0].hot.numel(), np.uint8)
    kk = np.zeros_like(k)
    vv = np.zeros_like(v)
    kk[:, t0:t1], vv[:, t0:t1] = k[:, t0:t1], v[:, t0:t1]
    for l in range(l0, l0 + nl):
        oracle.pack_pool(want, NL, hkv, D, ORACLE_DTYPE[dtype], l, np.array(pages, np.int32), kk[l], vv[l])
    got = [p.hot_page_bytes().cpu().numpy().reshape(-1) for p in pools]
    assert np.array_equal(got[0], got[1])
    assert np.array_equal(got[0], want)
    from paper_2609_25782_amd import hotcold_kv as kv
    for bad in ((4, 2), (-1, 1), (0, 6)):                # layer ranges outside the pool
        with pytest.raises(kv.KVError) as e:
            kv.kv_write_tokens_layers(pools[0].handle, 0, bad[0], bad[1], 0, 1, 16, 16)
        assert e.value.status == kv.KV_ERR_INVALID
    for p in pools:
        p.close()


@pytest.mark.parametrize("cold", ["device", "host"])
def test_append_table_matches_packer_and_decodes(dev, cold):
    """Decode-step appends through the batch table, two layers per launch; a
    fifth of the pages spilled to the cold tier (written in place)."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, dtype = 2, 2, 128, "bf16"
    lens = [37, 16, 1, 50, 17, 90]
    n_pages = sum(synth.pages_for(L) for L in lens)
    hot = n_pages * 4 // 5
    pool = HotColdPool(NL, hkv, D, dtype, hot, n_pages + 4, len(lens), 8, cold_location=cold)
    pool.set_spill(True)
    B = len(lens)
    sids = [pool.create_session(0) for _ in lens]
    kvs = [_stack_layers(SEED, b, L, range(NL), hkv, D, dtype) for b, L in enumerate(lens)]
    table = torch.empty((B, pool.stride), dtype=torch.int32, device=dev)
    sid_t = torch.tensor(sids, dtype=torch.int32, device=dev)
    rows_t = torch.arange(B, dtype=torch.int32, device=dev)
    pos_t = torch.zeros(B, dtype=torch.int32, device=dev)
    for t in range(max(lens)):
        live = [i for i, L in enumerate(lens) if L > t]
        for i in live:
            pool.extend(sids[i], t + 1)
        pool.gather_table(sid_t, out=table)
        # rows that are done get a position past the table: the kernel skips them
        pos = [t if i in live else 16 * pool.stride for i in range(B)]
        pos_t.copy_(torch.tensor(pos, dtype=torch.int32))
        k = np.zeros((NL, B, hkv, D), np.uint16)
        v = np.zeros((NL, B, hkv, D), np.uint16)
        for i in live:
            k[:, i], v[:, i] = kvs[i][0][:, t], kvs[i][1][:, t]
        pool.append_tokens_table(0, table, rows_t, pos_t, to_device(k, dtype, dev), to_device(v, dtype, dev))
    torch.cuda.synchronize()
    st = pool.stats()
    assert st["cold_active_pages"] > 0
    # every page, hot or spilled, equals the packer's image
    pb = pool.page_bytes
    for b, L in enumerate(lens):
        _, _, hot_ids, cold_ids = pool.info(sids[b])
        img = np.zeros(synth.pages_for(L) * pb, np.uint8)
        for l in range(NL):
            oracle.pack_pool(img, NL, hkv, D, oracle.BF16, l, np.arange(synth.pages_for(L), dtype=np.int32),
                             kvs[b][0][l], kvs[b][1][l])
        img = img.reshape(-1, pb)
        for i, (h, c) in enumerate(zip(hot_ids, cold_ids)):
            src = pool.hot_page_bytes([h])[0] if h >= 0 else pool.cold.view(-1, pb)[c]
            got = src.cpu().numpy()
            # the tail page's slots past L were never written: compare the written tokens only
            mask = _token_mask(NL, hkv, D, pb, min(16, L - 16 * i))
            assert np.array_equal(got[mask], img[i][mask]), "session %d page %d" % (b, i)
    # decode of the batch table against the oracle, both layers
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    for l in range(NL):
        case = Case(NL, 8, hkv, D, dtype, lens, seed=SEED, layer=l)
        got = to_host(pool.decode(l, to_device(case.q, dtype, dev), sl, page_table=table))
        tolerance_check(got, case.oracle_out())
    pool.close()


def test_append_table_skips_entries_naming_no_page(dev):
    """Rows outside the table, positions outside a row, -1 entries, staged
    tags and out-of-range ids write nothing; valid entries in the same launch
    still land."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    pool = HotColdPool(1, 1, 64, "bf16", 6, 2, 2, 4)
    pool.hot.zero_()
    pool.cold.zero_()
    pool.create_session(40)
    table = torch.tensor([[0, 1, 2, -1], [5, kv.KV_PAGE_STAGED | 0, 999, kv.KV_PAGE_COLD | 7]],
                         dtype=torch.int32, device=dev)
    rows = torch.tensor([0, 1, 1, 1, 1, 1, 2, -1, 0, 0], dtype=torch.int32, device=dev)
    pos = torch.tensor([35, 3, 20, 40, 60, 64, 0, 0, 48, -1], dtype=torch.int32, device=dev)
    # valid: (0, 35) -> page 2 slot 3; (1, 3) -> page 5 slot 3.  Skipped: staged, id 999,
    # cold id 7 (the cold pool has 2 pages), position 64 (past the row), rows 2 and -1,
    # entry -1 of row 0 (position 48), negative position.
    k = torch.ones((1, 10, 1, 64), dtype=torch.bfloat16, device=dev)
    pool.append_tokens_table(0, table, rows, pos, k, k.clone())
    torch.cuda.synchronize()
    pb = pool.page_bytes
    hot = pool.hot_page_bytes().cpu().numpy()
    changed = sorted(set(np.flatnonzero(hot.any(axis=1)).tolist()))
    assert changed == [2, 5]
    assert not pool.cold.cpu().numpy().any()
    for p, slot in ((2, 3), (5, 3)):
        img = np.zeros(pb, np.uint8)
        one = np.full((1, 1, 64), 0x3F80, np.uint16)  # bf16 1.0
        full_k = np.concatenate([np.zeros((slot, 1, 64), np.uint16), one])
        oracle.pack_pool(img, 1, 1, 64, oracle.BF16, 0, np.array([0]), full_k, full_k)
        assert np.array_equal(hot[p], img)
    with pytest.raises(kv.KVError) as e:
        kv.kv_append_tokens_table(pool.handle, 0, 2, table.data_ptr(), 4, 2, rows.data_ptr(), pos.data_ptr(), 10,
                                  k.data_ptr(), k.data_ptr())
    assert e.value.status == kv.KV_ERR_INVALID        # layers [0, 2) of a 1-layer pool
    pool.close()


def test_extension_keeps_write_on_evict_exact_for_device_appends(dev):
    """A resumed session whose tail page is partly filled: extending it drops
    that page's cold copy, so after an append resolved on the device the next
    eviction writes exactly that page, and its cold copy holds the new token."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D = 1, 2, 64
    pool = HotColdPool(NL, hkv, D, "bf16", 8, 8, 1, 4)
    k, v = synth.session_kv(SEED, 0, 21, 0, hkv, D, 1.0, "bf16")
    sid = pool.create_session(20)
    pool.write_tokens(sid, 0, 0, to_device(k[:20], "bf16", dev), to_device(v[:20], "bf16", dev))
    pool.evict(sid)
    pool.resume(sid)
    before = pool.stats()["pages_to_cold"]
    pool.extend(sid, 21)
    _, _, hot_ids, cold_ids = pool.info(sid)
    assert cold_ids[0] >= 0 and cold_ids[1] == -1
    table = pool.page_table[:1].contiguous()
    pool.append_tokens_table(0, table, torch.zeros(1, dtype=torch.int32, device=dev),
                             torch.tensor([20], dtype=torch.int32, device=dev),
                             to_device(k[20:21][None], "bf16", dev), to_device(v[20:21][None], "bf16", dev))
    pool.evict(sid)
    torch.cuda.synchronize()
    assert pool.stats()["pages_to_cold"] - before == 1
    _, _, _, cold_ids = pool.info(sid)
    pb = pool.page_bytes
    img = np.zeros(2 * pb, np.uint8)
    oracle.pack_pool(img, NL, hkv, D, oracle.BF16, 0, np.arange(2, dtype=np.int32), k, v)
    got = pool.cold.view(-1, pb)[cold_ids[1]].cpu().numpy()
    mask = _token_mask(NL, hkv, D, pb, 5)               # tokens 16..20 of page 1
    assert np.array_equal(got[mask], img[pb:][mask])
    pool.close()


@pytest.mark.parametrize("append", ["table", "fused"])
def test_serving_step_graph_matches_eager_steps(dev, append):
    """One captured graph per step shape: gather the batch table, then for each
    of 4 layers append the step's token (resolved on the device: a separate
    launch through the table, or fused into the decode launch) and decode.
    Replayed for 40 steps with the host's extensions and the new tokens' values
    written in place between replays; the same steps done eagerly (host-
    resolved appends) on a second pool give bitwise equal outputs and pages,
    and the last step matches the oracle."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, hq, dtype = 4, 2, 128, 16, "bf16"
    start = [100, 17, 333, 40, 250]
    steps = 40
    final = [L + steps for L in start]
    B = len(start)
    stride = max(synth.pages_for(L) for L in final) + 1
    n_pages = sum(synth.pages_for(L) for L in final) + 8
    pools = [HotColdPool(NL, hkv, D, dtype, n_pages, 0, B, stride) for _ in range(2)]
    kvs = [_stack_layers(SEED, b, L, range(NL), hkv, D, dtype) for b, L in enumerate(final)]
    for p in pools:
        p.hot.zero_()
        for b, L in enumerate(start):
            assert p.create_session(L) == b
            p.write_tokens_layers(b, 0, 0, to_device(np.ascontiguousarray(kvs[b][0][:, :L]), dtype, dev),
                                  to_device(np.ascontiguousarray(kvs[b][1][:, :L]), dtype, dev))
    cases = [Case(NL, hq, hkv, D, dtype, final, seed=SEED, layer=l) for l in range(NL)]
    qs = [to_device(c.q, dtype, dev) for c in cases]
    sid_t = torch.arange(B, dtype=torch.int32, device=dev)
    rows_t = torch.arange(B, dtype=torch.int32, device=dev)
    pos_t = torch.zeros(B, dtype=torch.int32, device=dev)
    sl_t = torch.zeros(B, dtype=torch.int32, device=dev)
    k_new = torch.zeros((NL, B, hkv, D), dtype=torch.bfloat16, device=dev)
    v_new = torch.zeros_like(k_new)
    table = torch.empty((B, stride), dtype=torch.int32, device=dev)
    outs = [torch.empty_like(q) for q in qs]
    eager_outs = [torch.empty_like(q) for q in qs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = None
    with torch.cuda.stream(s):
        for step in range(steps):
            lens = [L + step + 1 for L in start]
            for p in pools:
                for b in range(B):
                    p.extend(b, lens[b])
            pos_t.copy_(torch.tensor([L - 1 for L in lens], dtype=torch.int32))
            sl_t.copy_(torch.tensor(lens, dtype=torch.int32))
            k_new.copy_(to_device(np.stack([kvs[b][0][:, lens[b] - 1] for b in range(B)], axis=1), dtype, dev))
            v_new.copy_(to_device(np.stack([kvs[b][1][:, lens[b] - 1] for b in range(B)], axis=1), dtype, dev))

            def graph_step():
                pools[0].gather_table(sid_t, out=table, stream=s)
                for l in range(NL):
                    if append == "table":
                        pools[0].append_tokens_table(l, table, rows_t, pos_t, k_new[l:l + 1], v_new[l:l + 1],
                                                     stream=s)
                        pools[0].decode(l, qs[l], sl_t, page_table=table, out=outs[l], stream=s)
                    else:
                        pools[0].decode(l, qs[l], sl_t, page_table=table, out=outs[l], stream=s,
                                        k_new=k_new[l], v_new=v_new[l])

            if g is None:
                graph_step()                             # eager once: workspace allocated before capture
                torch.cuda.synchronize()
                # undo nothing: the step wrote the same bytes the replay will write again
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s):
                    graph_step()
            g.replay()
            # the eager path on the second pool: host-resolved appends
            for l in range(NL):
                pools[1].append_tokens(l, list(range(B)), [L - 1 for L in lens], k_new[l].contiguous(),
                                       v_new[l].contiguous(), stream=s)
                pools[1].decode(l, qs[l], sl_t, page_table=pools[1].page_table[:B], out=eager_outs[l], stream=s)
            torch.cuda.synchronize()
            for l in range(NL):
                assert torch.equal(outs[l], eager_outs[l]), "step %d layer %d" % (step, l)
    assert torch.equal(pools[0].hot, pools[1].hot)
    for l in range(NL):
        tolerance_check(to_host(outs[l]), cases[l].oracle_out())
    for p in pools:
        p.close()


@pytest.mark.parametrize("dtype,D,hq,hkv,waves,vector", [
    ("bf16", 128, 32, 4, None, False), ("bf16", 128, 32, 4, 5, False), ("bf16", 64, 8, 2, None, False),
    ("f32", 64, 8, 2, None, False), ("f32", 128, 16, 1, 7, False), ("bf16", 128, 32, 4, None, True),
    ("bf16", 64, 16, 2, 3, True)])
def test_fused_append_equals_append_then_decode(dev, dtype, D, hq, hkv, waves, vector):
    """paged_decode_attention_append against kv_append_tokens followed by
    paged_decode_attention on a twin pool: bitwise equal outputs and pages, for
    tails in a fresh page (L - 1 = 16 k), mid-page and at a page end, rows of
    length 0 (nothing appended) and 1, both work-split shapes (workers of four
    waves, and of one), and both forms of the split kernel.  Unwritten slots
    hold NaN, so a token the decode did not see written would show.  The last
    step also matches the oracle."""
    from paper_2609_25782_amd.pool import HotColdPool
    NL, layer = 2, 1
    L0 = [0, 15, 16, 17, 31, 100, 1, 250]
    final = [L + 2 if L > 0 else 0 for L in L0]          # two fused steps
    B = len(L0)
    stride = max(synth.pages_for(L) for L in final) + 1
    n_pages = sum(synth.pages_for(L) for L in final) + 5
    pools = [HotColdPool(NL, hkv, D, dtype, n_pages, 0, B, stride) for _ in range(2)]
    kvs = [synth.session_kv(SEED, b, L, layer, hkv, D, 1.0, dtype) for b, L in enumerate(final)]
    perm = np.random.default_rng(SEED + 1).permutation(n_pages)
    for p in pools:
        if dtype == "bf16":
            p.hot.view(torch.int16).fill_(0x7FC0)
        else:
            p.hot.view(torch.float32).fill_(float("nan"))
        p.set_compute(vector)
        if waves:
            p.set_waves(waves)
        off = 0
        for b, L in enumerate(L0):
            n = synth.pages_for(final[b])
            # pages for the final length up front: placement as a random permutation
            assert p.create_session(16 * n, [int(x) for x in perm[off:off + n]]) == b
            off += n
            if L:
                p.write_tokens(b, layer, 0, to_device(kvs[b][0][:L], dtype, dev), to_device(kvs[b][1][:L], dtype, dev))
    case = Case(NL, hq, hkv, D, dtype, final, seed=SEED, layer=layer)
    q = to_device(case.q, dtype, dev)
    for step in (1, 2):
        lens = [L + step if L > 0 else 0 for L in L0]
        sl = torch.tensor(lens, dtype=torch.int32, device=dev)
        rows = [b for b in range(B) if lens[b] > 0]
        kn = np.zeros((B, hkv, D), kvs[0][0].dtype)
        vn = np.zeros((B, hkv, D), kvs[0][0].dtype)
        for b in rows:
            kn[b], vn[b] = kvs[b][0][lens[b] - 1], kvs[b][1][lens[b] - 1]
        kn_t, vn_t = to_device(kn, dtype, dev), to_device(vn, dtype, dev)
        fused = pools[0].decode(layer, q, sl, page_table=pools[0].page_table[:B], k_new=kn_t, v_new=vn_t).clone()
        pools[1].append_tokens(layer, rows, [lens[b] - 1 for b in rows], kn_t[rows].contiguous(),
                               vn_t[rows].contiguous())
        sep = pools[1].decode(layer, q, sl, page_table=pools[1].page_table[:B]).clone()
        torch.cuda.synchronize()
        assert torch.equal(fused, sep), "step %d" % step
        assert torch.isfinite(fused.float()).all()
    assert torch.equal(pools[0].hot.view(torch.int16), pools[1].hot.view(torch.int16))
    tolerance_check(to_host(fused), case.oracle_out(), max_norm=1e-2 if dtype == "bf16" else 1e-5)
    for p in pools:
        p.close()


@pytest.mark.parametrize("cold", ["device", "host"])
def test_fused_append_into_spilled_tail_pages(dev, cold):
    """With spill on, tail pages in the cold tier receive the fused append in
    place; the outputs equal the separate append's, and a layer decoded through
    staging refuses the fused append."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    NL, hkv, D, hq, dtype = 2, 2, 128, 16, "bf16"
    L0 = [40, 17, 90, 5]
    B = len(L0)
    need = sum(synth.pages_for(L + 1) for L in L0)
    pools = [HotColdPool(NL, hkv, D, dtype, need // 2, need + 4, B, 8, cold_location=cold) for _ in range(2)]
    kvs = [synth.session_kv(SEED, b, L + 1, 0, hkv, D, 1.0, dtype) for b, L in enumerate(L0)]
    for p in pools:
        p.set_spill(True)
        for b, L in enumerate(L0):
            assert p.create_session(L) == b
            p.write_tokens(b, 0, 0, to_device(kvs[b][0][:L], dtype, dev), to_device(kvs[b][1][:L], dtype, dev))
            p.extend(b, L + 1)
    assert pools[0].stats()["cold_active_pages"] > 0
    sids = torch.arange(B, dtype=torch.int32, device=dev)
    tables = [p.gather_table(sids) for p in pools]
    lens = [L + 1 for L in L0]
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    case = Case(NL, hq, hkv, D, dtype, lens, seed=SEED, layer=0)
    q = to_device(case.q, dtype, dev)
    kn = to_device(np.stack([kvs[b][0][L] for b, L in enumerate(L0)]), dtype, dev)
    vn = to_device(np.stack([kvs[b][1][L] for b, L in enumerate(L0)]), dtype, dev)
    fused = pools[0].decode(0, q, sl, page_table=tables[0], k_new=kn, v_new=vn).clone()
    pools[1].append_tokens(0, list(range(B)), L0, kn, vn)
    sep = pools[1].decode(0, q, sl, page_table=tables[1]).clone()
    torch.cuda.synchronize()
    assert torch.equal(fused, sep)
    tolerance_check(to_host(fused), case.oracle_out())
    # staging: the fused append is refused for a staged layer
    staging = torch.empty(2 * 16 * pools[0].slice_bytes, dtype=torch.uint8, device=dev)
    kv.kv_pool_set_staging(pools[0].handle, staging.data_ptr(), staging.numel())
    table = torch.empty((B, pools[0].stride), dtype=torch.int32, device=dev)
    assert kv.paged_decode_stage(pools[0].handle, list(range(B)), table.data_ptr()) > 0
    kv.paged_decode_prefetch(pools[0].handle, 0)
    with pytest.raises(kv.KVError) as e:
        pools[0].decode(0, q, sl, page_table=table, k_new=kn, v_new=vn)
    assert e.value.status == kv.KV_ERR_INVALID
    torch.cuda.synchronize()
    kv.kv_pool_set_staging(pools[0].handle, 0, 0)
    for p in pools:
        p.close()
