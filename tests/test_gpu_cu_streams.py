"""Streams confined to disjoint CU slots (kv_stream_create_cu_slots): a decode
running beside a resume gives the same bits as alone, and the calls that make
such streams refuse bad arguments."""

import sys

import numpy as np
import pytest
import torch

from helpers import Case, build_gpu, to_device, to_host, tolerance_check
import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_slots_cover_the_device_and_bad_ranges_are_refused(dev):
    from paper_2609_25782_amd import hotcold_kv as kv
    xcds, slots = kv.kv_device_cu_slots(0)
    _say("device: %d XCDs x %d CUs" % (xcds, slots))
    assert xcds * slots == torch.cuda.get_device_properties(0).multi_processor_count
    for a, b in ((-1, 2), (3, 3), (5, 2), (0, slots + 1)):
        with pytest.raises(kv.KVError) as e:
            kv.kv_stream_create_cu_slots(0, a, b)
        assert e.value.status == kv.KV_ERR_INVALID
    with pytest.raises(kv.KVError) as e:
        kv.kv_device_cu_slots(torch.cuda.device_count())
    assert e.value.status == kv.KV_ERR_INVALID
    with pytest.raises(kv.KVError):
        kv.kv_stream_destroy(0)


@pytest.mark.parametrize("copy_slots", [8, 2])
def test_decode_beside_resume_on_split_streams(dev, copy_slots):
    """Sessions 0-2 decode on the decode stream while sessions 3-5 resume on the
    copy stream: that decode equals the same decode alone bit for bit.  After
    both, all six decode exactly as before the eviction (P8), also on the copy
    stream's few CUs, where the default grid needs several rounds."""
    from paper_2609_25782_amd.pool import split_streams
    lens = [3000, 700, 16, 4099, 2500, 9000]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=71, slack=1.3)
    n_cold = sum(synth.pages_for(L) for L in lens)
    pool = build_gpu(case, dev, num_cold_pages=n_cold, pool_kwargs={"max_sessions": 8})
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    before = to_host(pool.decode(0, q, sl))
    tolerance_check(before, case.oracle_out())
    q3, sl3 = q[:3].contiguous(), sl[:3].contiguous()
    pt3 = pool.page_table[:3].contiguous()
    alone3 = to_host(pool.decode(0, q3, sl3, page_table=pt3))
    pool.evict([3, 4, 5])
    torch.cuda.synchronize()
    dec, cpy = split_streams(copy_slots)
    _say("decode stream %d CUs, copy stream %d CUs" % (dec.cus, cpy.cus))
    main = torch.cuda.current_stream()
    dec.stream.wait_stream(main)
    cpy.stream.wait_stream(main)
    out3 = torch.empty_like(q3)
    pool.resume([5, 3, 4], stream=cpy.stream)
    pool.decode(0, q3, sl3, page_table=pt3, out=out3, stream=dec.stream)
    main.wait_stream(dec.stream)
    main.wait_stream(cpy.stream)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(out3), alone3)
    after = to_host(pool.decode(0, q, sl, page_table=pool.page_table[:6].contiguous()))
    torch.cuda.synchronize()
    assert np.array_equal(after, before)
    few = torch.empty_like(q)
    pool.decode(0, q, sl, page_table=pool.page_table[:6].contiguous(), out=few, stream=cpy.stream)
    torch.cuda.synchronize()
    assert np.array_equal(to_host(few), before)
    dec.close()
    cpy.close()
    pool.close()


def test_two_batches_decode_concurrently_on_split_streams(dev):
    """Two batches of one pool decode at the same time on two streams with
    disjoint CU sets.  Separate-merge decodes share nothing of the pool's, so the
    library does not order them, and each keeps its own workspace: each output is
    bit-identical to the same batch decoded alone, and matches the oracle.
    Repeated with the calls issued in both orders."""
    from paper_2609_25782_amd.pool import split_streams
    lens = [5000, 300, 12000, 17, 2048, 7777, 900, 4100]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=73, slack=1.2)
    pool = build_gpu(case, dev, pool_kwargs={"max_sessions": 8})
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    ref = case.oracle_out()
    halves = []
    for rows in (slice(0, 4), slice(4, 8)):
        qa, sa = q[rows].contiguous(), sl[rows].contiguous()
        pa = pool.page_table[rows].contiguous()
        alone = pool.decode(0, qa, sa, page_table=pa).clone()
        torch.cuda.synchronize()
        tolerance_check(to_host(alone), ref[rows])
        halves.append((qa, sa, pa, alone))
    from paper_2609_25782_amd import hotcold_kv as kv
    _, slots = kv.kv_device_cu_slots(0)
    s_a, s_b = split_streams(slots // 2)
    main = torch.cuda.current_stream()
    for order in ((0, 1), (1, 0)):
        outs = [torch.empty_like(halves[0][0]), torch.empty_like(halves[1][0])]
        for s in (s_a, s_b):
            s.stream.wait_stream(main)
        for i in order:
            qa, sa, pa, _ = halves[i]
            for _ in range(3):
                pool.decode(0, qa, sa, page_table=pa, out=outs[i], stream=(s_a, s_b)[i].stream)
        for s in (s_a, s_b):
            main.wait_stream(s.stream)
        torch.cuda.synchronize()
        for i in (0, 1):
            assert torch.equal(outs[i], halves[i][3])
    s_a.close()
    s_b.close()
    pool.close()
