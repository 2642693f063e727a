"""GPU parity of paged decode attention (split + combine) against the fp64 oracle.

Every case goes through the C ABI (paged_decode_attention).  The pool is
written by the library (kv_write_tokens); the oracle reads the same logical K/V
packed by its own code.  Bar: max-abs error <= 1e-2 and normalised error <= 1e-2
(bf16), tighter for float32; structured cases (single token, V = 1, poison,
relocation, GQA rows) are exact.
"""

import math
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


def _run(case: Case, dev, poison=False, waves=None, scale=None, pool=None, fused=True):
    _say("decode case: dtype=%s D=%d Hq=%d Hkv=%d NL=%d layer=%d lens=%s waves=%s fused=%s" % (
        case.dtype, case.head_dim, case.num_q_heads, case.num_kv_heads, case.num_layers, case.layer,
        case.seq_lens[:8], waves, fused))
    own = pool is None
    if own:
        pool = build_gpu(case, dev, poison=poison)
    if waves:
        pool.set_waves(waves)
    pool.set_combine(fused)
    q = to_device(case.q, case.dtype, dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    out = pool.decode(case.layer, q, sl, scale=scale)
    torch.cuda.synchronize()
    res = to_host(out)
    if own:
        pool.close()
    return res


def test_tiny_config_f32(dev):
    """One layer, 4 query / 1 KV heads, d=64, fp32, 4 sessions with L in [100, 500]."""
    w = synth.config_tiny(0)
    case = Case(1, 4, 1, 64, "f32", [int(x) for x in w.seq_lens], seed=0, slack=2.0)
    got = _run(case, dev)
    ref = case.oracle_out()
    err, norm = tolerance_check(got, ref, 1e-2, 1e-5)
    _say("tiny f32: max abs %.3g normalised %.3g" % (err, norm))


@pytest.mark.parametrize("dtype,D,hq,hkv", [("bf16", 128, 32, 4), ("bf16", 64, 8, 2),
                                           ("bf16", 128, 16, 1), ("bf16", 64, 4, 4),
                                           ("f32", 128, 8, 1), ("f32", 64, 6, 2),
                                           ("bf16", 128, 32, 8), ("bf16", 64, 16, 16),
                                           ("f32", 64, 16, 8)])
def test_ragged_lengths(dev, dtype, D, hq, hkv):
    lens = [1, 15, 16, 17, 31, 33, 100, 1000, 4097, 250]
    case = Case(1, hq, hkv, D, dtype, lens, seed=3)
    got = _run(case, dev)
    ref = case.oracle_out()
    err, norm = tolerance_check(got, ref, 1e-2, 1e-2 if dtype == "bf16" else 1e-5)
    _say("ragged %s D=%d: abs %.3g norm %.3g" % (dtype, D, err, norm))


def test_group_of_16_and_multilayer(dev):
    case = Case(3, 32, 2, 128, "bf16", [300, 2000, 17], seed=4, layer=2)
    got = _run(case, dev)
    tolerance_check(got, case.oracle_out())


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("waves", [1, 3, 7, 64, 1000, 5000])
def test_split_invariance(dev, waves, fused):
    """Any number of waves, either merge of the partials: the oracle's answer
    within tolerance (P10)."""
    case = Case(1, 32, 4, 128, "bf16", [5000, 16, 1, 777, 3000, 48], seed=5)
    got = _run(case, dev, waves=waves, fused=fused)
    tolerance_check(got, case.oracle_out())


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("waves", [8, 64, 1000, 4096])
def test_split_invariance_two_head_groups(dev, waves, fused):
    """Eight KV heads: workers of four waves take two head groups per row."""
    case = Case(1, 32, 8, 128, "bf16", [5000, 16, 1, 777, 3000, 48], seed=19)
    got = _run(case, dev, waves=waves, fused=fused)
    tolerance_check(got, case.oracle_out())


@pytest.mark.parametrize("fused", [True, False])
@pytest.mark.parametrize("waves", [3, 4, 8, 64, 256])
def test_every_row_written_many_short_rows(dev, waves, fused):
    """96 short rows, two of them empty, and fewer waves than (row, KV head)
    segments: most segments sit whole in one piece, whose wave writes the
    output itself, a few are cut between workers and merged by the combine,
    whose grid then walks the workers' split-segment entries.  The output starts
    as NaN: every row must be written, the empty ones as zeros, the rest within
    the oracle's tolerance."""
    rng = np.random.default_rng(23)
    lens = [int(x) for x in rng.integers(1, 400, size=96)]
    lens[5] = lens[40] = 0
    case = Case(1, 16, 4, 128, "bf16", lens, seed=23)
    pool = build_gpu(case, dev)
    pool.set_waves(waves)
    pool.set_combine(fused)
    _say("short rows: waves=%d fused=%s" % (waves, fused))
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    out = torch.full((len(lens), 16, 128), float("nan"), dtype=torch.bfloat16, device=dev)
    pool.decode(0, q, sl, out=out)
    torch.cuda.synchronize()
    got = to_host(out)
    pool.close()
    assert not np.isnan(got).any()
    assert np.all(got[[5, 40]] == 0)
    rows = [b for b in range(len(lens)) if lens[b] > 0]
    tolerance_check(got[rows], case.oracle_out(rows=rows))


@pytest.mark.parametrize("dtype,D,hq,hkv", [("bf16", 128, 32, 4), ("f32", 64, 16, 1), ("bf16", 64, 16, 1)])
def test_separate_combine(dev, dtype, D, hq, hkv):
    case = Case(1, hq, hkv, D, dtype, [1, 15, 16, 17, 100, 3000, 250], seed=16)
    got = _run(case, dev, fused=False)
    tolerance_check(got, case.oracle_out(), 1e-2, 1e-2 if dtype == "bf16" else 1e-5)


def test_layer_shape_scaled_values(dev):
    """Qwen3-Coder-30B-A3B-shaped layer at reduced batch, values N(0,1)/sqrt(128)."""
    rng = np.random.default_rng(6)
    lens = [int(x) for x in rng.integers(8192, 32768, size=4, endpoint=True)]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=6, value_scale=1 / math.sqrt(128), slack=1.25)
    got = _run(case, dev)
    err, norm = tolerance_check(got, case.oracle_out())
    _say("layer shape scaled: abs %.3g norm %.3g" % (err, norm))


@pytest.mark.parametrize("waves", [0, 1, 4])
@pytest.mark.parametrize("fused", [True, False])
def test_zero_and_invalid_lengths(dev, fused, waves):
    """Zero, negative and over-long lengths.  With one wave every segment is
    one piece, so the split writes the NaN rows itself; with four, some
    segments are cut between waves; with the default grid every page is a
    piece of its own."""
    case = Case(1, 8, 2, 64, "bf16", [40, 0, 70], seed=7)
    pool = build_gpu(case, dev)
    pool.set_combine(fused)
    pool.set_waves(waves)
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor([40, 0, 70], dtype=torch.int32, device=dev)
    out = to_host(pool.decode(0, q, sl))
    torch.cuda.synchronize()
    assert np.all(out[1] == 0)
    tolerance_check(out[[0, 2]], case.oracle_out(rows=[0, 2]))
    # a length beyond the row stride and a negative one give NaN rows, others unchanged
    bad = torch.tensor([40, -5, 16 * case.stride + 1], dtype=torch.int32, device=dev)
    out2 = to_host(pool.decode(0, q, bad))
    torch.cuda.synchronize()
    assert np.all(np.isnan(out2[1])) and np.all(np.isnan(out2[2]))
    if waves == 4:
        # the longer row 2 moves the boundaries between the waves' ranges, so row
        # 0 is cut differently: equal to the oracle, not bit for bit to the first call
        tolerance_check(out2[[0]], case.oracle_out(rows=[0]))
    else:
        assert np.array_equal(out2[0], out[0])
    # the next call is clean again (the fused merge's counters reset themselves)
    out3 = to_host(pool.decode(0, q, sl))
    torch.cuda.synchronize()
    assert np.array_equal(out3, out)
    pool.close()


@pytest.mark.parametrize("waves", [0, 1, 4])
@pytest.mark.parametrize("fused", [True, False])
def test_out_of_range_page_id_gives_nan(dev, fused, waves):
    case = Case(1, 8, 2, 64, "bf16", [40, 70], seed=8)
    pool = build_gpu(case, dev)
    pool.set_combine(fused)
    pool.set_waves(waves)
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    pt = pool.page_table[:2].clone()
    pt[1, 2] = case.hot_pages + 1000
    out = to_host(pool.decode(0, q, sl, page_table=pt))
    torch.cuda.synchronize()
    assert np.all(np.isnan(out[1])) and np.all(np.isfinite(out[0]))
    pool.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_poison_outside_valid_tokens(dev, dtype):
    """NaN in every slot that is not a valid token: output finite and bitwise equal (P6)."""
    case = Case(1, 16, 2, 128 if dtype == "bf16" else 64, dtype, [1, 17, 45, 300, 16], seed=9)
    clean = _run(case, dev)
    dirty = _run(case, dev, poison=True)
    assert np.all(np.isfinite(dirty))
    assert np.array_equal(clean, dirty)


def test_relocation_is_bitwise_invariant(dev):
    """The same logical KV under two different page placements: identical bits (P7)."""
    lens = [3000, 17, 900, 4096]
    a = Case(1, 32, 4, 128, "bf16", lens, seed=10, slack=3.0)
    rng = np.random.default_rng(99)
    perm = rng.permutation(a.hot_pages).astype(np.int32)
    placement, off = [], 0
    for L in lens:
        n = synth.pages_for(L)
        placement.append(perm[off:off + n])
        off += n
    b = Case(1, 32, 4, 128, "bf16", lens, seed=10, placement=placement, hot_pages=a.hot_pages)
    assert not all(np.array_equal(x, y) for x, y in zip(a.placement, b.placement))
    assert np.array_equal(_run(a, dev), _run(b, dev))


def test_single_token_returns_v_exactly(dev):
    """L = 1: the output is v_0 exactly (P2)."""
    case = Case(1, 32, 4, 128, "bf16", [1, 1, 1], seed=11)
    got = _run(case, dev)
    for b in range(3):
        v0 = synth.bf16_bits_to_f32(case.kv[b][1][0]).astype(np.float64)  # [Hkv, D]
        for h in range(32):
            assert np.array_equal(got[b, h], v0[h // 8])


def test_constant_v_gives_constant_output(dev):
    """V = 1 everywhere: every output element is exactly 1 (weights sum to one, P4)."""
    case = Case(1, 32, 4, 128, "bf16", [5, 333, 4099, 16], seed=12)
    for b in range(case.batch):
        k, v = case.kv[b]
        case.kv[b] = (k, np.full_like(v, synth.f32_to_bf16_bits(np.float32(1.0))))
    got = _run(case, dev)
    assert np.all(got == 1.0)


def test_identical_keys_give_mean_of_values(dev):
    """All keys of a (row, KV head) equal: every weight is 1/L and the output is
    the mean of V (P3).  The scores are then bitwise equal, every exp2 is exactly
    1, the weight sums are exact integers and every merge factor is 1, so the
    only roundings are the float32 sums of V and the bf16 output: within one
    bf16 half-unit (2^-9 relative, bounded here by 2^-8) of the fp64 mean."""
    lens = [1000, 37, 5000, 16, 1]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=16)
    for b in range(case.batch):
        k, v = case.kv[b]
        case.kv[b] = (np.broadcast_to(k[:1], k.shape).copy(), v)
    got = _run(case, dev, fused=False)
    for b in range(case.batch):
        mean = synth.bf16_bits_to_f32(case.kv[b][1]).astype(np.float64).mean(axis=0)  # [Hkv, D]
        for h in range(32):
            want = mean[h // 8]
            assert np.all(np.abs(got[b, h] - want) <= 2 ** -8 * np.abs(want) + 1e-6)


def test_key_shift_leaves_output_unchanged(dev):
    """Adding the same vector c to every key of a (row, KV head) adds q.c to
    every score of a query head, which the softmax removes (P9).  float32 pool;
    keys and c on a 2^-8 grid, so k + c is exact and only the scores' float32
    rounding differs (about 1e-5 absolute at |q.c| ~ 24, 1e-6 relative in the
    weights): the outputs agree within 1e-5 of the largest output."""
    lens = [700, 33, 2500]
    a = Case(1, 8, 2, 64, "f32", lens, seed=17)
    b = Case(1, 8, 2, 64, "f32", lens, seed=17)
    rng = np.random.default_rng(18)
    shift = (np.round(rng.standard_normal((2, 64)) * 3 * 256) / 256).astype(np.float32)
    for i in range(len(lens)):
        k, v = a.kv[i]
        kq = (np.round(k.astype(np.float64) * 256) / 256).astype(np.float32)
        a.kv[i] = (kq, v)
        b.kv[i] = ((kq + shift[None]).astype(np.float32), v)
    ga, gb = _run(a, dev), _run(b, dev)
    tolerance_check(ga, a.oracle_out())
    diff = float(np.max(np.abs(ga - gb)))
    _say("key shift: max difference %.3g, max |out| %.3g" % (diff, float(np.max(np.abs(ga)))))
    assert diff <= 1e-5 * float(np.max(np.abs(ga)))


def test_gqa_rows_identical_for_equal_queries(dev):
    """Equal queries within a group give bitwise identical output rows (P11)."""
    case = Case(1, 32, 4, 128, "bf16", [2500, 60], seed=13)
    for b in range(case.batch):
        for g in range(4):
            case.q[b, g * 8:(g + 1) * 8] = case.q[b, g * 8]
    got = _run(case, dev)
    for b in range(case.batch):
        for g in range(4):
            for h in range(g * 8 + 1, (g + 1) * 8):
                assert np.array_equal(got[b, h], got[b, g * 8])


@pytest.mark.parametrize("where", ["first", "page_end", "page_start", "last", "middle"])
def test_needle(dev, where):
    """One key aligned with the query and a score gap of 40+: output = its value (P5).
    Catches page-table and offset mistakes that the tolerance cannot see."""
    L = 20000
    case = Case(1, 32, 4, 128, "bf16", [L, 4000], seed=14, value_scale=0.05)
    t_star = {"first": 0, "page_end": 15, "page_start": 16, "last": L - 1, "middle": 12345}[where]
    g = 2
    q = synth.bf16_bits_to_f32(case.q[0, g * 8]).astype(np.float64)
    case.q[0, g * 8:(g + 1) * 8] = case.q[0, g * 8]
    k, v = case.kv[0]
    k = k.copy()
    needle = (60.0 * math.sqrt(128) * q / np.dot(q, q)).astype(np.float32)
    k[t_star, g] = synth.f32_to_bf16_bits(needle)
    v = v.copy()
    v[t_star, g] = synth.f32_to_bf16_bits(np.linspace(-1, 1, 128).astype(np.float32))
    case.kv[0] = (k, v)
    got = _run(case, dev)
    want = synth.bf16_bits_to_f32(v[t_star, g]).astype(np.float64)
    for h in range(g * 8, (g + 1) * 8):
        assert np.max(np.abs(got[0, h] - want)) <= 2 ** -8 * np.max(np.abs(want))
    tolerance_check(got, case.oracle_out())


def test_partition_table_matches_reference(dev):
    from oracle import partition
    from paper_2609_25782_amd.pool import HotColdPool
    rng = np.random.default_rng(15)
    for hkv in (4, 8, 16, 2):
        pool = HotColdPool(1, hkv, 64, "bf16", 8, 0, 1, 4096)
        for trial in range(6):
            B = int(rng.integers(1, 40))
            lens = [int(x) for x in rng.integers(0, 20000, size=B)]
            waves = int(rng.choice([1, 5, 64, 300, 2048]))
            _say("partition trial %d: Hkv=%d B=%d waves=%d" % (trial, hkv, B, waves))
            sl = torch.tensor(lens, dtype=torch.int32, device=dev)
            got = pool.partition(sl, waves).cpu().numpy()
            want = np.array(partition.slot_table(lens, hkv, waves), dtype=np.int32)
            assert np.array_equal(got, want)
        pool.close()


def test_repeated_calls_and_batch_changes_are_consistent(dev):
    """Back-to-back calls with different batches on one pool: every call matches
    its own first result (the merge counters return to zero after each call)."""
    case = Case(1, 32, 4, 128, "bf16", [3000, 17, 900, 4096, 1, 64], seed=17)
    pool = build_gpu(case, dev)
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    first = to_host(pool.decode(0, q, sl))
    sub = to_host(pool.decode(0, q[2:5].contiguous(), sl[2:5].contiguous(),
                              page_table=pool.page_table[2:5].contiguous()))
    for _ in range(5):
        again = to_host(pool.decode(0, q, sl))
        assert np.array_equal(again, first)
    assert np.array_equal(to_host(pool.decode(0, q[2:5].contiguous(), sl[2:5].contiguous(),
                                              page_table=pool.page_table[2:5].contiguous())), sub)
    torch.cuda.synchronize()
    tolerance_check(first, case.oracle_out())
    pool.close()


def test_maximum_batch_and_full_rows(dev):
    """The largest batch the decode kernels take (8,192 rows) with ragged
    lengths of 1 to 48 tokens; the longest rows fill their page-table row (3
    pages) exactly.  Every row against the oracle; one row more is refused."""
    from paper_2609_25782_amd import hotcold_kv as kv
    rng = np.random.default_rng(11)
    lens = [int(x) for x in rng.integers(1, 49, size=8192)]
    lens[0] = lens[-1] = 48
    case = Case(1, 4, 1, 64, "bf16", lens, seed=11, extra_stride=0)
    assert case.stride == 3
    pool = build_gpu(case, dev)
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor(lens, dtype=torch.int32, device=dev)
    got = to_host(pool.decode(0, q, sl))
    torch.cuda.synchronize()
    tolerance_check(got, case.oracle_out())
    with pytest.raises(kv.KVError) as e:
        kv.paged_decode_attention(pool.handle, 0, q.data_ptr(), pool.page_table.data_ptr(), pool.stride,
                                  sl.data_ptr(), 8193, 4, 0.125, q.data_ptr(), q.data_ptr(), 1 << 20, 0)
    assert e.value.status == kv.KV_ERR_INVALID
    pool.close()
