"""GPU parity of the vector-ALU form of the decode split kernel.

kv_pool_set_decode_compute(KV_DECODE_VECTOR) runs both products of the split
kernel as bf16 dot2 on the vector ALU, with the matrix-core form's work split,
page loads and partial format.  The same bar as the matrix-core form: the fp64
oracle within max-abs 1e-2 and normalised 1e-2, and the exact structured cases
(single token, V = 1, poison, relocation, equal queries).  Calls that the form
cannot serve are refused.
"""

import math
import sys

import numpy as np
import pytest
import torch

import synth
from helpers import Case, build_gpu, to_device, to_host, tolerance_check

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda", 0)


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run(case: Case, dev, poison=False, waves=None, vector=True):
    _say("vector decode case: D=%d Hq=%d Hkv=%d NL=%d layer=%d lens=%s waves=%s vector=%s" % (
        case.head_dim, case.num_q_heads, case.num_kv_heads, case.num_layers, case.layer,
        case.seq_lens[:8], waves, vector))
    pool = build_gpu(case, dev, poison=poison)
    pool.set_combine(False)
    pool.set_compute(vector)
    if waves:
        pool.set_waves(waves)
    q = to_device(case.q, case.dtype, dev)
    sl = torch.tensor(case.seq_lens, dtype=torch.int32, device=dev)
    out = pool.decode(case.layer, q, sl)
    torch.cuda.synchronize()
    res = to_host(out)
    pool.close()
    return res


@pytest.mark.parametrize("D,hq,hkv", [(128, 32, 4), (64, 8, 2), (128, 4, 4), (64, 6, 2), (128, 7, 1),
                                      (128, 32, 8), (64, 16, 16)])
def test_ragged_lengths(dev, D, hq, hkv):
    """Groups of 8, 4, 1, 3 and 7 query heads; lengths across page boundaries."""
    case = Case(1, hq, hkv, D, "bf16", [1, 15, 16, 17, 31, 33, 100, 1000, 4097, 250], seed=31)
    err, norm = tolerance_check(_run(case, dev), case.oracle_out())
    _say("vector ragged D=%d G=%d: abs %.3g norm %.3g" % (D, hq // hkv, err, norm))


@pytest.mark.parametrize("waves", [1, 7, 768, 5000])
def test_split_invariance(dev, waves):
    """One wave for everything, a few, the default grid, and more waves than
    pages (one page per wave): the oracle's answer within tolerance."""
    case = Case(1, 32, 4, 128, "bf16", [5000, 16, 1, 777, 3000, 48], seed=32)
    tolerance_check(_run(case, dev, waves=waves), case.oracle_out())


def test_agrees_with_matrix_cores(dev):
    """Layer shape at reduced batch with the benchmark's value scale: both forms
    match the oracle, and they differ by at most one bf16 unit in the last place
    of the largest output (they round different float32 sums)."""
    rng = np.random.default_rng(33)
    lens = [int(x) for x in rng.integers(8192, 32768, size=4, endpoint=True)]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=33, value_scale=1 / math.sqrt(128), slack=1.25)
    vec = _run(case, dev, vector=True)
    mat = _run(case, dev, vector=False)
    ref = case.oracle_out()
    tolerance_check(vec, ref)
    tolerance_check(mat, ref)
    diff = float(np.max(np.abs(vec - mat)) / np.max(np.abs(ref)))
    _say("vector vs matrix: normalised difference %.3g" % diff)
    assert diff <= 2 ** -7


def test_poison_outside_valid_tokens(dev):
    """NaN in every slot that is not a valid token: finite, bitwise equal output."""
    case = Case(1, 16, 2, 128, "bf16", [1, 17, 45, 300, 16], seed=34)
    clean = _run(case, dev)
    dirty = _run(case, dev, poison=True)
    assert np.all(np.isfinite(dirty))
    assert np.array_equal(clean, dirty)


def test_relocation_is_bitwise_invariant(dev):
    lens = [3000, 17, 900, 4096]
    a = Case(1, 32, 4, 128, "bf16", lens, seed=35, slack=3.0)
    rng = np.random.default_rng(36)
    perm = rng.permutation(a.hot_pages).astype(np.int32)
    placement, off = [], 0
    for L in lens:
        n = synth.pages_for(L)
        placement.append(perm[off:off + n])
        off += n
    b = Case(1, 32, 4, 128, "bf16", lens, seed=35, placement=placement, hot_pages=a.hot_pages)
    assert np.array_equal(_run(a, dev), _run(b, dev))


def test_single_token_and_constant_v(dev):
    """L = 1 returns v_0 exactly; V = 1 everywhere gives exactly 1."""
    case = Case(1, 32, 4, 128, "bf16", [1, 1, 1], seed=37)
    got = _run(case, dev)
    for b in range(3):
        v0 = synth.bf16_bits_to_f32(case.kv[b][1][0]).astype(np.float64)
        for h in range(32):
            assert np.array_equal(got[b, h], v0[h // 8])
    case = Case(1, 32, 4, 128, "bf16", [5, 333, 4099, 16], seed=38)
    for b in range(case.batch):
        k, v = case.kv[b]
        case.kv[b] = (k, np.full_like(v, synth.f32_to_bf16_bits(np.float32(1.0))))
    assert np.all(_run(case, dev) == 1.0)


def test_identical_keys_give_mean_of_values(dev):
    """All keys of a (row, KV head) equal: the output is the mean of V within a
    bf16 half-unit (P3); see the matrix-core test for the rounding argument."""
    lens = [1000, 37, 5000, 16, 1]
    case = Case(1, 32, 4, 128, "bf16", lens, seed=42)
    for b in range(case.batch):
        k, v = case.kv[b]
        case.kv[b] = (np.broadcast_to(k[:1], k.shape).copy(), v)
    got = _run(case, dev)
    for b in range(case.batch):
        mean = synth.bf16_bits_to_f32(case.kv[b][1]).astype(np.float64).mean(axis=0)
        for h in range(32):
            want = mean[h // 8]
            assert np.all(np.abs(got[b, h] - want) <= 2 ** -8 * np.abs(want) + 1e-6)


def test_gqa_rows_identical_for_equal_queries(dev):
    case = Case(1, 32, 4, 128, "bf16", [2500, 60], seed=39)
    for b in range(case.batch):
        for g in range(4):
            case.q[b, g * 8:(g + 1) * 8] = case.q[b, g * 8]
    got = _run(case, dev)
    for b in range(case.batch):
        for h in range(32):
            assert np.array_equal(got[b, h], got[b, (h // 8) * 8])


@pytest.mark.parametrize("where", [0, 15, 16, 19999])
def test_needle(dev, where):
    """One key aligned with the query with a score gap of 40+: the output is its value."""
    L = 20000
    case = Case(1, 32, 4, 128, "bf16", [L, 4000], seed=40, value_scale=0.05)
    g = 1
    q = synth.bf16_bits_to_f32(case.q[0, g * 8]).astype(np.float64)
    case.q[0, g * 8:(g + 1) * 8] = case.q[0, g * 8]
    k, v = case.kv[0]
    k, v = k.copy(), v.copy()
    k[where, g] = synth.f32_to_bf16_bits((60.0 * math.sqrt(128) * q / np.dot(q, q)).astype(np.float32))
    v[where, g] = synth.f32_to_bf16_bits(np.linspace(-1, 1, 128).astype(np.float32))
    case.kv[0] = (k, v)
    got = _run(case, dev)
    want = synth.bf16_bits_to_f32(v[where, g]).astype(np.float64)
    for h in range(g * 8, (g + 1) * 8):
        assert np.max(np.abs(got[0, h] - want)) <= 2 ** -8 * np.max(np.abs(want))
    tolerance_check(got, case.oracle_out())


def test_zero_length_and_bad_rows(dev):
    """L = 0 gives zeros; an out-of-range page id and a length beyond the row
    give NaN rows; the other rows are unchanged."""
    case = Case(1, 8, 2, 64, "bf16", [40, 0, 70], seed=41)
    pool = build_gpu(case, dev)
    pool.set_compute(True)
    q = to_device(case.q, "bf16", dev)
    sl = torch.tensor([40, 0, 70], dtype=torch.int32, device=dev)
    out = to_host(pool.decode(0, q, sl))
    torch.cuda.synchronize()
    assert np.all(out[1] == 0)
    tolerance_check(out[[0, 2]], case.oracle_out(rows=[0, 2]))
    pt = pool.page_table[:3].clone()
    pt[2, 1] = case.hot_pages + 1000
    bad = torch.tensor([40, 16 * case.stride + 1, 70], dtype=torch.int32, device=dev)
    out2 = to_host(pool.decode(0, q, bad, page_table=pt))
    torch.cuda.synchronize()
    assert np.all(np.isnan(out2[1])) and np.all(np.isnan(out2[2]))
    assert np.array_equal(out2[0], out[0])
    pool.close()


@pytest.mark.parametrize("cold", ["device", "host"])
def test_reads_spilled_pages(dev, cold):
    """The tiered form: pages named KV_PAGE_COLD are read from the cold tier."""
    from test_gpu_spill import LENS, _oracle, _spilled_pool
    _say("vector decode of spilled pages, cold tier in %s memory" % cold)
    pool = _spilled_pool(dev, cold, LENS, hot_pages=30)
    pool.set_compute(True)
    table = pool.gather_table(torch.arange(len(LENS), dtype=torch.int32, device=dev))
    sl = torch.tensor(LENS, dtype=torch.int32, device=dev)
    for layer in (0, 1):
        case = _oracle(LENS, layer)
        got = to_host(pool.decode(layer, to_device(case.q, "bf16", dev), sl, page_table=table))
        torch.cuda.synchronize()
        tolerance_check(got, case.oracle_out())
    pool.close()


def test_refused_calls(dev):
    """More than 8 query heads per KV head, a float32 pool and the fused merge
    are refused with KV_ERR_INVALID; the matrix-core form serves the same calls."""
    from paper_2609_25782_amd import hotcold_kv as kv
    from paper_2609_25782_amd.pool import HotColdPool
    for dtype, hq, fused in (("bf16", 32, False), ("f32", 8, False), ("bf16", 8, True)):
        pool = HotColdPool(1, 2, 64, dtype, 8, 0, 1, 4)
        pool.hot.zero_()
        pool.set_compute(True)
        pool.set_combine(fused)
        assert pool.create_session(20) == 0
        q = torch.zeros((1, hq, 64), dtype=pool.torch_dtype, device=dev)
        sl = torch.tensor([20], dtype=torch.int32, device=dev)
        with pytest.raises(kv.KVError) as e:
            pool.decode(0, q, sl)
        assert e.value.status == kv.KV_ERR_INVALID
        pool.set_compute(False)
        out = pool.decode(0, q, sl)
        torch.cuda.synchronize()
        assert torch.all(out.float() == 0)
        with pytest.raises(kv.KVError):
            kv.kv_pool_set_decode_compute(pool.handle, 2)
        pool.close()
