"""Pins for the fp64 paged-attention oracle (CPU only).

Each test fixes the oracle against something other than itself: a separately
written dense routine on tiny inputs, closed forms, invariants, the paper's
printed shape numbers and hand-computed layout offsets.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_case(rng, dtype, num_layers, hkv, g, d, lens, layer, poison=False, shift=None):
    """Build a host pool for random logical K/V; returns everything the oracle needs
    plus the logical tensors for the dense check."""
    e = oracle.elt_bytes(dtype)
    npages_needed = sum((L + 15) // 16 for L in lens)
    num_pages = npages_needed + 3
    pb = oracle.page_bytes(num_layers, hkv, d, dtype)
    pool = np.zeros(num_pages * pb, dtype=np.uint8)
    if poison:
        # every byte of the pool starts as NaN; only valid tokens get overwritten
        if dtype == oracle.BF16:
            pool.view(np.uint16)[:] = 0x7FC0
        else:
            pool.view(np.float32)[:] = np.nan
    perm = rng.permutation(num_pages)
    stride = max((L + 15) // 16 for L in lens) + 2
    pt = np.full((len(lens), stride), -1, dtype=np.int32)
    ks, vs, off = [], [], 0
    for b, L in enumerate(lens):
        n = (L + 15) // 16
        pages = perm[off:off + n]
        off += n
        pt[b, :n] = pages
        k = rng.standard_normal((L, hkv, d)).astype(np.float32)
        v = rng.standard_normal((L, hkv, d)).astype(np.float32)
        if shift is not None:
            # keys and shift on a 2^-8 grid well inside float32 range: k + c is exact
            k = np.round(k * 256) / 256 + shift[None, :, :]
        if dtype == oracle.BF16:
            kb, vb = synth.f32_to_bf16_bits(k), synth.f32_to_bf16_bits(v)
            oracle.pack_pool(pool, num_layers, hkv, d, dtype, layer, pages, kb, vb)
            k, v = synth.bf16_bits_to_f32(kb), synth.bf16_bits_to_f32(vb)
        else:
            oracle.pack_pool(pool, num_layers, hkv, d, dtype, layer, pages, k, v)
        ks.append(k.astype(np.float64))
        vs.append(v.astype(np.float64))
    q = rng.standard_normal((len(lens), hkv * g, d)).astype(np.float32)
    if dtype == oracle.BF16:
        qs = synth.f32_to_bf16_bits(q)
        q64 = synth.bf16_bits_to_f32(qs).astype(np.float64)
    else:
        qs, q64 = q, q.astype(np.float64)
    return pool, num_pages, pt, np.array(lens, np.int32), qs, q64, ks, vs


def _dense(q64, ks, vs, g, scale):
    """Textbook attention on dense per-session K/V: softmax(scale q K^T) V, by numpy."""
    B, Hq, D = q64.shape
    out = np.zeros((B, Hq, D))
    for b in range(B):
        for h in range(Hq):
            K = ks[b][:, h // g, :]
            V = vs[b][:, h // g, :]
            if K.shape[0] == 0:
                continue
            s = scale * (K @ q64[b, h])
            w = np.exp(s - s.max())
            out[b, h] = (w / w.sum()) @ V
    return out


@pytest.mark.parametrize("dtype", [oracle.BF16, oracle.F32])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("hkv,g", [(1, 1), (1, 4), (2, 2), (4, 8)])
def test_p1_brute_force_dense(dtype, d, hkv, g):
    rng = np.random.default_rng(1000 + d + 10 * hkv + g + 7 * dtype)
    lens = [1, 15, 16, 17, 31, 32, 33, int(rng.integers(40, 200))]
    num_layers, layer = 3, 2
    scale = 1.0 / math.sqrt(d)
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, dtype, num_layers, hkv, g, d, lens, layer)
    got = oracle.paged_attention(pool, npg, num_layers, hkv, d, dtype, layer, qs, pt, sl, scale)
    ref = _dense(q64, ks, vs, g, scale)
    assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


def test_p1_other_layers_untouched():
    """Writing layer 0 and reading layer 1 must see only layer 1's data."""
    rng = np.random.default_rng(5)
    d, hkv, g = 64, 2, 2
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, oracle.F32, 2, hkv, g, d, [20, 40], 1)
    # overwrite layer 0 with different values: layer-1 results must not change
    before = oracle.paged_attention(pool, npg, 2, hkv, d, oracle.F32, 1, qs, pt, sl, 0.125)
    for b, L in enumerate([20, 40]):
        n = (L + 15) // 16
        junk = rng.standard_normal((L, hkv, d)).astype(np.float32) * 100
        oracle.pack_pool(pool, 2, hkv, d, oracle.F32, 0, pt[b, :n], junk, junk)
    after = oracle.paged_attention(pool, npg, 2, hkv, d, oracle.F32, 1, qs, pt, sl, 0.125)
    assert np.array_equal(before, after)


@pytest.mark.parametrize("dtype", [oracle.BF16, oracle.F32])
def test_p2_single_token_returns_v(dtype):
    rng = np.random.default_rng(2)
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, dtype, 1, 2, 4, 128, [1, 1], 0)
    got = oracle.paged_attention(pool, npg, 1, 2, 128, dtype, 0, qs, pt, sl, 0.3)
    for b in range(2):
        for h in range(8):
            assert np.array_equal(got[b, h], vs[b][0, h // 4])


def test_p3_identical_keys_give_mean_of_v():
    rng = np.random.default_rng(3)
    d, hkv, g, L = 128, 1, 8, 77
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, oracle.F32, 1, hkv, g, d, [L], 0)
    k0 = rng.standard_normal((1, hkv, d)).astype(np.float32)
    v = rng.standard_normal((L, hkv, d)).astype(np.float32)
    oracle.pack_pool(pool, 1, hkv, d, oracle.F32, 0, pt[0, :(L + 15) // 16],
                     np.repeat(k0, L, axis=0), v)
    got = oracle.paged_attention(pool, npg, 1, hkv, d, oracle.F32, 0, qs, pt, sl, 0.5)
    mean = v.astype(np.float64).mean(axis=0)[0]
    for h in range(g):
        assert np.max(np.abs(got[0, h] - mean)) <= 1e-13


@pytest.mark.parametrize("dtype", [oracle.BF16, oracle.F32])
def test_p4_weights_sum_to_one(dtype):
    rng = np.random.default_rng(4)
    lens = [1, 16, 33, 150]
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, dtype, 1, 2, 2, 64, lens, 0)
    out, w = oracle.paged_attention(pool, npg, 1, 2, 64, dtype, 0, qs, pt, sl, 2.0,
                                    return_weights=True)
    for b, L in enumerate(lens):
        for h in range(4):
            assert abs(w[b, h, :L].sum() - 1.0) <= 1e-12
            assert np.all(w[b, h, :L] >= 0) and np.all(w[b, h, L:] == 0)


def test_two_token_closed_form():
    """L = 2: out = sigma(s0 - s1) v0 + sigma(s1 - s0) v1 with s_t = scale q.k_t."""
    rng = np.random.default_rng(6)
    d = 64
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, oracle.F32, 1, 1, 1, d, [2], 0)
    scale = 0.37
    s0 = scale * float(np.dot(q64[0, 0], ks[0][0, 0]))
    s1 = scale * float(np.dot(q64[0, 0], ks[0][1, 0]))
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    w1 = 1.0 / (1.0 + math.exp(s0 - s1))
    expect = w0 * vs[0][0, 0] + w1 * vs[0][1, 0]
    got = oracle.paged_attention(pool, npg, 1, 1, d, oracle.F32, 0, qs, pt, sl, scale)
    assert np.max(np.abs(got[0, 0] - expect)) <= 1e-13


@pytest.mark.parametrize("where", ["first", "page_end", "page_start", "last", "random"])
def test_p5_needle(where):
    """A key aligned with the query and a score gap of 40+ picks out its value."""
    rng = np.random.default_rng(7)
    d, hkv, g, L = 128, 2, 4, 300
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, oracle.F32, 1, hkv, g, d, [L], 0)
    t_star = {"first": 0, "page_end": 15, "page_start": 16, "last": L - 1,
              "random": int(rng.integers(0, L))}[where]
    k = (rng.standard_normal((L, hkv, d)) * 0.01).astype(np.float32)
    v = rng.standard_normal((L, hkv, d)).astype(np.float32)
    gq = 1
    qvec = q64[0, gq * g]
    # same query for the whole group so the needle is strongest for each head of it
    q_all = np.array(qs, copy=True)
    q_all[0, gq * g:(gq + 1) * g] = qs[0, gq * g]
    k[t_star, gq] = (60.0 * qvec / np.dot(qvec, qvec)).astype(np.float32)
    oracle.pack_pool(pool, 1, hkv, d, oracle.F32, 0, pt[0, :(L + 15) // 16], k, v)
    got = oracle.paged_attention(pool, npg, 1, hkv, d, oracle.F32, 0, q_all, pt, sl, 1.0)
    for h in range(gq * g, (gq + 1) * g):
        ref = v[t_star, gq].astype(np.float64)
        assert np.max(np.abs(got[0, h] - ref)) <= 1e-6 * np.max(np.abs(ref))


@pytest.mark.parametrize("dtype", [oracle.BF16, oracle.F32])
def test_p6_poison_outside_valid_tokens(dtype):
    rng = np.random.default_rng(8)
    lens = [1, 17, 45]
    case_clean = _rand_case(np.random.default_rng(8), dtype, 2, 2, 2, 64, lens, 1)
    case_poison = _rand_case(np.random.default_rng(8), dtype, 2, 2, 2, 64, lens, 1, poison=True)
    outs = []
    for pool, npg, pt, sl, qs, q64, ks, vs in (case_clean, case_poison):
        outs.append(oracle.paged_attention(pool, npg, 2, 2, 64, dtype, 1, qs, pt, sl, 0.125))
    assert np.all(np.isfinite(outs[1]))
    assert np.array_equal(outs[0], outs[1])


def test_p9_key_shift_invariance():
    rng = np.random.default_rng(9)
    d, hkv, g = 64, 2, 2
    lens = [5, 40, 97]
    shift = (np.round(rng.standard_normal((hkv, d)) * 3 * 256) / 256).astype(np.float32)
    a = _rand_case(np.random.default_rng(10), oracle.F32, 1, hkv, g, d, lens, 0,
                   shift=np.zeros((hkv, d), np.float32))
    b = _rand_case(np.random.default_rng(10), oracle.F32, 1, hkv, g, d, lens, 0, shift=shift)
    oa = oracle.paged_attention(a[0], a[1], 1, hkv, d, oracle.F32, 0, a[4], a[2], a[3], 0.2)
    ob = oracle.paged_attention(b[0], b[1], 1, hkv, d, oracle.F32, 0, b[4], b[2], b[3], 0.2)
    assert np.max(np.abs(oa - ob)) <= 1e-12 * max(1.0, np.max(np.abs(oa)))


def test_zero_length_gives_zero_and_bad_page_rejected():
    rng = np.random.default_rng(11)
    pool, npg, pt, sl, qs, q64, ks, vs = _rand_case(rng, oracle.F32, 1, 1, 2, 64, [3, 20], 0)
    sl2 = sl.copy()
    sl2[0] = 0
    out = oracle.paged_attention(pool, npg, 1, 1, 64, oracle.F32, 0, qs, pt, sl2, 1.0)
    assert np.all(out[0] == 0)
    pt2 = pt.copy()
    pt2[1, 1] = npg + 5
    with pytest.raises(ValueError):
        oracle.paged_attention(pool, npg, 1, 1, 64, oracle.F32, 0, qs, pt2, sl, 1.0)


def test_layout_offsets_hand_computed():
    """Documented page layout, evaluated by hand for a few elements."""
    # bf16, 2 layers, 4 KV heads, d=128: tile = 16*128*2 = 4096 B, page = 2*4*2*4096 = 65536 B
    assert oracle.page_bytes(2, 4, 128, oracle.BF16) == 65536
    # K of page 3, layer 1, head 2, token 5, dim 9: x = 8 -> ((9//8)*16 + 5)*8 + 1 = 169 elements
    expect = 3 * 65536 + ((1 * 4 + 2) * 2 + 0) * 4096 + 169 * 2
    assert oracle.elem_offset(2, 4, 128, oracle.BF16, 3, 1, 2, 0, 5, 9) == expect
    # V of the same element: d * 16 + t = 9*16 + 5 = 149 elements after the K tile
    expect_v = 3 * 65536 + ((1 * 4 + 2) * 2 + 1) * 4096 + 149 * 2
    assert oracle.elem_offset(2, 4, 128, oracle.BF16, 3, 1, 2, 1, 5, 9) == expect_v
    # f32, d=64: x = 4; K(t=15, d=63) -> ((63//4)*16 + 15)*4 + 3 = (240+15)*4+3 = 1023 elements
    assert oracle.elem_offset(1, 1, 64, oracle.F32, 0, 0, 0, 0, 15, 63) == 1023 * 4


def test_pack_pool_matches_accessor():
    rng = np.random.default_rng(12)
    num_layers, hkv, d, dtype = 3, 2, 64, oracle.BF16
    pb = oracle.page_bytes(num_layers, hkv, d, dtype)
    pool = np.zeros(6 * pb, np.uint8)
    L = 40
    pages = np.array([4, 0, 2])
    k = rng.integers(0, 65535, size=(L, hkv, d), dtype=np.uint16)
    v = rng.integers(0, 65535, size=(L, hkv, d), dtype=np.uint16)
    oracle.pack_pool(pool, num_layers, hkv, d, dtype, 2, pages, k, v)
    for _ in range(200):
        t, g, dd = int(rng.integers(L)), int(rng.integers(hkv)), int(rng.integers(d))
        for kind, arr in ((0, k), (1, v)):
            off = oracle.elem_offset(num_layers, hkv, d, dtype, int(pages[t // 16]), 2, g, kind, t % 16, dd)
            assert pool[off:off + 2].view(np.uint16)[0] == arr[t, g, dd]


def test_c_packer_equals_numpy_packer():
    """The C packer (used for the full-size workloads) writes exactly the numpy
    packer's bytes, over random page lists, both dtypes, ragged lengths and
    every layer of a 3-layer pool; untouched bytes stay untouched."""
    rng = np.random.default_rng(13)
    for dtype, store, hkv, d in ((oracle.BF16, np.uint16, 4, 128), (oracle.F32, np.float32, 2, 64),
                                 (oracle.BF16, np.uint16, 1, 64)):
        pb = oracle.page_bytes(3, hkv, d, dtype)
        for L in (1, 15, 16, 17, 100):
            n = (L + 15) // 16
            pages = rng.permutation(n + 3)[:n].astype(np.int32)
            for layer in range(3):
                if store is np.uint16:
                    k = rng.integers(0, 65535, size=(L, hkv, d), dtype=np.uint16)
                    v = rng.integers(0, 65535, size=(L, hkv, d), dtype=np.uint16)
                else:
                    k = rng.standard_normal((L, hkv, d)).astype(np.float32)
                    v = rng.standard_normal((L, hkv, d)).astype(np.float32)
                a = rng.integers(0, 256, size=(n + 3) * pb, dtype=np.uint8)
                b = a.copy()
                oracle.pack_pool(a, 3, hkv, d, dtype, layer, pages, k, v)
                oracle.pack_session(b, 3, hkv, d, dtype, layer, pages, k, v)
                assert np.array_equal(a, b)


def test_p12_paper_shape_numbers():
    """96 KiB of KV per token and 1.5 MiB per 16-token page at 48 layers x 4 KV heads x 128, bf16."""
    with open(os.path.join(GOLDEN, "paper_numbers.json")) as f:
        gold = json.load(f)
    assert oracle.kv_bytes_per_token(48, 4, 128, oracle.BF16) == gold["kv_bytes_per_token"]["value"]
    assert oracle.page_bytes(48, 4, 128, oracle.BF16) == gold["kv_block_bytes"]["value"]
    assert gold["kv_block_bytes"]["value"] // gold["kv_bytes_per_token"]["value"] == oracle.PAGE_SIZE
