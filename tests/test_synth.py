"""The seeded input generator: SplitMix64 against its published outputs, bf16
rounding, and the distribution of the generated values (CPU only)."""

import numpy as np

import synth


def test_splitmix64_reference_outputs():
    # SplitMix64 seeded with 0 produces 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, ...
    # (Steele, Lea and Flood 2014; the same values as Vigna's splitmix64.c)
    z0 = synth._mix(np.array([0], np.uint64))[0]
    z1 = synth._mix(np.array([synth.GOLDEN], np.uint64))[0]
    assert int(z0) == 0xE220A8397B1DCDAF
    assert int(z1) == 0x6E789E6AA1B965F4


def test_bf16_round_to_nearest_even():
    f = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -9, -2.5], np.float32)
    b = synth.f32_to_bf16_bits(f)
    back = synth.bf16_bits_to_f32(b)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6
    assert list(back) == [1.0, 1.0, 1.0 + 2.0 ** -6, 1.0, -2.5]


def test_values_are_roughly_standard_normal():
    c = synth.coord(synth.KIND_K, 3, 0, 1, np.arange(200000, dtype=np.uint64), 5)
    v = synth.values_f32(123, c, 1.0).astype(np.float64)
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1.0) < 0.01
    assert np.abs(v).max() < 3.47


def test_workload_placements_are_disjoint():
    w = synth.config_layer(0)
    pages = np.concatenate(w.placement)
    assert len(pages) == len(set(pages.tolist())) and pages.max() < w.hot_pages
    assert all(len(p) == synth.pages_for(L) for p, L in zip(w.placement, w.seq_lens))
    assert w.seq_lens.min() >= 8192 and w.seq_lens.max() <= 32768


def test_c_generator_equals_numpy_generator():
    """The C form of the generator gives the numpy form's bits: bf16 and f32, odd
    sizes, high session, layer and token fields, several scales."""
    for seed, sid, L, layer, hkv, d, scale, dt in (
            (0, 0, 1, 0, 1, 64, 1.0, "f32"), (7, 3, 37, 2, 4, 128, 0.0884, "bf16"),
            (2 ** 40 + 5, 1048575, 19, 63, 2, 64, 1.0, "bf16"), (11, 900, 300, 47, 4, 128, 1.0, "f32"),
            (3, 5, 5000, 0, 4, 128, 1 / 128 ** 0.5, "bf16")):
        a = synth.session_kv(seed, sid, L, layer, hkv, d, scale, dt)
        b = synth.session_kv_numpy(seed, sid, L, layer, hkv, d, scale, dt)
        for x, y in zip(a, b):
            assert x.dtype == y.dtype and x.shape == y.shape == (L, hkv, d)
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    # token fields up to 2^23 - 1
    a = synth.session_kv(1, 2, 1, 3, 1, 64, 1.0, "bf16")
    c = synth.coord(synth.KIND_K, 2, 3, 0, 0, np.arange(64, dtype=np.uint64))
    assert np.array_equal(a[0][0, 0], synth.f32_to_bf16_bits(synth.values_f32(1, c, 1.0)))
