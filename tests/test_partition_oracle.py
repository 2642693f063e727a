"""Pins for the reference work split (CPU only): exact cover, balance, and the
closed form for the first and last wave of a segment that the GPU uses."""

import numpy as np
import pytest

from oracle import partition


def _closed_form_waves(a, e, T, N):
    # wave containing unit u: the largest k with floor(k T / N) <= u
    first = ((a + 1) * N - 1) // T
    last = (e * N - 1) // T
    return first, last


@pytest.mark.parametrize("seed", range(6))
def test_exact_cover_and_balance(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 9))
    hkv = int(rng.choice([1, 2, 4]))
    lens = [int(x) for x in rng.integers(0, 300, size=B)]
    if seed == 0:
        lens[0] = 0
    N = int(rng.integers(1, 40))
    ps = partition.pieces(lens, hkv, N)
    seen = set()
    per_wave = [0] * N
    slots = set()
    for slot, k, b, g, p0, p1 in ps:
        assert p0 < p1 and slot == k + b * hkv + g and slot not in slots
        slots.add(slot)
        for i in range(p0, p1):
            assert (b, g, i) not in seen
            seen.add((b, g, i))
        per_wave[k] += p1 - p0
    total = sum(hkv * ((L + 15) // 16) for L in lens)
    assert len(seen) == total
    assert all(x in (total // N, -(-total // N)) for x in per_wave)


def test_closed_form_matches_enumeration():
    rng = np.random.default_rng(11)
    for _ in range(300):
        B, hkv, N = int(rng.integers(1, 6)), int(rng.choice([1, 4])), int(rng.integers(1, 120))
        lens = [int(x) for x in rng.integers(1, 200, size=B)]
        n = [(L + 15) // 16 for L in lens]
        T = hkv * sum(n)
        ps = partition.pieces(lens, hkv, N)
        base = 0
        for b in range(B):
            for g in range(hkv):
                a = base + g * n[b]
                e = a + n[b]
                waves = sorted(k for _s, k, bb, gg, _p0, _p1 in ps if (bb, gg) == (b, g))
                first, last = _closed_form_waves(a, e, T, N)
                # waves in [first, last] with an empty range of their own (N > T) make no piece
                nonempty = [k for k in range(first, last + 1) if (k * T) // N < ((k + 1) * T) // N]
                assert waves == nonempty
            base += hkv * n[b]


def test_slot_table_small_example():
    # two sessions of 20 and 40 tokens (2 and 3 pages), one KV head, two waves:
    # units = (0,0,0) (0,0,1) (1,0,0) (1,0,1) (1,0,2); T = 5; wave 0 = [0,2), wave 1 = [2,5)
    t = partition.slot_table([20, 40], 1, 2)
    assert t == [(0, 0, 0, 2), (-1, -1, 0, 0), (1, 0, 0, 3), (-1, -1, 0, 0)]
    # three waves: bounds 0,1,3,5 -> wave 0: (0,0,0); wave 1: (0,0,1),(1,0,0); wave 2: (1,0,1..2)
    t = partition.slot_table([20, 40], 1, 3)
    assert t == [(0, 0, 0, 1), (0, 0, 1, 2), (1, 0, 0, 1), (1, 0, 1, 3), (-1, -1, 0, 0)]
