"""Pins for the reference work split (CPU only): exact cover, balance, the
closed form for the first and last worker of a segment that the GPU uses, and
hand-worked tables for both group widths."""

import numpy as np
import pytest

from oracle import partition


def _closed_form_workers(a, e, T, N):
    # worker containing unit u: the largest k with floor(k T / N) <= u
    first = ((a + 1) * N - 1) // T
    last = (e * N - 1) // T
    return first, last


def test_group_width_rule():
    assert partition.group_waves(4, 768) == 4
    assert partition.group_waves(8, 4) == 4
    assert partition.group_waves(4, 7) == 1
    assert partition.group_waves(2, 768) == 1
    assert partition.group_waves(1, 8) == 1


@pytest.mark.parametrize("seed", range(10))
def test_exact_cover_and_balance(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 9))
    hkv = int(rng.choice([1, 2, 4, 8]))
    lens = [int(x) for x in rng.integers(0, 300, size=B)]
    if seed == 0:
        lens[0] = 0
    N = int(rng.integers(1, 40)) * (4 if seed % 2 else 1)
    L = partition.group_waves(hkv, N)
    ps = partition.pieces(lens, hkv, N)
    seen = set()
    per_wave = [0] * N
    slots = set()
    last_slot = -1
    for slot, k, b, g, p0, p1 in ps:
        worker, w = divmod(k, L)
        assert w == g % L
        assert p0 < p1 and slot == (worker + b * (hkv // L) + g // L) * L + w and slot not in slots
        assert slot > last_slot and slot < N + B * hkv
        last_slot = slot
        slots.add(slot)
        for i in range(p0, p1):
            assert (b, g, i) not in seen
            seen.add((b, g, i))
        per_wave[k] += p1 - p0
    total = sum(hkv * ((x + 15) // 16) for x in lens)
    assert len(seen) == total
    units, workers = total // L, N // L
    assert all(x in (units // workers, -(-units // workers)) for x in per_wave)
    # the waves of one worker take the same pages of their own KV heads
    for k in range(0, N, L):
        runs = [sorted((b, p0, p1) for _s, kk, b, _g, p0, p1 in ps if kk == k + w) for w in range(L)]
        assert all(r == runs[0] for r in runs)


def test_closed_form_matches_enumeration():
    rng = np.random.default_rng(11)
    for _ in range(300):
        B, hkv = int(rng.integers(1, 6)), int(rng.choice([1, 4, 8]))
        N = int(rng.integers(1, 120))
        lens = [int(x) for x in rng.integers(1, 200, size=B)]
        L = partition.group_waves(hkv, N)
        groups, workers = hkv // L, N // L
        n = [(x + 15) // 16 for x in lens]
        T = groups * sum(n)
        ps = partition.pieces(lens, hkv, N)
        base = 0
        for b in range(B):
            for g in range(hkv):
                a = base + (g // L) * n[b]
                e = a + n[b]
                got = sorted(k // L for _s, k, bb, gg, _p0, _p1 in ps if (bb, gg) == (b, g))
                first, last = _closed_form_workers(a, e, T, workers)
                # workers in [first, last] with an empty range of their own (N > T) make no piece
                nonempty = [k for k in range(first, last + 1) if (k * T) // workers < ((k + 1) * T) // workers]
                assert got == nonempty
            base += groups * n[b]


def test_slot_table_small_examples():
    # two sessions of 20 and 40 tokens (2 and 3 pages), one KV head, two waves:
    # units = (0,0,0) (0,0,1) (1,0,0) (1,0,1) (1,0,2); T = 5; wave 0 = [0,2), wave 1 = [2,5)
    t = partition.slot_table([20, 40], 1, 2)
    assert t == [(0, 0, 0, 2), (-1, -1, 0, 0), (1, 0, 0, 3), (-1, -1, 0, 0)]
    # three waves: bounds 0,1,3,5 -> wave 0: (0,0,0); wave 1: (0,0,1),(1,0,0); wave 2: (1,0,1..2)
    t = partition.slot_table([20, 40], 1, 3)
    assert t == [(0, 0, 0, 1), (0, 0, 1, 2), (1, 0, 0, 1), (1, 0, 1, 3), (-1, -1, 0, 0)]
    # four KV heads, eight waves: two workers of four waves over the same 5 units
    # (one head group); worker 0 = session 0's 2 pages, worker 1 = session 1's 3;
    # wave w takes head w; slots (k + s) * 4 + w with s = b
    t = partition.slot_table([20, 40], 4, 8)
    hole = (-1, -1, 0, 0)
    assert t == [(0, 0, 0, 2), (0, 1, 0, 2), (0, 2, 0, 2), (0, 3, 0, 2),
                 hole, hole, hole, hole,
                 (1, 0, 0, 3), (1, 1, 0, 3), (1, 2, 0, 3), (1, 3, 0, 3),
                 hole, hole, hole, hole]
