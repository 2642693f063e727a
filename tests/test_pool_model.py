"""Pins for the oracle's pool/session model (CPU only).

The model is fixed by a hand-worked trace of the documented policy, by the
invariants the paper states (write-on-evict writes an unmodified page to the
cold tier at most once, Sec. III; KV never changes once written, Sec. II) and
by conservation properties checked on random call sequences.
"""

import copy

import numpy as np
import pytest

from oracle.pool_model import (ACTIVE, ERR_INVALID, ERR_NO_COLD, ERR_NO_HOT, ERR_STATE, PAUSED,
                               ModelError, PoolModel)


def test_hand_worked_trace():
    m = PoolModel(num_hot=8, num_cold=6, max_sessions=3, max_pages_per_session=4)
    a = m.create(40)                 # 3 pages: lowest free hot ids
    b = m.create(16)                 # 1 page
    assert (a, b) == (0, 1)
    assert m.row(a) == [0, 1, 2, -1] and m.row(b) == [3, -1, -1, -1]
    copies = m.evict(a)              # all 3 pages dirty -> cold 0,1,2
    assert copies == [(0, 0), (1, 1), (2, 2)] and m.cold_writes == 3
    assert m.row(a) == [-1] * 4 and m.free_hot() == 7
    c = m.create(33)                 # reuses hot 0,1,2 (lowest)
    assert c == 2 and m.row(c) == [0, 1, 2, -1]
    res = m.resume([a])              # needs 3 hot pages: 4,5,6
    assert res == [[(0, 4), (1, 5), (2, 6)]] and m.row(a) == [4, 5, 6, -1]
    assert m.evict(a) == [] and m.cold_writes == 3      # clean: nothing written
    m.resume([a])
    m.write_tokens(a, 20, 1)         # token 20 lives in page 1 -> its cold copy dropped
    assert m.sessions[a].cold == [0, -1, 2]
    assert m.evict(a) == [(5, 1)] and m.cold_writes == 4  # page 1 rewritten into cold id 1


def test_exhaustion_leaves_state_unchanged():
    m = PoolModel(num_hot=4, num_cold=2, max_sessions=4, max_pages_per_session=4)
    a = m.create(48)
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:
        m.create(33)
    assert e.value.code == ERR_NO_HOT and m.__dict__ == before
    with pytest.raises(ModelError) as e:
        m.evict(a)                   # 3 dirty pages, 2 cold pages
    assert e.value.code == ERR_NO_COLD and m.__dict__ == before
    with pytest.raises(ModelError) as e:
        m.resume([a])
    assert e.value.code == ERR_STATE and m.__dict__ == before
    with pytest.raises(ModelError) as e:
        m.create(16 * 5)             # longer than a row
    assert e.value.code == ERR_INVALID and m.__dict__ == before


def test_batched_resume_is_atomic_and_ordered():
    m = PoolModel(num_hot=10, num_cold=10, max_sessions=4, max_pages_per_session=4)
    a, b = m.create(32), m.create(48)
    m.evict(a), m.evict(b)
    x = m.create(64)                 # takes hot 0..3, leaves 6 free
    before = copy.deepcopy(m.__dict__)
    m2 = copy.deepcopy(m)
    with pytest.raises(ModelError):
        m2.resume([a, b, x])         # x is active -> whole batch refused
    assert m2.__dict__ == before
    res = m.resume([b, a])           # b first: 3 lowest, then a: next 2
    assert res[0] == [(2, 4), (3, 5), (4, 6)] and res[1] == [(0, 7), (1, 8)]


def test_write_on_evict_at_most_once_per_page():
    """Paper Sec. III: an unmodified page is written to the cold tier once,
    however many times its session is evicted and resumed."""
    m = PoolModel(num_hot=64, num_cold=64, max_sessions=4, max_pages_per_session=16)
    sid = m.create(16 * 7 + 3)       # 8 pages
    for _ in range(5):
        m.evict(sid)
        m.resume([sid])
    assert m.cold_writes == 8


def test_random_sequences_conserve_pages():
    rng = np.random.default_rng(0)
    nh, nc, ms, stride = 40, 30, 6, 8
    m = PoolModel(nh, nc, ms, stride)
    for step in range(3000):
        op = rng.integers(0, 6)
        sid = int(rng.integers(0, ms))
        before = copy.deepcopy(m.__dict__)
        try:
            if op == 0:
                m.create(int(rng.integers(0, 16 * stride + 1)))
            elif op == 1:
                m.evict(sid)
            elif op == 2:
                k = int(rng.integers(1, 3))
                m.resume([int(x) for x in rng.choice(ms, size=k, replace=False)])
            elif op == 3:
                s = m.sessions[sid]
                if s.state == ACTIVE and s.seq_len:
                    t0 = int(rng.integers(0, s.seq_len))
                    m.write_tokens(sid, t0, int(rng.integers(0, s.seq_len - t0 + 1)))
            elif op == 4:
                m.destroy(sid)
            else:
                n = int(rng.integers(0, stride + 1))
                m.import_cold(16 * n, rng.choice(nc, size=n, replace=False))
        except ModelError:
            assert m.__dict__ == before
        # conservation and disjointness
        hot_used = [p for s in m.sessions if s.state == ACTIVE for p in s.hot]
        assert len(hot_used) == len(set(hot_used))
        assert len(hot_used) + m.free_hot() == nh
        assert set(hot_used).isdisjoint(m.hot_free)
        refs = [0] * nc
        for s in m.sessions:
            for c in s.cold:
                if c >= 0:
                    refs[c] += 1
        assert refs == m.cold_ref
        assert all((refs[c] == 0) == (c in m.cold_free) for c in range(nc))
        for s in m.sessions:
            if s.state == PAUSED:
                assert all(c >= 0 for c in s.cold)
            if s.state == ACTIVE:
                assert len(s.hot) == (s.seq_len + 15) // 16 == len(s.cold)


def test_batched_evict_is_atomic():
    m = PoolModel(num_hot=10, num_cold=5, max_sessions=4, max_pages_per_session=4)
    a, b = m.create(48), m.create(48)      # 3 + 3 dirty pages, only 5 cold pages
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:
        m.evict_many([a, b])
    assert e.value.code == ERR_NO_COLD and m.__dict__ == before
    assert m.evict_many([b]) == [(3, 0), (4, 1), (5, 2)]


def test_lru_hand_worked_trace():
    """Page-granular LRU (Sec. III): the longest-paused session's pages go first,
    in logical order; pages that still have a cold copy cost no write."""
    m = PoolModel(num_hot=8, num_cold=16, max_sessions=4, max_pages_per_session=8)
    a = m.create(16 * 3)          # hot 0,1,2
    b = m.create(16 * 3)          # hot 3,4,5
    m.pause(a)                    # paused first: least recently used
    m.pause(b)
    c = m.create(16 * 4)          # 2 free (6,7) -> evict a's pages 0,1 (hot 0,1)
    assert m.sessions[c].hot == [0, 1, 6, 7]
    assert m.sessions[a].hot == [-1, -1, 2] and m.sessions[a].cold == [0, 1, -1]
    assert m.cold_writes == 2 and m.lru_evicted == 2
    # resume a: fetches its 2 missing pages; a's resident page stays (hit 1 of 3)
    m.destroy(c)
    per = m.resume([a])
    assert per == [[(0, 0), (1, 1)]] and m.sessions[a].hot == [0, 1, 2]
    assert (m.resume_resident, m.resume_total) == (1, 3)
    # pause a again: now b is older; pages 0,1 of a are clean (cold copies valid)
    m.pause(a)
    n, copies = m.evict_pages(5)
    # b's three pages (dirty: written), then a's pages 0 and 1 (clean: no write)
    assert n == 5 and copies == [(3, 2), (4, 3), (5, 4)]
    assert m.sessions[a].hot == [-1, -1, 2] and m.sessions[a].cold == [0, 1, -1]
    assert m.cold_writes == 2 + 3 and m.lru_evicted == 2 + 5


def test_resume_hit_rate_and_no_self_eviction():
    m = PoolModel(num_hot=6, num_cold=16, max_sessions=3, max_pages_per_session=8)
    a = m.create(16 * 4)
    m.pause(a)
    assert m.resume([a]) == [[]] and (m.resume_resident, m.resume_total) == (4, 4)
    m.pause(a)
    assert m.evict_pages(3)[0] == 3           # a keeps page 3 resident
    b = m.create(16 * 5)                      # fills the pool: 5 of 5 free
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:      # needs 3 pages; only a's own page is evictable
        m.resume([a])
    assert e.value.code == ERR_NO_HOT and m.__dict__ == before
    m.pause(b)                                # now b's pages are evictable
    per = m.resume([a])
    assert [len(x) for x in per] == [3] and m.resume_resident == 4 + 1


def test_residency_invariant_on_random_sequences():
    rng = np.random.default_rng(7)
    nh, nc, ms, stride = 30, 60, 6, 8
    m = PoolModel(nh, nc, ms, stride)
    for step in range(4000):
        op, sid = int(rng.integers(0, 7)), int(rng.integers(0, ms))
        before = copy.deepcopy(m.__dict__)
        try:
            if op == 0:
                m.create(int(rng.integers(0, 16 * stride + 1)))
            elif op == 1:
                m.pause(sid)
            elif op == 2:
                m.resume([sid])
            elif op == 3:
                m.extend(sid, int(rng.integers(0, 16 * stride + 1)))
            elif op == 4:
                m.evict_pages(int(rng.integers(0, 6)))
            elif op == 5:
                m.evict(sid)
            else:
                m.destroy(sid)
        except ModelError:
            assert m.__dict__ == before
        used = [p for s in m.sessions for p in s.hot if p >= 0]
        assert len(used) == len(set(used)) and len(used) + m.free_hot() == nh
        for s in m.sessions:
            if s.state == ACTIVE:
                assert all(p >= 0 for p in s.hot) and len(s.hot) == (s.seq_len + 15) // 16
            if s.state == PAUSED:
                assert all(p >= 0 or c >= 0 for p, c in zip(s.hot, s.cold))


def test_spill_hand_worked_trace():
    """Spill (Sec. III: no pinning; blocks spill instead of failing): pages that
    find no hot page live in the cold tier, named in the row with the cold bit;
    promote brings them back by evicting paused pages first."""
    from oracle.pool_model import COLD_BIT as C
    m = PoolModel(num_hot=4, num_cold=10, max_sessions=3, max_pages_per_session=4, spill=True)
    a = m.create(16 * 3)                          # hot 0,1,2
    b = m.create(16 * 3)                          # hot 3, then two pages spill to cold 0,1
    assert m.row(b) == [3, 0 | C, 1 | C, -1] and m.sessions[b].cold == [-1, 0, 1]
    assert m.spilled_pages == 2 and m.free_hot() == 0
    m.pause(a)
    copies = m.promote(5)                         # evicts a's pages 0,1 (dirty -> cold 2,3)
    assert m.last_victim_copies == [(0, 2), (1, 3)] and copies == [(0, 0), (1, 1)]
    assert m.row(b) == [3, 0, 1, -1] and m.sessions[b].cold == [-1, 0, 1]
    assert m.row(a) == [-1, -1, 2, -1] and m.sessions[a].cold == [2, 3, -1]
    assert (m.cold_writes, m.lru_evicted, m.promoted_pages, m.pages_to_hot) == (2, 2, 2, 2)
    m.write_tokens(b, 16, 1)                      # resident page 1 loses its cold copy 0
    assert m.sessions[b].cold == [-1, -1, 1] and 0 in m.cold_free
    assert m.resume([a]) == [[]]                  # nothing evictable: both pages stay cold
    assert m.row(a) == [2 | C, 3 | C, 2, -1] and m.spilled_pages == 4
    assert (m.resume_resident, m.resume_total) == (1, 3)
    m.write_tokens(a, 0, 1)                       # in place in cold page 2
    assert m.sessions[a].cold == [2, 3, -1]
    assert m.evict(a) == [(2, 0)]                 # only the resident dirty page is written
    assert m.row(a) == [-1, -1, -1, -1] and m.sessions[a].cold == [2, 3, 0]
    assert m.cold_writes == 3


def test_spill_refusals_change_nothing():
    from oracle.pool_model import COLD_BIT as C
    m = PoolModel(num_hot=2, num_cold=4, max_sessions=4, max_pages_per_session=8, spill=True)
    a = m.create(16 * 4)                          # 2 hot + 2 spilled (cold 0,1)
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:
        m.create(16 * 3)                          # 3 pages to spill, 2 cold pages free
    assert e.value.code == ERR_NO_COLD and m.__dict__ == before
    b = m.import_cold(16, [2])
    c = m.import_cold(16, [2])                    # cold page 2 shared by b and c
    m.resume([b])                                 # no free or evictable hot page: stays cold
    assert m.row(b)[0] == 2 | C and m.sessions[a].hot == [0, 1, -1, -1]
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:          # a shared spilled page is not written in place
        m.write_tokens(b, 0, 1)
    assert e.value.code == ERR_STATE and m.__dict__ == before
    m.destroy(c)
    m.write_tokens(b, 0, 1)
    assert m.row(b)[0] == 2 | C and m.sessions[b].cold == [2]
    m.pause(a)
    assert m.promote(3) == [(2, 0)]               # a's page 0 is written to cold 3 first
    assert m.last_victim_copies == [(0, 3)] and m.row(b)[0] == 0
    before = copy.deepcopy(m.__dict__)
    with pytest.raises(ModelError) as e:          # a's dirty page 1 and one spilled page need
        m.extend(b, 16 * 3)                       # two cold pages; none is free
    assert e.value.code == ERR_NO_COLD and m.__dict__ == before


@pytest.mark.parametrize("seed", range(3))
def test_spill_invariants_on_random_sequences(seed):
    from oracle.pool_model import COLD_BIT as C
    rng = np.random.default_rng(100 + seed)
    nh, nc, ms, stride = 12, 80, 6, 8
    m = PoolModel(nh, nc, ms, stride, spill=True)
    spills = 0
    for step in range(3000):
        op, sid = int(rng.integers(0, 8)), int(rng.integers(0, ms))
        before = copy.deepcopy(m.__dict__)
        try:
            if op == 0:
                m.create(int(rng.integers(0, 16 * stride + 1)))
            elif op == 1:
                m.pause(sid)
            elif op == 2:
                m.resume([sid])
            elif op == 3:
                m.extend(sid, int(rng.integers(0, 16 * stride + 1)))
            elif op == 4:
                m.promote(int(rng.integers(0, 6)))
            elif op == 5:
                m.evict(sid)
            elif op == 6:
                s = m.sessions[sid]
                if s.state == ACTIVE and s.seq_len:
                    t0 = int(rng.integers(0, s.seq_len))
                    m.write_tokens(sid, t0, int(rng.integers(0, s.seq_len - t0 + 1)))
            else:
                m.destroy(sid)
        except ModelError:
            assert m.__dict__ == before
        spills = max(spills, m.spilled_pages)
        used = [p for s in m.sessions for p in s.hot if p >= 0]
        assert len(used) == len(set(used)) and len(used) + m.free_hot() == nh
        refs = [0] * nc
        for s in m.sessions:
            for c in s.cold:
                if c >= 0:
                    refs[c] += 1
        assert refs == m.cold_ref
        for sid2, s in enumerate(m.sessions):
            if s.state == ACTIVE:
                assert len(s.hot) == (s.seq_len + 15) // 16
                assert all(h >= 0 or (sp and c >= 0) for h, c, sp in zip(s.hot, s.cold, s.spilled))
            if s.state != 0:
                for e, h, c, sp in zip(m.row(sid2), s.hot, s.cold, s.spilled):
                    assert e == (h if h >= 0 else (c | C if sp else -1))
                    assert not (sp and h >= 0)
    assert spills > 20


def test_lazy_resume_hand_worked():
    """Lazy resume: nothing is fetched; missing pages are named in the cold tier
    until promote moves them, lowest hot ids first."""
    from oracle.pool_model import COLD_BIT as C
    m = PoolModel(num_hot=6, num_cold=10, max_sessions=3, max_pages_per_session=4, spill=True)
    a = m.create(16 * 3)                          # hot 0,1,2
    m.evict(a)                                    # cold 0,1,2; hot free
    m.resume([a]); m.pause(a)                     # resident again (hot 0,1,2), cold copies valid
    assert m.evict_pages(2)[0] == 2               # pages 0,1 of a leave HBM (clean)
    m.resume_lazy([a])
    assert m.row(a) == [0 | C, 1 | C, 2, -1] and m.pages_to_hot == 3
    assert (m.resume_resident, m.resume_total) == (0 + 1, 3 + 3) and m.spilled_pages == 2
    assert m.promote(1) == [(0, 0)] and m.row(a) == [0, 1 | C, 2, -1]
    assert m.promote(5) == [(1, 1)] and m.row(a) == [0, 1, 2, -1]
    with pytest.raises(ModelError):
        PoolModel(4, 4, 2, 2).resume_lazy([0])    # needs spill


def test_extend_drops_the_tail_page_cold_copy_hand_worked():
    """Extending a session writes its partially filled tail page (the new tokens
    go there first): that page's cold copy is dropped and the next eviction
    writes it again; full pages keep theirs.  A full tail page is left alone.  A
    spilled tail page shared with another session cannot take new tokens."""
    m = PoolModel(num_hot=8, num_cold=8, max_sessions=3, max_pages_per_session=4)
    a = m.create(20)                 # pages 0, 1 (tokens 16..19 in page 1)
    assert m.evict(a) == [(0, 0), (1, 1)]
    m.resume([a])                    # hot 0, 1 again; cold copies 0, 1 valid
    assert m.sessions[a].cold == [0, 1]
    m.extend(a, 21)                  # token 20 goes into page 1: its copy is stale
    assert m.sessions[a].cold == [0, -1] and m.free_cold() == 7
    m.extend(a, 40)                  # tokens 21..39: page 1 again, and a new page 2
    assert m.row(a) == [0, 1, 2, -1] and m.sessions[a].cold == [0, -1, -1]
    assert m.evict(a) == [(1, 1), (2, 2)] and m.cold_writes == 4
    m.resume([a])
    b = m.create(32)                 # two full pages
    m.evict(b)
    m.resume([b])
    m.extend(b, 33)                  # the tail page was full: the new token opens page 2
    assert m.sessions[b].cold[:2] != [-1, -1] and m.sessions[b].cold[2] == -1
    # spill: a lazily resumed session whose spilled tail page is shared
    s = PoolModel(num_hot=2, num_cold=8, max_sessions=3, max_pages_per_session=4, spill=True)
    x = s.import_cold(20, [5, 6])
    y = s.import_cold(20, [7, 6])    # cold page 6 shared by both tails
    s.resume_lazy([x])
    before = copy.deepcopy(s.__dict__)
    with pytest.raises(ModelError) as e:
        s.extend(x, 21)
    assert e.value.code == ERR_STATE and s.__dict__ == before
    s.extend(x, 20)                  # no new tokens: nothing is written, accepted
    assert y == 1 and s.sessions[x].seq_len == 20
