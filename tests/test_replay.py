"""The agentic replay driver (CPU only: a metadata-only pool).

Pins: a hand-worked timeline whose counters follow from the scheduling rule,
write-back LRU and the resume hit rate; the library pool and the oracle's pool
model driven by the same replay reach identical summaries and session states;
preemption keeps an over-full active set from stalling; the idle-gap draws have
the median and mean the paper gives (Sec. IV, Methodology).
"""

import math

import numpy as np
import pytest

from oracle.pool_model import ERR_NO_COLD, ERR_NO_HOT, ModelError, PoolModel
from paper_2609_25782_amd import replay as rp


class ModelPool:
    """The oracle's pool model behind the replay's pool interface."""

    def __init__(self, cfg):
        self.m = PoolModel(cfg.num_hot_pages, cfg.num_cold_pages, cfg.max_sessions, cfg.stride,
                           spill=cfg.spill)

    def refused(self, e):
        return isinstance(e, ModelError) and e.code in (ERR_NO_HOT, ERR_NO_COLD)

    def create(self, n):
        return self.m.create(n)

    def extend(self, sid, n):
        self.m.extend(sid, n)

    def write(self, sid, t0, n):
        self.m.write_tokens(sid, t0, n)

    def pause(self, sid):
        self.m.pause(sid)

    def resume(self, sid):
        self.m.resume([sid])

    def destroy(self, sid):
        self.m.destroy(sid)

    def promote(self, n):
        return len(self.m.promote(n))

    def stats(self):
        m = self.m
        return {"free_hot_pages": m.free_hot(), "free_cold_pages": m.free_cold(),
                "pages_to_cold": m.cold_writes, "pages_to_hot": m.pages_to_hot,
                "resumes": m.resumes, "resume_pages_resident": m.resume_resident,
                "resume_pages_total": m.resume_total, "lru_evicted_pages": m.lru_evicted,
                "spilled_pages": m.spilled_pages, "promoted_pages": m.promoted_pages,
                "cold_active_pages": m.cold_active()}

    def close(self):
        pass


def _tiny(**kw):
    """Page-sized everything: 1 layer, 1 head, D 64, f32 -> 8 KiB pages."""
    base = dict(num_layers=1, num_kv_heads=1, head_dim=64, elt_bytes=4, weight_bytes=0.0,
                max_sessions=64, sample_s=1.0, tbt_s=1.0)
    base.update(kw)
    cfg = rp.ReplayConfig(**base)
    return cfg


def _pages_bytes(cfg, n):
    return n * cfg.page_bytes


def test_hand_worked_cycle():
    """N_a = 1, every draw fixed: prompt 16, later prompts 16, 16 decoded tokens
    per turn, peak 64, idle gap one step, HBM of 4 pages.  Sessions A and B
    alternate in a 64-step cycle:
      0  A created (1 page), its first decoded token opens page 2;  15 A pauses
      16 B created likewise (HBM now full);                          31 B pauses
      32 A resumes (both pages resident), grows to 4 pages: LRU evicts B's two
         dirty pages (2 cold writes);                                47 A ends
      48 B resumes with nothing resident (2 pages fetched), grows to 4; 63 B ends
    so per cycle: 2 resumes, 2 of 4 resumed pages resident (hit rate 1/2),
    2 pages written, 2 fetched, 2 evicted by LRU, 128 tokens produced."""
    cfg = _tiny(n_active=1, prompt0=(16, 16), turn_prompt=(16, 16), turn_decode=(16, 16),
                peak=(64, 64), gap_median_s=1.0, gap_mean_s=1.0, warmup_s=64, plateau_s=128)
    cfg.hbm_bytes = _pages_bytes(cfg, 4)
    cfg.cold_bytes = _pages_bytes(cfg, 4)
    for pool in (None, ModelPool(cfg)):
        r = rp.Replay(cfg, pool)
        s = r.run()
        assert s["plateau_counts"] == {                          # plateau: two cycles
            "resumes": 4, "resume_pages_resident": 4, "resume_pages_total": 8,
            "pages_to_cold": 4, "pages_to_hot": 4, "lru_evicted_pages": 4, "produced_tokens": 256,
            "spilled_pages": 0, "promoted_pages": 0}
        assert s["resume_hit_rate"] == 0.5
        st = r.pool.stats()                                       # three cycles in all
        assert (st["resumes"], st["pages_to_cold"], st["pages_to_hot"]) == (6, 6, 6)
        assert (st["resume_pages_resident"], st["resume_pages_total"]) == (6, 12)
        assert st["lru_evicted_pages"] == 6
        assert (r.sessions_started, r.sessions_finished) == (6, 6)
        assert s["preemptions"] == 0 and s["refused_admissions"] == 0
        assert st["free_hot_pages"] == 4 and st["free_cold_pages"] == 4
        r.close()


def _final_state(r):
    return sorted((a.sid, a.length, a.target, a.turn, a.preempted) for a in r.agents.values())


@pytest.mark.parametrize("hot_pages,n_active,seed", [(40, 4, 0), (26, 4, 1), (100, 12, 2)])
def test_library_pool_matches_oracle_model(hot_pages, n_active, seed):
    """The same replay over the library and over the oracle's model: every
    decision depends on the pool, so equal summaries and states mean the
    library's allocation, LRU, write-back and resume followed the model."""
    cfg = _tiny(n_active=n_active, prompt0=(10, 40), turn_prompt=(5, 30), turn_decode=(5, 40),
                peak=(60, 160), gap_median_s=6.0, gap_mean_s=15.0, warmup_s=150, plateau_s=600,
                seed=seed)
    cfg.hbm_bytes = _pages_bytes(cfg, hot_pages)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    lib = rp.Replay(cfg)
    a = lib.run()
    model = rp.Replay(cfg, ModelPool(cfg))
    b = model.run()
    assert a == b
    assert _final_state(lib) == _final_state(model)
    c = a["plateau_counts"]        # each case has LRU pressure and partial residency
    assert 0 < c["resume_pages_resident"] < c["resume_pages_total"] and c["lru_evicted_pages"] > 0
    # the pool holds exactly the pages of the live sessions' hot and cold copies
    for sid_state in range(cfg.max_sessions):
        st, L, hot, cold = rp.kv.kv_session_info(lib.pool.h, sid_state)
        if st:
            ms = model.pool.m.sessions[sid_state]
            assert (L, hot, cold) == (ms.seq_len, ms.hot, ms.cold)
    live = sum(rp._pages(x.length) for x in lib.agents.values())
    assert live == lib.live_pages
    lib.close()


def test_preemption_keeps_an_overfull_active_set_moving():
    """HBM smaller than the active set's growth: sessions are paused mid-turn
    instead of stalling, and every turn still finishes."""
    cfg = _tiny(n_active=4, prompt0=(30, 40), turn_prompt=(10, 20), turn_decode=(60, 80),
                peak=(150, 200), gap_median_s=2.0, gap_mean_s=4.0, warmup_s=50, plateau_s=800)
    cfg.hbm_bytes = _pages_bytes(cfg, 18)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    lib = rp.Replay(cfg)
    a = lib.run()
    b = rp.Replay(cfg, ModelPool(cfg)).run()
    assert a == b
    assert a["preemptions"] > 0 and a["sessions_finished"] > 5
    lib.close()


def test_full_tiers_stop_the_replay_instead_of_spinning():
    """A cold tier too small to take the evictions: the active set can neither
    grow nor make room, so after stall_steps steps with nothing decoding the
    replay raises, for the library pool and for the oracle's model alike (the
    same configuration with a large cold tier runs to the end)."""
    cfg = _tiny(n_active=4, prompt0=(30, 40), turn_prompt=(10, 20), turn_decode=(60, 80),
                peak=(150, 200), gap_median_s=2.0, gap_mean_s=4.0, warmup_s=50, plateau_s=800)
    cfg.hbm_bytes = _pages_bytes(cfg, 18)
    cfg.cold_bytes = _pages_bytes(cfg, 6)
    cfg.stall_steps = 500
    for pool in (None, ModelPool(cfg)):
        r = rp.Replay(cfg, pool)
        with pytest.raises(rp.ReplayStalled, match="cold tier is too small"):
            r.run()
        r.close()
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    r = rp.Replay(cfg)
    assert r.run()["sessions_finished"] > 5
    r.close()


def test_replay_is_deterministic():
    cfg = _tiny(n_active=6, prompt0=(10, 40), turn_prompt=(5, 30), turn_decode=(5, 40),
                peak=(60, 160), gap_median_s=6.0, gap_mean_s=15.0, warmup_s=100, plateau_s=300)
    cfg.hbm_bytes = _pages_bytes(cfg, 80)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    assert rp.run(cfg) == rp.run(cfg)
    cfg.seed = 1
    assert rp.run(cfg) != rp.run(rp.ReplayConfig(**{**cfg.__dict__, "seed": 2}))


def test_gap_draws_have_the_papers_median_and_mean():
    cfg = rp.ReplayConfig(tbt_s=0.001)
    r = rp.Replay(cfg)
    g = np.array([r._gap_steps() for _ in range(200000)]) * cfg.step_s
    assert np.median(g) == pytest.approx(8.0, rel=0.02)
    assert g.mean() == pytest.approx(23.0, rel=0.04)
    assert r.sigma == pytest.approx(math.sqrt(2 * math.log(23 / 8)))
    r.close()


def test_tbt_line_through_the_printed_points():
    assert rp.tbt_for(48) == pytest.approx(0.014)
    assert rp.tbt_for(128) == pytest.approx(0.027)


def test_paper_scale_footprint_and_eviction_onset():
    """At the paper's shape (96 KiB of KV per token, 1.5 MiB pages, 192 GiB HBM
    minus 56.8 GiB of weights, 3 TiB flash) a resident agent holds about
    0.82 GiB (Sec. IV) and low concurrency evicts nothing (Sec. IV, Endurance).
    The per-turn prompt and decode lengths are a reading: the paper does not
    print them; they are set so that writing every produced block gives its
    all-KV-to-flash lifetime of about 11 years at N_a = 48."""
    low = rp.run(rp.ReplayConfig(n_active=16, warmup_s=600, plateau_s=300))
    assert low["cold_write_GBps"] == 0 and low["resume_hit_rate"] == 1.0
    assert low["kv_per_resident_session_gib"] == pytest.approx(0.82, rel=0.08)
    mid = rp.run(rp.ReplayConfig(n_active=48, warmup_s=600, plateau_s=300))
    assert 0.5 < mid["resume_hit_rate"] < 1.0 and mid["cold_write_GBps"] > 0
    assert 9.5 < mid["lifetime_years"]["all_kv_to_flash"] < 13.5
    assert mid["lifetime_years"]["write_on_evict"] > mid["lifetime_years"]["all_kv_to_flash"]
    assert mid["sessions_per_device"]["hbm_only"] == pytest.approx(165, rel=0.08)


@pytest.mark.parametrize("hot_pages,n_active", [(26, 4), (18, 4), (100, 12)])
def test_decode_lengths_stay_within_resident_pages(hot_pages, n_active):
    """What a device decode would read: every length handed to the decode hook
    belongs to an ACTIVE session, grows by one token a step, and stays within
    the session's allocated pages, all of them resident."""
    cfg = _tiny(n_active=n_active, prompt0=(10, 40), turn_prompt=(5, 30), turn_decode=(5, 40),
                peak=(60, 160), gap_median_s=6.0, gap_mean_s=15.0, warmup_s=20, plateau_s=500)
    cfg.hbm_bytes = _pages_bytes(cfg, hot_pages)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    r = rp.Replay(cfg)
    last = {}
    seen = [0]

    def check(lengths):
        sids = [s for s, _ in lengths]
        assert len(sids) == len(set(sids)) and len(sids) <= n_active
        aid_of = {a.sid: aid for aid, a in r.running.items()}   # session ids are reused
        for sid, n in lengths:
            state, L, hot, _ = rp.kv.kv_session_info(r.pool.h, sid)
            assert state == rp.kv.KV_SESSION_ACTIVE
            assert 0 < n <= 16 * len(hot) and all(p >= 0 for p in hot)
            assert n >= L
            assert last.get(aid_of[sid], 0) <= n
            last[aid_of[sid]] = n
            seen[0] += 1

    r.run(check)
    assert seen[0] > 1000
    r.close()


def test_spill_replaces_preemption_and_follows_the_model():
    """The over-full configuration of the preemption test with spill on: no
    session is paused mid-turn; pages spill to the cold tier and are promoted
    back, with the library and the model taking the same decisions."""
    cfg = _tiny(n_active=4, prompt0=(30, 40), turn_prompt=(10, 20), turn_decode=(60, 80),
                peak=(150, 200), gap_median_s=2.0, gap_mean_s=4.0, warmup_s=50, plateau_s=800,
                spill=True, promote_s=3.0)
    cfg.hbm_bytes = _pages_bytes(cfg, 18)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    lib = rp.Replay(cfg)
    a = lib.run()
    b = rp.Replay(cfg, ModelPool(cfg)).run()
    assert a == b
    assert a["preemptions"] == 0 and a["sessions_finished"] > 5
    c = a["plateau_counts"]
    assert c["spilled_pages"] > 0 and c["promoted_pages"] > 0
    assert 0 < a["spill"]["cold_share_of_hot_set"] < 1
    lib.close()


def test_spill_decode_lengths_stay_within_allocated_pages():
    cfg = _tiny(n_active=4, prompt0=(30, 40), turn_prompt=(10, 20), turn_decode=(60, 80),
                peak=(150, 200), gap_median_s=2.0, gap_mean_s=4.0, warmup_s=20, plateau_s=400,
                spill=True)
    cfg.hbm_bytes = _pages_bytes(cfg, 18)
    cfg.cold_bytes = _pages_bytes(cfg, 400)
    r = rp.Replay(cfg)
    spilled_seen = [0]

    def check(lengths):
        for sid, n in lengths:
            state, L, hot, cold = rp.kv.kv_session_info(r.pool.h, sid)
            assert state == rp.kv.KV_SESSION_ACTIVE and 0 < n <= 16 * len(hot)
            assert all(h >= 0 or c >= 0 for h, c in zip(hot, cold))
            spilled_seen[0] += sum(h < 0 for h in hot)

    r.run(check)
    assert spilled_seen[0] > 0
    r.close()
