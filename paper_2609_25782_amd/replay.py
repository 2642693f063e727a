"""Agentic replay on synthetic trajectories, with the paper's accounting.

The paper replays recorded agent trajectories through a trace-driven simulator
(Sec. IV, Methodology).  Those recordings are not available here; this driver
generates seeded synthetic trajectories with the statistics the paper prints and
drives them through the library's pool, so every allocation, LRU eviction,
write-on-evict and resume is the library's own decision:

* a session starts from a prompt and grows turn by turn (tool output or user
  text appended, then a decoded reply) until it reaches its peak context, about
  16.7k tokens on average (Sec. IV, Methodology);
* between turns it idles for a heavy-tailed gap with median about 8 s and mean
  about 23 s; the paper does not name the family, here it is lognormal with
  those two moments (mu = ln 8, sigma^2 = 2 ln(23/8));
* a batching scheduler keeps N_a sessions decoding and admits another whenever
  one pauses (Sec. IV, Methodology): first a paused session whose gap is over,
  in the order the gaps ended, else a new session (new trajectories arrive
  without limit, each with its own phase);
* a paused session keeps its pages in HBM until LRU eviction needs them, with
  write-back of pages that have no valid cold copy (Sec. III and IV).

Time advances in decode steps of one TBT.  Each step first admits sessions,
then every active session produces one token; a page is allocated when a token
starts it, and a turn ends with a pause (or, at the peak context, with the
session's end).  Prefill is instantaneous: the paper's resume overhead is
measured on top of it.

Accounting over the plateau after a warm-up (Sec. IV): HBM and flash
footprint, mean resident KV per session, resume hit rate, cold-fetch and
cold-write rates, Eq. (1) lifetime for write-on-evict and for writing every
produced block (all-KV-to-flash), read power by tier, sessions per device, and
the resume overhead each cold tier's bandwidth implies for the measured misses.
"""

from __future__ import annotations

import heapq
import math
from collections import deque
from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import accounting as acc
from . import hotcold_kv as kv

PAGE = kv.KV_PAGE_TOKENS

_EXT, _END = 0, 1


def _pages(n: int) -> int:
    return (n + PAGE - 1) // PAGE


def tbt_for(n_active: int) -> float:
    """Seconds per decode step: the straight line through the two points the
    paper gives for its design (14 ms at N_a = 48, 27 ms at N_a = 128; Sec. IV,
    "Capacity and latency")."""
    return 0.014 + (n_active - 48) * (0.027 - 0.014) / (128 - 48)


@dataclass
class ReplayConfig:
    n_active: int = 48                    # N_a, sessions decoding at once
    hbm_bytes: float = 192 * acc.GIB      # fast tier of the modelled device
    weight_bytes: float = 56.8 * acc.GIB  # model weights resident in HBM
    cold_bytes: float = 3 * acc.TIB       # the capacity tier
    num_layers: int = 48
    num_kv_heads: int = 4
    head_dim: int = 128
    elt_bytes: int = 2
    tbt_s: Optional[float] = None         # None: tbt_for(n_active)
    warmup_s: float = 900.0
    plateau_s: float = 900.0
    sample_s: float = 1.0                 # footprint sampling period
    prompt0: Tuple[int, int] = (1000, 2000)      # first prompt of a session
    turn_prompt: Tuple[int, int] = (280, 1280)   # tokens appended at each later turn
    turn_decode: Tuple[int, int] = (200, 800)     # tokens decoded per turn
    peak: Tuple[int, int] = (12400, 21000)       # peak context, uniform (mean 16.7k)
    gap_median_s: float = 8.0
    gap_mean_s: float = 23.0
    max_sessions: int = 4096              # rows of the pool's page table
    spill: bool = False                   # no pinning: spill to the cold tier instead of preempting
    promote_s: float = 0.5                # with spill: move spilled active pages back this often
    pe_cycles: float = 1e5
    waf: float = 1.02
    hbm_pj_per_bit: float = 3.5
    flash_pj_per_bit: float = 20.0
    # cold tiers for the resume-overhead estimate: (name, bytes/s, access latency s)
    tiers: Tuple[Tuple[str, float, float], ...] = (("hbf", 8e12, 25e-6),
                                                   ("nvlink_c2c", 450e9, 0.0),
                                                   ("pcie5", 64e9, 0.0))
    seed: int = 0
    stall_steps: int = 2000               # steps with nothing decoding before the replay gives up

    @property
    def step_s(self) -> float:
        return self.tbt_s if self.tbt_s is not None else tbt_for(self.n_active)

    @property
    def token_bytes(self) -> int:
        return acc.kv_bytes_per_token(self.num_layers, self.num_kv_heads, self.head_dim, self.elt_bytes)

    @property
    def page_bytes(self) -> int:
        return PAGE * self.token_bytes

    @property
    def num_hot_pages(self) -> int:
        return int((self.hbm_bytes - self.weight_bytes) // self.page_bytes)

    @property
    def num_cold_pages(self) -> int:
        return int(self.cold_bytes // self.page_bytes)

    @property
    def stride(self) -> int:
        return _pages(self.peak[1] + self.turn_prompt[1] + self.turn_decode[1])


class ReplayStalled(RuntimeError):
    """The replay cannot make progress: every tier is full."""


class LibraryPool:
    """The replay's pool: a metadata-only pool of the C library (host
    bookkeeping, no device), or the handle of a device pool."""

    def __init__(self, cfg: ReplayConfig, handle: Optional[int] = None):
        self.own = handle is None
        if handle is None:
            desc = kv.kv_pool_desc(cfg.num_layers, cfg.num_kv_heads, cfg.head_dim, PAGE,
                                   kv.KV_DTYPE_BF16 if cfg.elt_bytes == 2 else kv.KV_DTYPE_F32,
                                   cfg.num_hot_pages, cfg.num_cold_pages, kv.KV_COLD_DEVICE,
                                   cfg.max_sessions, cfg.stride, 0, kv.KV_POOL_METADATA_ONLY)
            handle = kv.kv_pool_create(desc, 0, 0, 0, 0, 0)
        self.h = handle
        kv.kv_pool_set_spill(self.h, cfg.spill)

    REFUSED = (kv.KV_ERR_NO_HOT_PAGES, kv.KV_ERR_NO_COLD_PAGES)

    def refused(self, e: Exception) -> bool:
        return isinstance(e, kv.KVError) and e.status in self.REFUSED

    def create(self, n: int) -> int:
        return kv.kv_session_create(self.h, n)

    def extend(self, sid: int, n: int) -> None:
        kv.kv_session_extend(self.h, sid, n)

    def write(self, sid: int, t0: int, n: int) -> None:
        kv.kv_write_tokens(self.h, sid, 0, t0, n, 0, 0)

    def pause(self, sid: int) -> None:
        kv.kv_session_pause(self.h, sid)

    def resume(self, sid: int) -> None:
        kv.kv_resume_session(self.h, sid)

    def destroy(self, sid: int) -> None:
        kv.kv_session_destroy(self.h, sid)

    def promote(self, n: int) -> int:
        return kv.kv_promote_pages(self.h, n)

    def stats(self) -> Dict[str, int]:
        return kv.kv_pool_stats(self.h)

    def close(self) -> None:
        if self.own and self.h:
            kv.kv_pool_destroy(self.h)
        self.h = None


class DevicePool(LibraryPool):
    """A device pool (paper_2609_25782_amd.pool.HotColdPool) under the replay:
    the same pool calls, now moving real pages, plus the KV itself.  Each
    session gets a generator id when it is created, and every page it is given
    is filled (all layers, every slot) with the counter-based values of that
    id, so the contents of any resident page are known without reading it."""

    def __init__(self, cfg: ReplayConfig, pool, seed: int, value_mult: float):
        super().__init__(cfg, pool.handle)
        self.dev = pool
        self.seed, self.mult = seed, value_mult
        self.gen: Dict[int, int] = {}       # session id -> generator id
        self.npages: Dict[int, int] = {}
        self.next_gen = 0

    def _fill(self, sid: int, first: int, n: int) -> None:
        if n > 0:
            kv.kv_fill_synthetic_pages(self.h, sid, self.gen[sid], self.seed, self.mult, first, n)

    def create(self, n: int) -> int:
        sid = kv.kv_session_create(self.h, n)
        self.gen[sid] = self.next_gen % (1 << 20)
        self.next_gen += 1
        self.npages[sid] = _pages(n)
        self._fill(sid, 0, _pages(n))
        return sid

    def extend(self, sid: int, n: int) -> None:
        kv.kv_session_extend(self.h, sid, n)
        old = self.npages[sid]
        self.npages[sid] = max(old, _pages(n))
        self._fill(sid, old, self.npages[sid] - old)

    def write(self, sid: int, t0: int, n: int) -> None:
        # Pages past the old tail were filled when extend allocated them.  The
        # tail page that already held tokens is filled again (its values do not
        # change) and so loses its cold copy, as a write records it.
        if n > 0 and t0 % PAGE:
            self._fill(sid, t0 // PAGE, 1)

    def destroy(self, sid: int) -> None:
        kv.kv_session_destroy(self.h, sid)
        del self.gen[sid], self.npages[sid]

    def close(self) -> None:
        self.h = None                        # the HotColdPool owns the handle


class DeviceDecode:
    """The decode of one replay step on a device pool: the page-table rows of
    the sessions decoding are gathered into a batch table once (one launch),
    then every layer's paged attention runs over that batch.  Batch row i uses
    query row i of q.  Records, per step, HIP events around the whole step and
    around its decode."""

    def __init__(self, pool, q, layers=None):
        import torch
        self.torch = torch
        self.pool = pool
        self.q = q                           # [max batch, num_q_heads, head_dim]
        cap = q.shape[0]
        self.out = torch.empty_like(q)
        self.table = torch.empty((cap, pool.stride), dtype=torch.int32, device=pool.device)
        self.meta = torch.zeros((2, cap), dtype=torch.int32, device=pool.device)   # lengths, ids
        self.host = np.zeros((2, cap), np.int32)
        self.n = 0
        self.layers = list(range(pool.num_layers)) if layers is None else list(layers)
        self.marks: List = []                # per step: (step start, decode start, decode end)
        self.batch: List[int] = []
        self.tokens: List[int] = []
        self._start = None

    def _event(self):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def step_begin(self) -> None:
        self._start = self._event()

    def __call__(self, lengths: List[Tuple[int, int]]) -> None:
        n = len(lengths)
        if n > self.q.shape[0]:
            raise ValueError("batch of %d sessions exceeds the %d query rows" % (n, self.q.shape[0]))
        self.n = n
        self.host[0, :n] = [length for _, length in lengths]
        self.host[1, :n] = [sid for sid, _ in lengths]
        d0 = self._event()
        if n:
            self.meta[:, :n].copy_(self.torch.from_numpy(self.host[:, :n]))   # pageable: host-synchronous
            self.pool.gather_table(self.meta[1, :n], out=self.table)
            for layer in self.layers:
                self.pool.decode(layer, self.q[:n], self.meta[0, :n], page_table=self.table[:n],
                                 out=self.out[:n])
        self.marks.append((self._start, d0, self._event()))
        self.batch.append(n)
        self.tokens.append(int(self.host[0, :n].sum()))

    def last_batch(self) -> Tuple[List[int], List[int]]:
        """(session ids, lengths) of the last decoded step, in batch order."""
        return [int(x) for x in self.host[1, :self.n]], [int(x) for x in self.host[0, :self.n]]

    def timings(self) -> Dict:
        """Per-step GPU times in ms: the whole step (from its first launch to the
        end of its decode: admissions, resumes, evictions, page fills, decode)
        and the decode alone."""
        self.torch.cuda.synchronize()
        step = np.array([a.elapsed_time(c) for a, b, c in self.marks])
        dec = np.array([b.elapsed_time(c) for a, b, c in self.marks])
        return {"step_ms": step, "decode_ms": dec, "batch": np.array(self.batch),
                "tokens": np.array(self.tokens)}


@dataclass
class _Agent:
    peak: int
    sid: int = -1          # pool session id, -1 before the first turn
    length: int = 0        # tokens the pool holds for the session
    target: int = 0        # length at the end of the current turn
    turn: int = 0          # turn counter (stale events carry an older value)
    decode: int = 0        # tokens decoded in the current turn
    preempted: bool = False  # paused mid-turn; the turn continues on admission
    len0: int = 0          # length when the current (part of the) turn was admitted
    step0: int = 0         # step of that admission


class Replay:
    def __init__(self, cfg: ReplayConfig, pool=None):
        self.cfg = cfg
        self.pool = pool if pool is not None else LibraryPool(cfg)
        self.rng = np.random.Generator(np.random.PCG64(cfg.seed))
        self.mu = math.log(cfg.gap_median_s)
        self.sigma = math.sqrt(2.0 * math.log(cfg.gap_mean_s / cfg.gap_median_s))
        self.step = 0
        self.events: List[Tuple[int, int, int, int, int]] = []   # (step, kind, seq, agent, turn)
        self.gaps: List[Tuple[int, int, int]] = []               # (ready step, seq, agent)
        self.ready: deque = deque()       # paused sessions whose idle gap is over
        self.preempted: deque = deque()   # sessions paused mid-turn, admitted first
        self.agents: Dict[int, _Agent] = {}
        self.running: Dict[int, _Agent] = {}      # decoding this step
        self.active = 0
        self.next_id = 0
        self.seq = 0
        # running totals (in tokens or pages) for the accounting
        self.live_pages = 0
        self.active_pages = 0
        self.produced_tokens = 0
        self.refused_admissions = 0
        self.refused_pages = 0
        self.sessions_started = 0
        self.sessions_finished = 0
        self.plateau_start = 0

    # -- trajectory draws ----------------------------------------------------
    def _uniform(self, lo_hi) -> int:
        return int(self.rng.integers(lo_hi[0], lo_hi[1] + 1))

    def _gap_steps(self) -> int:
        return max(1, int(round(float(self.rng.lognormal(self.mu, self.sigma)) / self.cfg.step_s)))

    # -- bookkeeping helpers -------------------------------------------------
    def _push(self, step: int, kind: int, aid: int) -> None:
        self.seq += 1
        heapq.heappush(self.events, (step, kind, self.seq, aid, self.agents[aid].turn))

    def _set_length(self, a: _Agent, n: int, active: bool) -> None:
        d = _pages(n) - _pages(a.length)
        self.live_pages += d
        if active:
            self.active_pages += d
        a.length = n

    # -- scheduler -----------------------------------------------------------
    def _admit(self, aid: int) -> bool:
        """Start agent aid's next turn (create or resume its session and append
        the turn's prompt), or continue a turn that was preempted."""
        a, pool = self.agents[aid], self.pool
        new = a.sid < 0
        try:
            if new:
                n = self._uniform(self.cfg.prompt0)
                a.sid = pool.create(n)
                self.sessions_started += 1
                self._set_length(a, n, False)
                added = n
            else:
                pool.resume(a.sid)
                added = 0 if a.preempted else self._uniform(self.cfg.turn_prompt)
        except Exception as e:
            if pool.refused(e):
                return False
            raise
        if added and not new:                     # a later turn: its prompt is appended
            try:
                pool.extend(a.sid, a.length + added)
            except Exception as e:
                if pool.refused(e):
                    pool.pause(a.sid)
                    return False
                raise
            pool.write(a.sid, a.length, added)
            self._set_length(a, a.length + added, False)
        self.active_pages += _pages(a.length)
        if self.step >= self.plateau_start:
            self.produced_tokens += added
        if a.preempted:
            a.preempted = False
        else:
            a.decode = self._uniform(self.cfg.turn_decode)
            a.target = a.length + a.decode
        a.turn += 1
        a.len0, a.step0 = a.length, self.step
        self.running[aid] = a
        remaining = a.target - a.length
        first_new = PAGE * _pages(a.length) - a.length   # decoded tokens before the next page
        if first_new < remaining:
            self._push(self.step + first_new, _EXT, aid)
        self._push(self.step + remaining - 1, _END, aid)
        self.active += 1
        return True

    def _on_ext(self, aid: int) -> None:
        a = self.agents[aid]
        n = PAGE * _pages(a.length) + 1          # the token that starts the next page
        try:
            self.pool.extend(a.sid, n)
        except Exception as e:
            if not self.pool.refused(e):
                raise
            self._preempt(a, n - 1)
            del self.running[aid]
            self.preempted.append(aid)
            return
        self._set_length(a, n, True)
        if n + PAGE <= a.target:
            self._push(self.step + PAGE, _EXT, aid)

    def _preempt(self, a: _Agent, length: int) -> None:
        """Every hot page is held and the session needs another: pause it mid-turn
        (its pages become evictable) and let it continue before anyone else is
        admitted.  Without this the active set could outgrow HBM and stall."""
        self.refused_pages += 1
        self.pool.extend(a.sid, length)           # fills the pages it holds; allocates nothing
        self._set_length(a, length, True)
        self.pool.pause(a.sid)
        self.active_pages -= _pages(a.length)
        self.active -= 1
        a.turn += 1                               # drops the turn's pending events
        a.preempted = True

    def _on_end(self, aid: int) -> None:
        a = self.agents[aid]
        self.pool.extend(a.sid, a.target)         # no new page: _on_ext allocated it
        if self.step >= self.plateau_start:
            self.produced_tokens += a.decode
        self._set_length(a, a.target, True)
        self.active_pages -= _pages(a.length)
        self.active -= 1
        del self.running[aid]
        if a.length >= a.peak:
            self.pool.destroy(a.sid)
            self.live_pages -= _pages(a.length)
            self.sessions_finished += 1
            del self.agents[aid]
        else:
            self.pool.pause(a.sid)
            self.seq += 1
            heapq.heappush(self.gaps, (self.step + 1 + self._gap_steps(), self.seq, aid))

    def _new_agent(self) -> int:
        aid = self.next_id
        self.next_id += 1
        self.agents[aid] = _Agent(peak=self._uniform(self.cfg.peak))
        return aid

    def decode_lengths(self) -> List[Tuple[int, int]]:
        """(session id, context length) of every session decoding this step,
        counting the token it produces."""
        return [(a.sid, a.len0 + self.step - a.step0 + 1) for a in self.running.values()]

    def _events(self, through_kind: int) -> None:
        while self.events and self.events[0][0] <= self.step and self.events[0][1] <= through_kind:
            _, kind, _, aid, turn = heapq.heappop(self.events)
            a = self.agents.get(aid)
            if a is None or a.turn != turn:
                continue
            if kind == _EXT:
                self._on_ext(aid)
            else:
                self._on_end(aid)

    def _advance(self, decode_fn=None) -> None:
        """One decode step: admissions, page allocations for this step's tokens,
        the decode itself (decode_fn, given decode_lengths()), turn ends."""
        while self.gaps and self.gaps[0][0] <= self.step:
            self.ready.append(heapq.heappop(self.gaps)[2])
        while self.active < self.cfg.n_active:
            queue = self.preempted or self.ready
            if queue:
                aid = queue[0]
                if not self._admit(aid):
                    self.refused_admissions += 1
                    break
                queue.popleft()
            elif len(self.agents) >= self.cfg.max_sessions:   # every page-table row in use
                self.refused_admissions += 1
                break
            else:
                aid = self._new_agent()
                if not self._admit(aid):
                    del self.agents[aid]
                    self.refused_admissions += 1
                    break
        self._events(_EXT)
        if decode_fn is not None:
            decode_fn(self.decode_lengths())
        self._events(_END)

    # -- run -----------------------------------------------------------------
    def run(self, decode_fn=None) -> Dict:
        """Warm-up, then the plateau; decode_fn (if any) runs the decode of each
        plateau step on a device pool."""
        cfg = self.cfg
        warm = int(round(cfg.warmup_s / cfg.step_s))
        total = warm + int(round(cfg.plateau_s / cfg.step_s))
        every = max(1, int(round(cfg.sample_s / cfg.step_s)))
        promote_every = max(1, int(round(cfg.promote_s / cfg.step_s)))
        self.plateau_start = warm
        base = None
        samples = []
        stalled = 0
        for self.step in range(total):
            if self.step == warm:
                base = self.pool.stats()
            if self.step >= warm and hasattr(decode_fn, "step_begin"):
                decode_fn.step_begin()
            self._advance(decode_fn if self.step >= warm else None)
            # Nothing decoding while sessions wait: both tiers are full (a page
            # for the next token needs an eviction, which needs a free cold page),
            # and preempting and re-admitting would go on forever.
            stalled = stalled + 1 if self.active == 0 and (self.preempted or self.ready) else 0
            if stalled > cfg.stall_steps:
                st = self.pool.stats()
                raise ReplayStalled("no session has decoded for %d steps at step %d: %d free hot and %d free "
                                    "cold pages; the cold tier is too small for this load" % (
                                        stalled, self.step, st["free_hot_pages"], st["free_cold_pages"]))
            if cfg.spill and self.step % promote_every == 0:
                self.pool.promote(1 << 30)
            if self.step >= warm and (self.step - warm) % every == 0:
                st = self.pool.stats()
                samples.append((cfg.num_hot_pages - st["free_hot_pages"],
                                cfg.num_cold_pages - st["free_cold_pages"],
                                len(self.agents), self.live_pages, self.active_pages, self.active,
                                st.get("cold_active_pages", 0)))
        return self._summary(base, self.pool.stats(), np.array(samples, dtype=np.float64),
                             (total - warm) * cfg.step_s)

    def _summary(self, base, end, samples, secs) -> Dict:
        cfg = self.cfg
        pb = cfg.page_bytes
        d = {k: end[k] - base[k] for k in ("pages_to_cold", "pages_to_hot", "resumes",
                                          "resume_pages_resident", "resume_pages_total",
                                          "lru_evicted_pages")}
        for k in ("spilled_pages", "promoted_pages"):
            if k in end:
                d[k] = end[k] - base[k]
        hot_used, cold_used, live, live_pages, active_pages, batch, cold_active = samples.mean(axis=0)
        write_bps = d["pages_to_cold"] * pb / secs
        fetch_bps = d["pages_to_hot"] * pb / secs
        produced_bps = self.produced_tokens * cfg.token_bytes / secs
        hot_read_bps = active_pages * pb / cfg.step_s        # every step's decode reads all active KV
        per_session = live_pages * pb / live if live else 0.0
        miss_bytes = d["pages_to_hot"] * pb / d["resumes"] if d["resumes"] else 0.0
        e_hbm, e_fl = cfg.hbm_pj_per_bit, cfg.flash_pj_per_bit
        power_tiered = acc.read_power_watts([hot_read_bps, fetch_bps], [e_hbm, e_fl])
        power_flash = acc.read_power_watts([hot_read_bps], [e_fl])
        return {
            "n_active": cfg.n_active,
            "tbt_ms": round(cfg.step_s * 1e3, 3),
            "plateau_s": round(secs, 1),
            "sessions_resident": round(float(live), 1),
            "kv_per_resident_session_gib": round(per_session / acc.GIB, 3),
            "hot_set_gib": round(active_pages * pb / acc.GIB, 2),
            "hbm_kv_gib": round(hot_used * pb / acc.GIB, 2),
            "hbm_kv_capacity_gib": round(cfg.num_hot_pages * pb / acc.GIB, 2),
            "flash_kv_gib": round(cold_used * pb / acc.GIB, 2),
            "resumes_per_s": round(d["resumes"] / secs, 2),
            "resume_hit_rate": round(d["resume_pages_resident"] / d["resume_pages_total"], 4)
            if d["resume_pages_total"] else None,
            "resume_miss_mib": round(miss_bytes / 2 ** 20, 1),
            "resume_overhead_ms": {name: round((lat + miss_bytes / bw) * 1e3, 3) if miss_bytes else 0.0
                                   for name, bw, lat in cfg.tiers},
            "cold_fetch_GBps": round(fetch_bps / 1e9, 3),
            "cold_write_GBps": round(write_bps / 1e9, 4),
            "produced_kv_GBps": round(produced_bps / 1e9, 4),
            "lru_evicted_pages_per_s": round(d["lru_evicted_pages"] / secs, 1),
            "lifetime_years": {
                "write_on_evict": round(acc.flash_lifetime_years(cfg.cold_bytes, cfg.pe_cycles,
                                                                 write_bps, cfg.waf), 1),
                "all_kv_to_flash": round(acc.flash_lifetime_years(cfg.cold_bytes, cfg.pe_cycles,
                                                                  produced_bps, cfg.waf), 1)},
            "read_power_w": {"write_on_evict": round(power_tiered, 1),
                             "all_kv_to_flash": round(power_flash, 1),
                             "saving": round(power_flash - power_tiered, 1)},
            "sessions_per_device": {
                "hbm_only": round(acc.sessions_per_device(cfg.hbm_bytes, cfg.weight_bytes, per_session), 1)
                if per_session else None,
                "with_flash": round(acc.sessions_per_device(cfg.hbm_bytes, cfg.weight_bytes, per_session,
                                                            cfg.cold_bytes), 1) if per_session else None},
            "mean_batch": round(float(batch), 2),
            "spill": self._spill_summary(cold_active, active_pages) if cfg.spill else None,
            "decode_tokens_per_s": round(batch / cfg.step_s, 1),
            "plateau_counts": dict(d, produced_tokens=self.produced_tokens),
            "refused_admissions": self.refused_admissions,
            "preemptions": self.refused_pages,
            "sessions_started": self.sessions_started,
            "sessions_finished": self.sessions_finished,
        }

    def _spill_summary(self, cold_active: float, active_pages: float) -> Dict:
        """Decode reads of spilled pages: the share of the hot set living in the
        cold tier and the step time each tier's bandwidth adds to read it."""
        cfg = self.cfg
        cold_bytes = cold_active * cfg.page_bytes
        return {"cold_share_of_hot_set": round(cold_active / active_pages, 4) if active_pages else 0.0,
                "cold_read_per_step_mib": round(cold_bytes / 2 ** 20, 1),
                "added_tbt_ms": {name: round((cold_bytes / bw + (lat if cold_bytes else 0.0)) * 1e3, 3)
                                 for name, bw, lat in cfg.tiers}}

    def close(self) -> None:
        self.pool.close()


def run(cfg: ReplayConfig, pool=None) -> Dict:
    r = Replay(cfg, pool)
    try:
        return r.run()
    finally:
        if pool is None:
            r.close()


def sweep(n_actives=(8, 16, 32, 48, 64, 96, 128), **overrides) -> List[Dict]:
    return [run(ReplayConfig(n_active=n, **overrides)) for n in n_actives]


if __name__ == "__main__":
    import argparse
    import json

    ap = argparse.ArgumentParser(description="Agentic replay over a metadata-only pool")
    ap.add_argument("--n-active", type=int, nargs="+", default=[8, 16, 32, 48, 64, 96, 128])
    ap.add_argument("--warmup", type=float, default=900.0)
    ap.add_argument("--plateau", type=float, default=900.0)
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args()
    for n in args.n_active:
        print(json.dumps(run(ReplayConfig(n_active=n, warmup_s=args.warmup, plateau_s=args.plateau,
                                          seed=args.seed))), flush=True)
