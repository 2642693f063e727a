"""Oracle model of the hot/cold page pools and session states — TEST INFRASTRUCTURE ONLY.

It replays the documented policy on plain Python sets and lists and predicts,
for every call, the resulting page-table rows, the pages copied in each
direction and the counters.  Nothing here touches a GPU or the library.

Policy being modelled (paper Sec. III):

* Active sessions keep their KV in the hot tier; paused sessions' KV drains to
  the cold tier (Sec. III, first paragraph; data paths 2 and 4).
* Write-on-evict: a page is written to the cold tier only when it is evicted,
  and a cold copy stays valid after the session is resumed, because written KV
  never changes; an unmodified page is therefore written to the cold tier at
  most once (Sec. III, "Memory hierarchy and write policy").
* Eviction is least-recently-used at page granularity; active pages are read
  every step, so the pages of the longest-paused sessions go first (Sec. III,
  "Eviction, resume and decode").
* A resumed session's missing KV is brought back before it runs; pages still
  resident are not fetched, and the share found resident is the resume hit
  rate (Sec. III, "Eviction, resume and decode"; Sec. IV, Methodology).

Readings where the paper is silent:

* Hot and cold pages are handed out lowest id first; pages needed by one call
  go to its sessions in argument order and logical page order; session ids are
  handed out lowest first.
* LRU order: paused sessions by pause time, oldest first; within a session,
  logical page order.  Only paused sessions' pages are evicted page by page
  (no spilling of active pages); a call that would have to evict pages of the
  sessions it resumes fails instead.
* Writing tokens into a page that has a cold copy invalidates that copy, so the
  next eviction writes the page again.  Extending a session counts as writing
  its partially filled tail page, which the new tokens go into: the extension
  drops that page's cold copy (and, for a spilled tail page shared with another
  session, is refused), so appends whose page is resolved on the device need no
  bookkeeping of their own.
* Cold pages may be shared by several paused sessions (a virtualised cold
  pool); they are reference counted and freed when the last user lets go.
* Every failing call leaves the whole state unchanged.

Spill (a pool option; Sec. III: no hard pinning, blocks spill under extreme
pressure instead of failing):

* When a call needs more hot pages than are free plus evictable (the resident
  pages of paused sessions), it first evicts all of those, then places the rest
  in the cold tier: new pages (create, extend) get fresh cold pages, lowest id
  first after the victims' write-back pages; missing pages of resumed sessions
  stay where they are.  Pages are taken for hot residence in call order and
  logical page order, the remainder spills.
* A spilled page's page-table entry is its cold id with the cold tier bit set;
  decode reads it from the cold tier.  Its cold copy is the page itself, so
  evicting it writes nothing.  The entry keeps naming the cold page while the
  session is paused, until the page is fetched or the whole session evicted.
* Writing tokens into a spilled page writes the cold page in place; a cold page
  shared with another session cannot be written (state error).
* promote(n) moves up to n spilled pages of active sessions (session id order,
  logical page order) into hot pages, evicting paused pages by LRU if needed,
  since active pages are the more recently used.  Cold copies stay valid.
* resume_lazy resumes without fetching: missing pages are read in place from
  the cold tier and promoted later, so the copy work can be spread over steps.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

PAGE_TOKENS = 16

FREE, ACTIVE, PAUSED = 0, 1, 2

OK, ERR_INVALID, ERR_STATE, ERR_NO_HOT, ERR_NO_COLD = 0, -1, -2, -3, -4

COLD_BIT = 1 << 30     # page-table entry names a cold-tier page


class ModelError(Exception):
    def __init__(self, code: int, msg: str = ""):
        super().__init__(msg or str(code))
        self.code = code


@dataclass
class _Session:
    state: int = FREE
    seq_len: int = 0
    stamp: int = 0
    hot: List[int] = field(default_factory=list)   # -1 = not resident
    cold: List[int] = field(default_factory=list)  # -1 = no valid cold copy
    spilled: List[bool] = field(default_factory=list)  # row entry names the cold page


def _pages(seq_len: int) -> int:
    return (seq_len + PAGE_TOKENS - 1) // PAGE_TOKENS


class PoolModel:
    def __init__(self, num_hot: int, num_cold: int, max_sessions: int, max_pages_per_session: int,
                 spill: bool = False):
        self.spill = spill
        self.num_hot, self.num_cold = num_hot, num_cold
        self.max_sessions, self.stride = max_sessions, max_pages_per_session
        self.hot_free = set(range(num_hot))
        self.cold_free = set(range(num_cold))
        self.cold_ref = [0] * num_cold
        self.sessions = [_Session() for _ in range(max_sessions)]
        self.clock = 0
        self.cold_writes = 0          # pages written to the cold tier
        self.pages_to_hot = 0         # pages copied cold -> hot
        self.resumes = 0
        self.evicts = 0
        self.resume_resident = 0      # pages found resident by resumes
        self.resume_total = 0         # pages of resumed sessions
        self.lru_evicted = 0          # pages evicted page by page
        self.spilled_pages = 0        # pages placed or left in the cold tier by spill
        self.promoted_pages = 0       # spilled pages moved back to the hot tier

    # -- helpers -----------------------------------------------------------
    @staticmethod
    def _lowest(free: set, n: int) -> List[int]:
        return sorted(free)[:n]

    def _new_sid(self) -> int:
        for sid, s in enumerate(self.sessions):
            if s.state == FREE:
                return sid
        raise ModelError(ERR_INVALID, "no free session slot")

    def _session(self, sid: int) -> _Session:
        if not (0 <= sid < self.max_sessions):
            raise ModelError(ERR_INVALID, "bad session id")
        return self.sessions[sid]

    def _release_cold(self, page: int) -> None:
        self.cold_ref[page] -= 1
        assert self.cold_ref[page] >= 0
        if self.cold_ref[page] == 0:
            self.cold_free.add(page)

    def _tick(self) -> int:
        self.clock += 1
        return self.clock

    def _lru(self, need: int, exclude=()) -> List[Tuple[int, int]]:
        """Up to `need` (sid, page) resident pages of paused sessions, LRU first."""
        order = sorted((s.stamp, sid) for sid, s in enumerate(self.sessions)
                       if s.state == PAUSED and sid not in exclude and any(p >= 0 for p in s.hot))
        out = []
        for _stamp, sid in order:
            for i, p in enumerate(self.sessions[sid].hot):
                if len(out) == need:
                    return out
                if p >= 0:
                    out.append((sid, i))
        return out

    def _plan(self, k: int, exclude=(), fresh_spill: bool = True, spill: Optional[bool] = None):
        """k pages, hot ones with the LRU victims to evict first.  Changes nothing.
        Returns (victims, cold pages for the dirty victims, the hot pages, and
        the fresh cold pages of the spilled remainder).  Without spill the hot
        pages number k or the call fails; with it, fewer hot pages leave the
        remainder spilled (fresh cold pages only if fresh_spill)."""
        spill = self.spill if spill is None else spill
        victims = []
        if k > len(self.hot_free):
            victims = self._lru(k - len(self.hot_free), exclude)
            if len(victims) < k - len(self.hot_free) and not spill:
                raise ModelError(ERR_NO_HOT, "hot pool exhausted")
        dirty = sum(1 for sid, i in victims if self.sessions[sid].cold[i] < 0)
        n_hot = min(k, len(self.hot_free) + len(victims))
        n_spill = (k - n_hot) if fresh_spill else 0
        if dirty + n_spill > len(self.cold_free):
            raise ModelError(ERR_NO_COLD, "cold pool exhausted")
        both = self._lowest(self.cold_free, dirty + n_spill)
        after = set(self.hot_free) | {self.sessions[sid].hot[i] for sid, i in victims}
        return victims, both[:dirty], self._lowest(after, n_hot), both[dirty:]

    def _evict_victims(self, victims, cold):
        """Apply the victims; returns their (hot_src, cold_dst) copies."""
        copies, it = [], iter(cold)
        for sid, i in victims:
            s = self.sessions[sid]
            if s.cold[i] < 0:
                c = next(it)
                self.cold_free.remove(c)
                self.cold_ref[c] = 1
                s.cold[i] = c
                copies.append((s.hot[i], c))
                self.cold_writes += 1
            self.hot_free.add(s.hot[i])
            s.hot[i] = -1
            self.lru_evicted += 1
        return copies

    def _take_hot(self, pages):
        for p in pages:
            self.hot_free.remove(p)

    def _take_cold(self, pages):
        for c in pages:
            self.cold_free.remove(c)
            self.cold_ref[c] = 1
        self.spilled_pages += len(pages)

    # -- calls ---------------------------------------------------------------
    def create(self, seq_len: int, pages: Optional[Sequence[int]] = None) -> int:
        if seq_len < 0 or _pages(seq_len) > self.stride:
            raise ModelError(ERR_INVALID, "bad length")
        n = _pages(seq_len)
        sid = self._new_sid()
        victims, cold = [], []
        if pages is not None:
            pages = [int(p) for p in pages]
            if len(pages) != n or len(set(pages)) != n or any(p not in self.hot_free for p in pages):
                raise ModelError(ERR_INVALID, "pages not free/distinct")
            spill = []
        else:
            victims, cold, pages, spill = self._plan(n)
        self.last_victim_copies = self._evict_victims(victims, cold)
        self._take_hot(pages)
        self._take_cold(spill)
        self.sessions[sid] = _Session(ACTIVE, seq_len, 0, list(pages) + [-1] * len(spill),
                                      [-1] * len(pages) + list(spill),
                                      [False] * len(pages) + [True] * len(spill))
        return sid

    def extend(self, sid: int, new_len: int) -> None:
        s = self._session(sid)
        if s.state != ACTIVE:
            raise ModelError(ERR_STATE, "not active")
        if new_len < s.seq_len or _pages(new_len) > self.stride:
            raise ModelError(ERR_INVALID, "bad length")
        tail = s.seq_len // PAGE_TOKENS if new_len > s.seq_len and s.seq_len % PAGE_TOKENS else -1
        if tail >= 0 and s.hot[tail] < 0 and self.cold_ref[s.cold[tail]] > 1:
            raise ModelError(ERR_STATE, "tail page spilled to a cold page shared with another session")
        add = _pages(new_len) - len(s.hot)
        victims, cold, pages, spill = self._plan(add)
        self.last_victim_copies = self._evict_victims(victims, cold)
        self._take_hot(pages)
        self._take_cold(spill)
        if tail >= 0 and s.hot[tail] >= 0 and s.cold[tail] >= 0:   # the new tokens modify it
            self._release_cold(s.cold[tail])
            s.cold[tail] = -1
        s.hot += list(pages) + [-1] * len(spill)
        s.cold += [-1] * len(pages) + list(spill)
        s.spilled += [False] * len(pages) + [True] * len(spill)
        s.seq_len = new_len

    def pause(self, sid: int) -> None:
        s = self._session(sid)
        if s.state != ACTIVE:
            raise ModelError(ERR_STATE, "not active")
        s.state = PAUSED
        s.stamp = self._tick()

    def evict_pages(self, n: int):
        """Returns (number evicted, their copies)."""
        if n < 0:
            raise ModelError(ERR_INVALID, "negative count")
        victims = self._lru(n)
        dirty = sum(1 for sid, i in victims if self.sessions[sid].cold[i] < 0)
        if dirty > len(self.cold_free):
            raise ModelError(ERR_NO_COLD, "cold pool exhausted")
        copies = self._evict_victims(victims, self._lowest(self.cold_free, dirty))
        return len(victims), copies

    def import_cold(self, seq_len: int, cold_pages: Sequence[int]) -> int:
        n = _pages(seq_len)
        cold_pages = [int(p) for p in cold_pages]
        if seq_len < 0 or n > self.stride or len(cold_pages) != n or len(set(cold_pages)) != n \
                or any(not (0 <= p < self.num_cold) for p in cold_pages):
            raise ModelError(ERR_INVALID, "bad cold page list")
        sid = self._new_sid()
        for p in cold_pages:
            self.cold_free.discard(p)
            self.cold_ref[p] += 1
        self.sessions[sid] = _Session(PAUSED, seq_len, self._tick(), [-1] * n, list(cold_pages),
                                      [False] * n)
        return sid

    def evict(self, sid: int):
        return self.evict_many([sid])

    def evict_many(self, sids: Sequence[int]):
        """Whole-session eviction, atomic as a whole, sessions in argument order.
        Returns the (hot_src, cold_dst) copies of all of them."""
        sids = [int(x) for x in sids]
        if len(set(sids)) != len(sids):
            raise ModelError(ERR_INVALID, "duplicate session")
        dirty = 0
        for sid in sids:
            s = self._session(sid)
            if s.state != ACTIVE:
                raise ModelError(ERR_STATE, "not active")
            dirty += sum(1 for c in s.cold if c < 0)
        if dirty > len(self.cold_free):
            raise ModelError(ERR_NO_COLD, "cold pool exhausted")
        copies = []
        fresh = iter(self._lowest(self.cold_free, dirty))  # lowest first, in call and page order
        for sid in sids:
            s = self.sessions[sid]
            for i in range(len(s.hot)):
                if s.cold[i] < 0:
                    c = next(fresh)
                    self.cold_free.remove(c)
                    self.cold_ref[c] = 1
                    s.cold[i] = c
                    copies.append((s.hot[i], c))
                    self.cold_writes += 1
                if s.hot[i] >= 0:
                    self.hot_free.add(s.hot[i])
                s.hot[i] = -1
                s.spilled[i] = False
            s.state = PAUSED
            s.stamp = self._tick()
            self.evicts += 1
        return copies

    def resume(self, sids: Sequence[int]):
        """Batched resume, atomic as a whole.  Fetches only non-resident pages.
        Returns, per session, the (cold_src, hot_dst) copies in logical page order;
        the LRU victims' copies of the call are in `last_victim_copies`."""
        sids = [int(x) for x in sids]
        if len(set(sids)) != len(sids):
            raise ModelError(ERR_INVALID, "duplicate session")
        need = 0
        for sid in sids:
            s = self._session(sid)
            if s.state != PAUSED:
                raise ModelError(ERR_STATE, "not paused")
            need += sum(1 for p in s.hot if p < 0)
        victims, cold, pages, _ = self._plan(need, exclude=set(sids), fresh_spill=False)
        self.last_victim_copies = self._evict_victims(victims, cold)
        self._take_hot(pages)
        self.spilled_pages += need - len(pages)
        out, it = [], iter(pages)
        for sid in sids:
            s = self.sessions[sid]
            per = []
            resident = sum(1 for p in s.hot if p >= 0)
            for i, p in enumerate(s.hot):
                if p < 0:
                    h = next(it, None)
                    if h is None:                 # stays in the cold tier
                        s.spilled[i] = True
                        continue
                    s.hot[i] = h
                    s.spilled[i] = False
                    per.append((s.cold[i], s.hot[i]))
            self.pages_to_hot += len(per)
            self.resume_resident += resident
            self.resume_total += len(s.hot)
            s.state = ACTIVE
            self.resumes += 1
            out.append(per)
        return out

    def resume_lazy(self, sids: Sequence[int]) -> None:
        """Resume without fetching: every non-resident page stays in the cold tier
        (spilled, read in place) until promoted.  Needs the spill option.
        Atomic as a whole."""
        sids = [int(x) for x in sids]
        if not self.spill:
            raise ModelError(ERR_INVALID, "lazy resume needs spill")
        if len(set(sids)) != len(sids):
            raise ModelError(ERR_INVALID, "duplicate session")
        for sid in sids:
            if self._session(sid).state != PAUSED:
                raise ModelError(ERR_STATE, "not paused")
        for sid in sids:
            s = self.sessions[sid]
            missing = [i for i, p in enumerate(s.hot) if p < 0]
            for i in missing:
                s.spilled[i] = True
            self.spilled_pages += len(missing)
            self.resume_resident += len(s.hot) - len(missing)
            self.resume_total += len(s.hot)
            s.state = ACTIVE
            self.resumes += 1

    def write_tokens(self, sid: int, tok_begin: int, n_tok: int) -> None:
        s = self._session(sid)
        if s.state != ACTIVE or tok_begin < 0 or n_tok < 0 or tok_begin + n_tok > s.seq_len:
            raise ModelError(ERR_INVALID if s.state == ACTIVE else ERR_STATE, "bad write")
        if n_tok == 0:
            return
        span = range(tok_begin // PAGE_TOKENS, (tok_begin + n_tok - 1) // PAGE_TOKENS + 1)
        if any(s.hot[i] < 0 and self.cold_ref[s.cold[i]] > 1 for i in span):
            raise ModelError(ERR_STATE, "spilled page shared with another session")
        for i in span:
            if s.hot[i] >= 0 and s.cold[i] >= 0:
                self._release_cold(s.cold[i])
                s.cold[i] = -1

    def destroy(self, sid: int) -> None:
        s = self._session(sid)
        if s.state == FREE:
            raise ModelError(ERR_STATE, "not in use")
        self.hot_free.update(p for p in s.hot if p >= 0)
        for c in s.cold:
            if c >= 0:
                self._release_cold(c)
        self.sessions[sid] = _Session()

    def promote(self, n: int):
        """Move up to n spilled pages of active sessions to the hot tier.
        Returns the (cold_src, hot_dst) copies."""
        if n < 0:
            raise ModelError(ERR_INVALID, "negative count")
        want = [(sid, i) for sid, s in enumerate(self.sessions) if s.state == ACTIVE
                for i, p in enumerate(s.hot) if p < 0][:n]
        victims, cold, pages, _ = self._plan(len(want), fresh_spill=False, spill=True)
        self.last_victim_copies = self._evict_victims(victims, cold)
        self._take_hot(pages)
        copies = []
        for (sid, i), h in zip(want, pages):
            s = self.sessions[sid]
            s.hot[i] = h
            s.spilled[i] = False
            copies.append((s.cold[i], h))
        self.promoted_pages += len(copies)
        self.pages_to_hot += len(copies)
        return copies

    # -- views ---------------------------------------------------------------
    def row(self, sid: int) -> List[int]:
        """Expected page-table row (length = row stride)."""
        s = self.sessions[sid]
        r = [] if s.state == FREE else [
            h if h >= 0 else (c | COLD_BIT if sp else -1) for h, c, sp in zip(s.hot, s.cold, s.spilled)]
        return r + [-1] * (self.stride - len(r))

    def table(self) -> List[List[int]]:
        return [self.row(sid) for sid in range(self.max_sessions)]

    def free_hot(self) -> int:
        return len(self.hot_free)

    def free_cold(self) -> int:
        return len(self.cold_free)

    def cold_active(self) -> int:
        """Pages of active sessions living in the cold tier (spilled)."""
        return sum(1 for s in self.sessions if s.state == ACTIVE for h in s.hot if h < 0)
