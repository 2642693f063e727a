"""Oracle model of the hot/cold page pools and session states — TEST INFRASTRUCTURE ONLY.

It replays the documented policy on plain Python sets and lists and predicts,
for every call, the resulting page-table rows, the pages copied in each
direction and the number of cold-tier writes.  Nothing here touches a GPU or
the library.

Policy being modelled (paper Sec. III):

* Active sessions keep their KV in the hot tier; paused sessions keep it in the
  cold tier (Sec. III, first paragraph; data paths 2 and 4).
* Write-on-evict: a page is written to the cold tier only when it is evicted,
  and a cold copy stays valid after the session is resumed, because written KV
  never changes; an unmodified page is therefore written to the cold tier at
  most once (Sec. III, "Memory hierarchy and write policy").
* A resumed session's KV is brought back into the hot tier before it runs
  (Sec. III, "Eviction, resume and decode").

Readings where the paper is silent (each is stated in the design notes):

* Hot and cold pages are handed out lowest id first; a session's logical pages
  0..n-1 get the n lowest free ids in ascending order; batched calls process
  sessions in argument order; session ids are also handed out lowest first.
* Resume restores every page of the session (no partial residency).
* Writing tokens into a page that has a cold copy invalidates that copy, so the
  next eviction writes the page again.
* Cold pages may be shared by several paused sessions (a virtualised cold
  pool); they are reference counted and freed when the last user lets go.
* Every failing call leaves the whole state unchanged.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

PAGE_TOKENS = 16

FREE, ACTIVE, PAUSED = 0, 1, 2

OK, ERR_INVALID, ERR_STATE, ERR_NO_HOT, ERR_NO_COLD = 0, -1, -2, -3, -4


class ModelError(Exception):
    def __init__(self, code: int, msg: str = ""):
        super().__init__(msg or str(code))
        self.code = code


@dataclass
class _Session:
    state: int = FREE
    seq_len: int = 0
    hot: List[int] = field(default_factory=list)
    cold: List[int] = field(default_factory=list)  # -1 = no valid cold copy


def _pages(seq_len: int) -> int:
    return (seq_len + PAGE_TOKENS - 1) // PAGE_TOKENS


class PoolModel:
    def __init__(self, num_hot: int, num_cold: int, max_sessions: int, max_pages_per_session: int):
        self.num_hot, self.num_cold = num_hot, num_cold
        self.max_sessions, self.stride = max_sessions, max_pages_per_session
        self.hot_free = set(range(num_hot))
        self.cold_free = set(range(num_cold))
        self.cold_ref = [0] * num_cold
        self.sessions = [_Session() for _ in range(max_sessions)]
        self.cold_writes = 0          # pages written to the cold tier
        self.pages_to_hot = 0         # pages copied cold -> hot
        self.resumes = 0
        self.evicts = 0

    # -- helpers -----------------------------------------------------------
    def _take(self, free: set, n: int) -> List[int]:
        got = sorted(free)[:n]
        for p in got:
            free.remove(p)
        return got

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

    # -- calls ---------------------------------------------------------------
    def create(self, seq_len: int, pages: Optional[Sequence[int]] = None) -> int:
        if seq_len < 0 or _pages(seq_len) > self.stride:
            raise ModelError(ERR_INVALID, "bad length")
        n = _pages(seq_len)
        if pages is not None:
            pages = [int(p) for p in pages]
            if len(pages) != n or len(set(pages)) != n or any(p not in self.hot_free for p in pages):
                raise ModelError(ERR_INVALID, "pages not free/distinct")
        elif n > len(self.hot_free):
            raise ModelError(ERR_NO_HOT, "hot pool exhausted")
        sid = self._new_sid()
        if pages is None:
            pages = self._take(self.hot_free, n)
        else:
            for p in pages:
                self.hot_free.remove(p)
        self.sessions[sid] = _Session(ACTIVE, seq_len, list(pages), [-1] * n)
        return sid

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
        self.sessions[sid] = _Session(PAUSED, seq_len, [], list(cold_pages))
        return sid

    def evict(self, sid: int):
        """Returns the list of (hot_src, cold_dst) copies the eviction performs."""
        s = self._session(sid)
        if s.state != ACTIVE:
            raise ModelError(ERR_STATE, "not active")
        dirty = [i for i, c in enumerate(s.cold) if c < 0]
        if len(dirty) > len(self.cold_free):
            raise ModelError(ERR_NO_COLD, "cold pool exhausted")
        dst = self._take(self.cold_free, len(dirty))
        copies = []
        for i, c in zip(dirty, dst):
            s.cold[i] = c
            self.cold_ref[c] += 1
            copies.append((s.hot[i], c))
        self.cold_writes += len(dirty)
        self.hot_free.update(s.hot)
        s.hot = []
        s.state = PAUSED
        self.evicts += 1
        return copies

    def evict_many(self, sids: Sequence[int]):
        """Batched eviction, atomic as a whole: sessions in argument order.
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
        out = []
        for sid in sids:
            out += self.evict(sid)
        return out

    def resume(self, sids: Sequence[int]):
        """Batched resume, atomic as a whole.  Returns, per session, the list of
        (cold_src, hot_dst) copies in logical page order."""
        sids = [int(x) for x in sids]
        if len(set(sids)) != len(sids):
            raise ModelError(ERR_INVALID, "duplicate session")
        need = 0
        for sid in sids:
            s = self._session(sid)
            if s.state != PAUSED:
                raise ModelError(ERR_STATE, "not paused")
            need += len(s.cold)
        if need > len(self.hot_free):
            raise ModelError(ERR_NO_HOT, "hot pool exhausted")
        out = []
        for sid in sids:
            s = self.sessions[sid]
            dst = self._take(self.hot_free, len(s.cold))
            s.hot = dst
            s.state = ACTIVE
            out.append(list(zip(s.cold, dst)))
            self.pages_to_hot += len(dst)
            self.resumes += 1
        return out

    def write_tokens(self, sid: int, tok_begin: int, n_tok: int) -> None:
        s = self._session(sid)
        if s.state != ACTIVE or tok_begin < 0 or n_tok < 0 or tok_begin + n_tok > s.seq_len:
            raise ModelError(ERR_INVALID if s.state == ACTIVE else ERR_STATE, "bad write")
        if n_tok == 0:
            return
        for i in range(tok_begin // PAGE_TOKENS, (tok_begin + n_tok - 1) // PAGE_TOKENS + 1):
            if s.cold[i] >= 0:
                self._release_cold(s.cold[i])
                s.cold[i] = -1

    def destroy(self, sid: int) -> None:
        s = self._session(sid)
        if s.state == FREE:
            raise ModelError(ERR_STATE, "not in use")
        self.hot_free.update(s.hot)
        for c in s.cold:
            if c >= 0:
                self._release_cold(c)
        self.sessions[sid] = _Session()

    # -- views ---------------------------------------------------------------
    def row(self, sid: int) -> List[int]:
        """Expected page-table row (length = row stride)."""
        s = self.sessions[sid]
        r = list(s.hot) if s.state == ACTIVE else []
        return r + [-1] * (self.stride - len(r))

    def table(self) -> List[List[int]]:
        return [self.row(sid) for sid in range(self.max_sessions)]

    def free_hot(self) -> int:
        return len(self.hot_free)

    def free_cold(self) -> int:
        return len(self.cold_free)
