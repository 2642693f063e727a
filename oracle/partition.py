"""Reference split of decode-attention work over waves — TEST INFRASTRUCTURE ONLY.

The paper's decode simply reads every active session's KV each step (Sec. II;
Sec. III, data path 1).  How that read is divided among GPU waves is this
library's own design, not the paper's; this module states the rule by brute
force so that the GPU's closed-form version can be checked.

Rule:

* Group width ``L``: 4 when the KV heads come in fours (``Hkv % 4 == 0``) and
  the waves too (``N % 4 == 0``), else 1.  ``L`` consecutive waves form one
  *worker*; wave ``w`` of a worker takes KV head ``L * hg + w`` of each head
  group ``hg`` it meets (``Hkv / L`` groups per session).
* A *unit* is one page of one (session b, head group hg) pair.  Session b has
  ``n_b = ceil(L_b / 16)`` pages (0 when ``L_b <= 0``).
* Units are ordered by (b, hg, page).  Super-segment ``s = b * Hkv / L + hg``
  is the run of units of that pair; ``T`` is the total number of units.
* Worker ``k`` of ``N / L`` takes units ``[floor(k T / (N / L)),
  floor((k + 1) T / (N / L)))``.
* Where a worker's range meets a super-segment, each of its waves produces one
  *piece*: a partial result for its (b, g) over a contiguous page range.  Wave
  ``w``'s piece is stored in slot ``(k + s) * L + w`` of a table with
  ``N + B * Hkv`` slots; the slot numbers of the pieces increase strictly
  along the unit order, so no two pieces share one.  With ``L = 1`` a worker
  is a single wave and a unit one page of one KV head.
"""

from __future__ import annotations

from typing import List, Tuple

PAGE_TOKENS = 16


def group_waves(num_kv_heads: int, waves: int) -> int:
    """Waves sharing one unit, one KV head each."""
    return 4 if num_kv_heads % 4 == 0 and waves % 4 == 0 else 1


def pieces(seq_lens, num_kv_heads: int, waves: int) -> List[Tuple[int, int, int, int, int, int]]:
    """All pieces as (slot, wave, b, g, page_begin, page_end), in unit order and,
    within a unit run, in wave order.

    Enumerates every unit one by one.
    """
    L = group_waves(num_kv_heads, waves)
    groups = num_kv_heads // L
    workers = waves // L
    units = []  # (b, hg, page)
    for b, length in enumerate(seq_lens):
        n = (int(length) + PAGE_TOKENS - 1) // PAGE_TOKENS if int(length) > 0 else 0
        for hg in range(groups):
            for i in range(n):
                units.append((b, hg, i))
    T = len(units)
    bounds = [(k * T) // workers for k in range(workers + 1)]
    owner = []
    k = 0
    for u in range(T):
        while not (bounds[k] <= u < bounds[k + 1]):
            k += 1
        owner.append(k)
    out = []
    u = 0
    while u < T:
        b, hg, i0 = units[u]
        k = owner[u]
        v = u
        while v < T and owner[v] == k and units[v][0] == b and units[v][1] == hg:
            v += 1
        s = b * groups + hg
        for w in range(L):
            out.append(((k + s) * L + w, k * L + w, b, hg * L + w, i0, units[v - 1][2] + 1))
        u = v
    return out


def slot_table(seq_lens, num_kv_heads: int, waves: int):
    """Dense table of ``waves + B * Hkv`` records (b, g, page_begin, page_end);
    slots without a piece hold (-1, -1, 0, 0)."""
    n_slots = waves + len(seq_lens) * num_kv_heads
    table = [(-1, -1, 0, 0)] * n_slots
    for slot, _k, b, g, p0, p1 in pieces(seq_lens, num_kv_heads, waves):
        assert table[slot][0] == -1, "two pieces in one slot"
        table[slot] = (b, g, p0, p1)
    return table
