"""Reference split of decode-attention work over waves — TEST INFRASTRUCTURE ONLY.

The paper's decode simply reads every active session's KV each step (Sec. II;
Sec. III, data path 1).  How that read is divided among GPU waves is this
library's own design, not the paper's; this module states the rule by brute
force so that the GPU's closed-form version can be checked.

Rule:

* A *unit* is one page of one (session b, KV head g) pair.  Session b has
  ``n_b = ceil(L_b / 16)`` pages (0 when ``L_b <= 0``).
* Units are ordered by (b, g, page).  Segment ``j = b * Hkv + g`` is the run of
  units of that pair; ``T`` is the total number of units.
* Wave ``k`` of ``N`` takes units ``[floor(k T / N), floor((k + 1) T / N))``.
* Where a wave's range meets a segment it produces one *piece*: a partial
  result for (b, g) over a contiguous page range.  The piece is stored in slot
  ``k + j`` of a table with ``N + B * Hkv`` slots; the slot numbers of the
  pieces increase strictly along the unit order, so no two pieces share one.
"""

from __future__ import annotations

from typing import List, Tuple

PAGE_TOKENS = 16


def pieces(seq_lens, num_kv_heads: int, waves: int) -> List[Tuple[int, int, int, int, int, int]]:
    """All pieces as (slot, wave, b, g, page_begin, page_end), in unit order.

    Enumerates every unit one by one.
    """
    units = []  # (b, g, page)
    for b, L in enumerate(seq_lens):
        n = (int(L) + PAGE_TOKENS - 1) // PAGE_TOKENS if int(L) > 0 else 0
        for g in range(num_kv_heads):
            for i in range(n):
                units.append((b, g, i))
    T = len(units)
    bounds = [(k * T) // waves for k in range(waves + 1)]
    owner = []
    k = 0
    for u in range(T):
        while not (bounds[k] <= u < bounds[k + 1]):
            k += 1
        owner.append(k)
    out = []
    u = 0
    while u < T:
        b, g, i0 = units[u]
        k = owner[u]
        v = u
        while v < T and owner[v] == k and units[v][0] == b and units[v][1] == g:
            v += 1
        j = b * num_kv_heads + g
        out.append((k + j, k, b, g, i0, units[v - 1][2] + 1))
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
