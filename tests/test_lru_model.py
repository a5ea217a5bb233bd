"""The reference model of the cache tier's policy, pinned to the textbook
least-recently-used cache: with one matched row per lookup call it must hit
and miss exactly like an LRU cache of the same size, and its statistics must
follow their definitions."""
import collections

import numpy as np

from oracle.lru import LruModel


def textbook_lru(capacity, prefill, seq):
    """Classic LRU over rows: hit if present (becomes most recent), else the
    least recent row leaves and the new row enters as most recent."""
    c = collections.OrderedDict()
    for r in range(prefill - 1, -1, -1):  # least recent = highest row
        c[r] = None
    out = []
    for r in seq:
        if r in c:
            c.move_to_end(r)
            out.append(True)
        else:
            if len(c) >= capacity:
                c.popitem(last=False)
            c[r] = None
            out.append(False)
    return out


def test_single_row_calls_are_textbook_lru():
    rng = np.random.default_rng(0)
    for capacity, prefill in ((8, 8), (8, 0), (16, 5), (64, 64)):
        seq = [int(x) for x in rng.zipf(1.3, 3000) % 200]
        m = LruModel(capacity, prefill, row_bytes=1)
        got = []
        for r in seq:
            before = m.stats["cache_hits"]
            m.lookup([r])
            got.append(m.stats["cache_hits"] > before)
        assert got == textbook_lru(capacity, prefill, seq)


def test_statistics_definitions():
    m = LruModel(4, 2, row_bytes=10)
    # rows 0, 1 cached; 5 and 6 miss and take the two empty slots; 0 hits twice.
    m.lookup([0, 5, -1, 0, 6, 5])
    assert m.stats["positions"] == 6
    assert m.stats["hits"] == 5
    assert m.stats["cache_hits"] == 2
    assert m.stats["cache_misses"] == 3
    # host bytes: 3 positions served from host (5, 6, 5); the fill copies the
    # rows those reads brought in.
    assert m.stats["host_bytes"] == 10 * 3
    assert set(m.resident()) == {0, 1, 5, 6}
    # A fill that reads the rows again adds the 2 filled rows.
    m2 = LruModel(4, 2, row_bytes=10, fill_rereads=True)
    m2.lookup([0, 5, -1, 0, 6, 5])
    assert m2.stats["host_bytes"] == 10 * (2 + 3)
    # Cache full; 7 evicts the least recent slot that is not referenced: row 1.
    m.lookup([7, 0])
    assert set(m.resident()) == {0, 5, 6, 7}
    # Prefetch fills a non-cached row and marks it; its first lookup counts.
    m.prefetch([9, 9, 0, -1])
    assert m.stats["prefetch_keys"] == 4 and m.stats["prefetch_found"] == 3
    assert m.stats["prefetch_filled"] == 1 and 9 in m.resident()
    m.lookup([9, 9])
    assert m.stats["prefetch_used"] == 1


def test_no_free_slot_reads_from_host_without_caching():
    m = LruModel(2, 2, row_bytes=1)
    src = m.lookup([0, 1, 7])      # 0, 1 referenced: 7 finds no victim
    assert src[2] == ("host", None) and 7 not in m.resident()


def test_long_call_never_evicts_a_row_it_uses_later():
    """A call of more than 4096 positions whose first position misses while
    the least recent cached row is named only at its last position: the miss
    must take the next least recent slot, and the late position is a cache
    hit.  (An implementation that chose the first position's victim before
    looking at the rest of the call would evict row 3 and miss it again.)"""
    T = 5000
    m = LruModel(4, 4, row_bytes=1)   # rows 0..3 cached; least recent: row 3
    rows = [100] + [-1] * (T - 2) + [3]
    src = m.lookup(rows)
    assert src[0] == ("fill", 2) and src[-1] == ("cache", 3)
    assert m.resident() == {0: 0, 1: 1, 3: 3, 100: 2}
    assert m.stats["cache_hits"] == 1 and m.stats["cache_misses"] == 1
    assert m.stats["host_bytes"] == 1
    # Recency after the call: by first position, row 100 (slot 2) before row 3.
    assert list(m.order) == [1, 0, 2, 3]


def test_repeated_missed_row_is_filled_once_per_call():
    m = LruModel(8, 0, row_bytes=1)
    rows = [5, 6] * 3000 + [7]
    src = m.lookup(rows)
    assert src[0] == ("fill", 0) and src[1] == ("fill", 1) and src[-1] == ("fill", 2)
    assert src[2] == ("fill", 0)          # later positions of a filled row
    assert m.stats["cache_hits"] == 0
    # Every position was served from host (its row was not cached when the
    # call began); a re-reading fill adds the three filled rows once.
    assert m.stats["host_bytes"] == len(rows)
    m2 = LruModel(8, 0, row_bytes=1, fill_rereads=True)
    m2.lookup(rows)
    assert m2.stats["host_bytes"] == len(rows) + 3


def test_full_cache_long_call_matches_brute_force_definition():
    """Against the policy stated from scratch on a recency list: the set of
    slots a call references is fixed before any victim is chosen."""
    rng = np.random.default_rng(7)
    C, pre = 12, 12
    m = LruModel(C, pre, row_bytes=1)
    # Independent statement: list of (slot, row) least recent first.
    order = [(s, s) for s in range(pre - 1, -1, -1)]
    for call in range(40):
        rows = [int(x) if x < 30 else -1 for x in rng.integers(0, 34, 4100 + call)]
        firsts = list(dict.fromkeys(r for r in rows if r >= 0))
        held = {r: s for s, r in order}
        ref = {held[r] for r in firsts if r in held}
        newly = {}
        for r in firsts:
            if r in held:
                newly[r] = held[r]
        for r in firsts:
            if r in held:
                continue
            free = [s for s, _ in order if s not in ref]
            if not free:
                continue
            v = free[0]
            order = [(s, rr) for s, rr in order if s != v] + []
            order.insert(0, (v, r))       # provisional place; moved below
            ref.add(v)
            newly[r] = v
        moved = sorted(newly, key=firsts.index)
        keep = [(s, r) for s, r in order if s not in set(newly.values())]
        order = keep + [(newly[r], r) for r in moved]
        m.lookup(rows)
        assert m.resident() == {r: s for s, r in order}
        assert list(m.order) == [s for s, _ in order]


def test_scored_prefetch_orders_by_score_and_respects_budget():
    import numpy as np
    m = LruModel(8, 0, row_bytes=1)
    rows = [10, 11, 12, 10, 13, -1]
    lens = [2, 3, 2, 3, 2, 0]
    prob = np.array([0.5, 0.1, 0.2, 0.3, 0.0, 0.9], np.float32)
    # scores: 10 -> max(1.0, 0.9) = 1.0; 11 -> 0.3; 12 -> 0.4; 13 -> 0 (not fetched)
    m.prefetch_scored(rows, lens, prob, budget=2)
    assert set(m.resident()) == {10, 12}
    assert m.stats["prefetch_filled"] == 2 and m.stats["prefetch_dropped"] == 1
    # Recency: 10 then 12 were filled in score order (10 first = less recent).
    assert list(m.order)[-2:] == [m.resident()[10], m.resident()[12]]


def test_prefetch_never_evicts_a_row_it_names():
    """A prefetch references its cached candidate rows like a lookup does:
    the least recent slot holds a candidate row, so the fill takes the next
    one, and both become most recent in candidate order."""
    m = LruModel(2, 2, row_bytes=1)          # rows 0, 1 cached; least recent: row 1
    m.prefetch([5, 1, -1, 5])
    assert m.resident() == {1: 1, 5: 0}
    assert m.stats["prefetch_filled"] == 1 and m.stats["prefetch_found"] == 3
    assert list(m.order) == [0, 1]
    assert m.stats["hits"] == 0 and m.stats["cache_hits"] == 0
    m.lookup([5])                             # the prefetched row is used once
    assert m.stats["prefetch_used"] == 1
    # No unreferenced slot left: the row stays in host memory.
    m4 = LruModel(2, 2, row_bytes=1)
    m4.prefetch([0, 1, 7])
    assert m4.resident() == {0: 0, 1: 1} and m4.stats["prefetch_filled"] == 0


def test_scored_prefetch_references_cached_rows_with_positive_score():
    m = LruModel(2, 2, row_bytes=1)
    m.prefetch_scored([5, 1], [2, 2], np.array([0.5, 0.25], np.float32), budget=4)
    assert m.resident() == {1: 1, 5: 0}
    # Recency: the referenced row first (by candidate), then the fill.
    assert list(m.order) == [1, 0]
    # A cached row whose candidates all have probability 0 is not referenced.
    m3 = LruModel(2, 2, row_bytes=1)
    m3.prefetch_scored([5, 1, 6], [2, 2, 2], np.array([0.5, 0.0, 0.25], np.float32), budget=4)
    assert m3.resident() == {5: 1, 6: 0}
    assert m3.stats["prefetch_filled"] == 2 and m3.stats["prefetch_dropped"] == 0
