"""The reference model of the cache tier's policy, pinned to the textbook
least-recently-used cache: with one matched row per lookup call it must hit
and miss exactly like an LRU cache of the same size, and its statistics must
follow their definitions."""
import collections

import numpy as np

from oracle.lru import GROUP, LruModel


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


def test_groups_split_long_calls():
    m = LruModel(GROUP, 0, row_bytes=1)
    rows = list(range(GROUP)) + [0]
    m.lookup(rows)
    # Row 0 was filled in the first group: cached when the second began, but
    # still served from host memory (it was not cached when the call began).
    assert m.stats["cache_hits"] == 1
    assert m.stats["host_bytes"] == GROUP + 1
    m2 = LruModel(GROUP, 0, row_bytes=1, fill_rereads=True)
    m2.lookup(rows)
    assert m2.stats["host_bytes"] == GROUP + (GROUP + 1)


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
