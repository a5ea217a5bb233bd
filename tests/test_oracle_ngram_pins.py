"""Pins of the oracle's phrase-table construction (Sec. 4.2: candidate
phrases selected by corpus frequency): a hand-counted stream, a brute-force
Counter over random streams with invalid tokens and many equal counts, the
skip/top windows of one ranking, the window-count invariant, and agreement
with the input generator's independent partitioned implementation (on small
streams here, and at the full 2^26-token workload size through the digests
of the oracle's ranking in tests/golden/ngram_top_workload2.json)."""
import collections
import hashlib
import json
import os

import numpy as np
import pytest

import oracle
import synth


def brute(tokens, vocab, n):
    c = collections.Counter()
    for i in range(len(tokens) - n + 1):
        w = tuple(int(x) for x in tokens[i:i + n])
        if all(0 <= x < vocab for x in w):
            c[w] += 1
    return sorted(c.items(), key=lambda kv: (-kv[1], kv[0]))


def test_hand_counted():
    tup, cnt = oracle.ngram_top(np.array([1, 2, 1, 2, 1, 2, 3]), 10, 2, 0, 10)
    assert tup.tolist() == [[1, 2], [2, 1], [2, 3]]
    assert cnt.tolist() == [3, 2, 1]
    tup, cnt = oracle.ngram_top(np.array([5, 5, 5, 5]), 10, 3, 0, 10)
    assert tup.tolist() == [[5, 5, 5]] and cnt.tolist() == [2]


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_matches_counter_with_invalid_tokens(n):
    rng = np.random.default_rng(30 + n)
    vocab = 5
    tokens = rng.integers(-1, vocab + 1, 3000).astype(np.int32)
    want = brute(tokens, vocab, n)
    tup, cnt = oracle.ngram_top(tokens, vocab, n, 0, len(want) + 5)
    assert [tuple(t) for t in tup.tolist()] == [w for w, _ in want]
    assert cnt.tolist() == [c for _, c in want]
    # Every valid window is counted exactly once.
    valid = sum(all(0 <= x < vocab for x in tokens[i:i + n]) for i in range(len(tokens) - n + 1))
    assert int(cnt.sum()) == valid


def test_skip_and_top_are_windows_of_one_ranking():
    rng = np.random.default_rng(7)
    tokens = rng.integers(0, 6, 5000).astype(np.int32)
    full_t, full_c = oracle.ngram_top(tokens, 6, 3, 0, 10 ** 6)
    assert len(full_t) == 216
    for skip, top in [(0, 5), (10, 20), (200, 50), (216, 3), (300, 3)]:
        t, c = oracle.ngram_top(tokens, 6, 3, skip, top)
        np.testing.assert_array_equal(t, full_t[skip:skip + top])
        np.testing.assert_array_equal(c, full_c[skip:skip + top])


def test_empty_cases():
    t, c = oracle.ngram_top(np.array([1], np.int32), 10, 2, 0, 5)
    assert t.shape == (0, 2)
    t, c = oracle.ngram_top(np.array([1, 2, 3], np.int32), 10, 2, 0, 0)
    assert t.shape == (0, 2)
    with pytest.raises(oracle.OracleError):
        oracle.ngram_top(np.array([1, 2, 3], np.int32), 10, 5, 0, 1)


@pytest.mark.parametrize("n", [2, 3])
def test_agrees_with_the_generators_partitioned_count(n):
    toks = synth.zipf_tokens(11, 77, 1 << 18, 1.1)
    want_t, want_c = synth.ngram_top(toks, n, 3000, skip=100)
    t, c = oracle.ngram_top(toks, synth.V, n, 100, 3000)
    np.testing.assert_array_equal(t, want_t)
    np.testing.assert_array_equal(c, want_c)


def test_generator_matches_oracle_digests_at_full_size():
    """The stored digests come from the oracle's ranking of the full
    2^26-token workload-2 stream (tests/golden/make_ngram_digests.py, which
    calls only the oracle and the generator).  The generator's stream and
    its partitioned count -- the GPU tests' second reference -- reproduce
    them; the head ranks are checked in clear against the stream."""
    golden = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                         "ngram_top_workload2.json")))
    sha = lambda a: hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
    toks = synth.workload2_stream()
    assert sha(toks) == golden["stream_sha256"] and toks.size == golden["stream_tokens"]
    for n in (2, 3, 4):
        g = golden["n"][str(n)]
        t, c = synth.ngram_top(toks, n, golden["top"])
        assert sha(t.astype("<i4")) == g["tuples_sha256"]
        assert sha(c.astype("<i8")) == g["counts_sha256"]
        # The most frequent tuple's count, by a direct scan of the stream.
        head = np.array(g["head"][0][0], np.int32)
        hits = np.ones(toks.size - n + 1, bool)
        for j in range(n):
            hits &= toks[j:toks.size - n + 1 + j] == head[j]
        assert int(hits.sum()) == g["head"][0][1]
