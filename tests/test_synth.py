"""The seeded input generator: its counter-based draws are re-derived here in
plain numpy, its Zipf sampler is checked against the law it samples, and its
n-gram ranking against collections.Counter."""
import collections

import numpy as np

import synth

M64 = (1 << 64) - 1


def mix(x):
    x ^= x >> 30
    x = (x * 0xBF58476D1CE4E5B9) & M64
    x ^= x >> 27
    x = (x * 0x94D049BB133111EB) & M64
    return x ^ (x >> 31)


def draw(k, i):
    return mix((k + (i + 1) * 0x9E3779B97F4A7C15) & M64)


def test_stream_key_and_normal_draws_match_python_twin():
    seed, tag = 7, 3
    key = draw(seed, tag)
    assert synth.stream_key(seed, tag) == key
    cols = 5
    got = synth.normal_rows(seed, tag, [0, 3, 11], cols, 0.02, synth.F32)
    scale = np.float32(0.02 / 65536)
    for r, row in enumerate([0, 3, 11]):
        for c in range(cols):
            e = row * cols + c
            s = 0
            for d in range(3):
                w = draw(key, 3 * e + d)
                s += sum((w >> (16 * q)) & 0xFFFF for q in range(4))
            want = np.float32(s - 393210) * scale
            assert got[r, c] == want
    b = synth.normal_rows(seed, tag, [3], cols, 0.02, synth.BF16)
    f = synth.normal_rows(seed, tag, [3], cols, 0.02, synth.F32)
    u = f.view(np.uint32).astype(np.uint64)
    np.testing.assert_array_equal(b, ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16))


def test_normal_moments():
    x = synth.normal_range(3, 9, 0, 256, 1024, 1.0, synth.F32).ravel().astype(np.float64)
    assert abs(x.mean()) < 0.01
    assert abs(x.std() - 1.0) < 0.01
    assert np.abs(x).max() <= 6.0


def test_zipf_frequencies():
    n, s = 2_000_000, 1.1
    t = synth.zipf_tokens(0, 99, n, s)
    assert t.min() >= 0 and t.max() < synth.V
    r = np.arange(1, synth.V + 1, dtype=np.float64)
    p = r ** -s
    p /= p.sum()
    cnt = np.bincount(t, minlength=synth.V)
    for k in range(20):
        sd = np.sqrt(n * p[k] * (1 - p[k]))
        assert abs(cnt[k] - n * p[k]) < 5 * sd
    # Mass of the head and of the tail.
    assert abs(cnt[:1000].sum() / n - p[:1000].sum()) < 0.005


def test_ngram_top_matches_counter():
    t = synth.zipf_tokens(1, 98, 200_000, 1.1, vocab=300)
    for n in (2, 3, 4):
        c = collections.Counter(tuple(t[i:i + n].tolist()) for i in range(t.size - n + 1))
        ranked = sorted(c.items(), key=lambda kv: (-kv[1], kv[0]))
        for skip in (0, 37):
            tup, cnt = synth.ngram_top(t, n, 500, skip=skip, vocab=300)
            want = ranked[skip:skip + 500]
            assert [tuple(x) for x in tup.tolist()] == [w for w, _ in want]
            assert cnt.tolist() == [k for _, k in want]
