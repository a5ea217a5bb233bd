"""Pins of the oracle's multi-match path (Eq. 4, Eq. 11: every matched
phrase is retained and the rows are combined with weights that add up to 1):
a brute-force scan of every phrase for every window, closed-form weighted
sums on rows whose products are exact, the reduction to single-match
injection, and the gate evaluated on the aggregated signal (Eq. 5)."""
import math

import numpy as np
import pytest

import oracle
import synth

from .test_oracle_pins import table_of


def brute_force_all(toks, lens, tokens, ctx, S, n_min, n_max, vocab):
    """Scan every stored phrase for every window of every length."""
    B = tokens.shape[0]
    L = n_max - n_min + 1
    mask = np.zeros(B * S, np.uint8)
    rows = np.full((B * S, L), -1, np.int32)
    for b in range(B):
        for s in range(S):
            c = ctx + s
            p = b * S + s
            for j, n in enumerate(range(n_min, n_max + 1)):
                if c - n + 1 < 0:
                    continue
                w = tokens[b, c - n + 1:c + 1]
                if np.any(w < 0) or np.any(w >= vocab):
                    continue
                idx = np.flatnonzero((lens == n) & np.all(toks[:, :n] == w[None, :], axis=1))
                assert idx.size <= 1
                if idx.size:
                    rows[p, j] = idx[0]
                    mask[p] |= 1 << j
    return mask, rows


def test_lookup_all_matches_brute_force_with_pads_and_4grams():
    rng = np.random.default_rng(12)
    vocab = 5
    phrases = set()
    for n, want in ((2, 15), (3, 60), (4, 300)):
        got = set()
        while len(got) < want:
            got.add(tuple(int(x) for x in rng.integers(0, vocab, n)))
        phrases |= got
    phrases = sorted(phrases, key=lambda w: (len(w) * 7919 + sum(w) * 31) % 997)
    t, toks, lens = table_of(phrases, 2, 4, vocab)
    tokens = rng.integers(-1, vocab + 1, (8, 3 + 29)).astype(np.int32)
    mask, rows = t.lookup_all(tokens, 3, 29)
    emask, erows = brute_force_all(toks, lens, tokens, 3, 29, 2, 4, vocab)
    np.testing.assert_array_equal(mask, emask)
    np.testing.assert_array_equal(rows, erows)
    # Every subset of lengths occurs, including all three at once.
    assert set(mask.tolist()) >= {0, 1, 3, 7}
    # The longest retained phrase is the longest-match selection.
    hit, row, ln = t.lookup(tokens, 3, 29)
    top = np.where(mask > 0, np.floor(np.log2(np.maximum(mask, 1))).astype(int), -1)
    np.testing.assert_array_equal(hit, (mask > 0).astype(np.uint8))
    np.testing.assert_array_equal(ln, np.where(top >= 0, top + 2, 0))
    sel = np.where(top >= 0, rows[np.arange(rows.shape[0]), np.maximum(top, 0)], -1)
    np.testing.assert_array_equal(row, sel)


def test_lookup_all_hand_enumerated():
    # (7,9) -> 0, (5,7,9) -> 1, (9,7) -> 2, (3,5) -> 3
    t, _, _ = table_of([(7, 9), (5, 7, 9), (9, 7), (3, 5)])
    mask, rows = t.lookup_all(np.array([[3, 5, 7, 9, 7]], np.int32), 0, 5)
    np.testing.assert_array_equal(mask, [0, 1, 0, 3, 1])
    np.testing.assert_array_equal(rows, [[-1, -1], [3, -1], [-1, -1], [0, 1], [2, -1]])


def unit(D, k, c):
    v = np.zeros(D, np.float32)
    v[k] = c
    return v


@pytest.mark.parametrize("weighting,lens_present,scale,want", [
    # by length: alpha_j = n_j / sum n
    (oracle.WEIGHT_LENGTH, (2, 3), 5.0, {0: 2.0, 1: 3.0}),
    (oracle.WEIGHT_LENGTH, (2, 3, 4), 9.0, {0: 2.0, 1: 3.0, 2: 4.0}),
    (oracle.WEIGHT_LENGTH, (3, 4), 7.0, {1: 3.0, 2: 4.0}),
    (oracle.WEIGHT_LENGTH, (2, 4), 6.0, {0: 2.0, 2: 4.0}),
    # uniform: alpha_j = 1 / count
    (oracle.WEIGHT_UNIFORM, (2, 3), 2.0, {0: 1.0, 1: 1.0}),
    (oracle.WEIGHT_UNIFORM, (2, 3, 4), 3.0, {0: 1.0, 1: 1.0, 2: 1.0}),
])
def test_weighted_sum_closed_form(weighting, lens_present, scale, want):
    """Row of length n is scale * e_{n-2}; with the constant gate the output
    is h + lambda * sum alpha_n * scale * e_{n-2}, exact in float32."""
    D, n_min = 64, 2
    values = np.stack([unit(D, n - 2, scale) for n in (2, 3, 4)])
    h = (np.arange(D, dtype=np.float32) - 20.0)[None]
    idx = np.full((1, 3), -1, np.int64)
    for n in lens_present:
        idx[0, n - n_min] = n - 2
    for lam in (1.0, 0.5):
        out = oracle.inject_multi(h, values, idx, n_min, synth.F32, weighting, oracle.GATE_CONST,
                                  lam)
        exp = h[0].copy()
        for k, c in want.items():
            exp[k] += lam * c
        np.testing.assert_array_equal(out[0], exp)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
@pytest.mark.parametrize("gate", [oracle.GATE_SIGMOID, oracle.GATE_CONST])
@pytest.mark.parametrize("weighting", [oracle.WEIGHT_LENGTH, oracle.WEIGHT_UNIFORM])
def test_single_retained_row_is_single_match_injection(dtype, gate, weighting):
    D, T = 1024, 6
    h = synth.normal_range(3, 910, 0, T, D, 1.0, dtype)
    v = synth.normal_range(3, 911, 0, T, D, 0.02, dtype)
    idx = np.full((T, 3), -1, np.int64)
    idx[np.arange(T), np.arange(T) % 3] = np.arange(T)
    got = oracle.inject_multi(h, v, idx, 2, dtype, weighting, gate, 0.8)
    want = oracle.inject(h, v, np.arange(T), dtype, gate, 0.8)
    assert got.tobytes() == want.tobytes()


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_equal_rows_aggregate_to_the_row(dtype):
    """Weights add up to 1: retaining the same vector several times gives the
    vector itself (exact for uniform halves)."""
    D, T = 1024, 4
    h = synth.normal_range(4, 912, 0, T, D, 1.0, dtype)
    v = synth.normal_range(4, 913, 0, 1, D, 0.02, dtype)
    v2 = np.concatenate([v, v, v])
    want = oracle.inject(h, v, np.zeros(T, np.int64), dtype)
    idx = np.array([[0, 1, -1]] * T, np.int64)
    got = oracle.inject_multi(h, v2, idx, 2, dtype, oracle.WEIGHT_UNIFORM)
    assert got.tobytes() == want.tobytes()
    idx3 = np.array([[0, 1, 2]] * T, np.int64)
    got = oracle.inject_multi(h, v2, idx3, 2, dtype, oracle.WEIGHT_LENGTH)
    a = synth.bf16_to_f32(got) if dtype == synth.BF16 else got
    b = synth.bf16_to_f32(want) if dtype == synth.BF16 else want
    # alpha sums to 1 up to double rounding: outputs equal, or one unit apart
    # in the last place of the output type.
    step = np.spacing(np.abs(b).astype(np.float32)) * (256 if dtype == synth.BF16 else 1)
    assert np.all(np.abs(a.astype(np.float64) - b) <= step)
    assert np.mean(a == b) > 0.99


def test_gate_is_evaluated_on_the_aggregated_signal():
    """h parallel to m = 0.4 v2 + 0.6 v3 but not to either row: the sigmoid
    gate reaches its parallel limit sigmoid(sqrt(D)) only for the aggregate
    (D = 16 keeps the logistic function away from saturation)."""
    D = 16
    a = synth.normal_range(6, 914, 0, 1, D, 1.0, synth.F32)[0].astype(np.float64)
    b = synth.normal_range(6, 915, 0, 1, D, 1.0, synth.F32)[0].astype(np.float64)
    a[1::2] = 0
    b[0::2] = 0
    v2, v3 = (5.0 * a).astype(np.float32), (5.0 * b).astype(np.float32)
    m = 0.4 * v2.astype(np.float64) + 0.6 * v3.astype(np.float64)
    h = (3.0 * m).astype(np.float32)
    lam = 1.5
    out = oracle.inject_multi(h[None], np.stack([v2, v3]), np.array([[0, 1]]), 2, synth.F32,
                              oracle.WEIGHT_LENGTH, oracle.GATE_SIGMOID, lam)[0]
    nz = np.abs(m) > 1e-3
    g = (out[nz].astype(np.float64) - h[nz]) / m[nz]
    want = lam / (1.0 + math.exp(-math.sqrt(D)))
    assert np.all(np.abs(g - want) < 1e-5)
    # With only the longer row retained the gate is far from that limit.
    out3 = oracle.inject(h[None], v3[None], np.array([0]), synth.F32, oracle.GATE_SIGMOID, lam)[0]
    g3 = oracle.gate_value(h, v3, synth.F32, lam=lam)
    assert abs(g3 - want) > 1e-3 and out3.tobytes() != out.tobytes()


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_multi_noop_invariants(dtype):
    D, T = 512, 5
    h = synth.normal_range(7, 916, 0, T, D, 1.0, dtype)
    v = synth.normal_range(7, 917, 0, 3, D, 0.02, dtype)
    out = oracle.inject_multi(h, v, np.full((T, 3), -1), 2, dtype)
    assert out.tobytes() == h.tobytes()
    z = np.zeros_like(v)
    idx = np.tile(np.array([0, 1, 2]), (T, 1))
    for w in (oracle.WEIGHT_LENGTH, oracle.WEIGHT_UNIFORM):
        for gate in (oracle.GATE_SIGMOID, oracle.GATE_CONST):
            assert oracle.inject_multi(h, z, idx, 2, dtype, w, gate).tobytes() == h.tobytes()
    # Opposite rows of equal weight cancel: uniform over +v and -v.
    vv = np.concatenate([v[:1], v[:1]])
    if dtype == synth.F32:
        vv[1] = -vv[1]
    else:
        vv[1] ^= 0x8000
    out = oracle.inject_multi(h, vv, np.tile(np.array([0, 1, -1]), (T, 1)), 2, dtype,
                              oracle.WEIGHT_UNIFORM, oracle.GATE_CONST)
    assert out.tobytes() == h.tobytes()


def test_multi_rejects_bad_arguments():
    h = np.zeros((2, 8), np.float32)
    v = np.zeros((2, 8), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.inject_multi(h, v, np.array([[0, 2], [0, 1]]), 2, synth.F32)
    with pytest.raises(oracle.OracleError):
        oracle.inject_multi(h, v, np.array([[0, 1], [0, 1]]), 2, synth.F32, weighting=7)
