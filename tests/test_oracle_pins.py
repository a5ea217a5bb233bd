"""Pins of the CPU oracle against facts fixed by the paper and by arithmetic,
not against the oracle itself: hand-enumerated windows, a brute-force scan of
every phrase, closed forms of the gate, exact rounding, and the no-op
invariants of gated residual injection (Eq. 5)."""
import fractions
import math

import numpy as np
import pytest
import torch

import oracle
import synth

V = synth.V


def bf16_bits_of_f32(x):
    """float32 -> bfloat16 bits, nearest-even, by integer rounding of the
    float32 bit pattern (finite inputs)."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def table_of(phrases, n_min=2, n_max=3, vocab=V):
    toks = np.full((len(phrases), n_max), -1, np.int32)
    lens = np.zeros(len(phrases), np.uint8)
    for i, w in enumerate(phrases):
        k = min(len(w), n_max)
        toks[i, :k] = w[:k]
        lens[i] = len(w)
    return oracle.Table(toks, lens, n_min, n_max, vocab), toks, lens


# ---------------------------------------------------------------- windows ---

def test_hand_enumerated_windows():
    # Phrases: (7,9) -> 0, (5,7,9) -> 1, (9,7) -> 2, (3,5) -> 3.
    t, _, _ = table_of([(7, 9), (5, 7, 9), (9, 7), (3, 5)])
    toks = np.array([[5, 7, 9, 7, 9]], np.int32)
    hit, row, ln = t.lookup(toks, 0, 5)
    # col 0: no window; col 1: (5,7) absent; col 2: (5,7,9) beats (7,9);
    # col 3: (7,9,7) absent, (9,7) present; col 4: (9,7,9) absent, (7,9).
    assert hit.tolist() == [0, 0, 1, 1, 1]
    assert row.tolist() == [-1, -1, 1, 2, 0]
    assert ln.tolist() == [0, 0, 3, 2, 2]


def test_history_columns_and_row_boundaries():
    t, _, _ = table_of([(7, 9), (5, 7, 9), (9, 3)])
    # Two rows, ctx = 2 history columns, S = 2 injected columns.  The window
    # of row 1's first injected column may use row 1's history but never row 0.
    toks = np.array([[1, 5, 7, 9],
                     [9, 3, 7, 9]], np.int32)
    hit, row, ln = t.lookup(toks, 2, 2)
    # row 0: col 2 -> (1,5,7),(5,7) absent; col 3 -> (5,7,9).
    # row 1: col 2 -> (9,3,7),(3,7) absent; col 3 -> (3,7,9) absent, (7,9).
    assert row.tolist() == [-1, 1, -1, 0]
    assert ln.tolist() == [0, 3, 0, 2]
    # History columns are never outputs: 4 positions for B*S = 4.
    assert hit.size == 4


def test_pads_and_out_of_range_tokens_break_windows():
    t, _, _ = table_of([(7, 9), (5, 7, 9), (9, 7)])
    toks = np.array([[5, 7, 9, -1, 7, 9, V, 9, 7]], np.int32)
    hit, row, ln = t.lookup(toks, 0, 9)
    # col 2: (5,7,9); col 3: pad -> nothing; col 4: (-1,7) and (9,-1,7)
    # broken -> nothing; col 5: (7,9) (3-gram has the pad); col 6: V is out
    # of range -> nothing; col 7: windows hold V -> nothing; col 8: (9,7).
    assert row.tolist() == [-1, -1, 1, -1, -1, 0, -1, -1, 2]
    assert ln.tolist() == [0, 0, 3, 0, 0, 2, 0, 0, 2]


def test_window_count_closed_form():
    # A table holding every window of the input matches every position whose
    # windows are formed: sum over b of max(0, ctx+S-n_min+1) minus history.
    rng = np.random.default_rng(5)
    B, ctx, S = 3, 2, 6
    toks = rng.integers(0, 50, (B, ctx + S)).astype(np.int32)
    phrases = set()
    for b in range(B):
        for c in range(ctx + S):
            for n in (2, 3):
                if c - n + 1 >= 0:
                    phrases.add(tuple(toks[b, c - n + 1:c + 1].tolist()))
    t, _, _ = table_of(sorted(phrases))
    hit, _, ln = t.lookup(toks, ctx, S)
    assert int(hit.sum()) == B * S          # ctx >= 1: every position has a 2-gram
    assert set(ln.tolist()) == {3}          # ctx >= 2: the 3-gram always exists


# ------------------------------------------------------------ brute force ---

def brute_force_lookup(toks, lens, tokens, ctx, S, n_min, n_max, vocab):
    """Scan every stored phrase for every window; keep the longest match."""
    B = tokens.shape[0]
    hit = np.zeros(B * S, np.uint8)
    row = np.full(B * S, -1, np.int32)
    ln = np.zeros(B * S, np.uint8)
    for b in range(B):
        for s in range(S):
            c = ctx + s
            best = (-1, 0)
            for n in range(n_min, n_max + 1):
                if c - n + 1 < 0:
                    continue
                w = tokens[b, c - n + 1:c + 1]
                if np.any(w < 0) or np.any(w >= vocab):
                    continue
                eq = (lens == n) & np.all(toks[:, :n] == w[None, :], axis=1)
                idx = np.flatnonzero(eq)
                assert idx.size <= 1
                if idx.size and n > best[1]:
                    best = (int(idx[0]), n)
            p = b * S + s
            if best[0] >= 0:
                hit[p], row[p], ln[p] = 1, best[0], best[1]
    return hit, row, ln


def test_oracle_matches_brute_force_on_workload1():
    table, batch = synth.config1()
    t = oracle.Table(table.tokens, table.lens, 2, 3, V)
    got = t.lookup(batch.tokens, batch.ctx, batch.S)
    exp = brute_force_lookup(table.tokens, table.lens, batch.tokens, batch.ctx, batch.S, 2, 3, V)
    for g, e in zip(got, exp):
        np.testing.assert_array_equal(g, e)
    assert 0 < int(got[0].sum()) < batch.S


def test_oracle_matches_brute_force_with_pads_and_4grams():
    rng = np.random.default_rng(11)
    vocab = 6   # tiny vocabulary: many windows repeat and many phrases match
    phrases = set()
    for n, want in ((2, 20), (3, 100), (4, 500)):
        got = set()
        while len(got) < want:
            got.add(tuple(int(x) for x in rng.integers(0, vocab, n)))
        phrases |= got
    phrases = sorted(phrases, key=lambda w: (len(w) * 7919 + sum(w) * 31) % 997)
    t, toks, lens = table_of(phrases, 2, 4, vocab)
    tokens = rng.integers(-1, vocab + 1, (8, 3 + 29)).astype(np.int32)
    got = t.lookup(tokens, 3, 29)
    exp = brute_force_lookup(toks, lens, tokens, 3, 29, 2, 4, vocab)
    for g, e in zip(got, exp):
        np.testing.assert_array_equal(g, e)
    assert set(got[2].tolist()) >= {0, 2, 3, 4}


def test_self_lookup_and_absent_keys():
    table, _ = synth.config1()
    t = oracle.Table(table.tokens, table.lens, 2, 3, V)
    for n in (2, 3):
        rows = np.flatnonzero(table.lens == n)
        q = table.tokens[rows, :n]
        hit, row, ln = t.lookup(q, n - 1, 1)
        assert hit.all()
        np.testing.assert_array_equal(row, rows)
        assert (ln == n).all()
    # Random tuples verified absent by a scan miss.
    rng = np.random.default_rng(3)
    q = rng.integers(0, V, (200, 3)).astype(np.int32)
    stored = {tuple(r[:l]) for r, l in zip(table.tokens.tolist(), table.lens.tolist())}
    keep = [i for i in range(200)
            if tuple(q[i, 1:].tolist()) not in stored and tuple(q[i].tolist()) not in stored]
    hit, row, _ = t.lookup(q[keep], 2, 1)
    assert not hit.any() and (row == -1).all()


def test_empty_table_misses_everywhere():
    t = oracle.Table(np.zeros((0, 3), np.int32), np.zeros(0, np.uint8), 2, 3, V)
    hit, row, ln = t.lookup(np.arange(12, dtype=np.int32).reshape(2, 6), 1, 5)
    assert not hit.any() and (row == -1).all() and not ln.any()


@pytest.mark.parametrize("phrases,n_min,n_max,status", [
    ([(1, 2), (1, 2)], 2, 3, oracle.DUPLICATE),
    ([(1, 2, 3), (4, 5), (1, 2, 3)], 2, 3, oracle.DUPLICATE),
    ([(1,)], 2, 3, oracle.INVALID),
    ([(1, 2, 3, 4)], 2, 3, oracle.INVALID),
    ([(1, V)], 2, 3, oracle.INVALID),
    ([(1, -5)], 2, 3, oracle.INVALID),
])
def test_load_errors(phrases, n_min, n_max, status):
    with pytest.raises(oracle.OracleError) as e:
        table_of(phrases, n_min, n_max)
    assert e.value.status == status


def test_bad_length_range_rejected():
    for n_min, n_max in [(1, 3), (2, 5), (3, 2)]:
        with pytest.raises(oracle.OracleError):
            oracle.Table(np.zeros((0, max(n_max, 1)), np.int32), np.zeros(0, np.uint8), n_min,
                         n_max, V)


# --------------------------------------------------------------- rounding ---

def test_bf16_rounding_of_float32_values_matches_integer_rounding():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                        (rng.standard_normal(2000) * 1e-30).astype(np.float32),
                        (rng.standard_normal(2000) * 1e30).astype(np.float32)])
    # Exact ties (low 16 bits == 0x8000) with odd and even bfloat16 significands.
    sign = rng.integers(0, 2, 1000).astype(np.uint32) << 31
    expo = rng.integers(100, 150, 1000).astype(np.uint32) << 23
    mant = rng.integers(0, 128, 1000).astype(np.uint32) << 16
    ties = (sign | expo | mant | 0x8000).view(np.float32)
    assert {0, 1} <= set(((mant >> 16) & 1).tolist())
    x = np.concatenate([x, ties])
    got = np.array([oracle.round_bf16(float(v)) for v in x], np.uint16)
    np.testing.assert_array_equal(got, bf16_bits_of_f32(x))
    np.testing.assert_array_equal(
        got, torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))


def test_bf16_rounding_of_doubles_by_exact_rationals():
    """Doubles that are not float32 values: compare against the nearest of
    the two neighbouring bfloat16 values found with exact rational
    arithmetic (ties to the even significand)."""
    rng = np.random.default_rng(1)
    xs = list(rng.standard_normal(300) * 3.0) + [1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8),
                                                  1.0 + 2**-8 + 2**-40, 2**-130 * 1.5]
    for x in xs:
        f = fractions.Fraction(x)
        e = math.floor(math.log2(abs(x)))
        q = max(e - 7, -133)
        step = fractions.Fraction(2) ** q
        lo = (f / step).__floor__()
        cands = [lo, lo + 1]
        d = [abs(f - c * step) for c in cands]
        if d[0] < d[1]:
            k = cands[0]
        elif d[1] < d[0]:
            k = cands[1]
        else:
            k = cands[0] if cands[0] % 2 == 0 else cands[1]
        want = float(k * step)
        got_bits = oracle.round_bf16(x)
        got = float(np.array([got_bits], np.uint16).astype(np.uint32).__lshift__(16)
                    .view(np.float32)[0])
        assert got == want, (x, got, want)


# ------------------------------------------------------------ gate & inject --

def test_gate_disjoint_supports_is_half_lambda_and_output_is_exact():
    D = 1024
    h = synth.normal_range(0, 900, 0, 1, D, 1.0, synth.BF16)[0].copy()
    m = synth.normal_range(0, 901, 0, 1, D, 0.02, synth.BF16)[0].copy()
    h[1::2] = 0
    m[0::2] = 0
    for lam in (1.0, 0.5, 2.0):
        assert oracle.gate_value(h, m, synth.BF16, lam=lam) == lam / 2
        out = oracle.inject(h[None], m[None], np.array([0]), synth.BF16, lam=lam)[0]
        hf, mf = synth.bf16_to_f32(h), synth.bf16_to_f32(m)
        want = np.where(np.arange(D) % 2 == 0, hf, np.float32(lam / 2) * mf)
        np.testing.assert_array_equal(synth.bf16_to_f32(out), want)


def test_gate_parallel_and_antiparallel_limits():
    D = 1024
    h = synth.normal_range(0, 902, 0, 1, D, 1.0, synth.F32)[0]
    sig32 = 1.0 / (1.0 + math.exp(-math.sqrt(D)))
    for c in (0.5, 3.0):
        g = oracle.gate_value(h, (c * h).astype(np.float32), synth.F32, lam=1.0)
        assert abs(g - sig32) < 1e-9
        g = oracle.gate_value(h, (-c * h).astype(np.float32), synth.F32, lam=2.0)
        assert 0 < g < 2.0 * 1e-13


def test_gate_is_a_sigmoid_of_the_scaled_cosine():
    # With eps negligible the gate is lambda * sigmoid(sqrt(D) * cos(h, m)).
    D = 256
    h = synth.normal_range(1, 903, 0, 1, D, 1.0, synth.F32)[0].astype(np.float64)
    m = synth.normal_range(1, 904, 0, 1, D, 5.0, synth.F32)[0].astype(np.float64)
    m = m + 0.3 * h * 5.0
    cos = float(h @ m) / (np.linalg.norm(h) * np.linalg.norm(m))
    want = 0.7 / (1.0 + math.exp(-math.sqrt(D) * cos))
    got = oracle.gate_value(h.astype(np.float32), m.astype(np.float32), synth.F32, lam=0.7)
    assert abs(got - want) < 1e-6


def test_constant_gate_is_axpy():
    table, batch = synth.config1()
    h = batch.hidden()
    rows = np.arange(batch.T) % table.n_phrases
    m = table.value_rows(rows)
    lam = 0.75
    out = oracle.inject(h, m, np.arange(batch.T), synth.F32, oracle.GATE_CONST, lam)
    want = torch.add(torch.from_numpy(h).double(), torch.from_numpy(m).double(), alpha=lam).float()
    np.testing.assert_array_equal(out, want.numpy())
    # bf16 with lambda = 1: where the float32 sum of the two bf16 values is
    # exact, torch's float32-add-then-round is the correctly rounded sum.
    hb = synth.normal_range(5, 905, 0, 8, 1024, 1.0, synth.BF16)
    mb = synth.normal_range(5, 906, 0, 8, 1024, 0.02, synth.BF16)
    hf, mf = torch.from_numpy(synth.bf16_to_f32(hb)), torch.from_numpy(synth.bf16_to_f32(mb))
    s32 = hf + mf
    exact = (s32.double() == hf.double() + mf.double()).numpy()
    assert exact.mean() > 0.99
    want = s32.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    out = oracle.inject(hb, mb, np.arange(8), synth.BF16, oracle.GATE_CONST, 1.0)
    np.testing.assert_array_equal(out[exact], want[exact])


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_noop_invariants(dtype):
    D, T = 1024, 6
    h = synth.normal_range(2, 907, 0, T, D, 1.0, dtype)
    m = synth.normal_range(2, 908, 0, T, D, 0.02, dtype)
    # Miss: the output bytes are the input bytes.
    out = oracle.inject(h, m, np.full(T, -1), dtype)
    assert out.tobytes() == h.tobytes()
    # Zero value row: no-op for both gates.
    z = np.zeros_like(m)
    for gate in (oracle.GATE_SIGMOID, oracle.GATE_CONST):
        out = oracle.inject(h, z, np.arange(T), dtype, gate, 1.0)
        assert out.tobytes() == h.tobytes()
    # lambda = 0: no-op.
    out = oracle.inject(h, m, np.arange(T), dtype, oracle.GATE_SIGMOID, 0.0)
    assert out.tobytes() == h.tobytes()


def test_injection_changes_hits_only():
    table, batch = synth.config1()
    t = oracle.Table(table.tokens, table.lens, 2, 3, V)
    h = batch.hidden()
    vals = table.all_values()
    hit, row, ln, out = oracle.lookup_inject(t, batch.tokens, batch.ctx, batch.S, h, vals,
                                             synth.F32)
    miss = hit == 0
    assert out[miss].tobytes() == h[miss].tobytes()
    assert np.all(np.any(out[~miss] != h[~miss], axis=1))


# ------------------------------------------------------- workload recipe ---

def test_workload1_has_both_match_lengths():
    table, batch = synth.config1()
    t = oracle.Table(table.tokens, table.lens, 2, 3, V)
    seq = batch.tokens[0]
    stored = {tuple(r[:l]) for r, l in zip(table.tokens.tolist(), table.lens.tolist())}
    both = only2 = 0
    for c in range(2, 64):
        w2, w3 = tuple(seq[c - 1:c + 1].tolist()), tuple(seq[c - 2:c + 1].tolist())
        both += (w2 in stored) and (w3 in stored)
        only2 += (w2 in stored) and (w3 not in stored)
    assert both >= 1 and only2 >= 1
    _, _, ln = t.lookup(batch.tokens, 0, 64)
    assert {2, 3} <= set(ln.tolist())
    assert table.n_phrases == 4096


@pytest.mark.slow
def test_workload3_hit_rate_in_range():
    """Workload 3 asks for a hit rate of about 30-40%; the oracle measures it."""
    table = synth.config3_table()
    t = oracle.Table(table.tokens, table.lens, 2, 4, V)
    batch = synth.prefill_batch(2, 8, 4096)
    hit, _, ln = t.lookup(batch.tokens, batch.ctx, batch.S)
    assert 0.30 <= hit.mean() <= 0.40
    assert np.bincount(ln, minlength=5)[4] > 0
