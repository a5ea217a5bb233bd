"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs.  Hit masks, slot (row) ids and match lengths must be
bit-exact; fp32 outputs within 1e-5 absolute, bf16 within 2e-2 relative."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu


def check(table, gt, ot, tokens, ctx, S, hidden, gate=tfe.TFE_GATE_SIGMOID, scale=1.0,
          inplace=False, positions=None, row_map=None):
    B = tokens.shape[0]
    T = B * S
    tok_d = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    h_d = H.to_device(hidden, table.dtype)
    outs = H.Outputs(T, table.dim, table.dtype)
    hout = H.run(gt, tok_d, B, ctx, S, h_d, outs, gate, scale, inplace)
    torch.cuda.synchronize()
    hit, row, ln, want = H.oracle_answer(table, ot, tokens, ctx, S, hidden, gate, scale, positions,
                                         row_map)
    np.testing.assert_array_equal(outs.hit.cpu().numpy(), hit)
    np.testing.assert_array_equal(outs.slot.cpu().numpy(), row)
    np.testing.assert_array_equal(outs.len.cpu().numpy(), ln)
    got = H.to_host(hout, table.dtype)
    if positions is not None:
        got = got[positions]
    H.assert_close(got, want, table.dtype)
    # Rows without a match keep their bytes.
    miss = hit == 0 if positions is None else hit[positions] == 0
    src = hidden if positions is None else hidden[positions]
    assert got[miss].tobytes() == src[miss].tobytes()
    return hit, got


@pytest.fixture(scope="module")
def w1():
    table, batch = synth.config1()
    gt = H.GpuTable(table)
    yield table, batch, gt, H.oracle_table(table)
    gt.close()


@pytest.mark.parametrize("gate,scale", [(tfe.TFE_GATE_SIGMOID, 1.0), (tfe.TFE_GATE_CONST, 1.0),
                                        (tfe.TFE_GATE_SIGMOID, 0.37)])
def test_workload1_fp32(w1, gate, scale):
    table, batch, gt, ot = w1
    hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(), gate, scale)
    assert 0 < hit.sum() < batch.T


def test_workload1_in_place(w1):
    table, batch, gt, ot = w1
    check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(), inplace=True)


def test_workload1_const_gate_is_index_select_add(w1):
    """Gather pin: with g = 1 in fp32 the output is the IEEE sum of the hidden
    row and the gathered value row, i.e. h + index_select(values, slot)."""
    table, batch, gt, _ = w1
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), synth.F32)
    outs = H.Outputs(batch.T, table.dim, synth.F32)
    H.run(gt, tok, 1, 0, batch.S, h, outs, tfe.TFE_GATE_CONST, 1.0)
    vals = H.device_values(table)
    slot = outs.slot.long()
    hitm = slot >= 0
    want = h.clone()
    want[hitm] = h[hitm] + torch.index_select(vals, 0, slot[hitm])
    torch.cuda.synchronize()
    assert torch.equal(outs.out, want)


def test_determinism(w1):
    table, batch, gt, _ = w1
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), synth.F32)
    res = []
    for _ in range(2):
        outs = H.Outputs(batch.T, table.dim, synth.F32)
        H.run(gt, tok, 1, 0, batch.S, h, outs)
        torch.cuda.synchronize()
        res.append((outs.out.cpu().numpy().tobytes(), outs.slot.cpu().numpy().tobytes()))
    assert res[0] == res[1]


def test_noop_cases(w1):
    table, batch, gt, _ = w1
    tok = torch.from_numpy(batch.tokens).cuda()
    hid = batch.hidden()
    h = H.to_device(hid, synth.F32)
    outs = H.Outputs(batch.T, table.dim, synth.F32)
    H.run(gt, tok, 1, 0, batch.S, h, outs, tfe.TFE_GATE_SIGMOID, 0.0)   # scale 0
    torch.cuda.synchronize()
    assert outs.out.cpu().numpy().tobytes() == hid.tobytes()
    # Zero value rows: every hit is a no-op.
    zt = synth.PhraseTable(table.tokens, table.lens, 2, 3, synth.F32, table.seed, sigma=0.0)
    gz = H.GpuTable(zt)
    outs = H.Outputs(batch.T, table.dim, synth.F32)
    H.run(gz, tok, 1, 0, batch.S, h, outs)
    torch.cuda.synchronize()
    assert outs.hit.sum().item() > 0
    assert outs.out.cpu().numpy().tobytes() == hid.tobytes()
    gz.close()


def small_table(seed, vocab, counts, dtype, dim, n_max):
    rng = np.random.default_rng(seed)
    phrases = set()
    for n, want in counts:
        got = set()
        while len(got) < want:
            got.add(tuple(int(x) for x in rng.integers(0, vocab, n)))
        phrases |= got
    phrases = sorted(phrases)
    perm = rng.permutation(len(phrases))
    toks = np.full((len(phrases), n_max), -1, np.int32)
    lens = np.zeros(len(phrases), np.uint8)
    for r, i in enumerate(perm):
        w = phrases[i]
        toks[r, :len(w)] = w
        lens[r] = len(w)
    n_min = min(n for n, _ in counts)
    return synth.PhraseTable(toks, lens, n_min, n_max, dtype, seed, dim=dim, vocab=vocab)


@pytest.mark.parametrize("dtype,dim", [(synth.BF16, 1024), (synth.BF16, 512), (synth.BF16, 4096),
                                       (synth.F32, 256), (synth.F32, 2048)])
def test_4grams_pads_ragged_tail(dtype, dim):
    """Small vocabulary, 2/3/4-grams, pad and out-of-range tokens, history
    columns, and B*S = 3*37 = 111 positions (not a multiple of the 4 waves
    of a block)."""
    vocab = 7
    table = small_table(21 + dim, vocab, [(2, 20), (3, 150), (4, 900)], dtype, dim, 4)
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    rng = np.random.default_rng(dim)
    B, ctx, S = 3, 3, 37
    tokens = rng.integers(-1, vocab + 1, (B, ctx + S)).astype(np.int32)
    hidden = synth.normal_range(7, 77, 0, B * S, dim, 1.0, dtype)
    hit, _ = check(table, gt, ot, tokens, ctx, S, hidden)
    _, _, ln = ot.lookup(tokens, ctx, S)
    assert {0, 2, 3, 4} <= set(ln.tolist())
    gt.close()


@pytest.mark.parametrize("lengths", [(2,), (3,), (4,), (3, 4), (2, 4)])
def test_length_ranges(lengths):
    """n_min..n_max covering one length, a range without 2-grams, and 2/4-gram
    tables with no 3-grams (that lane group probes and never matches); both
    entry points, the multi-match one with its n_max - n_min + 1 columns."""
    from .test_gpu_multi import check_multi
    vocab = 7
    want = {2: 20, 3: 150, 4: 900}
    table = small_table(500 + sum(lengths) * 7 + len(lengths), vocab,
                        [(n, want[n]) for n in lengths], synth.BF16, 1024, max(lengths))
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    rng = np.random.default_rng(len(lengths) * 10 + lengths[0])
    B, ctx, S = 3, 3, 37
    tokens = rng.integers(-1, vocab + 1, (B, ctx + S)).astype(np.int32)
    hidden = synth.normal_range(7, 90 + lengths[0], 0, B * S, 1024, 1.0, synth.BF16)
    check(table, gt, ot, tokens, ctx, S, hidden)
    _, _, ln = ot.lookup(tokens, ctx, S)
    assert set(ln.tolist()) == {0} | set(lengths)
    mask, _ = check_multi(table, gt, ot, tokens, ctx, S, hidden, tfe.TFE_WEIGHT_LENGTH)
    if len(lengths) == 2:  # both lengths matched at some position
        assert (mask == (1 | 1 << (lengths[1] - lengths[0]))).any()
    gt.close()


def test_empty_table_and_empty_batch():
    table = synth.PhraseTable(np.zeros((0, 3), np.int32), np.zeros(0, np.uint8), 2, 3, synth.BF16,
                              0)
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    tokens = synth.zipf_tokens(0, 50, 4 * 9, 1.1).reshape(4, 9)
    hidden = synth.normal_range(0, 51, 0, 4 * 7, 1024, 1.0, synth.BF16)
    hit, _ = check(table, gt, ot, tokens, 2, 7, hidden)
    assert hit.sum() == 0
    # B = 0 and S = 0 enqueue nothing and succeed.
    outs = H.Outputs(1, 1024, synth.BF16)
    tfe.tfe_lookup_inject(gt.handle, None, 0, 2, 7, None, None, None, None, None, 0, 1.0, None)
    tfe.tfe_lookup_inject(gt.handle, None, 4, 2, 0, None, None, None, None, None, 0, 1.0, None)
    del outs
    gt.close()


@pytest.fixture(scope="module")
def w2():
    table = synth.config2_table()
    gt = H.GpuTable(table)
    yield table, gt, H.oracle_table(table)
    gt.close()


def test_workload2_decode_batch64(w2):
    table, gt, ot = w2
    batch = synth.decode_batch(1, 64)
    hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden())
    assert 0.4 < hit.mean() < 0.9


def test_workload2_stacked_decode_16384_rows(w2):
    """The benchmark's launch: 256 batch-64 decode steps in one call."""
    table, gt, ot = w2
    batch = synth.decode_batch(1, 64 * 256, set_index=1)
    hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden())
    assert 0.5 < hit.mean() < 0.8


def test_workload2_in_place_const_gate(w2):
    table, gt, ot = w2
    batch = synth.decode_batch(1, 1000, set_index=2)
    check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(), tfe.TFE_GATE_CONST,
          0.5, inplace=True)


def test_workload3_prefill_full():
    """8 x 4096 prefill against the 4M-phrase 2/3/4-gram table (8 GiB of
    values): every position compared; hit rate in [0.30, 0.40]."""
    table = synth.config3_table()
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    batch = synth.prefill_batch(2, 8, 4096)
    hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden())
    assert 0.30 <= hit.mean() <= 0.40
    _, _, ln = ot.lookup(batch.tokens, batch.ctx, batch.S)
    assert {0, 2, 3, 4} <= set(ln.tolist())
    gt.close()


def test_workload4_large_table():
    """Batch-256 decode against the 2^25-phrase table (64 GiB of values);
    the oracle holds the phrases that can match the query (found by exact
    tuple comparison over the whole table)."""
    table = synth.config4_table()
    gt = H.GpuTable(table)
    batch = synth.decode_batch(3, 256, s=1.05)
    rows = H.subset_rows(table, batch.tokens, batch.ctx, batch.S)
    ot = oracle.Table(table.tokens[rows], table.lens[rows], 2, 3, synth.V)
    hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(), row_map=rows)
    assert 0.5 < hit.mean() < 0.95
    gt.close()


def test_negative_zero_is_value_equal_on_noop_hits(w1):
    """Zero value rows make every hit a no-op by value, but signed zeros
    follow IEEE addition: h = -0 plus g * (+0) gives +0 (the zero rows hold
    both +0 and -0).  So: equal to the input by value, byte-identical to the
    oracle (same signed-zero arithmetic), and misses keep their bytes."""
    table, batch, _, _ = w1
    zt = synth.PhraseTable(table.tokens, table.lens, 2, 3, synth.F32, table.seed, sigma=0.0)
    gz = H.GpuTable(zt)
    hid = batch.hidden().copy()
    hid[:, ::7] = -0.0
    tok = torch.from_numpy(batch.tokens).cuda()
    outs = H.Outputs(batch.T, table.dim, synth.F32)
    H.run(gz, tok, 1, 0, batch.S, H.to_device(hid, synth.F32), outs)
    torch.cuda.synchronize()
    out = outs.out.cpu().numpy()
    hit = outs.hit.cpu().numpy().astype(bool)
    assert hit.any() and (~hit).any()
    assert np.array_equal(out, hid)
    assert out[~hit].tobytes() == hid[~hit].tobytes()
    _, _, _, want = H.oracle_answer(zt, H.oracle_table(zt), batch.tokens, 0, batch.S, hid)
    assert out.tobytes() == want.tobytes()
    flipped = np.signbit(hid) & ~np.signbit(out)
    assert flipped.any() and (hid[flipped] == 0).all()
    gz.close()


def test_vocab_boundary_ids_pack_and_match():
    """vocab = 2^18 (18-bit token fields fully used): phrases over the ids
    {0, 1, 2^17, 2^18 - 2, 2^18 - 1} in every length 2-4, queried with
    those ids, ids in no phrase (5, 2^18 - 3), the first invalid id (2^18)
    and -1; both entry points against the oracle, bit-exact rows."""
    from .test_gpu_multi import check_multi
    vocab = 1 << 18
    ids = np.array([0, 1, 1 << 17, vocab - 2, vocab - 1], np.int64)
    rng = np.random.default_rng(18)
    tuples = [tuple(int(x) for x in ids[list(ix)]) for ix in np.ndindex(5, 5)]
    tuples += [tuple(int(x) for x in ids[list(ix)]) for ix in np.ndindex(5, 5, 5)]
    four = {tuple(int(x) for x in rng.choice(ids, 4)) for _ in range(400)}
    tuples += sorted(four)
    perm = rng.permutation(len(tuples))
    toks = np.full((len(tuples), 4), -1, np.int32)
    lens = np.zeros(len(tuples), np.uint8)
    for r, i in enumerate(perm):
        toks[r, :len(tuples[i])] = tuples[i]
        lens[r] = len(tuples[i])
    table = synth.PhraseTable(toks, lens, 2, 4, synth.BF16, 18, dim=1024, vocab=vocab)
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    pool = np.concatenate([ids, [5, vocab - 3, vocab, -1]]).astype(np.int32)
    weights = np.array([4, 4, 4, 4, 4, 1, 1, 1, 1], np.float64)
    tokens = rng.choice(pool, size=(4, 64), p=weights / weights.sum()).astype(np.int32)
    hidden = synth.normal_range(8, 1818, 0, 4 * 61, 1024, 1.0, synth.BF16)
    hit, _ = check(table, gt, ot, tokens, 3, 61, hidden)
    _, _, ln = ot.lookup(tokens, 3, 61)
    assert {0, 2, 3, 4} <= set(ln.tolist())
    check_multi(table, gt, ot, tokens, 3, 61, hidden, tfe.TFE_WEIGHT_LENGTH)
    gt.close()


def test_resident_hit_count_in_stats(w2):
    """tfe_get_stats on a resident table: hits equals the oracle's matched
    positions over a sequence of calls of several sizes (one launch of 16384
    rows spreads its counts over the table's counters), calls and positions
    count API calls, and tfe_reset_stats clears them."""
    table, _, ot = w2
    gt = H.GpuTable(table)
    want_hits = want_pos = 0
    for k, T in enumerate([64, 16384, 1, 1000]):
        batch = synth.decode_batch(1, T, set_index=50 + k)
        hit, _ = check(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden())
        want_hits += int(hit.sum())
        want_pos += T
        st = tfe.tfe_get_stats(gt.handle)
        assert st["hits"] == want_hits and st["positions"] == want_pos and st["calls"] == k + 1
    tfe.tfe_reset_stats(gt.handle)
    st = tfe.tfe_get_stats(gt.handle)
    assert st["hits"] == 0 and st["positions"] == 0 and st["calls"] == 0
    # Multi-match calls count positions with any retained phrase.
    batch = synth.decode_batch(1, 4096, set_index=60)
    T = 4096
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), table.dtype)
    mask = torch.zeros(T, dtype=torch.uint8, device="cuda")
    slots = torch.zeros((T, 2), dtype=torch.int32, device="cuda")
    out = torch.empty_like(h)
    tfe.tfe_lookup_inject_multi(gt.handle, tok, T, batch.ctx, batch.S, h, out, mask, slots,
                                tfe.TFE_WEIGHT_LENGTH, tfe.TFE_GATE_SIGMOID, 1.0, H.cur_stream())
    hit, _, _ = ot.lookup(batch.tokens, batch.ctx, batch.S)
    assert tfe.tfe_get_stats(gt.handle)["hits"] == int(hit.sum())
    gt.close()
