"""GPU parity of the multi-match path (Eq. 4, Eq. 11): tfe_lookup_inject_multi
through the C ABI against the oracle's all-matches lookup and weighted
injection on the same seeded inputs.  Match masks and row ids bit-exact;
fp32 outputs within 1e-5 absolute, bf16 within 2e-2 relative.  Where a
single phrase matches, the output must equal the longest-match entry
point's byte for byte."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2607_07388_amd import tfe

from . import harness as H
from .test_gpu_parity import small_table

pytestmark = pytest.mark.gpu

WEIGHTINGS = [tfe.TFE_WEIGHT_LENGTH, tfe.TFE_WEIGHT_UNIFORM]


def run_multi(gt, tokens, ctx, S, hidden, dtype, dim, L, weighting, gate, scale, inplace=False):
    B = tokens.shape[0]
    T = B * S
    tok_d = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    h_d = H.to_device(hidden, dtype)
    out = h_d if inplace else torch.empty((T, dim), dtype=H.TORCH_DT[dtype], device="cuda")
    mask = torch.full((T,), 0xEE, dtype=torch.uint8, device="cuda")
    slots = torch.full((T, L), -7, dtype=torch.int32, device="cuda")
    tfe.tfe_lookup_inject_multi(gt.handle, tok_d, B, ctx, S, h_d, out, mask, slots, weighting,
                                gate, scale, H.cur_stream())
    torch.cuda.synchronize()
    return mask.cpu().numpy(), slots.cpu().numpy(), H.to_host(out, dtype)


def oracle_multi(table, ot, tokens, ctx, S, hidden, weighting, gate, scale, positions=None,
                 row_map=None):
    mask, rows = ot.lookup_all(tokens, ctx, S)
    if row_map is not None:
        rows = np.where(rows >= 0, row_map[np.maximum(rows, 0)], -1).astype(np.int32)
    if positions is None:
        positions = np.arange(mask.size)
    sel = rows[positions].astype(np.int64)
    uniq, inv = np.unique(sel[sel >= 0], return_inverse=True)
    vals = table.value_rows(uniq) if uniq.size else np.zeros((0, table.dim), np.float32)
    idx = np.full(sel.shape, -1, np.int64)
    idx[sel >= 0] = inv
    out = oracle.inject_multi(hidden[positions], vals, idx, table.n_min, table.dtype, weighting,
                              gate, scale)
    return mask, rows, out


def check_multi(table, gt, ot, tokens, ctx, S, hidden, weighting, gate=tfe.TFE_GATE_SIGMOID,
                scale=1.0, inplace=False, positions=None, row_map=None):
    L = table.n_max - table.n_min + 1
    gmask, gslots, got = run_multi(gt, tokens, ctx, S, hidden, table.dtype, table.dim, L,
                                   weighting, gate, scale, inplace)
    mask, rows, want = oracle_multi(table, ot, tokens, ctx, S, hidden, weighting, gate, scale,
                                    positions, row_map)
    np.testing.assert_array_equal(gmask, mask)
    np.testing.assert_array_equal(gslots, rows)
    if positions is not None:
        got = got[positions]
    H.assert_close(got, want, table.dtype)
    miss = (mask if positions is None else mask[positions]) == 0
    src = hidden if positions is None else hidden[positions]
    assert got[miss].tobytes() == src[miss].tobytes()
    return mask, got


def longest_match_output(gt, tokens, ctx, S, hidden, dtype, dim, gate, scale):
    B = tokens.shape[0]
    tok_d = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    h_d = H.to_device(hidden, dtype)
    outs = H.Outputs(B * S, dim, dtype)
    H.run(gt, tok_d, B, ctx, S, h_d, outs, gate, scale)
    torch.cuda.synchronize()
    return H.to_host(outs.out, dtype)


def popcount(m):
    return np.unpackbits(m[:, None], axis=1).sum(axis=1)


@pytest.fixture(scope="module")
def w1():
    table, batch = synth.config1()
    gt = H.GpuTable(table)
    yield table, batch, gt, H.oracle_table(table)
    gt.close()


@pytest.mark.parametrize("weighting", WEIGHTINGS)
@pytest.mark.parametrize("gate,scale", [(tfe.TFE_GATE_SIGMOID, 1.0), (tfe.TFE_GATE_CONST, 1.0),
                                        (tfe.TFE_GATE_SIGMOID, 0.37)])
def test_workload1_fp32_multi(w1, weighting, gate, scale):
    table, batch, gt, ot = w1
    mask, _ = check_multi(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(),
                          weighting, gate, scale)
    assert (mask == 3).any() and (mask == 1).any()


def test_workload1_multi_in_place(w1):
    table, batch, gt, ot = w1
    check_multi(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(),
                tfe.TFE_WEIGHT_LENGTH, inplace=True)


@pytest.mark.parametrize("weighting", WEIGHTINGS)
@pytest.mark.parametrize("dtype,dim", [(synth.BF16, 1024), (synth.F32, 1024),
                                       (synth.BF16, 4096), (synth.F32, 256)])
def test_single_match_equals_longest_match_entry_point(weighting, dtype, dim):
    vocab = 7
    table = small_table(31 + dim, vocab, [(2, 20), (3, 150), (4, 900)], dtype, dim, 4)
    gt = H.GpuTable(table)
    rng = np.random.default_rng(dim + 1)
    B, ctx, S = 3, 3, 37
    tokens = rng.integers(-1, vocab + 1, (B, ctx + S)).astype(np.int32)
    hidden = synth.normal_range(8, 78, 0, B * S, dim, 1.0, dtype)
    for gate in (tfe.TFE_GATE_SIGMOID, tfe.TFE_GATE_CONST):
        mask, _, got = run_multi(gt, tokens, ctx, S, hidden, dtype, dim, 3, weighting, gate, 0.9)
        ref = longest_match_output(gt, tokens, ctx, S, hidden, dtype, dim, gate, 0.9)
        one = popcount(mask) <= 1
        assert one.any() and (~one).any()
        assert got[one].tobytes() == ref[one].tobytes()
    gt.close()


@pytest.mark.parametrize("weighting", WEIGHTINGS)
@pytest.mark.parametrize("dtype,dim,B,ctx,S", [
    (synth.BF16, 1024, 3, 3, 37),      # 111 positions: ragged for any block size
    (synth.F32, 2048, 2, 0, 53),       # no history: early columns lack long windows
    (synth.BF16, 512, 9, 3, 1000),     # 9000 positions: the 4-wave launch shape, ragged tail
])
def test_4grams_all_subsets(weighting, dtype, dim, B, ctx, S):
    """Tiny vocabulary so that every subset of {2, 3, 4} matches somewhere,
    with pad and out-of-range tokens breaking windows."""
    vocab = 6
    table = small_table(41 + dim + S, vocab, [(2, 20), (3, 120), (4, 700)], dtype, dim, 4)
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    rng = np.random.default_rng(S + dim)
    tokens = rng.integers(-1, vocab + 1, (B, ctx + S)).astype(np.int32)
    hidden = synth.normal_range(9, 79, 0, B * S, dim, 1.0, dtype)
    mask, _ = check_multi(table, gt, ot, tokens, ctx, S, hidden, weighting)
    assert {0, 1, 3, 7} <= set(mask.tolist())
    gt.close()


def test_multi_errors_and_empty():
    table, batch = synth.config1()
    gt = H.GpuTable(table)
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), synth.F32)
    out = torch.empty_like(h)
    mask = torch.zeros(batch.T, dtype=torch.uint8, device="cuda")
    slots = torch.zeros((batch.T, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(tfe.TfeError) as e:
        tfe.tfe_lookup_inject_multi(gt.handle, tok, 1, 0, batch.S, h, out, mask, slots, 5, 0, 1.0)
    assert e.value.status == -1
    with pytest.raises(tfe.TfeError):
        tfe.tfe_lookup_inject_multi(gt.handle, tok, 1, 0, batch.S, h, out, mask, None, 0, 0, 1.0)
    # Empty batches enqueue nothing.
    tfe.tfe_lookup_inject_multi(gt.handle, None, 0, 0, 5, None, None, None, None, 0, 0, 1.0)
    tfe.tfe_lookup_inject_multi(gt.handle, None, 3, 2, 0, None, None, None, None, 0, 0, 1.0)
    gt.close()


def test_multi_rejected_on_tiered_table():
    table, batch = synth.config1()
    vals = table.all_values()
    desc = tfe.make_desc(table.tokens, table.lens, 2, 3, table.vocab, vals, table.dim,
                         table.dtype, False, 0.5, hbm_cache_rows=64)
    handle = tfe.tfe_table_load(desc, H.cur_stream())
    tok = torch.from_numpy(batch.tokens).cuda()
    h = H.to_device(batch.hidden(), synth.F32)
    out = torch.empty_like(h)
    mask = torch.zeros(batch.T, dtype=torch.uint8, device="cuda")
    slots = torch.zeros((batch.T, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(tfe.TfeError) as e:
        tfe.tfe_lookup_inject_multi(handle, tok, 1, 0, batch.S, h, out, mask, slots, 0, 0, 1.0)
    assert e.value.status == -5
    tfe.tfe_table_free(handle)


@pytest.fixture(scope="module")
def w2():
    table = synth.config2_table()
    gt = H.GpuTable(table)
    yield table, gt, H.oracle_table(table)
    gt.close()


@pytest.mark.parametrize("weighting", WEIGHTINGS)
def test_workload2_stacked_decode_multi(w2, weighting):
    """The benchmark's launch of the multi-match kernel: 256 batch-64 decode
    steps (16384 rows) in one call, every position compared."""
    table, gt, ot = w2
    batch = synth.decode_batch(1, 64 * 256, set_index=3)
    mask, _ = check_multi(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(),
                          weighting)
    assert 0.15 < (mask == 3).mean() < 0.5 and not (mask == 2).any()


def test_workload3_prefill_multi_sampled():
    """8 x 4096 prefill against the 4M-phrase 2/3/4-gram table: masks and row
    ids at every position, outputs at a 4096-position sample."""
    table = synth.config3_table()
    gt = H.GpuTable(table)
    ot = H.oracle_table(table)
    batch = synth.prefill_batch(2, 8, 4096)
    pos = np.random.default_rng(5).choice(batch.T, 4096, replace=False)
    pos.sort()
    mask, _ = check_multi(table, gt, ot, batch.tokens, batch.ctx, batch.S, batch.hidden(),
                          tfe.TFE_WEIGHT_LENGTH, positions=pos)
    assert (popcount(mask) >= 2).mean() > 0.01
    gt.close()
