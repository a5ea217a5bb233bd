"""Tiered tables whose rows are not all pinned (Sec. 4.3: value rows in a
hierarchy of memories; rows the GPU cannot read in place are staged first).

Rows [0, pinned_rows) are in pinned host memory; rows [pinned_rows, P) stay
in the caller's pageable memory and reach the GPU through the table's
staging queue and host threads.  Where a row comes from changes nothing a
caller sees: every output must be byte-identical to a resident table's, and
the cache statistics must equal the policy model's (oracle/lru.py) exactly,
for decode steps, long calls, both prefetches and both fill modes, with the
cache prefill reaching into the pageable rows."""
import numpy as np
import pytest
import torch

import synth
from oracle.lru import LruModel
from paper_2607_07388_amd import tfe

from . import harness as H
from .test_gpu_tiered import FILLS, check_stats, pinned_values, run_both

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def w2():
    table = synth.config2_table()
    res = H.GpuTable(table)
    host = table.all_values()  # [P x D] bf16 bit patterns, pageable
    yield table, res, H.oracle_table(table), host
    res.close()
    H.release_pinned()


class SplitTable:
    """Rows [0, pinned) pinned (a library copy, or the caller's adopted
    buffer), rows [pinned, P) read in place from pageable memory."""

    def __init__(self, table, host, pinned, cache_rows, prefill_rows, fill, adopt):
        self.pageable = np.ascontiguousarray(host[pinned:])
        self.pinned_buf = pinned_values(table) if adopt else None
        head = self.pinned_buf if adopt else np.ascontiguousarray(host[:pinned])
        desc = tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab,
                             head, table.dim, table.dtype, 0, 0.5, hbm_cache_rows=cache_rows,
                             adopt_host_values=int(adopt), prefill_rows=prefill_rows,
                             miss_fill=fill, pinned_rows=pinned, pageable_values=self.pageable)
        self.handle = tfe.tfe_table_load(desc, H.cur_stream())

    def close(self):
        if self.handle:
            tfe.tfe_table_free(self.handle)
            self.handle = None


@pytest.mark.parametrize("fill", FILLS)
@pytest.mark.parametrize("adopt", [False, True])
def test_pageable_rows_decode_long_call_and_prefetch(w2, fill, adopt):
    table, res, ot, host = w2
    P = table.n_phrases
    C, pre, pinned = 4096, 2048, P // 4
    print("# split table: %d pinned of %d rows, fill %d, adopt %d" % (pinned, P, fill, adopt),
          flush=True)
    tier = SplitTable(table, host, pinned, C, pre, fill, adopt)
    model = LruModel(C, pre, table.dim * 2, fill_rereads=fill == tfe.TFE_FILL_SIDE_STREAM)
    B, K = 64, 8
    seqs = synth.zipf_tokens(1, 940, B * 12, 1.1).reshape(B, 12)
    side = torch.cuda.Stream()
    pageable_used = 0
    for s in range(6):
        window = np.ascontiguousarray(seqs[:, s:s + 3])
        hidden = synth.normal_range(1, 941 + s, 0, B, table.dim, 1.0, synth.BF16)
        o = run_both(res, tier, window, 2, 1, hidden, table.dtype, table.dim)
        rows = [int(r) for r in o.slot.cpu().numpy()]
        pageable_used += sum(1 for r in rows if r >= pinned)
        model.lookup(rows)
        check_stats(tier, model)
        tail = np.ascontiguousarray(seqs[:, s + 1:s + 3])
        cand = synth.workloads.candidates(1, B, K, seqs[:, s + 3], step=s)
        win = np.concatenate([np.repeat(tail, K, axis=0), cand.reshape(-1, 1)], axis=1)
        _, crow, clen = ot.lookup(win, 2, 1)
        tail_d, cand_d = torch.from_numpy(tail).cuda(), torch.from_numpy(cand).cuda()
        if s % 2 == 0:
            tfe.tfe_prefetch(tier.handle, tail_d, 2, cand_d, B, K, side)
            model.prefetch([int(r) for r in crow])
        else:
            prob = np.random.default_rng(s).dirichlet(np.ones(K) * 0.5, B).astype(np.float32)
            tfe.tfe_prefetch_scored(tier.handle, tail_d, 2, cand_d, torch.from_numpy(prob).cuda(),
                                    B, K, 64, side)
            model.prefetch_scored([int(r) for r in crow], [int(x) for x in clen], prob.ravel(), 64)
        check_stats(tier, model)
    assert pageable_used > 0
    # A 16384-position call: thousands of rows from both host tiers.
    pb = synth.prefill_batch(2, 4, 4096, set_index=5)
    o = run_both(res, tier, pb.tokens, pb.ctx, pb.S, pb.hidden(), table.dtype, table.dim)
    rows = [int(r) for r in o.slot.cpu().numpy()]
    assert sum(1 for r in rows if r >= pinned) > 1000
    model.lookup(rows)
    check_stats(tier, model)
    st = tfe.tfe_get_stats(tier.handle)  # raises if a staging wait ran out
    assert st["cache_misses"] > 0 and st["prefetch_filled"] > 0
    tier.close()
    H.release_pinned()


def test_prefill_reaching_into_pageable_rows(w2):
    """Cache prefill of rows beyond the pinned ones (copied from pageable
    memory at load): the first decode steps hit them in the cache."""
    table, res, ot, host = w2
    C, pre, pinned = 4096, 3000, 1000
    tier = SplitTable(table, host, pinned, C, pre, tfe.TFE_FILL_INLINE, False)
    model = LruModel(C, pre, table.dim * 2)
    for s in range(4):
        batch = synth.decode_batch(1, 64, set_index=950 + s)
        o = run_both(res, tier, batch.tokens, batch.ctx, batch.S, batch.hidden(), table.dtype,
                     table.dim)
        model.lookup([int(r) for r in o.slot.cpu().numpy()])
        check_stats(tier, model)
    assert tfe.tfe_get_stats(tier.handle)["cache_hits"] > 0
    tier.close()


def test_split_arguments_are_checked(w2):
    table, _, _, host = w2
    P = table.n_phrases

    def load(**kw):
        desc = tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab,
                             host, table.dim, table.dtype, 0, 0.5, **kw)
        return tfe.tfe_table_load(desc, H.cur_stream())

    for kw in (dict(hbm_cache_rows=4096, pinned_rows=P // 2),             # no pageable rows given
               dict(hbm_cache_rows=4096, pinned_rows=P + 1, pageable_values=host),
               dict(hbm_cache_rows=4096, pinned_rows=-1, pageable_values=host),
               dict(hbm_cache_rows=0, pinned_rows=P // 2, pageable_values=host)):
        with pytest.raises(tfe.TfeError) as e:
            load(**kw)
        assert e.value.status == tfe.TFE_ERR_INVALID_ARG
    # pinned_rows = P: every row pinned, pageable_values ignored.
    h = load(hbm_cache_rows=4096, pinned_rows=P, pageable_values=host[:1])
    tfe.tfe_table_free(h)
