"""Tiered table at the full workload-5 scale: 2^26 phrases, 128 GiB of bf16
values in host memory -- the 2^25 most frequent rows (64 GiB, what one
process can pin here) in pinned memory, the rest in pageable memory behind
the table's staging queue -- a 4M-row HBM cache prefilled with the most
frequent rows, batch-64 decode with prefetch on a side stream.  Every step's
outputs must be byte-identical to a resident copy of the same table (128 GiB
in HBM), and sampled positions must match the oracle (which holds the
phrases that can match the queries, found by exact tuple comparison over the
whole table)."""
import time

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu


def test_workload5_full_scale_tiered_equals_resident_and_oracle():
    t0 = time.time()
    table = synth.config5_table(26)
    print("# table %d phrases (%.0f s)" % (table.n_phrases, time.time() - t0), flush=True)
    P, D, C, B, K, steps = table.n_phrases, table.dim, 4 << 20, 64, 8, 6
    Pp = 1 << 25
    H.release_pinned()
    held = torch.cuda.host_memory_stats().get("allocated_bytes.current", 0)
    print("# pinned bytes still held by torch: %d" % held, flush=True)
    # Device memory that earlier tests freed stays reserved by torch's caching
    # allocator, out of reach of the library's allocations (the two tables
    # here need about 140 GB of HBM); idle construction scratch goes back too.
    H.release_device()
    free, total = torch.cuda.mem_get_info()
    print("# device memory: %.1f of %.1f GB free; library holds %d bytes"
          % (free / 1e9, total / 1e9, tfe.tfe_memory_held()[0]), flush=True)
    vals = torch.empty((Pp, D), dtype=torch.bfloat16, pin_memory=True)
    synth.normal_fill_device(synth.host_device_ptr(vals.data_ptr()), 0, Pp, D, table.seed,
                             synth.TAG_VALUES, table.sigma, synth.BF16, H.cur_stream())
    torch.cuda.synchronize()
    pageable = H.pageable_values(table, Pp)
    print("# host values ready: %d pinned, %d pageable rows (%.0f s)"
          % (Pp, P - Pp, time.time() - t0), flush=True)
    desc = tfe.make_desc(table.tokens, table.lens, 2, 3, table.vocab, vals, D, synth.BF16, 0,
                         0.5, hbm_cache_rows=C, adopt_host_values=1, prefill_rows=C,
                         pinned_rows=Pp, pageable_values=pageable)
    tiered = tfe.tfe_table_load(desc, H.cur_stream())
    resident = H.GpuTable(table, values_on_device=True)
    print("# tables loaded (%.0f s)" % (time.time() - t0), flush=True)
    seqs = synth.zipf_tokens(9, 810, B * (steps + 3), 1.1).reshape(B, steps + 3)
    side = torch.cuda.Stream()
    hits = pageable_hits = 0
    for s in range(steps):
        window = np.ascontiguousarray(seqs[:, s:s + 3])
        hidden = synth.normal_range(9, 811 + s, 0, B, D, 1.0, synth.BF16)
        tok = torch.from_numpy(window).cuda()
        h = H.to_device(hidden, synth.BF16)
        o1, o2 = H.Outputs(B, D, synth.BF16), H.Outputs(B, D, synth.BF16)
        H.run(resident, tok, B, 2, 1, h, o1)
        tfe.tfe_lookup_inject(tiered, tok, B, 2, 1, h, o2.out, o2.hit, o2.slot, o2.len, 0, 1.0,
                              H.cur_stream())
        torch.cuda.synchronize()
        assert torch.equal(o1.slot, o2.slot) and torch.equal(o1.len, o2.len)
        assert o1.out.view(torch.int16).equal(o2.out.view(torch.int16))
        rows = H.subset_rows(table, window, 2, 1)
        ot = oracle.Table(table.tokens[rows], table.lens[rows], 2, 3, synth.V)
        hit, row, ln, want = H.oracle_answer(table, ot, window, 2, 1, hidden, row_map=rows)
        np.testing.assert_array_equal(o2.slot.cpu().numpy(), row)
        np.testing.assert_array_equal(o2.len.cpu().numpy(), ln)
        H.assert_close(H.to_host(o2.out, synth.BF16), want, synth.BF16)
        hits += int(hit.sum())
        pageable_hits += int((row >= Pp).sum())
        tail = torch.from_numpy(np.ascontiguousarray(seqs[:, s + 1:s + 3])).cuda()
        cand = torch.from_numpy(synth.workloads.candidates(9, B, K, seqs[:, s + 3], step=s)).cuda()
        tfe.tfe_prefetch(tiered, tail, 2, cand, B, K, side)
        print("# step %d ok (%.0f s)" % (s, time.time() - t0), flush=True)
    st = tfe.tfe_get_stats(tiered)
    assert st["cache_misses"] > 0 and st["cache_hits"] > 0 and st["prefetch_filled"] > 0
    assert hits > steps * B // 2
    print("# %d matched positions, %d of them on pageable rows" % (hits, pageable_hits),
          flush=True)
    tfe.tfe_table_free(tiered)
    resident.close()
    del vals, pageable
    H.release_pinned()
