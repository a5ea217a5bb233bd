"""Allocation failures forced from the host (TFE_FAIL_ALLOC=k fails the k-th
allocation of a library call), on the GPU path.

- Every allocation of a resident load, a tiered load (with and without an
  adopted pinned buffer) and a head creation is failed in turn: each returns
  TFE_ERR_OOM naming it, returns no handle, and leaves the library holding
  exactly what it held before (device and pinned bytes).
- Lookups and prefetches whose scratch (or recency ring) cannot grow fail
  with TFE_ERR_OOM without enqueuing anything: their outputs stay untouched,
  repeated failures hold no more memory, and the table then runs the same
  call correctly, with outputs identical to a resident table's and
  statistics equal to the policy model's that never saw the failed calls.
- A construction whose buffers cannot be had fails and gives them back.
Every kernel still runs to completion: failures happen on the host before
anything is launched."""
import os
import types

import numpy as np
import pytest
import torch

import synth
from oracle.lru import LruModel
from paper_2607_07388_amd import tfe

from . import harness as H
from .test_gpu_tiered import TieredTable, check_stats, pinned_values, run_both

pytestmark = pytest.mark.gpu


class FailAt:
    def __init__(self, k):
        self.k = k

    def __enter__(self):
        os.environ["TFE_FAIL_ALLOC"] = str(self.k)

    def __exit__(self, *exc):
        os.environ.pop("TFE_FAIL_ALLOC", None)


def fail_every_allocation(call, max_k=64):
    """Runs call() with the k-th allocation failing, k = 1, 2, ..., until it
    succeeds; returns (its result, the failure messages in order)."""
    before = tfe.tfe_memory_held()
    msgs = []
    for k in range(1, max_k):
        try:
            with FailAt(k):
                res = call()
        except tfe.TfeError as e:
            assert e.status == tfe.TFE_ERR_OOM, (k, str(e))
            assert tfe.tfe_memory_held() == before, (k, str(e))
            msgs.append(str(e).split(": ", 1)[1])
            continue
        return res, msgs
    raise AssertionError("still failing after %d allocations" % max_k)


def names(msgs):
    return [m.split(" (")[0].split(" of ")[0] for m in msgs]


@pytest.fixture(scope="module")
def w2():
    table = synth.config2_table()
    res = H.GpuTable(table)
    yield table, res
    res.close()
    H.release_pinned()


def test_every_allocation_of_a_resident_load(w2):
    table, res = w2
    vals = H.device_values(table)
    torch.cuda.synchronize()
    base = tfe.tfe_memory_held()

    def load():
        desc = tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab,
                             vals, table.dim, table.dtype, 1)
        return tfe.tfe_table_load(desc, H.cur_stream())

    h, msgs = fail_every_allocation(load)
    assert names(msgs) == ["host index", "table object", "device index", "hit counters",
                           "device values"]
    # The table that finally loaded answers like the one loaded normally.
    gt = types.SimpleNamespace(handle=h)
    batch = synth.decode_batch(1, 64, set_index=900)
    tok = torch.from_numpy(batch.tokens).cuda()
    hid = H.to_device(batch.hidden(), table.dtype)
    o1, o2 = H.Outputs(64, table.dim, table.dtype), H.Outputs(64, table.dim, table.dtype)
    H.run(res, tok, 64, batch.ctx, batch.S, hid, o1)
    H.run(gt, tok, 64, batch.ctx, batch.S, hid, o2)
    torch.cuda.synchronize()
    assert torch.equal(o1.slot, o2.slot) and torch.equal(o1.out.view(torch.int16),
                                                         o2.out.view(torch.int16))
    tfe.tfe_table_free(h)
    assert tfe.tfe_memory_held() == base


@pytest.mark.parametrize("adopt,split", [(False, False), (True, False), (False, True)])
def test_every_allocation_of_a_tiered_load(w2, adopt, split):
    """split: the upper half of the rows stays in pageable memory behind the
    staging queue (its acknowledgement words, state and pinned queue)."""
    table, _ = w2
    P = table.n_phrases
    Pp = P // 2 if split else P
    pinned = pinned_values(table) if adopt else None
    host = None if adopt else table.all_values()
    pageable = np.ascontiguousarray(host[Pp:]) if split else None
    base = tfe.tfe_memory_held()

    def load():
        desc = tfe.make_desc(table.tokens, table.lens, table.n_min, table.n_max, table.vocab,
                             pinned if adopt else host[:Pp], table.dim, table.dtype, 0, 0.5,
                             hbm_cache_rows=4096, adopt_host_values=int(adopt),
                             prefill_rows=1024, pinned_rows=Pp if split else 0,
                             pageable_values=pageable)
        return tfe.tfe_table_load(desc, H.cur_stream())

    h, msgs = fail_every_allocation(load)
    want = ["host index", "table object", "device index"] + ([] if adopt else ["pinned host values"])
    if split:
        want += ["staging acknowledgements", "staging state", "staging queue", "staging queue"]
    want += ["HBM cache", "residency map", "slot owners", "slot stamps", "prefetch flags",
             "spare slots", "recency ring", "recency ring", "tier control block"]
    assert names(msgs) == want
    d, p = tfe.tfe_memory_held()
    esz = 2 if table.dtype == synth.BF16 else 4
    staging = 4096 * 16 + 4096 * table.dim * esz if split else 0
    assert d > base[0] and p == base[1] + (0 if adopt else Pp * table.dim * esz) + staging
    tfe.tfe_table_free(h)
    assert tfe.tfe_memory_held() == base
    del pinned
    H.release_pinned()


def test_failed_scratch_growth_leaves_the_table_usable(w2):
    table, res = w2
    ot = H.oracle_table(table)
    C, pre = 4096, 2048
    tier = TieredTable(table, C, pre)
    model = LruModel(C, pre, table.dim * 2)

    def failing_calls(call, outs, plan):
        """Runs call() once per (k, what) of `plan` with its k-th allocation
        failing: each fails naming `what`, enqueues nothing (outputs keep
        their fill) and returns nothing it allocated; returns the memory held
        after each."""
        held = []
        for k, what in plan:
            with FailAt(k):
                with pytest.raises(tfe.TfeError) as e:
                    call()
            assert e.value.status == tfe.TFE_ERR_OOM and what in str(e.value), (k, str(e.value))
            torch.cuda.synchronize()
            if outs is not None:
                assert bool((outs.hit == 0xEE).all()) and bool((outs.slot == -7).all())
            held.append(tfe.tfe_memory_held())
        return held

    # 1. The first decode call allocates the scratch (8 buffers).
    batch = synth.decode_batch(1, 64, set_index=910)
    tok = torch.from_numpy(batch.tokens).cuda()
    hid = H.to_device(batch.hidden(), table.dtype)
    outs = H.Outputs(64, table.dim, table.dtype)

    def decode():
        tfe.tfe_lookup_inject(tier.handle, tok, 64, batch.ctx, batch.S, hid, outs.out, outs.hit,
                              outs.slot, outs.len, 0, 1.0, H.cur_stream())

    before = tfe.tfe_memory_held()
    held = failing_calls(decode, outs, [(k, "scratch") for k in range(1, 9)])
    assert held == [before] * 8
    decode()
    assert tfe.tfe_memory_held()[0] > before[0]
    torch.cuda.synchronize()
    o1 = H.Outputs(64, table.dim, table.dtype)
    H.run(res, tok, 64, batch.ctx, batch.S, hid, o1)
    torch.cuda.synchronize()
    assert torch.equal(o1.slot, outs.slot) and torch.equal(o1.out.view(torch.int16),
                                                           outs.out.view(torch.int16))
    model.lookup([int(r) for r in outs.slot.cpu().numpy()])
    check_stats(tier, model)
    assert tfe.tfe_get_stats(tier.handle)["calls"] == 1

    # 2. A 16384-position call grows the scratch (8 buffers) and, since it
    # appends more recency entries than the ring holds beyond the cache
    # rows, the ring (2 buffers).  A scratch that grew before the ring
    # failed stays with the table; the ring's first buffer is returned when
    # its second cannot be had.
    pb = synth.prefill_batch(2, 4, 4096, set_index=3)
    ptok = torch.from_numpy(pb.tokens).cuda()
    phid = H.to_device(pb.hidden(), table.dtype)
    pouts = H.Outputs(4 * 4096, table.dim, table.dtype)

    def long_call():
        tfe.tfe_lookup_inject(tier.handle, ptok, 4, pb.ctx, pb.S, phid, pouts.out, pouts.hit,
                              pouts.slot, pouts.len, 0, 1.0, H.cur_stream())

    before = tfe.tfe_memory_held()
    held = failing_calls(long_call, pouts, [(k, "scratch") for k in range(1, 9)] +
                         [(9, "recency ring"), (2, "recency ring"), (1, "recency ring")])
    assert held[:8] == [before] * 8
    assert held[8][0] > before[0] and held[8:] == [held[8]] * 3
    long_call()
    torch.cuda.synchronize()
    _, row, _, _ = H.oracle_answer(table, ot, pb.tokens, pb.ctx, pb.S, pb.hidden(),
                                   positions=np.arange(4))
    np.testing.assert_array_equal(pouts.slot.cpu().numpy(), row)
    model.lookup([int(r) for r in row])
    check_stats(tier, model)

    # 3. The first prefetch allocates its own scratch (4 buffers).
    B, K = 64, 8
    seqs = synth.zipf_tokens(1, 920, B * 4, 1.1).reshape(B, 4)
    tail = np.ascontiguousarray(seqs[:, 1:3])
    cand = synth.workloads.candidates(1, B, K, seqs[:, 3], step=0)
    win = np.concatenate([np.repeat(tail, K, axis=0), cand.reshape(-1, 1)], axis=1)
    _, crow, _ = ot.lookup(win, 2, 1)
    tail_d, cand_d = torch.from_numpy(tail).cuda(), torch.from_numpy(cand).cuda()
    side = torch.cuda.Stream()

    def prefetch():
        tfe.tfe_prefetch(tier.handle, tail_d, 2, cand_d, B, K, side)

    before = tfe.tfe_memory_held()
    held = failing_calls(prefetch, None, [(k, "prefetch scratch") for k in range(1, 5)])
    assert held == [before] * 4
    prefetch()
    torch.cuda.synchronize()
    model.prefetch([int(r) for r in crow])
    check_stats(tier, model)
    # And a decode after it sees the prefetched rows as the model does.
    window = np.ascontiguousarray(seqs[:, 1:4])
    o = run_both(res, tier, window, 2, 1, synth.normal_range(1, 921, 0, B, table.dim, 1.0,
                                                             synth.BF16), table.dtype, table.dim)
    model.lookup([int(r) for r in o.slot.cpu().numpy()])
    check_stats(tier, model)
    tier.close()
    H.release_pinned()


def test_every_allocation_of_a_head(w2):
    V, D = 4096, 1024
    w = torch.randn(V, D, device="cuda").to(torch.bfloat16)
    base = tfe.tfe_memory_held()
    h, msgs = fail_every_allocation(lambda: tfe.tfe_head_create(w, V, D, 64, 16))
    assert names(msgs) == ["head"] + ["head scratch for 64 rows"] * 5
    tfe.tfe_head_free(h)
    assert tfe.tfe_memory_held() == base


def test_construction_gives_its_buffers_back_when_one_fails():
    """Construction buffers go back to the library's reuse cache when a call
    fails, and to the device allocator with tfe_ngram_release."""
    toks = torch.from_numpy(synth.zipf_tokens(3, 930, 1 << 16, 1.1).astype(np.int32)).cuda()
    top = 256
    ids = torch.empty((top, 2), dtype=torch.int32, device="cuda")
    cnt = torch.empty((top,), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()
    tfe.tfe_ngram_release()
    base = tfe.tfe_memory_held()
    want = tfe.tfe_ngram_top(toks, toks.numel(), synth.V, 2, 0, top, ids, cnt, H.cur_stream())
    torch.cuda.synchronize()
    ref_ids, ref_cnt = ids.clone(), cnt.clone()
    tfe.tfe_ngram_release()
    assert tfe.tfe_memory_held() == base
    n_fail = 0
    for k in range(1, 64):
        ids.fill_(-9)
        try:
            with FailAt(k):
                got = tfe.tfe_ngram_top(toks, toks.numel(), synth.V, 2, 0, top, ids, cnt,
                                        H.cur_stream())
        except tfe.TfeError as e:
            assert e.status == tfe.TFE_ERR_OOM, str(e)
            n_fail += 1
            tfe.tfe_ngram_release()
            assert tfe.tfe_memory_held() == base
            continue
        torch.cuda.synchronize()
        assert got == want and torch.equal(ids, ref_ids) and torch.equal(cnt, ref_cnt)
        break
    assert n_fail >= 3
    tfe.tfe_ngram_release()
    assert tfe.tfe_memory_held() == base
