"""Cache policy of tiered tables on calls of every length, against the
policy model (oracle/lru.py): statistics after every call and the residency
of every row (phrase id -> HBM cache slot, or host only), slot for slot.

Calls longer than 4096 positions are resolved over many blocks; the policy
must not depend on that: every cached row a call uses is referenced before
any victim is chosen (a row named only at the end of a long call is never
evicted by a miss at its start)."""
import os

import numpy as np
import pytest
import torch

import synth
from oracle.lru import LruModel
from paper_2607_07388_amd import tfe

from . import harness as H
from .test_gpu_tiered import STAT_KEYS, TieredTable, check_stats

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def w2():
    table = synth.config2_table()
    res = H.GpuTable(table)
    yield table, res, H.oracle_table(table)
    res.close()
    H.release_pinned()


def windows_for_rows(table, rows):
    """Decode windows (2 history tokens + 1) whose longest match is exactly
    the given row (-1: a window of absent tokens, no match)."""
    w = np.full((len(rows), 3), -1, np.int32)
    for i, r in enumerate(rows):
        if r >= 0:
            n = int(table.lens[r])
            w[i, 3 - n:] = table.tokens[r, :n]
    return w


def residency(tier, P):
    rows = torch.arange(P, dtype=torch.int32, device="cuda")
    out = torch.full((P,), -9, dtype=torch.int32, device="cuda")
    tfe.tfe_residency(tier.handle, rows, P, out, H.cur_stream())
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_residency(tier, model, P):
    """The phrases held in the HBM tier equal the model's cached rows, and
    every cached row has its own physical slot (slot numbers are placement:
    the cache has kDecodeMaxT = 64 physical slots beyond its rows)."""
    got = residency(tier, P)
    assert np.all(got >= -1)
    cached = np.flatnonzero(got >= 0)
    want = np.array(sorted(model.resident()), np.int64)
    missing = np.setdiff1d(want, cached)
    extra = np.setdiff1d(cached, want)
    assert missing.size == 0 and extra.size == 0, (missing[:8], extra[:8])
    slots = got[cached]
    assert np.unique(slots).size == slots.size
    assert slots.max(initial=0) < model.C + 64


def call(tier, res, table, tokens, hidden, inplace=False, stream=None):
    """One call on the tiered table and one on the resident table; outputs
    byte-identical; returns the matched rows."""
    T = tokens.shape[0]
    tok = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    h1 = H.to_device(hidden, synth.BF16)
    h2 = h1.clone()
    o1, o2 = H.Outputs(T, 1024, synth.BF16), H.Outputs(T, 1024, synth.BF16)
    out1 = H.run(res, tok, T, 2, 1, h1, o1, inplace=inplace)
    out2 = h2 if inplace else o2.out
    tfe.tfe_lookup_inject(tier.handle, tok, T, 2, 1, h2, out2, o2.hit, o2.slot, o2.len,
                          tfe.TFE_GATE_SIGMOID, 1.0,
                          stream.cuda_stream if stream is not None else H.cur_stream())
    torch.cuda.synchronize()
    assert torch.equal(o1.slot, o2.slot) and torch.equal(o1.hit, o2.hit)
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    return o2.slot.cpu().numpy()


@pytest.mark.parametrize("fill", [tfe.TFE_FILL_INLINE, tfe.TFE_FILL_SIDE_STREAM])
def test_late_reference_is_not_evicted_in_a_long_call(w2, fill):
    table, res, ot = w2
    C = 4
    tier = TieredTable(table, C, C, fill=fill)      # rows 0..3 cached; least recent: row 3
    model = LruModel(C, C, 2048, fill_rereads=fill == tfe.TFE_FILL_SIDE_STREAM)
    T = 5000
    rows = [100] + [-1] * (T - 2) + [3]
    tokens = windows_for_rows(table, rows)
    hidden = synth.normal_range(11, 1, 0, T, 1024, 1.0, synth.BF16)
    got = call(tier, res, table, tokens, hidden)
    np.testing.assert_array_equal(got, np.array(rows, np.int32))
    model.lookup(rows)
    check_stats(tier, model)
    check_residency(tier, model, table.n_phrases)
    assert model.resident() == {0: 0, 1: 1, 3: 3, 100: 2}
    st = tfe.tfe_get_stats(tier.handle)
    assert st["cache_hits"] == 1 and st["cache_misses"] == 1
    tier.close()


@pytest.mark.parametrize("fill", [tfe.TFE_FILL_INLINE, tfe.TFE_FILL_SIDE_STREAM])
def test_long_calls_of_every_shape_follow_the_model(w2, fill):
    """Calls of 4097 .. 20000 positions (ragged last blocks) drawn from a few
    hundred rows, so rows repeat within a call and across calls, cached rows
    recur late, and the cache (300 rows) is smaller than a call's distinct
    rows: victims, direct host reads and ring compaction all occur; one call
    in place.  Outputs equal the resident table byte for byte and the
    oracle's rows; stats and residency equal the model after every call."""
    table, res, ot = w2
    C, pre = 300, 120
    tier = TieredTable(table, C, pre, fill=fill)
    model = LruModel(C, pre, 2048, fill_rereads=fill == tfe.TFE_FILL_SIDE_STREAM)
    rng = np.random.default_rng(31 + fill)
    pool = np.concatenate([np.arange(0, 200), rng.choice(table.n_phrases, 400, replace=False)])
    for step, T in enumerate([4097, 6000, 9000, 5121, 20000, 4097, 8191]):
        pick = rng.zipf(1.3, T) % pool.size
        rows = pool[pick].astype(np.int64)
        rows[rng.random(T) < 0.2] = -1
        tokens = windows_for_rows(table, rows)
        hidden = synth.normal_range(12, step, 0, T, 1024, 1.0, synth.BF16)
        got = call(tier, res, table, tokens, hidden, inplace=step == 2)
        _, orow, _ = ot.lookup(tokens, 2, 1)
        np.testing.assert_array_equal(got, orow)
        np.testing.assert_array_equal(got, rows.astype(np.int32))
        model.lookup([int(r) for r in rows])
        check_stats(tier, model)
        check_residency(tier, model, table.n_phrases)
    tier.close()


def test_prefetch_then_long_lookup_without_sync(w2):
    """tfe_prefetch on a side stream, then at once (no synchronisation, no
    stats read) a lookup of 200 positions on the main stream, which runs the
    wide probe and the one-block resolve: the lookup must wait for the
    prefetch before any of its kernels touch the shared scratch, ring or
    residency.  A 16-row cache makes ring compaction fire along the way."""
    table, res, ot = w2
    C, pre, B, K, T = 16, 8, 64, 8, 200
    tier = TieredTable(table, C, pre)
    model = LruModel(C, pre, 2048)
    side = torch.cuda.Stream()
    rng = np.random.default_rng(99)
    seqs = synth.zipf_tokens(1, 900, T * 40, 1.1).reshape(T, 40)
    outs = []
    for s in range(30):
        tail = np.ascontiguousarray(seqs[:B, s + 1:s + 3])
        cand = synth.workloads.candidates(1, B, K, seqs[:B, s + 3], step=300 + s)
        win = np.concatenate([np.repeat(tail, K, axis=0), cand.reshape(-1, 1)], axis=1)
        _, crow, _ = ot.lookup(win, 2, 1)
        window = np.ascontiguousarray(seqs[:, s:s + 3])
        hidden = synth.normal_range(13, s, 0, T, 1024, 1.0, synth.BF16)
        tok = torch.from_numpy(window).cuda()
        h = H.to_device(hidden, synth.BF16)
        o = H.Outputs(T, 1024, synth.BF16)
        tail_d, cand_d = torch.from_numpy(tail).cuda(), torch.from_numpy(cand).cuda()
        torch.cuda.synchronize()
        tfe.tfe_prefetch(tier.handle, tail_d, 2, cand_d, B, K, side)
        tfe.tfe_lookup_inject(tier.handle, tok, T, 2, 1, h, o.out, o.hit, o.slot, o.len,
                              tfe.TFE_GATE_SIGMOID, 1.0, H.cur_stream())
        outs.append((window, hidden, o, tail_d, cand_d, tok, h))
        model.prefetch([int(r) for r in crow])
        _, row, _ = ot.lookup(window, 2, 1)
        model.lookup([int(r) for r in row])
    torch.cuda.synchronize()
    for window, hidden, o, *_ in outs:
        o1 = H.Outputs(T, 1024, synth.BF16)
        H.run(res, torch.from_numpy(window).cuda(), T, 2, 1, H.to_device(hidden, synth.BF16), o1)
        torch.cuda.synchronize()
        assert torch.equal(o1.slot, o.slot)
        assert torch.equal(o1.out.view(torch.int16), o.out.view(torch.int16))
    check_stats(tier, model)
    check_residency(tier, model, table.n_phrases)
    tier.close()


def test_recency_clock_restart(w2):
    """The 32-bit recency clock restarts (stamps renormalised, order kept)
    without changing the policy: a table whose clock starts 20 calls below
    the wrap runs 40 calls of mixed lengths with prefetches."""
    table, res, ot = w2
    C, pre = 64, 32
    os.environ["TFE_TIER_CLOCK_START"] = str(0xFFFFFFFF - 20)
    try:
        tier = TieredTable(table, C, pre)
    finally:
        del os.environ["TFE_TIER_CLOCK_START"]
    model = LruModel(C, pre, 2048)
    rng = np.random.default_rng(5)
    pool = np.arange(0, 400)
    side = torch.cuda.Stream()
    for step in range(40):
        T = [64, 300, 5000][step % 3]
        rows = pool[rng.zipf(1.2, T) % pool.size].astype(np.int64)
        tokens = windows_for_rows(table, rows)
        hidden = synth.normal_range(14, step, 0, T, 1024, 1.0, synth.BF16)
        call(tier, res, table, tokens, hidden)
        model.lookup([int(r) for r in rows])
        if step % 4 == 1:
            cr = pool[rng.zipf(1.2, 64) % pool.size].astype(np.int64)
            cw = windows_for_rows(table, cr)
            # Candidate = the window's last token, tail = the two before it:
            # the candidate's longest match is the row itself.
            cand = torch.from_numpy(np.ascontiguousarray(cw[:, 2:3])).cuda()
            tail = torch.from_numpy(np.ascontiguousarray(cw[:, 0:2])).cuda()
            tfe.tfe_prefetch(tier.handle, tail, 2, cand, 64, 1, side)
            model.prefetch([int(r) for r in cr])
        check_stats(tier, model)
    check_residency(tier, model, table.n_phrases)
    tier.close()


def test_prefetch_keeps_the_cached_rows_it_names(w2):
    """Candidates whose rows sit in the least recent slots: the prefetch
    references them (never its own victims) and fills the other rows into
    the next least recent slots, after lookups through each launch shape."""
    table, res, ot = w2
    for pattern in [(64, 300), (64, 64), (5000, 5000)]:
        C, pre = 64, 32
        tier = TieredTable(table, C, pre)
        model = LruModel(C, pre, 2048)
        rng = np.random.default_rng(5)
        pool = np.arange(0, 400)
        for step, T in enumerate(pattern):
            rows = pool[rng.zipf(1.2, T) % pool.size].astype(np.int64)
            call(tier, res, table, windows_for_rows(table, rows),
                 synth.normal_range(14, step, 0, T, 1024, 1.0, synth.BF16))
            model.lookup([int(r) for r in rows])
        cr = pool[rng.zipf(1.2, 64) % pool.size].astype(np.int64)
        cw = windows_for_rows(table, cr)
        cand = torch.from_numpy(np.ascontiguousarray(cw[:, 2:3])).cuda()
        tail = torch.from_numpy(np.ascontiguousarray(cw[:, 0:2])).cuda()
        tfe.tfe_prefetch(tier.handle, tail, 2, cand, 64, 1, torch.cuda.Stream())
        model.prefetch([int(r) for r in cr])
        check_stats(tier, model)
        check_residency(tier, model, table.n_phrases)
        tier.close()


def test_residency_of_resident_table_and_bad_ids(w2):
    table, res, ot = w2
    rows = torch.tensor([0, 5, table.n_phrases - 1, -1, table.n_phrases, 1 << 30],
                        dtype=torch.int32, device="cuda")
    out = torch.full((6,), -9, dtype=torch.int32, device="cuda")
    tfe.tfe_residency(res.handle, rows, 6, out, H.cur_stream())
    torch.cuda.synchronize()
    assert out.cpu().tolist() == [0, 5, table.n_phrases - 1, -2, -2, -2]
    tfe.tfe_residency(res.handle, rows, 0, out, H.cur_stream())  # empty query
    with pytest.raises(tfe.TfeError):
        tfe.tfe_residency(res.handle, rows, -1, out, H.cur_stream())


def continuations(table, need):
    """The table's 2-gram phrases grouped by first token: (first, seconds)
    for the first tokens with at least `need` continuations, most first."""
    two = np.flatnonzero(table.lens == 2)
    f, s = table.tokens[two, 0], table.tokens[two, 1]
    order = np.argsort(f, kind="stable")
    f, s = f[order], s[order]
    uniq, start, cnt = np.unique(f, return_index=True, return_counts=True)
    out = []
    for i in np.argsort(-cnt, kind="stable"):
        if cnt[i] < need:
            break
        out.append((int(uniq[i]), s[start[i]:start[i] + cnt[i]]))
    return out


@pytest.mark.parametrize("K,many", [(64, True), (80, False), (80, True)])
def test_scored_prefetch_selection_paths(w2, K, many):
    """Eq. 17's budgeted selection ranks a call's distinct uncached candidate
    rows by score: by counting when they number at most one per thread of
    the resolving block, else by radix select, gather and sort -- in the
    one-block prefetch (up to 4096 windows: K = 64) and in the global-memory
    resolution (K = 80: 5120 windows).  Each row's candidates continue its
    last token with 2-grams the table holds: all K of them (thousands of
    distinct rows), or 4 of them and absent tokens otherwise (a few
    hundred), so that each case takes the path it names (asserted from the
    model's count).  Statistics and residency equal the model after every
    call; outputs equal the resident table."""
    table, res, ot = w2
    B, C, pre, budget, steps = 64, 8192, 4096, 256, 4
    groups = continuations(table, K)
    assert len(groups) >= B * steps
    tier = TieredTable(table, C, pre)
    model = LruModel(C, pre, 2048)
    rng = np.random.default_rng(K + int(many))
    seqs = synth.zipf_tokens(1, 1500 + K, B * (steps + 3), 1.1).reshape(B, steps + 3)
    # Scores fall with the candidate's rank, in equal pairs (ties).
    prob = np.tile(((K - np.arange(K)) // 2 + 1).astype(np.float32), (B, 1))
    prob /= prob.sum(axis=1, keepdims=True)
    side = torch.cuda.Stream()
    for s in range(steps):
        hidden = synth.normal_range(17, s, 0, B, 1024, 1.0, synth.BF16)
        rows = call(tier, res, table, np.ascontiguousarray(seqs[:, s:s + 3]), hidden)
        model.lookup([int(r) for r in rows])
        tail = np.full((B, 2), -1, np.int32)
        cand = np.full((B, K), -1, np.int32)
        take = K if many else 4
        for b in range(B):
            first, nexts = groups[s * B + b]
            tail[b, 1] = first
            cand[b, :take] = rng.choice(nexts, take, replace=False)
        win = np.concatenate([np.repeat(tail, K, axis=0), cand.reshape(-1, 1)], axis=1)
        _, crow, clen = ot.lookup(win, 2, 1)
        cached = set(int(r) for r in model.resident())
        n = len({int(r) for r in crow if r >= 0 and int(r) not in cached})
        assert (n > 1024) if many else (0 < n <= 1024), n
        tfe.tfe_prefetch_scored(tier.handle, torch.from_numpy(tail).cuda(), 2,
                                torch.from_numpy(cand).cuda(), torch.from_numpy(prob).cuda(),
                                B, K, budget, side)
        model.prefetch_scored([int(r) for r in crow], [int(x) for x in clen], prob.ravel(),
                              budget)
        check_stats(tier, model)
        check_residency(tier, model, table.n_phrases)
    st = tfe.tfe_get_stats(tier.handle)
    assert st["prefetch_filled"] > 0
    if many:
        assert st["prefetch_dropped"] > 0
    tier.close()


@pytest.mark.parametrize("budget", [64, 1024])
def test_head_topk_feeds_scored_prefetch_at_batch64_k128(w2, budget):
    """The early-exit head's top 128 of a 151936-token vocabulary for 64 rows
    (Eq. 13, Eq. 14) goes straight into tfe_prefetch_scored (Eq. 17): 8192
    candidates per call, more candidate rows than the budget (the threshold
    is found by radix select), cached candidates referenced.  Alternate steps
    run the plain prefetch of the same 8192 candidates (the multi-block
    resolve).  Statistics and residency equal the model after every call;
    outputs equal the resident table."""
    table, res, ot = w2
    V, Dh, B, K, steps = synth.V, 1024, 64, 128, 6
    C, pre = 8192, 4096
    w = torch.empty((V, Dh), dtype=torch.bfloat16, device="cuda")
    synth.normal_fill_device(w.data_ptr(), 0, V, Dh, 3, 40, 0.1, synth.BF16, H.cur_stream())
    torch.cuda.synchronize()
    head = tfe.tfe_head_create(w, V, Dh, B, K)
    tier = TieredTable(table, C, pre)
    model = LruModel(C, pre, 2048)
    seqs = synth.zipf_tokens(1, 1200 + budget, B * (steps + 3), 1.1).reshape(B, steps + 3)
    side = torch.cuda.Stream()
    for s in range(steps):
        window = np.ascontiguousarray(seqs[:, s:s + 3])
        hidden = synth.normal_range(15, s, 0, B, 1024, 1.0, synth.BF16)
        rows = call(tier, res, table, window, hidden)
        model.lookup([int(r) for r in rows])
        hd = H.to_device(synth.normal_range(16, s, 0, B, Dh, 1.0, synth.BF16), synth.BF16)
        ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
        prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
        tfe.tfe_head_topk(head, hd, B, K, ids, prob, H.cur_stream())
        torch.cuda.synchronize()
        tail = np.ascontiguousarray(seqs[:, s + 1:s + 3])
        ids_h, prob_h = ids.cpu().numpy(), prob.cpu().numpy()
        win = np.concatenate([np.repeat(tail, K, axis=0), ids_h.reshape(-1, 1)], axis=1)
        _, crow, clen = ot.lookup(win, 2, 1)
        tail_d = torch.from_numpy(tail).cuda()
        if s % 2 == 0:
            tfe.tfe_prefetch_scored(tier.handle, tail_d, 2, ids, prob, B, K, budget, side)
            model.prefetch_scored([int(r) for r in crow], [int(x) for x in clen],
                                  prob_h.ravel(), budget)
        else:
            tfe.tfe_prefetch(tier.handle, tail_d, 2, ids, B, K, side)
            model.prefetch([int(r) for r in crow])
        check_stats(tier, model)
        check_residency(tier, model, table.n_phrases)
    st = tfe.tfe_get_stats(tier.handle)
    assert st["prefetch_filled"] > 0
    if budget == 64:
        assert st["prefetch_dropped"] > 0
    tier.close()
    tfe.tfe_head_free(head)


@pytest.mark.parametrize("scored", [False, True])
def test_decode_and_prefetch_overlapping_without_sync(w2, scored):
    """Decode steps on the main stream and a prefetch of 8 candidates per
    row on a side stream after each, 300 steps enqueued without any
    synchronisation, so that each prefetch's probe overlaps the decode
    before it and the next decode waits for the prefetch on the device.  A
    2048-row cache makes victims and ring compactions frequent.  Every
    step's output equals the resident table's; statistics and residency
    equal the model at the end."""
    table, res, ot = w2
    C, pre, B, K, steps = 2048, 1024, 64, 8, 300
    tier = TieredTable(table, C, pre)
    model = LruModel(C, pre, 2048)
    seqs = synth.zipf_tokens(1, 1300 + scored, B * (steps + 3), 1.1).reshape(B, steps + 3)
    seqs_d = torch.from_numpy(seqs).cuda()
    wins = [seqs_d[:, s:s + 3].contiguous() for s in range(steps)]
    tails = [seqs_d[:, s + 1:s + 3].contiguous() for s in range(steps)]
    cands = np.stack([synth.workloads.candidates(1, B, K, seqs[:, s + 3], step=500 + s)
                      for s in range(steps)])
    cands_d = torch.from_numpy(cands).cuda()
    prob = torch.from_numpy(np.tile((np.float32(0.5) ** np.arange(K)).astype(np.float32),
                                    (B, 1))).cuda()
    hid = H.to_device(synth.normal_range(17, 0, 0, B * steps, 1024, 1.0, synth.BF16), synth.BF16)
    out = torch.empty((steps, B, 1024), dtype=torch.bfloat16, device="cuda")
    slots = torch.full((steps, B), -7, dtype=torch.int32, device="cuda")
    hit = torch.zeros((steps, B), dtype=torch.uint8, device="cuda")
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    for s in range(steps):
        tfe.tfe_lookup_inject(tier.handle, wins[s], B, 2, 1, hid[s * B:(s + 1) * B], out[s],
                              hit[s], slots[s], None, tfe.TFE_GATE_SIGMOID, 1.0, H.cur_stream())
        if scored:
            tfe.tfe_prefetch_scored(tier.handle, tails[s], 2, cands_d[s], prob, B, K, 48, side)
        else:
            tfe.tfe_prefetch(tier.handle, tails[s], 2, cands_d[s], B, K, side)
    torch.cuda.synchronize()
    # The same steps on the resident table.
    o_res = H.Outputs(B * steps, 1024, synth.BF16)
    win_all = np.ascontiguousarray(np.concatenate([seqs[:, s:s + 3] for s in range(steps)]))
    H.run(res, torch.from_numpy(win_all).cuda(), B * steps, 2, 1, hid, o_res)
    torch.cuda.synchronize()
    assert torch.equal(o_res.slot, slots.view(-1))
    assert torch.equal(o_res.out.view(torch.int16), out.view(-1, 1024).view(torch.int16))
    # The model, call by call.
    pk = (np.float32(0.5) ** np.arange(K)).astype(np.float32)
    for s in range(steps):
        _, row, _ = ot.lookup(np.ascontiguousarray(seqs[:, s:s + 3]), 2, 1)
        model.lookup([int(r) for r in row])
        win = np.concatenate([np.repeat(seqs[:, s + 1:s + 3], K, axis=0),
                              cands[s].reshape(-1, 1)], axis=1)
        _, crow, clen = ot.lookup(win, 2, 1)
        if scored:
            model.prefetch_scored([int(r) for r in crow], [int(x) for x in clen],
                                  np.tile(pk, B), 48)
        else:
            model.prefetch([int(r) for r in crow])
    check_stats(tier, model)
    check_residency(tier, model, table.n_phrases)
    tier.close()


@pytest.mark.parametrize("fill", [tfe.TFE_FILL_INLINE, tfe.TFE_FILL_SIDE_STREAM])
def test_random_interleavings_of_every_call_kind(w2, fill):
    """A seeded random sequence of 400 calls on one tiered table: decode
    lookups (64 positions, one launch) and long lookups (65 to 6000
    positions, several kernels) on two streams; plain and scored prefetches
    of at most 4096 candidates (one block) and of more (several kernels) on
    any of three streams, scored ones with random budgets; now and then a
    device synchronisation or a statistics read.  Every input and output
    buffer is made first; the calls are then enqueued with no other
    synchronisation.  Calls on one table take effect in the order they are
    enqueued, whatever their streams, so every lookup's output equals the
    resident table's byte for byte, and the statistics (at every read and at
    the end) and the residency of every row equal the policy model fed the
    same calls in that order.  A 4096-row cache keeps victims and
    recency-ring compactions frequent."""
    table, res, ot = w2
    C, pre, B = 4096, 2048, 64
    print("# random interleavings, fill mode %d" % fill, flush=True)
    rng = np.random.default_rng(4242 + fill)
    kinds = ["decode", "long", "pf", "pf_big", "scored", "scored_big", "sync", "stats"]
    weights = np.array([30, 12, 14, 5, 14, 5, 6, 4], np.float64)
    plan = []
    for i in range(400):
        kind = kinds[rng.choice(len(kinds), p=weights / weights.sum())]
        c = {"kind": kind, "stream": int(rng.integers(0, 3))}
        if kind in ("decode", "long"):
            T = 64 if kind == "decode" else int(rng.integers(65, 6001))
            seq = synth.zipf_tokens(51, 100 + i, T + 2, 1.1)
            win = np.stack([seq[0:T], seq[1:T + 1], seq[2:T + 2]], axis=1).astype(np.int32)
            c.update(T=T, win=win, stream=int(rng.integers(0, 2)),
                     tok=torch.from_numpy(win).cuda(),
                     hid=H.to_device(synth.normal_range(52, i, 0, T, 1024, 1.0, synth.BF16),
                                     synth.BF16),
                     out=H.Outputs(T, 1024, synth.BF16))
        elif kind not in ("sync", "stats"):
            K = int(rng.integers(1, 65)) if kind in ("pf", "scored") else int(rng.integers(65, 129))
            tail = synth.zipf_tokens(53, 100 + i, B * 2, 1.1).reshape(B, 2)
            cand = synth.zipf_tokens(54, 100 + i, B * K, 1.1).reshape(B, K)
            c.update(K=K, tail=tail, cand=cand,
                     tail_d=torch.from_numpy(np.ascontiguousarray(tail)).cuda(),
                     cand_d=torch.from_numpy(np.ascontiguousarray(cand)).cuda())
            if kind.startswith("scored"):
                c["prob"] = rng.dirichlet(np.ones(K) * 0.5, B).astype(np.float32)
                c["prob_d"] = torch.from_numpy(c["prob"]).cuda()
                c["budget"] = int(rng.integers(8, 1025))
        plan.append(c)
    tier = TieredTable(table, C, pre, fill=fill)
    model = LruModel(C, pre, 2048, fill_rereads=fill == tfe.TFE_FILL_SIDE_STREAM)
    streams = [torch.cuda.current_stream(), torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for c in plan:
        kind, st = c["kind"], streams[c["stream"]]
        if kind == "sync":
            torch.cuda.synchronize()
        elif kind == "stats":
            check_stats(tier, model)
        elif kind in ("decode", "long"):
            o, T = c["out"], c["T"]
            tfe.tfe_lookup_inject(tier.handle, c["tok"], T, 2, 1, c["hid"], o.out, o.hit, o.slot,
                                  o.len, tfe.TFE_GATE_SIGMOID, 1.0, st)
            _, row, _ = ot.lookup(c["win"], 2, 1)
            model.lookup([int(r) for r in row])
        else:
            K = c["K"]
            win = np.concatenate([np.repeat(c["tail"], K, axis=0), c["cand"].reshape(-1, 1)],
                                 axis=1)
            _, crow, clen = ot.lookup(np.ascontiguousarray(win, np.int32), 2, 1)
            if kind.startswith("scored"):
                tfe.tfe_prefetch_scored(tier.handle, c["tail_d"], 2, c["cand_d"], c["prob_d"], B,
                                        K, c["budget"], st)
                model.prefetch_scored([int(r) for r in crow], [int(x) for x in clen],
                                      c["prob"].reshape(-1), c["budget"])
            else:
                tfe.tfe_prefetch(tier.handle, c["tail_d"], 2, c["cand_d"], B, K, st)
                model.prefetch([int(r) for r in crow])
    torch.cuda.synchronize()
    for c in plan:
        if c["kind"] not in ("decode", "long"):
            continue
        o, T = c["out"], c["T"]
        o_res = H.Outputs(T, 1024, synth.BF16)
        H.run(res, c["tok"], T, 2, 1, c["hid"], o_res)
        torch.cuda.synchronize()
        assert torch.equal(o_res.slot, o.slot) and torch.equal(o_res.hit, o.hit)
        assert torch.equal(o_res.out.view(torch.int16), o.out.view(torch.int16))
    check_stats(tier, model)
    check_residency(tier, model, table.n_phrases)
    tier.close()
