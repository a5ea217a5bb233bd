"""The one-launch head (tfe_head_topk for at most 64 rows and K at most the
number of compute units: logits held in registers, a bound of each row's
K-th largest logit from the blocks' maxima, only the logits above it
written) against the two-launch kernels (tfe_head_topk_noalloc, which
writes every logit), on the same inputs: ids bit-exact and probabilities
within 1e-5 relative (the two add the softmax denominator up in different
orders).  The shapes take every branch of the selection: the usual few
hundred candidates per row, K = 1 and K = 256, heavy ties (an all-zero
projection makes every logit a candidate, more than LDS holds, so the
selection first narrows in memory), the largest logits clustered in a few
blocks, vocabularies smaller than one tile per block, and every width.
Many calls in a row on one head, and calls of two heads interleaved on
one stream, check that the grid barriers' counters stay aligned; calls of
two heads on two streams without synchronisation run one after another;
calls captured in a HIP graph replay correctly between eager calls; a
call
whose barrier waits are forced to give up (TFE_HEAD_WAIT_LIMIT=0) answers
-1 and leaves the head working."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu


def two_launch(w, V, D, h, B, K):
    ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
    tfe.tfe_head_topk_noalloc(w, V, D, h, B, K, ids, prob, H.cur_stream())
    torch.cuda.synchronize()
    return ids.cpu().numpy(), prob.cpu().numpy()


def one_launch(head, h, B, K):
    ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
    tfe.tfe_head_topk(head, h, B, K, ids, prob, H.cur_stream())
    torch.cuda.synchronize()
    return ids.cpu().numpy(), prob.cpu().numpy()


def gaussian(seed, V, D, B, scale=0.1):
    w = torch.empty((V, D), dtype=torch.bfloat16, device="cuda")
    synth.normal_fill_device(w.data_ptr(), 0, V, D, seed, 40, scale, synth.BF16, H.cur_stream())
    h = H.to_device(synth.normal_range(seed, 41, 0, B, D, 1.0, synth.BF16), synth.BF16)
    torch.cuda.synchronize()
    return w, h


def small_ints(seed, V, D, B, lo, hi):
    rng = np.random.default_rng(seed)
    w = rng.integers(lo, hi, (V, D)).astype(np.float32)
    h = rng.integers(lo, hi, (B, D)).astype(np.float32)
    bits = lambda x: (x.view(np.uint32) >> 16).astype(np.uint16)
    return H.to_device(bits(w), synth.BF16), H.to_device(bits(h), synth.BF16)


def check(w, h, V, D, B, K, calls=1):
    print("# one launch vs two: V=%d D=%d B=%d K=%d" % (V, D, B, K), flush=True)
    want_ids, want_prob = two_launch(w, V, D, h, B, K)
    head = tfe.tfe_head_create(w, V, D, B, K)
    try:
        for _ in range(calls):
            ids, prob = one_launch(head, h, B, K)
            np.testing.assert_array_equal(ids, want_ids)
            np.testing.assert_allclose(prob, want_prob, rtol=1e-5, atol=1e-37)
    finally:
        tfe.tfe_head_free(head)
    assert np.all(want_ids >= 0) and np.all(want_ids < V)


@pytest.mark.parametrize("V,D,B,K", [
    (151936, 1024, 64, 128),   # the batch-64 decode step
    (151936, 1024, 64, 1),
    (151936, 1024, 64, 256),   # K = the number of blocks
    (151936, 1024, 1, 64),
    (151936, 1024, 13, 7),     # fewer groups than the 8 threads of a row
    (40000, 512, 64, 100),
    (3001, 256, 5, 17),        # ragged vocabulary
    (300, 512, 17, 256),       # fewer tiles than blocks: empty blocks
    (100, 1024, 64, 50),
])
def test_gaussian(V, D, B, K):
    w, h = gaussian(V + K, V, D, B)
    check(w, h, V, D, B, K)


def test_all_logits_equal_narrows_in_memory():
    V, D, B, K = 151936, 1024, 64, 128
    w = torch.zeros((V, D), dtype=torch.bfloat16, device="cuda")
    _, h = gaussian(3, 16, D, B)
    check(w, h, V, D, B, K)


def test_integer_ties():
    V, D, B = 151936, 256, 64
    w, h = small_ints(4, V, D, B, 0, 2)
    check(w, h, V, D, B, 128)
    w, h = small_ints(5, V, D, B, -2, 3)
    check(w, h, V, D, B, 256)


def test_largest_logits_clustered_in_a_few_blocks():
    V, D, B, K = 151936, 1024, 64, 256
    w, h = gaussian(6, V, D, B)
    w[:2000] *= 10
    check(w, h, V, D, B, K)


def test_many_calls_and_two_heads_interleaved():
    V, D, B, K = 151936, 1024, 64, 128
    w1, h1 = gaussian(7, V, D, B)
    w2, h2 = gaussian(8, V, D, B)
    want1 = two_launch(w1, V, D, h1, B, K)
    want2 = two_launch(w2, V, D, h2, B, K)
    a = tfe.tfe_head_create(w1, V, D, B, K)
    b = tfe.tfe_head_create(w2, V, D, B, K)
    try:
        for i in range(40):
            for head, h, want in ((a, h1, want1), (b, h2, want2)) if i % 3 else ((b, h2, want2),):
                ids, prob = one_launch(head, h, B, K)
                np.testing.assert_array_equal(ids, want[0])
                np.testing.assert_allclose(prob, want[1], rtol=1e-5, atol=1e-37)
        # Back to back without synchronising in between.
        outs = []
        for _ in range(20):
            ids = torch.empty((B, K), dtype=torch.int32, device="cuda")
            prob = torch.empty((B, K), dtype=torch.float32, device="cuda")
            tfe.tfe_head_topk(a, h1, B, K, ids, prob, H.cur_stream())
            outs.append((ids, prob))
        torch.cuda.synchronize()
        for ids, prob in outs:
            np.testing.assert_array_equal(ids.cpu().numpy(), want1[0])
    finally:
        tfe.tfe_head_free(a)
        tfe.tfe_head_free(b)


def test_two_heads_on_two_streams_without_sync():
    """One-launch calls of two heads on two streams, issued alternately with
    no synchronisation in between: the library runs them one after another
    on the device (side by side, each could hold compute units with blocks
    waiting at a barrier for blocks of its own that cannot start, until the
    bounded waits give up).  Every call matches the two-launch kernels."""
    V, D, B, K = 151936, 1024, 64, 128
    print("# two heads, two streams: V=%d D=%d B=%d K=%d" % (V, D, B, K), flush=True)
    w1, h1 = gaussian(12, V, D, B)
    w2, h2 = gaussian(13, V, D, B)
    want1 = two_launch(w1, V, D, h1, B, K)
    want2 = two_launch(w2, V, D, h2, B, K)
    a = tfe.tfe_head_create(w1, V, D, B, K)
    b = tfe.tfe_head_create(w2, V, D, B, K)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    try:
        outs = []
        for _ in range(16):
            for head, h, st, want in ((a, h1, s1, want1), (b, h2, s2, want2)):
                ids = torch.empty((B, K), dtype=torch.int32, device="cuda")
                prob = torch.empty((B, K), dtype=torch.float32, device="cuda")
                tfe.tfe_head_topk(head, h, B, K, ids, prob, st)
                outs.append((ids, prob, want))
        torch.cuda.synchronize()
        for ids, prob, want in outs:
            np.testing.assert_array_equal(ids.cpu().numpy(), want[0])
            np.testing.assert_allclose(prob.cpu().numpy(), want[1], rtol=1e-5, atol=1e-37)
    finally:
        tfe.tfe_head_free(a)
        tfe.tfe_head_free(b)


@pytest.mark.parametrize("B,K", [(64, 128), (100, 64)])
def test_captured_calls_replay_with_eager_calls_between(B, K):
    """Head calls captured in a HIP graph (through torch's CUDA-graph API):
    64 rows take the one-launch path, 100 rows the two launches.  The call
    epoch that the one-launch barriers count against lives on the device, so
    graph replays and eager calls of the same head stay aligned in any
    order: three calls on different inputs are captured, the graph is
    replayed three times with eager calls of the head and eager fills of the
    outputs between, and every output equals the eager calls' (for 64 rows,
    whose ids equal the two-launch kernels')."""
    V, D = 151936, 1024
    print("# captured head calls: V=%d D=%d B=%d K=%d" % (V, D, B, K), flush=True)
    w, h0 = gaussian(14, V, D, B)
    hs = [h0] + [H.to_device(synth.normal_range(14, 41 + k, 0, B, D, 1.0, synth.BF16),
                             synth.BF16) for k in (1, 2)]
    head = tfe.tfe_head_create(w, V, D, B, K)
    want = [one_launch(head, h, B, K) for h in hs]  # eager calls, the same path
    if B <= 64:
        for h, wnt in zip(hs, want):
            np.testing.assert_array_equal(two_launch(w, V, D, h, B, K)[0], wnt[0])
    outs = [(torch.empty((B, K), dtype=torch.int32, device="cuda"),
             torch.empty((B, K), dtype=torch.float32, device="cuda")) for _ in hs]

    def calls():
        s = torch.cuda.current_stream().cuda_stream
        for h, (ids, prob) in zip(hs, outs):
            tfe.tfe_head_topk(head, h, B, K, ids, prob, s)

    try:
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            calls()  # warm-up on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            calls()
        for rep in range(3):
            for ids, prob in outs:  # eager work between replays
                ids.fill_(-7)
                prob.fill_(-1.0)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for (ids, prob), wnt in zip(outs, want):
                np.testing.assert_array_equal(ids.cpu().numpy(), wnt[0])
                np.testing.assert_allclose(prob.cpu().numpy(), wnt[1], rtol=1e-5, atol=1e-37)
            ids, prob = one_launch(head, hs[rep], B, K)
            np.testing.assert_array_equal(ids, want[rep][0])
            np.testing.assert_allclose(prob, want[rep][1], rtol=1e-5, atol=1e-37)
        del g
    finally:
        tfe.tfe_head_free(head)


def test_a_barrier_wait_that_gives_up_fails_only_its_call(monkeypatch):
    """The one-launch barriers' waits are bounded; TFE_HEAD_WAIT_LIMIT=0
    makes every wait give up at once (forced from the host: every block
    still arrives, so no kernel waits forever).  That call answers every row
    with id -1 and probability 0, and tfe_head_last_fault names it; the next
    calls on the same head, with the default limit, are correct again (the
    barrier counters stayed aligned) and leave the fault record as it was."""
    V, D, B, K = 40000, 1024, 64, 64
    w, h = gaussian(11, V, D, B)
    want = two_launch(w, V, D, h, B, K)
    head = tfe.tfe_head_create(w, V, D, B, K)
    try:
        ids, prob = one_launch(head, h, B, K)
        np.testing.assert_array_equal(ids, want[0])
        assert tfe.tfe_head_last_fault(head) == 0
        monkeypatch.setenv("TFE_HEAD_WAIT_LIMIT", "0")
        ids, prob = one_launch(head, h, B, K)
        assert np.all(ids == -1) and np.all(prob == 0)
        assert tfe.tfe_head_last_fault(head) == 2  # the second one-launch call
        monkeypatch.delenv("TFE_HEAD_WAIT_LIMIT")
        for _ in range(3):
            ids, prob = one_launch(head, h, B, K)
            np.testing.assert_array_equal(ids, want[0])
            np.testing.assert_allclose(prob, want[1], rtol=1e-5, atol=1e-37)
        assert tfe.tfe_head_last_fault(head) == 2
    finally:
        tfe.tfe_head_free(head)
