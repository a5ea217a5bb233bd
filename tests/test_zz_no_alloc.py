"""The no-allocation entry point tfe_head_topk_noalloc (for callers that
cannot allocate) against tfe_head_topk on the same inputs: two calls in a
row, the second smaller (fewer rows, a ragged vocabulary, another width),
ids bit-exact and probabilities within 1e-5 relative (tfe_head_topk takes
the one-launch path for these shapes, which adds the softmax denominator up
per logits block instead of per tile); sizes beyond its scratch are
refused."""
import numpy as np
import pytest
import torch

import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu


def reference(w, V, D, h, B, K):
    head = tfe.tfe_head_create(w, V, D, B, K)
    ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
    tfe.tfe_head_topk(head, h, B, K, ids, prob, H.cur_stream())
    torch.cuda.synchronize()
    tfe.tfe_head_free(head)
    return ids.cpu().numpy(), prob.cpu().numpy()


def noalloc(w, V, D, h, B, K):
    ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
    prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
    tfe.tfe_head_topk_noalloc(w, V, D, h, B, K, ids, prob, H.cur_stream())
    torch.cuda.synchronize()
    return ids.cpu().numpy(), prob.cpu().numpy()


def inputs(seed, V, D, B):
    w = torch.empty((V, D), dtype=torch.bfloat16, device="cuda")
    synth.normal_fill_device(w.data_ptr(), 0, V, D, seed, 40, 0.1, synth.BF16, H.cur_stream())
    h = H.to_device(synth.normal_range(seed, 41, 0, B, D, 1.0, synth.BF16), synth.BF16)
    torch.cuda.synchronize()
    return w, h


def test_noalloc_matches_head_topk_on_two_calls():
    for V, D, B, K in [(151936, 1024, 64, 128), (40001, 512, 17, 33)]:
        w, h = inputs(V % 97, V, D, B)
        want_ids, want_prob = reference(w, V, D, h, B, K)
        got_ids, got_prob = noalloc(w, V, D, h, B, K)
        np.testing.assert_array_equal(got_ids, want_ids)
        np.testing.assert_allclose(got_prob, want_prob, rtol=1e-5, atol=0)
        assert np.all(got_ids >= 0) and np.all(got_ids < V)


def test_noalloc_refuses_sizes_beyond_its_scratch():
    V, D = 1000, 256
    w, h = inputs(5, V, D, 65)
    ids = torch.zeros((65, 8), dtype=torch.int32, device="cuda")
    prob = torch.zeros((65, 8), dtype=torch.float32, device="cuda")
    with pytest.raises(tfe.TfeError) as e:
        tfe.tfe_head_topk_noalloc(w, V, D, h, 65, 8, ids, prob)       # more than 64 rows
    assert "64" in str(e.value)
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_topk_noalloc(w, 1 << 19, D, h, 4, 8, ids, prob)  # vocab above 2^18
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_topk_noalloc(w, V, D, h, 4, 257, ids, prob)      # K above 256
    tfe.tfe_head_topk_noalloc(w, V, D, None, 0, 8, None, None)         # empty: nothing enqueued
