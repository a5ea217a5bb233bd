"""GPU parity of the early-exit prefetch head (Eq. 13, Eq. 14):
tfe_head_topk through the C ABI against the oracle.

With small-integer projections and hidden states every logit is an integer
below 2^24, so the float32 logits of the GPU are exact: token ids must then
match bit for bit (ties go to the lower id on both sides) and probabilities
within 1e-5 relative (float32 softmax with about 1-ulp exponentials).  With Gaussian inputs the float32 logits carry
rounding error: the GPU's candidates must be a valid top K of the exact
logits within the float32 accumulation bound eps = D 2^-24 max_v sum_d
|w_vd h_d|, identical to the oracle's wherever the oracle's K-th and
(K+1)-th logits are more than 2 eps apart, and each probability within
2 eps + 1e-5 relative of the exact one."""
import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2607_07388_amd import tfe

from . import harness as H

pytestmark = pytest.mark.gpu

TAG_W, TAG_H = 40, 41


def int_inputs(seed, V, D, B):
    rng = np.random.default_rng(seed)
    w = rng.integers(-2, 3, (V, D)).astype(np.float32)
    h = rng.integers(-3, 4, (B, D)).astype(np.float32)
    return bf16_bits(w), bf16_bits(h)


def bf16_bits(x):
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


class Head:
    def __init__(self, w_bits, max_batch, max_k):
        self.V, self.D = w_bits.shape
        self.w = H.to_device(w_bits, synth.BF16)
        self.h = tfe.tfe_head_create(self.w, self.V, self.D, max_batch, max_k)

    def topk(self, h_bits, K):
        B = h_bits.shape[0]
        hd = H.to_device(h_bits, synth.BF16)
        ids = torch.full((B, K), -7, dtype=torch.int32, device="cuda")
        prob = torch.full((B, K), -1.0, dtype=torch.float32, device="cuda")
        tfe.tfe_head_topk(self.h, hd, B, K, ids, prob, H.cur_stream())
        torch.cuda.synchronize()
        return ids.cpu().numpy(), prob.cpu().numpy()

    def close(self):
        if self.h:
            tfe.tfe_head_free(self.h)
            self.h = None


@pytest.mark.parametrize("V,D,B,K", [
    (3001, 256, 5, 17),        # ragged vocabulary (not a multiple of 16 or 4)
    (300, 512, 17, 256),       # one chunk, K close to V
    (200, 256, 3, 200),        # K = V: every token, in order
    (40000, 1024, 100, 64),    # two column groups (64 + 36 rows), ten chunks
    (151936, 1024, 64, 128),   # the backbone vocabulary, one batch-64 decode step
    (1 << 18, 256, 3, 256),    # the largest vocabulary (16384 tiles) and the largest K
])
def test_integer_logits_bit_exact_ids(V, D, B, K):
    w, h = int_inputs(V + D + B, V, D, B)
    head = Head(w, B, K)
    ids, prob = head.topk(h, K)
    rows = np.arange(B) if V * D * B <= 4e8 else np.array([0, 1, B // 2, B - 1])
    eids, eprob = oracle.head_topk(w, h[rows], K, synth.BF16)
    np.testing.assert_array_equal(ids[rows], eids)
    # Probabilities below ~1e-36 sit in float32's subnormal range.
    np.testing.assert_allclose(prob[rows], eprob, rtol=1e-5, atol=1e-36)
    head.close()


def test_integer_logits_with_many_ties():
    """Entries in {0, 1}: logits take few distinct values, so the K-th place
    falls inside a large group of equal logits resolved by token id."""
    V, D, B, K = 20000, 256, 8, 100
    rng = np.random.default_rng(7)
    w = bf16_bits(rng.integers(0, 2, (V, D)).astype(np.float32) * (rng.random((V, D)) < 0.05))
    h = bf16_bits(np.ones((B, D), np.float32))
    head = Head(w, B, K)
    ids, prob = head.topk(h, K)
    eids, eprob = oracle.head_topk(w, h, K, synth.BF16)
    np.testing.assert_array_equal(ids, eids)
    np.testing.assert_allclose(prob, eprob, rtol=1e-5, atol=1e-36)
    _, _, logits = oracle.head_topk(w, h[:1], 1, synth.BF16, with_logits=True)
    kth = np.sort(logits[0])[::-1][K - 1]
    assert (logits[0] == kth).sum() > 50
    head.close()


@pytest.mark.parametrize("V,D,B,K,sigma", [
    (151936, 1024, 64, 64, 0.1),
    (50000, 512, 20, 16, 0.05),
    (4097, 256, 3, 256, 0.3),
])
def test_gaussian_logits_valid_topk(V, D, B, K, sigma):
    seed = V % 1000
    w = synth.normal_range(seed, TAG_W, 0, V, D, sigma, synth.BF16)
    h = synth.normal_range(seed, TAG_H, 0, B, D, 1.0, synth.BF16)
    head = Head(w, B, K)
    ids, prob = head.topk(h, K)
    rows = np.arange(B) if V * B <= 2e6 else np.array([0, 7, 31, B - 1])
    eids, eprob, logits = oracle.head_topk(w, h[rows], K, synth.BF16, with_logits=True)
    wf = synth.bf16_to_f32(w).astype(np.float64)
    hf = synth.bf16_to_f32(h[rows]).astype(np.float64)
    eps = D * 2.0 ** -24 * (np.abs(hf) @ np.abs(wf).T).max(axis=1)
    for n, b in enumerate(rows):
        l = logits[n]
        got = ids[b].astype(np.int64)
        assert len(set(got.tolist())) == K and got.min() >= 0 and got.max() < V
        srt = np.sort(l)[::-1]
        kth, nxt = srt[K - 1], (srt[K] if K < V else -np.inf)
        # Valid top K within eps: chosen logits reach the K-th, the rest do not exceed it.
        assert l[got].min() >= kth - 2 * eps[n]
        rest = np.setdiff1d(np.arange(V), got)
        if rest.size:
            assert l[rest].max() <= kth + 2 * eps[n]
        if kth - nxt > 4 * eps[n]:
            assert set(got.tolist()) == set(eids[n].tolist())
        # Probabilities of the chosen tokens against the exact softmax.
        m = l.max()
        z = np.exp(l - m).sum()
        want = np.exp(l[got] - m) / z
        np.testing.assert_allclose(prob[b], want, rtol=2 * eps[n] + 1e-5, atol=1e-36)
        assert np.all(np.diff(prob[b]) <= 1e-6 * prob[b][:-1])
    head.close()


def test_head_feeds_scored_prefetch_arguments():
    """Candidate ids and probabilities come out in the layout tfe_prefetch_scored
    takes ([B x K] int32 and float32) and each row's probabilities are a
    sub-distribution."""
    V, D, B, K = 151936, 1024, 64, 8
    w = synth.normal_range(3, TAG_W, 0, V, D, 0.1, synth.BF16)
    h = synth.normal_range(3, TAG_H, 0, B, D, 1.0, synth.BF16)
    head = Head(w, B, K)
    ids, prob = head.topk(h, K)
    assert ids.dtype == np.int32 and prob.dtype == np.float32 and ids.shape == (B, K)
    assert np.all(prob > 0) and np.all(prob.sum(axis=1) <= 1.0 + 1e-5)
    head.close()


def test_head_errors():
    w = torch.zeros((1000, 512), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tfe.TfeError) as e:
        tfe.tfe_head_create(w, 1000, 384, 4, 8)
    assert e.value.status == -5
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_create(w, 1000, 512, 4, 300)          # max_k above 256
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_create(w.data_ptr() + 2, 1000, 512, 4, 8)   # misaligned
    wh = np.zeros((1000, 512), np.uint16)
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_create(wh, 1000, 512, 4, 8)           # host memory
    h = tfe.tfe_head_create(w, 1000, 512, 4, 8)
    hid = torch.zeros((5, 512), dtype=torch.bfloat16, device="cuda")
    ids = torch.zeros((5, 8), dtype=torch.int32, device="cuda")
    prob = torch.zeros((5, 8), dtype=torch.float32, device="cuda")
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_topk(h, hid, 5, 8, ids, prob)          # B above max_batch
    with pytest.raises(tfe.TfeError):
        tfe.tfe_head_topk(h, hid, 4, 9, ids, prob)          # K above max_k
    tfe.tfe_head_topk(h, None, 0, 8, None, None)            # empty: nothing enqueued
    tfe.tfe_head_topk(h, hid, 4, 8, ids, prob)
    torch.cuda.synchronize()
    # All-zero logits: uniform distribution, lowest ids first.
    assert ids[:4].cpu().numpy().tolist() == [list(range(8))] * 4
    np.testing.assert_allclose(prob[:4].cpu().numpy(), 1e-3, rtol=1e-5)
    tfe.tfe_head_free(h)
