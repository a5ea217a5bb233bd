"""Pins of the oracle's early-exit prefetch head (Eq. 13: p = softmax(W h);
Eq. 14: the K most likely next tokens, ties by lower id) against an
independent float64 computation (numpy's matrix product and a lexicographic
sort), closed forms (one-hot projections, two tokens, equal logits) and the
softmax invariants (probabilities add up to 1, a common logit shift changes
nothing)."""
import math

import numpy as np
import pytest

import oracle
import synth


def numpy_topk(w, h, K):
    """Independent reference: float64 matmul, stable softmax, lexsort by
    (-logit, id)."""
    l = h.astype(np.float64) @ w.astype(np.float64).T
    ids = np.empty((h.shape[0], K), np.int64)
    probs = np.empty((h.shape[0], K))
    for b in range(h.shape[0]):
        order = np.lexsort((np.arange(l.shape[1]), -l[b]))[:K]
        e = np.exp(l[b] - l[b].max())
        ids[b] = order
        probs[b] = e[order] / e.sum()
    return ids, probs, l


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_head_matches_numpy_reference(dtype):
    V, D, B, K = 3001, 128, 5, 17
    w = synth.normal_range(11, 930, 0, V, D, 0.1, dtype)
    h = synth.normal_range(11, 931, 0, B, D, 1.0, dtype)
    ids, probs, logits = oracle.head_topk(w, h, K, dtype, with_logits=True)
    wf = synth.bf16_to_f32(w) if dtype == synth.BF16 else w
    hf = synth.bf16_to_f32(h) if dtype == synth.BF16 else h
    eids, eprobs, el = numpy_topk(wf, hf, K)
    np.testing.assert_array_equal(ids, eids)
    np.testing.assert_allclose(probs, eprobs, rtol=1e-12)
    np.testing.assert_allclose(logits, el, rtol=1e-12, atol=1e-12)
    assert np.all(np.diff(probs, axis=1) <= 0)


def test_one_hot_projection_closed_form():
    """Row v of W is c_v e_{v mod D}: logit_v = c_v h[v mod D]."""
    V, D = 40, 8
    c = np.arange(1, V + 1, dtype=np.float32)
    w = np.zeros((V, D), np.float32)
    w[np.arange(V), np.arange(V) % D] = c
    h = np.array([[0.5, -1.0, 0.0, 2.0, 0.25, -0.5, 1.0, 0.125]], np.float32)
    ids, probs = oracle.head_topk(w, h, 4, synth.F32)
    # logits: v = 3 + 8k -> 2 (v+1); v = 6 + 8k -> v+1; v = 0 + 8k -> (v+1)/2 ...
    # largest: v=35 (72), v=27 (56), v=38 (39), v=19 (40) -> 72, 56, 40, 39
    np.testing.assert_array_equal(ids[0], [35, 27, 19, 38])
    l = np.array([c[v] * h[0, v % D] for v in range(V)], np.float64)
    z = np.exp(l - l.max()).sum()
    np.testing.assert_allclose(probs[0], np.exp(l[[35, 27, 19, 38]] - 72.0) / z, rtol=1e-14)


def test_two_tokens_is_a_logistic_function():
    w = np.array([[1.0, 2.0], [-0.5, 0.25]], np.float32)
    h = np.array([[0.3, -0.7], [2.0, 1.0]], np.float32)
    ids, probs = oracle.head_topk(w, h, 2, synth.F32)
    for b in range(2):
        l0 = float(w[0] @ h[b].astype(np.float64))
        l1 = float(w[1] @ h[b].astype(np.float64))
        p0 = 1.0 / (1.0 + math.exp(l1 - l0))
        top = 0 if l0 >= l1 else 1
        assert ids[b, 0] == top and ids[b, 1] == 1 - top
        assert abs(probs[b, 0] - max(p0, 1 - p0)) < 1e-15
        assert abs(probs[b].sum() - 1.0) < 1e-15


def test_equal_logits_uniform_and_tie_break_by_id():
    V, D = 1000, 16
    w = np.zeros((V, D), np.float32)
    h = synth.normal_range(1, 932, 0, 3, D, 1.0, synth.F32)
    ids, probs = oracle.head_topk(w, h, 10, synth.F32)
    np.testing.assert_array_equal(ids, np.tile(np.arange(10), (3, 1)))
    np.testing.assert_allclose(probs, 1.0 / V, rtol=1e-15)


def test_full_distribution_sums_to_one_and_shift_invariance():
    V, D = 500, 32
    # Entries on a 2^-10 grid, so that shifting them by small powers of two
    # stays exact in float32.
    w = np.round(synth.normal_range(2, 933, 0, V, D, 0.3, synth.F32) * 1024) / np.float32(1024)
    h = synth.normal_range(2, 934, 0, 4, D, 1.0, synth.F32)
    ids, probs = oracle.head_topk(w, h, V, synth.F32)
    np.testing.assert_allclose(probs.sum(axis=1), 1.0, rtol=1e-13)
    assert all(sorted(r) == list(range(V)) for r in ids.tolist())
    # Adding the same vector u to every row of W adds u.h to every logit:
    # the distribution and the ranking do not change.  u is a power of two on
    # a few coordinates so that the shifted float32 rows stay exact.
    u = np.zeros(D, np.float32)
    u[:4] = [4.0, -8.0, 2.0, 16.0]
    ids2, probs2 = oracle.head_topk(w + u[None], h, 20, synth.F32)
    ok = np.all((w + u[None]) - u[None] == w)
    assert ok
    np.testing.assert_array_equal(ids2, ids[:, :20])
    np.testing.assert_allclose(probs2, probs[:, :20], rtol=1e-9)


def test_head_rejects_bad_sizes():
    w = np.zeros((4, 8), np.float32)
    h = np.zeros((1, 8), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.head_topk(w, h, 5, synth.F32)
