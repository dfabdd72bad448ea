"""Pins of the oracle's selective speculation (CPU only).

Fixed against a worked example, brute force over every subset on tiny batches (with distinct
confidences the kept set is the one of the right size with the largest total score, and it is
prefix-closed), monotonicity in alpha, ties, and clamping.
"""
import itertools

import numpy as np
import pytest

import oracle


def batch(k):
    return np.concatenate([[0], np.cumsum(np.asarray(k) + 1)]).astype(np.int32)


def test_worked_example():
    # sequence 0: drafts with confidences 0.9, 0.5 (scores 0.9, 0.45); sequence 1: 0.4;
    # sequence 2: no draft.  alpha = 0.4 drops floor(1.2) = 1 draft: the 0.4 one.
    kept_k, kept_qsl, keep = oracle.select_drafts(batch([2, 1, 0]), np.array([0.9, 0.5, 0.4], np.float32), 0.4)
    assert kept_k.tolist() == [2, 0, 0]
    assert kept_qsl.tolist() == [0, 3, 4, 5]
    assert keep.tolist() == [1, 1, 0]


def test_alpha_zero_keeps_everything():
    rng = np.random.default_rng(1)
    k = rng.integers(0, 6, 30)
    conf = rng.random(int(k.sum()), dtype=np.float32)
    kept_k, kept_qsl, keep = oracle.select_drafts(batch(k), conf, 0.0)
    np.testing.assert_array_equal(kept_k, k)
    np.testing.assert_array_equal(kept_qsl, batch(k))
    assert keep.all()


@pytest.mark.parametrize("seed", range(20))
def test_brute_force_on_tiny_batches(seed):
    rng = np.random.default_rng(seed)
    k = rng.integers(0, 4, 4)
    N = int(k.sum())
    if N == 0:
        return
    conf = rng.uniform(0.05, 1.0, N).astype(np.float32)
    alpha = float(np.float32(rng.uniform(0, 0.99)))
    m = int(np.floor(np.float64(np.float32(alpha)) * N))
    # fp32 prefix products, as the definition states
    score = np.empty(N, np.float32)
    qsl = batch(k)
    for b in range(len(k)):
        s = np.float32(1.0)
        for i in range(k[b]):
            s = np.float32(s * conf[qsl[b] - b + i])
            score[qsl[b] - b + i] = s
    best = max(itertools.combinations(range(N), N - m), key=lambda c: (sum(float(score[i]) for i in c), [-i for i in c]))
    kept_k, kept_qsl, keep = oracle.select_drafts(qsl, conf, alpha)
    assert sorted(np.flatnonzero(keep).tolist()) == sorted(best)
    assert keep.sum() == N - m
    for b in range(len(k)):   # prefix-closed: the kept drafts of a sequence are its first kept_k
        d0 = qsl[b] - b
        assert keep[d0:d0 + kept_k[b]].all() and not keep[d0 + kept_k[b]:d0 + k[b]].any()


def test_larger_alpha_never_keeps_more():
    rng = np.random.default_rng(3)
    k = rng.integers(0, 9, 64)
    conf = rng.random(int(k.sum()), dtype=np.float32)
    prev = None
    for alpha in (0.0, 0.1, 0.15, 0.3, 0.6, 0.95):
        kept_k, _, _ = oracle.select_drafts(batch(k), conf, alpha)
        if prev is not None:
            assert (kept_k <= prev).all()
        prev = kept_k


def test_equal_scores_drop_the_highest_indices():
    k = [3, 2, 4]
    N = sum(k)
    kept_k, _, keep = oracle.select_drafts(batch(k), np.ones(N, np.float32), 0.5)   # drops floor(4.5) = 4
    assert keep.tolist() == [1] * 5 + [0] * 4
    assert kept_k.tolist() == [3, 2, 0]


def test_confidences_are_clamped():
    k = [3]
    conf = np.array([np.nan, 2.0, -1.0], np.float32)   # clamped to 0, 1, 0: scores 0, 0, 0
    kept_k, _, keep = oracle.select_drafts(batch(k), conf, 0.34)    # drops 1: the highest index
    assert keep.tolist() == [1, 1, 0] and kept_k.tolist() == [2]
