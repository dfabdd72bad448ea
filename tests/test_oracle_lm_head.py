"""Pins of the oracle's LM-head projection and row statistics (CPU only).

The oracle computes logits = h W^T over bf16 inputs in fp64 and, per row, mx = max(logits)/T and
z = sum(exp(logits/T - mx)).  These tests fix it to things outside itself: numpy's fp64 matmul of
the same bf16 values, unit vectors that select a column of W, scipy's logsumexp, and closed forms.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle


def bf16(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    t = (torch.randn(shape, generator=g, dtype=torch.float32) * scale).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16), t.double().numpy()


@pytest.mark.parametrize("rows,V,d", [(1, 7, 8), (5, 1000, 64), (3, 4099, 256)])
def test_logits_equal_fp64_matmul(rows, V, d):
    hb, h = bf16((rows, d), 1)
    wb, w = bf16((V, d), 2, 0.1)
    logits, mx, z = oracle.lm_head(hb, wb, 1.0)
    ref = h @ w.T
    np.testing.assert_allclose(logits, ref, rtol=1e-12, atol=1e-12)


def test_unit_hidden_state_selects_a_weight_column():
    d, V = 32, 50
    wb, w = bf16((V, d), 3)
    h = torch.zeros((d, d), dtype=torch.bfloat16)
    h[torch.arange(d), torch.arange(d)] = 1.0
    hb = h.view(torch.int16).numpy().view(np.uint16)
    logits, _, _ = oracle.lm_head(hb, wb, 1.0)
    np.testing.assert_array_equal(logits, w.T)   # row j of the output is column j of W


@pytest.mark.parametrize("T", [1.0, 0.7, 2.5])
def test_row_statistics_are_max_and_logsumexp(T):
    hb, h = bf16((6, 128), 4)
    wb, w = bf16((3000, 128), 5, 0.2)
    logits, mx, z = oracle.lm_head(hb, wb, T)
    t = np.float64(np.float32(T))
    np.testing.assert_array_equal(mx, (logits / t).max(axis=1))
    np.testing.assert_allclose(mx + np.log(z), logsumexp(logits / t, axis=1), rtol=1e-13)
    assert (z >= 1.0).all() and (z <= logits.shape[1]).all()


def test_temperature_scales_the_maximum():
    hb, _ = bf16((4, 64), 6)
    wb, _ = bf16((500, 64), 7)
    _, m1, _ = oracle.lm_head(hb, wb, 1.0)
    _, m2, _ = oracle.lm_head(hb, wb, 2.0)
    np.testing.assert_array_equal(m2, m1 / 2.0)


def test_zero_weights_give_uniform_statistics():
    hb, _ = bf16((3, 16), 8)
    wb = np.zeros((123, 16), np.uint16)
    logits, mx, z = oracle.lm_head(hb, wb, 1.0)
    assert (logits == 0).all() and (mx == 0).all() and (z == 123).all()


def test_statistics_only_mode_matches():
    hb, _ = bf16((4, 64), 9)
    wb, _ = bf16((700, 64), 10)
    _, m1, z1 = oracle.lm_head(hb, wb, 0.9)
    l2, m2, z2 = oracle.lm_head(hb, wb, 0.9, want_logits=False)
    assert l2 is None
    np.testing.assert_array_equal(m1, m2)
    np.testing.assert_array_equal(z1, z2)
