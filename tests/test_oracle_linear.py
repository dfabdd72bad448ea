"""Pins of the oracle's adapter linear layer and its bf16 rounding helper (CPU only).

Fixed against numpy's fp64 matmul of the same bf16 values, unit inputs that select a weight
column, the residual identity, and torch's own fp32 -> bf16 conversion (round to nearest even).
"""
import numpy as np
import pytest
import torch

import oracle


def bf16(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    t = (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16), t.double().numpy()


@pytest.mark.parametrize("rows,n_out,n_in", [(1, 8, 16), (5, 33, 64), (17, 100, 256)])
def test_linear_equals_fp64_matmul(rows, n_out, n_in):
    xb, x = bf16((rows, n_in), 1)
    wb, w = bf16((n_out, n_in), 2, 0.1)
    rb, r = bf16((rows, n_out), 3)
    np.testing.assert_allclose(oracle.linear(xb, wb), x @ w.T, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(oracle.linear(xb, wb, rb), x @ w.T + r, rtol=1e-13, atol=1e-13)


def test_unit_input_selects_a_weight_column_and_zero_weights_give_the_residual():
    wb, w = bf16((12, 32), 4)
    x = np.zeros((1, 32), np.float32)
    x[0, 7] = 1.0
    y = oracle.linear(oracle.to_bf16(x), wb)
    np.testing.assert_array_equal(y[0], w[:, 7])
    rb, r = bf16((3, 12), 5)
    xb, _ = bf16((3, 32), 6)
    y = oracle.linear(xb, np.zeros((12, 32), np.uint16), rb)
    np.testing.assert_array_equal(y, r)


def test_bf16_rounding_matches_torch():
    g = torch.Generator().manual_seed(7)
    v = torch.cat([torch.randn(100000, generator=g) * 10, torch.tensor([0.0, -0.0, 1.0, 3.0e38, -1e-40, 65504.0])])
    # ties: values exactly halfway between two bf16 numbers
    half = (torch.arange(1, 2000, dtype=torch.int32) << 16 | 0x8000).view(torch.float32)
    v = torch.cat([v, half, -half])
    ref = v.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(oracle.to_bf16(v.numpy()), ref)
    np.testing.assert_array_equal(oracle.bf16_value(ref), v.to(torch.bfloat16).double().numpy())
