"""The closed forms of the selective-speculation model (Sec. 5, Eq. 3 and 4) in the package,
pinned to the oracle's iteration of the recurrence, to the quantity the recurrence conserves
(B_t + alpha * the sum of the N-1 previous terms), and to the cases alpha = 0 and theta = 0, 1."""
import numpy as np
import pytest

import oracle
from paper_2609_34370_amd import schedule


@pytest.mark.parametrize("alpha", [0.0, 0.15, 0.3, 0.6])
@pytest.mark.parametrize("N", [1, 2, 4, 8])
def test_steady_batch_is_the_limit_of_the_recurrence(alpha, N):
    B = 256.0
    assert oracle.batch_recurrence(B, alpha, N) == pytest.approx(schedule.steady_batch(B, alpha, N), rel=1e-9)


def test_recurrence_conserves_its_invariant():
    B, alpha, N = 100.0, 0.3, 5
    hist = [0.0] * (N - 1) + [B]
    for _ in range(50):
        inv = hist[-1] + alpha * sum(hist[-N:-1])
        hist.append(alpha * hist[-N] + (1 - alpha) * hist[-1])
        assert hist[-1] + alpha * sum(hist[-N:-1]) == pytest.approx(inv, rel=1e-12)
    assert inv == pytest.approx(B)   # so the steady state is B / (1 + alpha (N - 1))


def test_effective_batch_special_cases():
    B, N = 128.0, 4
    for alpha in (0.0, 0.2):
        bs = schedule.steady_batch(B, alpha, N)
        assert schedule.effective_batch(B, alpha, N, 1.0) == pytest.approx(bs)   # every draft accepted
        assert schedule.effective_batch(B, alpha, N, 0.0) == pytest.approx(alpha * bs + (1 - alpha) * bs / N)
    assert schedule.steady_batch(B, 0.0, N) == B
    with pytest.raises(ValueError):
        schedule.steady_batch(B, 1.0, N)
