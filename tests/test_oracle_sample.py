"""Pins of the oracle's plain sampling (acceptance with no drafts), CPU only.

Over a uniform grid of 2^16 fp32 uniforms the emitted tokens must follow p to within one grid
step per token, the returned probability must be p[token], and degenerate rows behave as the
acceptance rule defines (a one-hot row always gives its token; a row with a NaN is refused).
"""
import numpy as np

import oracle


def test_grid_frequencies_follow_p():
    rng = np.random.default_rng(1)
    for V in (2, 8, 37):
        p = rng.dirichlet(np.ones(V)).astype(np.float32)
        n = 1 << 16
        u = (np.arange(n) / n).astype(np.float32)
        tok, prob, status = oracle.sample(np.tile(p, (n, 1)), u)
        assert (status == oracle.OK).all()
        freq = np.bincount(tok, minlength=V) / n
        w = p.astype(np.float64) / p.astype(np.float64).sum()
        assert np.abs(freq - w).max() <= 2.0 / n + 1e-9
        np.testing.assert_array_equal(prob, p[tok])
        # the inverse CDF is monotone in u
        assert (np.diff(tok) >= 0).all()


def test_one_hot_and_bad_rows():
    V = 10
    rows = np.zeros((3, V), np.float32)
    rows[0, 7] = 1.0
    rows[1] = 0.1
    rows[1, 3] = np.nan
    rows[2, :] = 0.0
    tok, prob, status = oracle.sample(rows, np.array([0.99, 0.5, 0.5], np.float32))
    assert tok[0] == 7 and prob[0] == 1.0 and status[0] == oracle.OK
    assert tok[1] == -1 and status[1] == oracle.BAD_ROW and prob[1] == 0
    assert tok[2] == -1 and status[2] == oracle.EMPTY_ROW
