"""Pins of the oracle's softmax and speculative-sampling acceptance.

Softmax: V = 2 reduces to the logistic function; equal logits give 1/V; a constant shift
of the logits changes nothing; probabilities sum to 1; dividing by T equals scaling the
logits by 1/T.

Acceptance, against the theorem of speculative sampling (Leviathan et al. 2023; Chen et
al. 2023; the paper's [sd]) rather than against a restatement of the rule:
* brute force over the entire grid of fp32 uniforms (2^24 points): the emitted token at
  position i, given that position i is reached, is distributed as the target p_i
  (k = 0, the bonus row, and positions 0 and 1 with k = 2 at V = 8);
* the acceptance frequency of draft x equals min(1, p(x)/q(x)) on that grid (to 2^-23);
* exact inverse-CDF agreement with a rational computation for plain sampling and for the
  residual of a rejected draft, up to the fixed-point resolution of the target row's scale;
  a residual below that resolution falls back to the target row;
* invariants: an identical draft accepts every token; p(x) = 0 always rejects;
  q(x) = 0 < p(x) always accepts; NaN rejects; lowering a uniform never shortens the
  accepted prefix; status codes and the sequence-length rollback.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2609_34370_amd import workloads as wl

GRID = 1 << 24          # fp32 uniforms from Philox(...).random(dtype=float32) are k / 2^24
BATCH = 1 << 20


def grid_u(s, e):
    return (np.arange(s, e, dtype=np.float64) / GRID).astype(np.float32)


def norm(x):
    x = np.asarray(x, np.float64)
    return x / x.sum()


# ------------------------------------------------------------------ softmax

def test_softmax_two_logits_is_logistic():
    rng = np.random.default_rng(1)
    x = rng.normal(0, 3, (200, 2)).astype(np.float32)
    p = oracle.softmax(x)
    d = x[:, 0].astype(np.float64) - x[:, 1].astype(np.float64)
    np.testing.assert_allclose(p[:, 0], 1 / (1 + np.exp(-d)), rtol=0, atol=1e-7)
    np.testing.assert_allclose(p[:, 1], 1 / (1 + np.exp(d)), rtol=0, atol=1e-7)


def test_softmax_equal_logits_uniform_and_shift_invariant():
    V = 1000
    p = oracle.softmax(np.full((3, V), 2.5, np.float32))
    np.testing.assert_array_equal(p, np.float32(1.0 / V))
    rng = np.random.default_rng(2)
    # logits on a 2^-10 grid, so that adding 64 is exact in fp32
    x = (np.round(rng.normal(0, 2, (4, V)) * 1024) / 1024).astype(np.float32)
    np.testing.assert_allclose(oracle.softmax(x + np.float32(64.0)), oracle.softmax(x), rtol=0, atol=2e-9)


def test_softmax_sums_to_one_and_temperature_is_division():
    rng = np.random.default_rng(3)
    x = rng.normal(0, 4, (6, 5000)).astype(np.float32)
    p = oracle.softmax(x, temperature=0.5)
    np.testing.assert_allclose(p.astype(np.float64).sum(axis=1), 1.0, atol=1e-6)
    np.testing.assert_allclose(p, oracle.softmax(x * np.float32(2.0), 1.0), rtol=0, atol=1e-9)
    # against the textbook formula in fp64
    xd = x.astype(np.float64) / 0.5
    ref = np.exp(xd - xd.max(1, keepdims=True))
    ref /= ref.sum(1, keepdims=True)
    np.testing.assert_allclose(p, ref, rtol=1e-6, atol=1e-12)


# ------------------------------------------------------- grid sweeps (brute force)

def sweep(rows_target, rows_draft, ids, u_accept, u_sample, vary):
    """Run the oracle once per grid point of one uniform; every other input is fixed.

    rows_target [k+1, V], rows_draft [k, V], ids [k], u_accept [k], u_sample: scalar.
    ``vary`` is "sample" (u_sample runs over the 2^24 grid) or an int i (u_accept[i] does).
    Returns (token counts per output position [k+1, V], accepted-length histogram [k+1]).
    """
    k = len(ids)
    V = rows_target.shape[1]
    qsl = (np.arange(BATCH + 1) * (k + 1)).astype(np.int32)
    tg = np.tile(np.asarray(rows_target, np.float32), (BATCH, 1))
    dr = np.tile(np.asarray(rows_draft, np.float32), (BATCH, 1)) if k else np.zeros((0, V), np.float32)
    di = np.tile(np.asarray(ids, np.int32), BATCH)
    counts = np.zeros((k + 1, V), np.int64)
    acc_hist = np.zeros(k + 1, np.int64)
    for s in range(0, GRID, BATCH):
        ua = np.tile(np.asarray(u_accept, np.float32), BATCH)
        us = np.full(BATCH, u_sample, np.float32)
        if vary == "sample":
            us = grid_u(s, s + BATCH)
        else:
            ua.reshape(BATCH, k)[:, vary] = grid_u(s, s + BATCH)
        a, tok, st, _ = oracle.accept(qsl, tg, dr, di, ua, us, max_k=k)
        assert (st == 0).all()
        acc_hist += np.bincount(a, minlength=k + 1)
        for i in range(k + 1):
            t = tok[:, i]
            counts[i] += np.bincount(t[t >= 0], minlength=V)
    return counts, acc_hist


P8 = np.array([0.31, 0.02, 0.17, 0.0, 0.09, 0.26, 0.05, 0.10], np.float32)
Q8 = np.array([0.12, 0.20, 0.17, 0.08, 0.01, 0.22, 0.15, 0.05], np.float32)
LAST_U = np.float32(1 - 1 / GRID)


def test_plain_sampling_distribution_is_target():
    counts, _ = sweep(P8[None], np.zeros((0, 8)), [], [], 0.0, "sample")
    np.testing.assert_allclose(counts[0] / GRID, norm(P8), rtol=0, atol=2e-7)
    assert counts[0][3] == 0   # a zero-probability token is never chosen


def emitted_at(p_rows, q_rows, i):
    """Distribution of the token emitted at position i, given positions < i were accepted.

    The drafts at positions < i are fixed tokens with p > 0 and u = 0 (always accepted).
    For each draft token x at position i, the acceptance frequency A(x) is measured over
    the uniform grid; after a forced rejection (the largest grid uniform on a token with
    p < q) the resampled distribution R is measured over the grid.  With x ~ q_i the
    emitted token has law sum_x q_i(x) [A(x) 1{m = x} + (1 - A(x)) R(m)].
    """
    k = len(q_rows)
    V = p_rows.shape[1]
    prefix = [int(np.argmax(p_rows[j])) for j in range(i)]
    A = np.zeros(V)
    for x in range(V):
        ids = prefix + [x] + [0] * (k - i - 1)
        _, hist = sweep(p_rows, q_rows, ids, [0.0] * k, 0.5, vary=i)
        assert hist[:i].sum() == 0
        A[x] = hist[i + 1:].sum() / GRID
        expect = 1.0 if q_rows[i][x] == 0 else min(1.0, float(p_rows[i][x]) / float(q_rows[i][x]))
        assert abs(A[x] - expect) <= 2.0 / GRID, (i, x, A[x], expect)
    xr = int(np.argmax(q_rows[i].astype(np.float64) - p_rows[i]))
    assert q_rows[i][xr] > p_rows[i][xr]
    ids = prefix + [xr] + [0] * (k - i - 1)
    ua = [0.0] * i + [LAST_U] + [0.0] * (k - i - 1)
    counts, hist = sweep(p_rows, q_rows, ids, ua, 0.0, "sample")
    assert hist[i] == GRID
    R = counts[i] / GRID
    resid = np.maximum(p_rows[i].astype(np.float64) - q_rows[i], 0)
    np.testing.assert_allclose(R, resid / resid.sum(), rtol=0, atol=2e-7)
    qn = norm(q_rows[i])
    return qn * A + (qn * (1 - A)).sum() * R


def test_speculative_sampling_preserves_target_distribution_position0():
    emitted = emitted_at(np.stack([P8, P8]), Q8[None], 0)
    np.testing.assert_allclose(emitted, norm(P8), rtol=0, atol=1e-6)


def three_rows():
    rng = np.random.default_rng(4)
    p = np.stack([P8, norm(rng.random(8) ** 2).astype(np.float32), norm(rng.random(8)).astype(np.float32)])
    q = np.stack([Q8, norm(rng.random(8)).astype(np.float32)])
    return p, q


def test_speculative_sampling_preserves_target_distribution_position1():
    p, q = three_rows()
    emitted = emitted_at(p, q, 1)
    np.testing.assert_allclose(emitted, norm(p[1]), rtol=0, atol=1e-6)


def test_bonus_token_comes_from_last_target_row():
    p, q = three_rows()
    x0, x1 = int(np.argmax(p[0])), int(np.argmax(p[1]))
    counts, hist = sweep(p, q, [x0, x1], [0.0, 0.0], 0.0, "sample")
    assert hist[2] == GRID
    assert counts[0][x0] == GRID and counts[1][x1] == GRID
    np.testing.assert_allclose(counts[2] / GRID, norm(p[2]), rtol=0, atol=2e-7)


# ----------------------------------------------------------- exact sampling

def exact_inverse_cdf(w, u):
    """Smallest m with sum_{v<=m} w_v > u * sum w, in rational arithmetic."""
    fw = [Fraction(float(x)) for x in w]
    tot = sum(fw)
    thr = Fraction(float(u)) * tot
    acc = Fraction(0)
    for m, x in enumerate(fw):
        acc += x
        if acc > thr:
            return m, min(abs(acc - thr), abs(acc - x - thr)) / tot
    return len(w) - 1, Fraction(0)


def test_plain_sampling_matches_rational_inverse_cdf():
    rng = np.random.default_rng(5)
    V = 64
    nseq = 300
    w = rng.random((nseq, V)).astype(np.float32) ** 3
    w[rng.random((nseq, V)) < 0.2] = 0
    u = rng.random(nseq, dtype=np.float32)
    qsl = np.arange(nseq + 1, dtype=np.int32)
    _, tok, st, _ = oracle.accept(qsl, w, np.zeros((0, V), np.float32), [], [], u, max_k=0)
    assert (st == 0).all()
    for b in range(nseq):
        m, margin = exact_inverse_cdf(w[b], u[b])
        # the fixed-point weights move a boundary by at most V * 2^-40 of the max weight
        if margin > V * 2.0 ** -39:
            assert tok[b, 0] == m, b
        assert w[b, tok[b, 0]] > 0


def test_extreme_uniforms_pick_first_and_last_positive_token():
    V = 1000
    w = np.zeros((2, V), np.float32)
    w[:, 7] = 1e-30
    w[:, 500] = 0.5
    w[:, 993] = 0.25
    qsl = np.arange(3, dtype=np.int32)
    _, tok, _, _ = oracle.accept(qsl, w, np.zeros((0, V), np.float32), [], [],
                                 np.array([0.0, 1 - 2.0 ** -24], np.float32), max_k=0)
    # 1e-30 is far below 2^-40 of the max weight: its fixed-point weight is 0, never sampled
    assert tok[0, 0] == 500 and tok[1, 0] == 993


def test_residual_sampling_matches_rational_inverse_cdf():
    # a rejected draft: the token is the rational inverse CDF of w = max(0, fp32(p - q)), except
    # within the fixed-point resolution: each weight is truncated to a multiple of 2^(e - 40),
    # e the exponent of the target row's largest probability
    rng = np.random.default_rng(11)
    V, nseq = 64, 200
    p = rng.random((2 * nseq, V)).astype(np.float32) ** 2
    q = rng.random((nseq, V)).astype(np.float32) ** 2
    ids = np.argmax(q - p[0::2], axis=1).astype(np.int32)   # q > p there: rejected at u near 1
    qsl = np.arange(0, 2 * nseq + 1, 2, dtype=np.int32)
    ua = np.full(nseq, 1 - 2.0 ** -24, np.float32)
    us = rng.random(nseq, dtype=np.float32)
    a, tok, st, _ = oracle.accept(qsl, p, q, ids, ua, us)
    assert (a == 0).all() and (st == 0).all()
    checked = 0
    for b in range(nseq):
        w = np.maximum(p[2 * b] - q[b], np.float32(0))
        e = np.frexp(np.float64(p[2 * b].max()))[1] - 1
        m, margin = exact_inverse_cdf(w, us[b])
        if margin > 4 * V * 2.0 ** (e - 40) / w.astype(np.float64).sum():
            assert tok[b, 0] == m, b
            checked += 1
        assert w[tok[b, 0]] > 0
    assert checked > nseq * 0.9


def test_sampling_scale_is_the_target_rows_largest_probability():
    # a positive residual below 2^-40 of max p has fixed-point weight 0: the sample falls back
    # to p (a scale taken from the residual itself would give token 3)
    V = 4
    p = np.array([[0.5, 0.25 - 2.0 ** -26, 0.25, 2.0 ** -45], [0.25] * V], np.float32)
    q = np.array([[0.5, 0.25, 0.25, 0.0]], np.float32)
    a, tok, st, _ = oracle.accept([0, 2], p, q, [1], [1 - 2.0 ** -24], [0.999])
    assert a[0] == 0 and st[0] == oracle.OK and tok[0, 0] == 2
    # a residual weight of 2^-40 = 2 units at that scale is sampled
    p[0, 3] = 2.0 ** -40
    a, tok, st, _ = oracle.accept([0, 2], p, q, [1], [1 - 2.0 ** -24], [0.999])
    assert a[0] == 0 and st[0] == oracle.OK and tok[0, 0] == 3


# --------------------------------------------------------------- invariants

def small_batch(wid=1, seed=None):
    spec = wl.WORKLOADS[wid]
    batch = wl.make_batch(spec, seed=seed)
    acc = wl.make_accept_inputs(spec, batch, device="cpu", seed=seed)
    return spec, batch, acc


def test_identical_draft_accepts_every_token():
    spec, batch, inp = small_batch()
    p = oracle.softmax(inp.target_logits.numpy(), inp.temperature)
    rows = wl.draft_row_index(batch)
    q = p[rows]                       # the draft distribution equals the target's
    # draft tokens drawn from q itself, so q(x) > 0
    rng = np.random.default_rng(0)
    ids = np.array([rng.choice(q.shape[1], p=norm(r)) for r in q], np.int32)
    a, tok, st, _ = oracle.accept(batch.qsl, p, q, ids, inp.u_accept.numpy(), inp.u_sample.numpy())
    np.testing.assert_array_equal(a, batch.k)
    assert (st == 0).all()


def test_zero_target_probability_always_rejects_and_zero_draft_always_accepts():
    V = 16
    p = np.full((2, V), 1.0 / V, np.float32)
    q = np.full((1, V), 1.0 / V, np.float32)
    p[0, 3] = 0.0
    for u in (0.0, 0.3, 0.999):
        a, tok, st, _ = oracle.accept([0, 2], p, q, [3], [u], [0.5])
        assert a[0] == 0 and tok[0, 0] != 3 and st[0] == 0
    q2 = q.copy()
    q2[0, 5] = 0.0
    for u in (0.0, 0.5, 0.99999994):
        a, tok, st, _ = oracle.accept([0, 2], np.full((2, V), 1.0 / V, np.float32), q2, [5], [u], [0.5])
        assert a[0] == 1 and tok[0, 0] == 5


def test_nan_in_test_rejects():
    V = 8
    p = np.full((2, V), 1.0 / V, np.float32)
    q = np.full((1, V), 1.0 / V, np.float32)
    q[0, 2] = np.nan
    a, tok, st, _ = oracle.accept([0, 2], p, q, [2], [0.0], [0.5])
    assert a[0] == 0
    assert st[0] == oracle.BAD_ROW   # the residual row then holds a NaN


def test_lowering_uniforms_never_shortens_prefix():
    spec, batch, inp = small_batch()
    p = oracle.softmax(inp.target_logits.numpy(), inp.temperature)
    q = oracle.softmax(inp.draft_logits.numpy(), inp.temperature)
    ids, ua, us = inp.draft_ids.numpy(), inp.u_accept.numpy(), inp.u_sample.numpy()
    a0, _, _, _ = oracle.accept(batch.qsl, p, q, ids, ua, us)
    rng = np.random.default_rng(6)
    for _ in range(5):
        a1, _, _, _ = oracle.accept(batch.qsl, p, q, ids, ua * rng.random(ua.shape).astype(np.float32), us)
        assert (a1 >= a0).all()


def test_status_codes_and_rollback():
    V = 8
    qsl = np.array([0, 3, 6, 9, 10], np.int32)     # k = 2, 2, 2, 0
    p = np.full((10, V), 1.0 / V, np.float32)
    q = np.full((6, V), 1.0 / V, np.float32)
    ids = np.array([1, 2, 1, 9, 0, 0], np.int32)    # seq 1 has an id outside [0, V)
    p[6, 0] = 0.0                                   # seq 2 rejects position 0 ...
    q[4:6] = 0.0
    q[4, 0] = 1.0                                   # ... with residual max(0, p - q)
    p[9] = 0.0                                      # seq 3 (k = 0): an all-zero row
    seq_lens = np.array([20, 30, 40, 50], np.int32)
    a, tok, st, sl = oracle.accept(qsl, p, q, ids, np.full(6, 0.5, np.float32), np.full(4, 0.5, np.float32),
                                   seq_lens=seq_lens)
    assert list(st) == [oracle.OK, oracle.BAD_TOKEN, oracle.OK, oracle.EMPTY_ROW]
    assert list(a) == [2, 0, 0, 0]
    assert list(tok[0, :2]) == [1, 2] and tok[0, 2] >= 0
    assert (tok[1] == -1).all()
    assert tok[2, 0] >= 1 and (tok[2, 1:] == -1).all()
    assert (tok[3] == -1).all()
    assert list(sl) == [20, 30, 40 - 2 + 0, 50]

    # negative value in a sampled row
    p2 = np.full((1, V), 1.0 / V, np.float32)
    p2[0, 4] = -1e-3
    _, tok2, st2, _ = oracle.accept([0, 1], p2, np.zeros((0, V), np.float32), [], [], [0.5])
    assert st2[0] == oracle.BAD_ROW and tok2[0, 0] == -1


def test_residual_all_zero_falls_back_to_target_row():
    V = 8
    p = np.tile(P8, (2, 1))
    q = P8[None].copy()
    # x = 3 has p = q = 0: rejected; the residual max(0, p - q) is then 0 everywhere
    counts, hist = sweep(p, q, [3], [0.25], 0.0, "sample")
    assert hist[0] == GRID
    np.testing.assert_allclose(counts[0] / GRID, norm(P8), rtol=0, atol=2e-7)
