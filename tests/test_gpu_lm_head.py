"""GPU parity of the LM-head projection with fused statistics, and of acceptance from them.

The oracle computes logits = h W^T in fp64 from the same bf16 bits and each row's max and
sum of exp at the temperature.  Bars:
  * logits: |gpu - oracle| <= 2 K 2^-24 sum_j |h_j W_vj| + 1e-6 per element: the worst case
    of an fp32 sum of K exact products, with room for the order of summation;
  * statistics: the row maximum (base e) within that bound / T, the sum of exponentials
    within 1e-4 relative (the statistics are combined per row on the host, in fp64);
  * acceptance from the fused statistics: the same decisions as the oracle's exact rule on its
    own fp64 logits, except within 1e-4 of a decision boundary (at most 1% of sequences).
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_34370_amd import spexis as sx

pytestmark = pytest.mark.gpu
LN2 = math.log(2.0)


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def bf16_pair(shape, seed, scale):
    g = torch.Generator().manual_seed(seed)
    t = (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)
    return t, t.view(torch.int16).numpy().view(np.uint16)


def run_lm_head(h, w, T, want_logits=True):
    rows, V = h.shape[0], w.shape[0]
    tiles = sx.spexis_lm_head_tiles(V)
    stats = torch.empty((rows, tiles, 2), dtype=torch.float32, device="cuda")
    logits = torch.empty((rows, V), dtype=torch.float32, device="cuda") if want_logits else None
    sx.spexis_lm_head(h.cuda(), sx.spexis_pack_weight(w.cuda()), stats, logits=logits, temperature=T, vocab=V)
    torch.cuda.synchronize()
    return (logits.cpu().numpy() if want_logits else None), stats.cpu().numpy()


def combine(stats):
    """Row (max, sum) in base e from the per-tile base-2 statistics, in fp64."""
    m = stats[..., 0].astype(np.float64)
    z = stats[..., 1].astype(np.float64)
    M = m.max(axis=1)
    Z = (z * np.exp2(m - M[:, None])).sum(axis=1)
    return M * LN2, Z


def check(h, hb, w, wb, T, rows_idx=None):
    logits, stats = run_lm_head(h, w, T)
    sel = np.arange(h.shape[0]) if rows_idx is None else np.asarray(rows_idx)
    ref, mx, z = oracle.lm_head(hb[sel], wb, T)
    hh = np.abs(h.double().numpy()[sel])
    ww = np.abs(w.double().numpy())
    bound = 2 * h.shape[1] * 2.0 ** -24 * (hh @ ww.T) + 1e-6
    err = np.abs(logits[sel].astype(np.float64) - ref)
    say(f"  max err {err.max():.3e}  max err/bound {(err / bound).max():.3f}")
    assert (err <= bound).all()
    M, Z = combine(stats[sel])
    t = float(np.float32(T))
    np.testing.assert_array_less(np.abs(M - mx), bound.max(axis=1) / t + 1e-6)
    np.testing.assert_allclose(Z, z, rtol=1e-4)
    return logits, stats


# (320, 2048), (200, 70001), (961, 4099), (1500, 9000) and (1100, 70001) run the eight-wave
# kernel: one group, a vocabulary whose last packed tile is part zeros, a last group of one row,
# a last group of 220 rows with a 40-column last tile, a last group of 140 rows with a
# part-zero last packed tile; (333, 3000) and (700, 130) the four-wave groups of 160 or 192 rows
@pytest.mark.parametrize("rows,V,d", [(1, 1000, 256), (37, 4101, 512), (320, 2048, 256), (333, 3000, 256),
                                      (700, 130, 512), (1500, 9000, 256), (200, 70001, 256), (961, 4099, 512),
                                      (1100, 70001, 512)])
def test_lm_head_small_shapes(rows, V, d):
    h, hb = bf16_pair((rows, d), 1, 1.0)
    w, wb = bf16_pair((V, d), 2, 0.05)
    say(f"[lm head] rows={rows} V={V} d={d}")
    check(h, hb, w, wb, 0.8)


@pytest.mark.parametrize("rows", [1, 40, 64, 100])
def test_lm_head_few_rows_wide_vocabulary(rows):
    # up to 128 rows, a vocabulary of at least 256 x 256 columns takes the 256-column
    # workgroups (two column tiles per wave); 70001 leaves a ragged last tile
    V, d = 70001, 256
    h, hb = bf16_pair((rows, d), 11, 1.0)
    w, wb = bf16_pair((V, d), 12, 0.05)
    say(f"[lm head] rows={rows} V={V} d={d}")
    check(h, hb, w, wb, 0.9)


def test_lm_head_four_row_tiles_narrow_vocabulary():
    rows, V, d = 100, 5000, 256
    h, hb = bf16_pair((rows, d), 13, 1.0)
    w, wb = bf16_pair((V, d), 14, 0.05)
    say(f"[lm head] rows={rows} V={V} d={d}")
    check(h, hb, w, wb, 1.1)


def test_lm_head_statistics_only_and_extreme_logits():
    rows, V, d = 64, 5000, 256
    h, hb = bf16_pair((rows, d), 3, 4.0)        # large logits: the maximum dominates each tile
    w, wb = bf16_pair((V, d), 4, 1.0)
    logits, stats = check(h, hb, w, wb, 0.5)
    _, stats2 = run_lm_head(h, w, 0.5, want_logits=False)
    np.testing.assert_array_equal(stats, stats2)


def test_lm_head_llama3_8b_shape_sampled_rows():
    # the shape of the verifying stage's LM head at the llama3-8b-layer workload: 320 query
    # tokens, hidden 4096, vocabulary 128256; the oracle checks 4 rows over the whole vocabulary
    rows, V, d = 320, 128256, 4096
    h, hb = bf16_pair((rows, d), 5, 1.0)
    w, wb = bf16_pair((V, d), 6, 0.02)
    say(f"[lm head] rows={rows} V={V} d={d} (rows 0, 31, 200, 319 checked)")
    check(h, hb, w, wb, 1.0, rows_idx=[0, 31, 200, 319])


def test_lm_head_large_row_count_sampled_rows():
    # many row groups: the acceptance-stress workload's shape (4608 query tokens, hidden 3584,
    # vocabulary 152064); rows on both sides of group boundaries checked over the whole vocabulary
    rows, V, d = 4608, 152064, 3584
    h, hb = bf16_pair((rows, d), 7, 1.0)
    w, wb = bf16_pair((V, d), 8, 0.02)
    sel = [0, 159, 160, 191, 192, 255, 256, 319, 320, 2301, 4351, 4352, 4479, 4480, 4607]
    say(f"[lm head] rows={rows} V={V} d={d} (rows {sel} checked)")
    check(h, hb, w, wb, 0.7, rows_idx=sel)


def test_accept_with_fused_statistics_agrees_with_oracle():
    # 24 sequences with 0..5 drafts; target rows from one hidden batch, draft rows from another
    # (a synthetic draft model sharing the LM head); both go through spexis_lm_head
    rng = np.random.default_rng(12)
    B, K, V, d, T = 24, 5, 20000, 512, 0.9
    k = rng.integers(0, K + 1, B)
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    Tt, Td = int(qsl[-1]), int(qsl[-1]) - B
    w, wb = bf16_pair((V, d), 7, 0.08)
    ht, htb = bf16_pair((Tt, d), 8, 1.0)
    g = torch.Generator().manual_seed(9)
    hd_f = ht.float()[np.concatenate([np.arange(qsl[b], qsl[b] + k[b]) for b in range(B)]).astype(np.int64)]
    hd = (hd_f + 0.4 * torch.randn(hd_f.shape, generator=g)).to(torch.bfloat16)
    hdb = hd.view(torch.int16).numpy().view(np.uint16)
    # oracle side: fp64 logits of both, rounded to fp32, probabilities by the oracle's softmax
    lt, _, _ = oracle.lm_head(htb, wb, T)
    ld, _, _ = oracle.lm_head(hdb, wb, T)
    p = oracle.softmax(lt.astype(np.float32), T)
    q = oracle.softmax(ld.astype(np.float32), T)
    ids = np.array([rng.choice(V, p=r / r.sum(dtype=np.float64)) for r in q.astype(np.float64)], np.int32)
    ua = rng.random(Td, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    # GPU side: logits and statistics from spexis_lm_head, then acceptance from them
    tiles = sx.spexis_lm_head_tiles(V)
    tl = torch.empty((Tt, V), dtype=torch.float32, device="cuda")
    dl = torch.empty((Td, V), dtype=torch.float32, device="cuda")
    ts = torch.empty((Tt, tiles, 2), dtype=torch.float32, device="cuda")
    ds = torch.empty((Td, tiles, 2), dtype=torch.float32, device="cuda")
    wp = sx.spexis_pack_weight(w.cuda())
    sx.spexis_lm_head(ht.cuda(), wp, ts, logits=tl, temperature=T)
    sx.spexis_lm_head(hd.cuda(), wp, ds, logits=dl, temperature=T)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    acc = torch.empty(B, dtype=torch.int32, device="cuda")
    tok = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    st = torch.empty(B, dtype=torch.int32, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    sx.spexis_accept_with_stats(dev(qsl), tl, dl, ts, ds, dev(ids), dev(ua), dev(us), K, acc, tok, st, ws,
                                temperature=T)
    torch.cuda.synchronize()
    a, t, s = acc.cpu().numpy(), tok.cpu().numpy(), st.cpu().numpy()
    # the same logits through spexis_accept (its own statistics) must decide identically
    acc2, tok2, st2 = torch.empty_like(acc), torch.empty_like(tok), torch.empty_like(st)
    sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, dev(qsl), tl, dl, dev(ids), dev(ua), dev(us), K, acc2, tok2, st2, ws,
                     temperature=T)
    torch.cuda.synchronize()
    say(f"[accept with stats] accepted={a.tolist()}")
    assert (s == 0).all() and (rs == 0).all()
    diff = [b for b in range(B) if a[b] != ra[b] or not np.array_equal(t[b], rt[b])]
    assert len(diff) <= 1, diff
    for b in diff:   # within fp32 rounding of a decision boundary
        t0, d0 = qsl[b], qsl[b] - b
        if a[b] != ra[b]:
            i = min(a[b], ra[b])
            x = ids[d0 + i]
            assert abs(float(ua[d0 + i]) * float(q[d0 + i, x]) - float(p[t0 + i, x])) <= 1e-4
    diff2 = [b for b in range(B) if a[b] != acc2.cpu().numpy()[b]]
    assert len(diff2) <= 1


def test_accept_with_fused_statistics_flags_bad_draft_ids():
    # a draft id past the vocabulary or negative marks its sequence (status 3, nothing accepted,
    # tokens -1) on both acceptance paths; the other sequences decide as they would without it
    rng = np.random.default_rng(31)
    B, K, V, d, T = 6, 3, 3000, 256, 1.0
    k = np.array([3, 0, 2, 3, 1, 3])
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    Tt, Td = int(qsl[-1]), int(qsl[-1]) - B
    w, _ = bf16_pair((V, d), 15, 0.08)
    ht, _ = bf16_pair((Tt, d), 16, 1.0)
    hd, _ = bf16_pair((Td, d), 17, 1.0)
    tiles = sx.spexis_lm_head_tiles(V)
    tl = torch.empty((Tt, V), dtype=torch.float32, device="cuda")
    dl = torch.empty((Td, V), dtype=torch.float32, device="cuda")
    ts = torch.empty((Tt, tiles, 2), dtype=torch.float32, device="cuda")
    ds = torch.empty((Td, tiles, 2), dtype=torch.float32, device="cuda")
    wp = sx.spexis_pack_weight(w.cuda())
    sx.spexis_lm_head(ht.cuda(), wp, ts, logits=tl, temperature=T)
    sx.spexis_lm_head(hd.cuda(), wp, ds, logits=dl, temperature=T)
    ids = rng.integers(0, V, Td).astype(np.int32)
    ua = rng.random(Td, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")

    def both(ids_h):
        out = []
        for fused in (True, False):
            acc = torch.empty(B, dtype=torch.int32, device="cuda")
            tok = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
            st = torch.empty(B, dtype=torch.int32, device="cuda")
            if fused:
                sx.spexis_accept_with_stats(dev(qsl), tl, dl, ts, ds, dev(ids_h), dev(ua), dev(us), K, acc, tok, st,
                                            ws, temperature=T)
            else:
                sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, dev(qsl), tl, dl, dev(ids_h), dev(ua), dev(us), K, acc, tok,
                                 st, ws, temperature=T)
            torch.cuda.synchronize()
            out.append((acc.cpu().numpy(), tok.cpu().numpy(), st.cpu().numpy()))
        return out

    clean = both(ids)
    bad = ids.copy()
    bad[qsl[0] - 0 + 2] = V + 5      # sequence 0, last draft
    bad[qsl[3] - 3 + 0] = -2         # sequence 3, first draft
    marked = both(bad)
    for (a0, t0, s0), (a1, t1, s1) in zip(clean, marked):
        assert (s0 == 0).all()
        assert s1[0] == sx.SPEXIS_ROW_BAD_TOKEN and s1[3] == sx.SPEXIS_ROW_BAD_TOKEN
        assert a1[0] == 0 and a1[3] == 0 and (t1[[0, 3]] == -1).all()
        keep = [1, 2, 4, 5]
        np.testing.assert_array_equal(a1[keep], a0[keep])
        np.testing.assert_array_equal(t1[keep], t0[keep])
        np.testing.assert_array_equal(s1[keep], 0)



@pytest.mark.parametrize("B,K,d", [(20, 5, 256), (64, 4, 512), (90, 4, 256)])
def test_lm_head_gathers_the_draft_logits(B, K, d):
    # target rows gather at the draft of the position they verify (spexis_verify_gather_columns), draft
    # rows at their own draft; the gathered values are the logits output bit for bit, rows with no
    # gather (bonus rows) or an id outside [0, V) are left alone, and acceptance from the fused
    # statistics gives the same outputs with or without them.  B sequences of 0..K drafts: about
    # 70, 290 and 400 target rows, so all three workgroup shapes of the projection run.
    rng = np.random.default_rng(B + d)
    V, T_ = 3000, 0.8
    k = rng.integers(0, K + 1, B)
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    Tt, Td = int(qsl[-1]), int(qsl[-1]) - B
    w, _ = bf16_pair((V, d), 31, 0.1)
    ht, _ = bf16_pair((Tt, d), 32, 1.0)
    hd, _ = bf16_pair((Td, d), 33, 1.0)
    ids = rng.integers(0, V, Td).astype(np.int32)
    if Td > 2:
        ids[1] = V + 5                       # out of range: gathered nowhere
    tiles = sx.spexis_lm_head_tiles(V)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    wp = sx.spexis_pack_weight(w.cuda())
    tl = torch.empty((Tt, V), dtype=torch.float32, device="cuda")
    dl = torch.empty((Td, V), dtype=torch.float32, device="cuda")
    ts = torch.empty((Tt, tiles, 2), dtype=torch.float32, device="cuda")
    ds = torch.empty((Td, tiles, 2), dtype=torch.float32, device="cuda")
    tg = torch.full((Tt,), float("nan"), device="cuda")
    dg = torch.full((Td,), float("nan"), device="cuda")
    cols = torch.full((Tt,), -9, dtype=torch.int32, device="cuda")
    sx.spexis_verify_gather_columns(dev(qsl), dev(ids), cols)
    torch.cuda.synchronize()
    expect = np.concatenate([np.append(ids[qsl[b] - b:qsl[b] - b + k[b]], -1) for b in range(B)])
    np.testing.assert_array_equal(cols.cpu().numpy(), expect)
    sx.spexis_lm_head_gather(ht.cuda(), wp, ts, cols, tg, logits=tl, temperature=T_)
    sx.spexis_lm_head_gather(hd.cuda(), wp, ds, dev(ids), dg, logits=dl, temperature=T_)
    ts2, ds2 = torch.empty_like(ts), torch.empty_like(ds)
    sx.spexis_lm_head(ht.cuda(), wp, ts2, temperature=T_, vocab=V)
    sx.spexis_lm_head(hd.cuda(), wp, ds2, temperature=T_, vocab=V)
    torch.cuda.synchronize()
    # the gathering pass writes the same statistics as the plain one
    assert torch.equal(ts, ts2) and torch.equal(ds, ds2)
    tln, dln, tgn, dgn = tl.cpu().numpy(), dl.cpu().numpy(), tg.cpu().numpy(), dg.cpu().numpy()
    for m in range(Td):
        x = ids[m]
        if 0 <= x < V:
            assert dgn[m].view(np.uint32) == dln[m, x].view(np.uint32), m
        else:
            assert np.isnan(dgn[m])
    for b in range(B):
        for i in range(k[b] + 1):
            m = qsl[b] + i
            x = ids[qsl[b] - b + i] if i < k[b] else -1
            if 0 <= x < V:
                assert tgn[m].view(np.uint32) == tln[m, x].view(np.uint32), (b, i)
            else:
                assert np.isnan(tgn[m]), (b, i)
    say(f"[lm_head gather] B={B} rows {Tt}/{Td}: gathered values equal the logits")
    ua = dev(rng.random(Td, dtype=np.float32))
    us = dev(rng.random(B, dtype=np.float32))
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    outs = []
    for gathered in ((None, None), (tg, dg)):
        acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        tok = torch.full((B, K + 1), -7, dtype=torch.int32, device="cuda")
        st = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        sx.spexis_accept_with_stats(dev(qsl), tl, dl, ts, ds, dev(ids), ua, us, K, acc, tok, st, ws, temperature=T_,
                                    target_gathered=gathered[0], draft_gathered=gathered[1])
        torch.cuda.synchronize()
        outs.append((acc.clone(), tok.clone(), st.clone()))
    for a, b_ in zip(*outs):
        assert torch.equal(a, b_)
    if Td > 2:   # the sequence holding the out-of-range draft id reports it
        d0 = qsl[:-1] - np.arange(B)
        bad = [b for b in range(B) if d0[b] <= 1 < d0[b] + k[b]][0]
        assert outs[1][2].cpu().numpy()[bad] == sx.SPEXIS_ROW_BAD_TOKEN
