"""GPU parity: the HIP path through the C ABI against the CPU oracle on the same seeded inputs.

Bars: append bit-exact; attention |gpu - oracle| <= 1e-2 + 1e-2 |oracle| per element (bf16
inputs, fp32 accumulation, bf16 output); softmax within 1e-5 absolute; acceptance (accepted
lengths, emitted tokens, row status) bit-exact when both sides get identical fp32
probabilities and uniforms; with logits, every disagreement must sit within 1e-5 of a
decision boundary.  The oracle's inputs are the generator's host copies, never anything the
GPU computed.  The five workloads are checked at their full sizes, every sequence and every
output element.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_34370_amd import spexis as sx
from paper_2609_34370_amd import workloads as wl
from paper_2609_34370_amd.step import VerifyStep, bf16_to_u16

pytestmark = pytest.mark.gpu

ATOL = RTOL = 1e-2


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def case(wid, seed=None, accept=True, **over):
    spec = wl.spec_with(wid, **over) if over else wl.WORKLOADS[wid]
    batch = wl.make_batch(spec, seed=seed)
    attn = wl.make_attention_inputs(spec, batch, device="cuda", seed=seed)
    acc = wl.make_accept_inputs(spec, batch, device="cuda", seed=seed) if accept else None
    return spec, batch, attn, acc


def pick_seqs(batch, n, rng):
    if batch.B <= n:
        return np.arange(batch.B)
    must = {int(np.argmax(batch.seq_lens)), int(np.argmin(batch.seq_lens)), int(np.argmax(batch.k)),
            int(np.argmin(batch.k))}
    rest = rng.choice(batch.B, size=n, replace=False)
    return np.array(sorted(must | set(int(x) for x in rest)))[: max(n, len(must))]


def oracle_pools_after_append(spec, batch, k0, v0, attn):
    kp, vp = k0.copy(), v0.copy()
    oracle.append_kv(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                     batch.seq_lens, batch.block_tables, bf16_to_u16(attn.new_k), bf16_to_u16(attn.new_v))
    return kp, vp


def bf16_out_to_f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


# ---------------------------------------------------------------------------- append

@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_append_bit_exact(wid):
    say(f"[append] workload {wid}")
    spec, batch, attn, _ = case(wid, accept=False)
    k0, v0 = bf16_to_u16(attn.k_pool), bf16_to_u16(attn.v_pool)
    step = VerifyStep(batch, attn, None)
    step.append()
    torch.cuda.synchronize()
    kp, vp = oracle_pools_after_append(spec, batch, k0, v0, attn)
    assert np.array_equal(bf16_to_u16(attn.k_pool), kp)
    assert np.array_equal(bf16_to_u16(attn.v_pool), vp)


@pytest.mark.parametrize("bs,D", [(16, 128), (32, 128), (16, 64), (32, 64)])
def test_append_long_queries_bit_exact(bs, D):
    # up to 150 new rows per sequence (more than the 64 V rows the kernel stages in LDS at a
    # time, so a 16-slot unit can be written by two chunks), empty caches and one-row queries
    say(f"[append] long queries bs={bs} D={D}")
    spec, batch, attn, _ = case(1, seed=50 + bs + D, accept=False, batch=9, block_size=bs, head_dim=D,
                                ctx=("uniform", 0, 70), k=("uniform", 0, 149))
    k0, v0 = bf16_to_u16(attn.k_pool), bf16_to_u16(attn.v_pool)
    step = VerifyStep(batch, attn, None)
    step.append()
    torch.cuda.synchronize()
    kp, vp = oracle_pools_after_append(spec, batch, k0, v0, attn)
    assert int(batch.k.max()) + 1 > 64
    assert np.array_equal(bf16_to_u16(attn.k_pool), kp)
    assert np.array_equal(bf16_to_u16(attn.v_pool), vp)


# ------------------------------------------------------------------------- attention

def check_attention(wid, nseq=None, seed=None, kv_chunk_tokens=0, **over):
    spec, batch, attn, _ = case(wid, seed=seed, accept=False, **over)
    say(f"[attention] workload {wid} B={batch.B} T={batch.T} max_S={batch.max_seq_len} chunk={kv_chunk_tokens}")
    k0, v0 = bf16_to_u16(attn.k_pool), bf16_to_u16(attn.v_pool)
    step = VerifyStep(batch, attn, None, kv_chunk_tokens=kv_chunk_tokens)
    step.append()
    step.attention()
    torch.cuda.synchronize()
    got = bf16_out_to_f64(step.out)
    kp, vp = oracle_pools_after_append(spec, batch, k0, v0, attn)
    seqs = np.arange(batch.B) if nseq is None else pick_seqs(batch, nseq, np.random.default_rng(wid))
    ref = oracle.attention(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                           batch.seq_lens, batch.block_tables, bf16_to_u16(attn.q), spec.num_q_heads,
                           float(np.float32(step.scale)), seqs=seqs)
    rows = np.concatenate([np.arange(batch.qsl[b], batch.qsl[b + 1]) for b in seqs])
    err = np.abs(got[rows] - ref[rows])
    bound = ATOL + RTOL * np.abs(ref[rows])
    worst = float((err / bound).max())
    say(f"  seqs={len(seqs)} max|err|={err.max():.3e} worst err/bound={worst:.3f}")
    assert np.isfinite(got[rows]).all()
    assert (err <= bound).all(), worst
    return step, got


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_attention_matches_oracle(wid):
    # every sequence of the full-size workload, so every item cut between wave shares (and
    # merged) is compared as well as the ones a wave covers whole
    check_attention(wid)


@pytest.mark.parametrize("chunk", [32, 96, 4096])
def test_attention_split_kv_settings(chunk):
    # many small chunks, an odd multiple of 32, and no split at all
    check_attention(1, 4, seed=77, kv_chunk_tokens=chunk, batch=6, ctx=("uniform", 1, 300))


def test_attention_short_contexts_and_tails():
    # empty caches, contexts shorter than one tile, block-size-32 pools, k = 0 rows
    check_attention(1, 8, seed=5, batch=8, ctx=("uniform", 0, 40), k=("uniform", 0, 6))
    check_attention(5, 8, seed=6, batch=8, ctx=("uniform", 0, 70), k=("uniform", 0, 8))


def test_attention_head_dim_64_block_32_and_wide_groups():
    check_attention(1, 6, seed=8, batch=6, block_size=32, num_q_heads=16, num_kv_heads=2, k=("fixed", 7))


@pytest.mark.parametrize("hq,hkv,D", [(4, 1, 128), (12, 3, 128), (20, 5, 64), (24, 12, 64)])
def test_attention_kv_head_counts(hq, hkv, D):
    # KV head counts whose grids round up to a multiple of 8 and of 2 Hkv waves (the map of
    # waves onto (share, head) for paired shares), padding waves included
    check_attention(1, 6, seed=30 + hkv, batch=12, num_q_heads=hq, num_kv_heads=hkv, head_dim=D,
                    ctx=("uniform", 100, 2000), k=("uniform", 0, 5))


def test_attention_skewed_share_pairs_odd_head_count():
    # 3 KV heads: 336 shares per head in 1008 waves; about 12500 tiles per head make shares of
    # 38 tiles, paired as 39 + 37, so every cut point moves off the equal split
    check_attention(1, 8, seed=41, batch=40, num_q_heads=12, num_kv_heads=3, head_dim=128,
                    ctx=("uniform", 9000, 11000), k=("fixed", 4))


def random_attention_geometry(seed):
    """One random attention geometry (seeded; the test's own draw): head size, block size, KV
    heads, group size and draft counts within the boundary's limits (G (k+1) <= 64 rows), batch,
    context range and KV split setting."""
    r = np.random.default_rng(1000 + seed)
    D = int(r.choice([64, 128]))
    bs = int(r.choice([16, 32]))
    hkv = int(r.choice([1, 2, 3, 4, 8]))
    G = int(r.choice([1, 2, 4, 7, 8]))
    kmax = int(r.integers(0, 64 // G))           # rows G (k+1) <= 64
    klo = int(r.integers(0, kmax + 1))
    lo = int(r.integers(0, 2000))
    hi = lo + int(r.integers(0, 2500))
    over = dict(batch=int(r.integers(1, 41)), num_q_heads=G * hkv, num_kv_heads=hkv, head_dim=D, block_size=bs,
                ctx=("uniform", lo, hi), k=("uniform", klo, kmax))
    return over, int(r.choice([0, 0, 32, 64, 160, 1024]))


@pytest.mark.parametrize("seed", range(10))
def test_attention_random_geometry(seed):
    # every row of every sequence against the oracle, over random mixes of the kernel's paths:
    # one or two row tiles, head sizes 64 and 128, block sizes 16 and 32, items whole or cut
    # between shares at random points, empty caches and k = 0 rows
    over, chunk = random_attention_geometry(seed)
    say(f"[attention random] seed {seed}: {over} kv_chunk_tokens={chunk}")
    check_attention(1, seed=2000 + seed, kv_chunk_tokens=chunk, **over)


def test_attention_block_permutation_invariance():
    spec, batch, attn, _ = case(1, seed=9, accept=False, batch=5, ctx=("uniform", 40, 200))
    step = VerifyStep(batch, attn, None)
    step.append()
    step.attention()
    base = step.out.clone()
    # move every physical block to a new id (whole (block, head) chunks are contiguous)
    nb = batch.num_blocks
    perm = torch.as_tensor(np.random.default_rng(3).permutation(nb), device="cuda")
    blk = spec.num_kv_heads * spec.block_size * spec.head_dim
    kp = torch.empty_like(attn.k_pool)
    vp = torch.empty_like(attn.v_pool)
    kp.view(nb, blk)[perm] = attn.k_pool.view(nb, blk)
    vp.view(nb, blk)[perm] = attn.v_pool.view(nb, blk)
    attn2 = wl.AttentionInputs(kp, vp, attn.q, attn.new_k, attn.new_v)
    tables = perm.cpu().numpy()[batch.block_tables].astype(np.int32)
    batch2 = wl.Batch(spec, batch.ctx_lens, batch.k, batch.qsl, batch.seq_lens, tables, nb)
    step2 = VerifyStep(batch2, attn2, None)
    step2.attention()
    torch.cuda.synchronize()
    assert torch.equal(base.view(torch.int16), step2.out.view(torch.int16))


def test_attention_ignores_garbage_past_sequence_end():
    # slots past S_b in a sequence's last block hold NaN: they must not leak into the output
    spec, batch, attn, _ = case(1, seed=10, accept=False, batch=4, ctx=("uniform", 20, 90))
    step = VerifyStep(batch, attn, None)
    step.append()
    step.attention()
    clean = step.out.clone()
    kp = bf16_to_u16(attn.k_pool).copy()
    vp = bf16_to_u16(attn.v_pool).copy()
    hkv, bs, D = spec.num_kv_heads, spec.block_size, spec.head_dim
    from tests import layout_ref as lr
    for b in range(batch.B):
        S = int(batch.seq_lens[b])
        last_blk = batch.block_tables[b, (S - 1) // bs]
        for slot in range(S % bs or bs, bs):
            for h in range(hkv):
                d = np.arange(D)
                kp[lr.k_offsets(last_blk, h, slot, d, hkv, bs, D)] = 0x7FC0   # bf16 NaN
                vp[lr.v_offsets(last_blk, h, slot, d, hkv, bs, D)] = 0x7FC0
    attn.k_pool.copy_(torch.as_tensor(kp.view(np.int16)).view(torch.bfloat16).cuda())
    attn.v_pool.copy_(torch.as_tensor(vp.view(np.int16)).view(torch.bfloat16).cuda())
    step.attention()
    torch.cuda.synchronize()
    assert torch.equal(clean.view(torch.int16), step.out.view(torch.int16))


# --------------------------------------------------------------------------- softmax

@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_softmax_matches_oracle(wid):
    # every target and draft row of the full-size workload
    spec, batch, _, acc = case(wid)
    for name, rows in (("target", acc.target_logits), ("draft", acc.draft_logits)):
        say(f"[softmax] workload {wid} {name} rows={rows.shape[0]} V={spec.vocab} T={acc.temperature}")
        probs = torch.empty_like(rows)
        sx.spexis_softmax_rows(rows, probs, acc.temperature)
        torch.cuda.synchronize()
        ref = oracle.softmax(rows.cpu().numpy(), acc.temperature)
        err = np.abs(probs.cpu().numpy() - ref).max()
        say(f"  max|err|={err:.3e}")
        assert err <= 1e-5


def test_softmax_odd_vocab_and_masked_logits():
    x = torch.randn((7, 1003), device="cuda") * 5
    x[:, 17] = -float("inf")
    p = torch.empty_like(x)
    sx.spexis_softmax_rows(x, p, 0.9)
    torch.cuda.synchronize()
    ref = oracle.softmax(x.cpu().numpy(), 0.9)
    assert np.abs(p.cpu().numpy() - ref).max() <= 1e-5
    assert (p[:, 17] == 0).all()


# ------------------------------------------------------------------------ acceptance

def oracle_probs(acc):
    return (oracle.softmax(acc.target_logits.cpu().numpy(), acc.temperature),
            oracle.softmax(acc.draft_logits.cpu().numpy(), acc.temperature))


def run_accept_probs(step, p_host, q_host, seq_lens=None):
    acc = step.acc
    tp = torch.as_tensor(p_host, device="cuda")
    dq = torch.as_tensor(q_host, device="cuda")
    sl = torch.as_tensor(seq_lens, device="cuda") if seq_lens is not None else None
    step.accept(target=tp, draft=dq, kind=sx.SPEXIS_INPUT_PROBS, seq_lens_inout=sl)
    torch.cuda.synchronize()
    a, t, s = step.accept_outputs()
    return a, t, s, (sl.cpu().numpy() if sl is not None else None)


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_accept_probs_bit_exact(wid):
    spec, batch, attn, acc = case(wid)
    say(f"[accept probs] workload {wid} B={batch.B} V={spec.vocab} max_k={batch.max_k}")
    p, q = oracle_probs(acc)
    step = VerifyStep(batch, attn, acc)
    a, t, s, sl = run_accept_probs(step, p, q, seq_lens=batch.seq_lens)
    ra, rt, rs, rsl = oracle.accept(batch.qsl, p, q, acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(),
                                    acc.u_sample.cpu().numpy(), max_k=batch.max_k, seq_lens=batch.seq_lens)
    say(f"  mean accepted={a.mean():.3f} emitted={int((a + 1).sum())}")
    np.testing.assert_array_equal(a, ra)
    np.testing.assert_array_equal(t, rt)
    np.testing.assert_array_equal(s, rs)
    np.testing.assert_array_equal(sl, rsl)


def test_accept_identical_draft_accepts_all():
    spec, batch, attn, acc = case(2, batch=32)
    p, _ = oracle_probs(acc)
    q = p[wl.draft_row_index(batch)]
    rng = np.random.default_rng(1)
    ids = np.array([rng.choice(q.shape[1], p=r / r.sum(dtype=np.float64)) for r in q.astype(np.float64)], np.int32)
    acc.draft_ids.copy_(torch.as_tensor(ids))
    step = VerifyStep(batch, attn, acc)
    a, t, s, _ = run_accept_probs(step, p, q)
    np.testing.assert_array_equal(a, batch.k)
    assert (s == 0).all()


def test_accept_status_codes_and_edge_rows():
    V = 5000
    qsl = np.array([0, 3, 6, 9, 10, 13], np.int32)      # k = 2, 2, 2, 0, 2
    B = 5
    rng = np.random.default_rng(2)
    p = rng.random((13, V)).astype(np.float32)
    p /= p.sum(1, keepdims=True)
    q = rng.random((8, V)).astype(np.float32)
    q /= q.sum(1, keepdims=True)
    ids = rng.integers(0, V, 8).astype(np.int32)
    ids[3] = V + 7                                      # seq 1: bad token id
    p[6, ids[4]] = 0.0                                  # seq 2: rejects position 0 ...
    p[6, 100] = np.nan                                  # ... and its residual row holds a NaN
    p[9] = 0.0                                          # seq 3 (k = 0): an all-zero bonus row
    q[6, :] = 0.0                                       # seq 4: a one-hot draft row
    q[6, ids[6]] = 1.0
    ua = rng.random(8, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=2)
    assert list(rs[:4]) == [0, 3, 2, 1]
    dev = lambda x: torch.as_tensor(x, device="cuda")
    accepted = torch.empty(B, dtype=torch.int32, device="cuda")
    toks = torch.empty((B, 3), dtype=torch.int32, device="cuda")
    stat = torch.empty(B, dtype=torch.int32, device="cuda")
    for kind in (sx.SPEXIS_INPUT_PROBS,):
        ws = torch.empty(sx.spexis_accept_workspace_size(B, V, 2), dtype=torch.uint8, device="cuda")
        sx.spexis_accept(kind, dev(qsl), dev(p), dev(q), dev(ids), dev(ua), dev(us), 2, accepted, toks, stat, ws)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(accepted.cpu().numpy(), ra)
        np.testing.assert_array_equal(toks.cpu().numpy(), rt)
        np.testing.assert_array_equal(stat.cpu().numpy(), rs)


def borderline(p, q, ids, ua, us, qsl, b, a_o, t_o, a_g, t_g, tol=1e-5):
    """True if a logits-mode disagreement sits within fp32 rounding of a decision boundary: the
    first test the two sides decide differently has |u q(x) - p(x)| <= tol, or the sampled
    tokens differ and the uniform lies within tol of the normalised CDF between them (t within
    tol * S of a prefix boundary)."""
    t0, d0 = qsl[b], qsl[b] - b
    if a_o != a_g:
        i = min(a_o, a_g)
        x = ids[d0 + i]
        return abs(float(ua[d0 + i]) * float(q[d0 + i, x]) - float(p[t0 + i, x])) <= tol
    k = qsl[b + 1] - qsl[b] - 1
    a = a_o
    w = np.maximum(p[t0 + a].astype(np.float64) - q[d0 + a], 0) if a < k else p[t0 + a].astype(np.float64)
    cdf = np.cumsum(w) / w.sum()
    m = min(t_o[a], t_g[a])
    return abs(cdf[m] - float(us[b])) <= tol


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_accept_logits_agrees_with_oracle(wid):
    spec, batch, attn, acc = case(wid)
    say(f"[accept logits] workload {wid} B={batch.B} V={spec.vocab} T={acc.temperature}")
    step = VerifyStep(batch, attn, acc)
    step.accept()
    torch.cuda.synchronize()
    a, t, s = step.accept_outputs()
    p, q = oracle_probs(acc)
    ids, ua, us = acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(), acc.u_sample.cpu().numpy()
    ra, rt, rs, _ = oracle.accept(batch.qsl, p, q, ids, ua, us, max_k=batch.max_k)
    assert (s == 0).all() and (rs == 0).all()
    diff = [b for b in range(batch.B) if a[b] != ra[b] or not np.array_equal(t[b], rt[b])]
    say(f"  mean accepted={a.mean():.3f} disagreements={len(diff)}")
    for b in diff:
        assert borderline(p, q, ids, ua, us, batch.qsl, b, ra[b], rt[b], a[b], t[b]), b


def test_accept_logits_rounds_with_ragged_drafts():
    # 128 sequences, k_b in 0..8, V = 128256: 590 MB of target rows, so the tests run in rounds,
    # and a first round over {0,1} would read 263 MB, so they are {0}, {1,2}, {3..8}; draft
    # noise spread U[0.1, 3] sends some sequences through all three
    spec, batch, attn, acc = case(4, vocab=128256)
    assert batch.B * (batch.max_k + 1) * spec.vocab * 4 > (192 << 20)
    say(f"[accept logits rounds] B={batch.B} V={spec.vocab} k in [{batch.k.min()}, {batch.k.max()}]")
    step = VerifyStep(batch, attn, acc)
    step.accept()
    torch.cuda.synchronize()
    a, t, s = step.accept_outputs()
    p, q = oracle_probs(acc)
    ids, ua, us = acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(), acc.u_sample.cpu().numpy()
    ra, rt, rs, _ = oracle.accept(batch.qsl, p, q, ids, ua, us, max_k=batch.max_k)
    assert (s == 0).all() and (rs == 0).all()
    assert (a >= 3).sum() > 0 and (a >= 7).sum() > 0, "some sequences must reach the later rounds"
    diff = [b for b in range(batch.B) if a[b] != ra[b] or not np.array_equal(t[b], rt[b])]
    say(f"  accepted histogram={np.bincount(a, minlength=9).tolist()} disagreements={len(diff)}")
    for b in diff:
        assert borderline(p, q, ids, ua, us, batch.qsl, b, ra[b], rt[b], a[b], t[b]), b


@pytest.mark.parametrize("seed", range(6))
def test_accept_random_geometry(seed):
    # random batch, vocabulary (not a multiple of 4 or of a sub-chunk), ragged draft counts up
    # to the boundary's 32, draft noise and temperature: probabilities bit-exact, logits equal
    # to the oracle's exact rule on its fp64 softmax (within 1e-5 of a decision boundary)
    r = np.random.default_rng(3000 + seed)
    V = int(r.integers(1000, 200000))
    kmax = int(r.integers(0, 33))
    over = dict(batch=int(r.integers(1, 41)), vocab=V, k=("uniform", int(r.integers(0, kmax + 1)), kmax),
                draft_noise=("uniform", 0.05, float(r.uniform(0.5, 4.0))), temperature=float(r.choice([0.5, 1.0, 1.7])),
                target_std=float(r.uniform(1.0, 4.0)), ctx=("uniform", 1, 64))
    spec, batch, attn, acc = case(1, seed=4000 + seed, **over)
    say(f"[accept random] seed {seed}: B={batch.B} V={V} k in [{batch.k.min()}, {batch.k.max()}] "
        f"T={spec.temperature}")
    p, q = oracle_probs(acc)
    ids, ua, us = acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(), acc.u_sample.cpu().numpy()
    ra, rt, rs, _ = oracle.accept(batch.qsl, p, q, ids, ua, us, max_k=batch.max_k)
    step = VerifyStep(batch, attn, acc)
    step.accept(target=torch.as_tensor(p, device="cuda"), draft=torch.as_tensor(q, device="cuda"),
                kind=sx.SPEXIS_INPUT_PROBS)
    torch.cuda.synchronize()
    a, t, s_ = step.accept_outputs()
    np.testing.assert_array_equal(a, ra)   # the oracle's rule on these same fp32 probabilities
    np.testing.assert_array_equal(t, rt)
    np.testing.assert_array_equal(s_, rs)
    step.accept()
    torch.cuda.synchronize()
    a, t, s_ = step.accept_outputs()
    assert (s_ == 0).all() and (rs == 0).all()
    diff = [b for b in range(batch.B) if a[b] != ra[b] or not np.array_equal(t[b], rt[b])]
    say(f"  mean accepted={a.mean():.3f} disagreements={len(diff)}")
    for b in diff:
        assert borderline(p, q, ids, ua, us, batch.qsl, b, ra[b], rt[b], a[b], t[b]), b


def test_accept_logits_edge_rows_across_rounds():
    # 64 sequences, max_k = 8, V = 100000: several rounds.  Special sequences:
    #   0: draft id out of range at position 5 (found before any test)   -> status 3
    #   1: draft equal to target at 0..2, a NaN target logit at 3        -> a = 3, status 2
    #   2: draft equal to target everywhere                              -> a = 8, bonus
    #   3: k = 0                                                         -> bonus row 0
    #   4: draft equal to target everywhere, bonus row all -inf          -> a = 8, status 2
    V, B, K = 100000, 64, 8
    rng = np.random.default_rng(11)
    k = rng.integers(0, K + 1, B)
    k[[0, 1, 2, 4]] = K
    k[3] = 0
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    T = int(qsl[-1])
    tl = (rng.standard_normal((T, V)) * 3).astype(np.float32)
    dl = np.empty((T - B, V), np.float32)
    for b in range(B):
        for i in range(k[b]):
            dl[qsl[b] - b + i] = tl[qsl[b] + i] + rng.standard_normal(V).astype(np.float32)
    for b, upto in ((1, 3), (2, K), (4, K)):
        for i in range(upto):
            dl[qsl[b] - b + i] = tl[qsl[b] + i]
    tl[qsl[1] + 3, 777] = np.nan
    tl[qsl[4] + K, :] = -np.inf
    ids = np.empty(T - B, np.int32)
    for b in range(B):                                  # drafts drawn from the draft rows
        for i in range(k[b]):
            row = dl[qsl[b] - b + i].astype(np.float64)
            g = row - np.log(-np.log(rng.random(V)))
            ids[qsl[b] - b + i] = int(np.argmax(g))
    ids[qsl[0] - 0 + 5] = V + 3
    ua = rng.random(T - B, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    assert B * (K + 1) * V * 4 > (192 << 20)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    accepted = torch.empty(B, dtype=torch.int32, device="cuda")
    toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    stat = torch.empty(B, dtype=torch.int32, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, dev(qsl), dev(tl), dev(dl), dev(ids), dev(ua), dev(us), K, accepted,
                     toks, stat, ws, temperature=1.0)
    torch.cuda.synchronize()
    a, t, s = accepted.cpu().numpy(), toks.cpu().numpy(), stat.cpu().numpy()
    p, q = oracle.softmax(tl, 1.0), oracle.softmax(dl, 1.0)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    say(f"[accept logits edges] status={s[:5].tolist()} a={a[:5].tolist()} oracle status={rs[:5].tolist()}")
    assert list(rs[:5]) == [3, 2, 0, 0, 2] and list(ra[:5]) == [0, 3, 8, 0, 8]
    np.testing.assert_array_equal(s, rs)
    np.testing.assert_array_equal(a[:5], ra[:5])
    np.testing.assert_array_equal(t[:2], rt[:2])
    np.testing.assert_array_equal(t[4], rt[4])
    np.testing.assert_array_equal(t[2, :K], rt[2, :K])
    diff = [b for b in range(2, B) if b != 4 and (a[b] != ra[b] or not np.array_equal(t[b], rt[b]))]
    for b in diff:
        assert borderline(p, q, ids, ua, us, qsl, b, ra[b], rt[b], a[b], t[b]), b


@pytest.mark.parametrize("V", [70001, 1100001])
def test_accept_most_drafts_every_round_odd_vocab(V):
    # max_k = 32 (the largest the boundary takes).  V = 70001: rows of 280 KB, logits-mode rounds
    # {0,1}, {2..5}, {6..13}, {14..32}; V = 1100001: a first round over {0,1} would read 282 MB,
    # so the rounds are {0}, {1,2}, {3..6}, {7..14}, {15..32}.  Sequence b has
    # k_b drafts and a draft row equal to the target row at positions below m_b (those tests
    # always pass), a noisy one after; the m_b sit on both sides of every round boundary of both
    # schedules.  Neither vocabulary is a multiple of 4 entries.
    K = 32
    km = [(32, 32), (32, 31), (32, 30), (31, 31), (30, 29), (29, 14), (14, 13), (13, 6), (6, 5), (5, 2),
          (2, 1), (1, 0), (0, 0), (32, 0), (20, 20), (7, 7), (16, 15), (8, 7), (4, 3), (3, 2)]
    B = len(km)
    k = np.array([x for x, _ in km])
    rng = np.random.default_rng(23)
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    T = int(qsl[-1])
    tl = (rng.standard_normal((T, V)) * 2.5).astype(np.float32)
    dl = np.empty((T - B, V), np.float32)
    ids = np.empty(T - B, np.int32)
    for b, (kb, m) in enumerate(km):
        for i in range(kb):
            r = qsl[b] - b + i
            dl[r] = tl[qsl[b] + i] if i < m else tl[qsl[b] + i] + (rng.standard_normal(V) * 2).astype(np.float32)
            g = dl[r].astype(np.float64) - np.log(-np.log(rng.random(V)))
            ids[r] = int(np.argmax(g))
    ua = rng.random(T - B, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    p, q = oracle.softmax(tl, 1.0), oracle.softmax(dl, 1.0)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    for kind, tg, dr in ((sx.SPEXIS_INPUT_PROBS, p, q), (sx.SPEXIS_INPUT_LOGITS, tl, dl)):
        accepted = torch.empty(B, dtype=torch.int32, device="cuda")
        toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        stat = torch.empty(B, dtype=torch.int32, device="cuda")
        sx.spexis_accept(kind, dev(qsl), dev(tg), dev(dr), dev(ids), dev(ua), dev(us), K, accepted, toks, stat, ws,
                         temperature=1.0)
        torch.cuda.synchronize()
        a, t, s = accepted.cpu().numpy(), toks.cpu().numpy(), stat.cpu().numpy()
        say(f"[accept max_k] kind={kind} a={a.tolist()} oracle={ra.tolist()}")
        assert (rs == 0).all()
        np.testing.assert_array_equal(s, rs)
        assert all(a[b] >= m for b, (_, m) in enumerate(km)), "an identical draft row must pass"
        if kind == sx.SPEXIS_INPUT_PROBS:
            np.testing.assert_array_equal(a, ra)
            np.testing.assert_array_equal(t, rt)
        else:
            diff = [b for b in range(B) if a[b] != ra[b] or not np.array_equal(t[b], rt[b])]
            for b in diff:
                assert borderline(p, q, ids, ua, us, qsl, b, ra[b], rt[b], a[b], t[b]), b
    assert (ra >= 30).sum() >= 3 and ra[0] == 32


def test_accept_largest_vocabulary():
    # V = 2^22, the largest vocabulary the boundary takes: fixed-point sums up to 2^22 weights of
    # under 2^41 each; 3 sequences with k = 2, 0, 1, both input kinds.  Sequence 0's draft rows
    # equal its target rows (both tests pass, the bonus row is sampled); sequence 2's are noisy.
    V, K = 1 << 22, 2
    k = np.array([2, 0, 1])
    B = len(k)
    rng = np.random.default_rng(29)
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    T = int(qsl[-1])
    tl = (rng.standard_normal((T, V)) * 1.5).astype(np.float32)
    dl = (tl[[qsl[b] + i for b in range(B) for i in range(k[b])]] +
          rng.standard_normal((T - B, V)).astype(np.float32) * 0.3)
    dl[:2] = tl[:2]
    ids = np.array([int(np.argmax(r)) for r in dl], np.int32)
    ua = rng.random(T - B, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    p, q = oracle.softmax(tl, 1.0), oracle.softmax(dl, 1.0)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    for kind, tg, dr in ((sx.SPEXIS_INPUT_PROBS, p, q), (sx.SPEXIS_INPUT_LOGITS, tl, dl)):
        accepted = torch.empty(B, dtype=torch.int32, device="cuda")
        toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        stat = torch.empty(B, dtype=torch.int32, device="cuda")
        sx.spexis_accept(kind, dev(qsl), dev(tg), dev(dr), dev(ids), dev(ua), dev(us), K, accepted, toks, stat, ws,
                         temperature=1.0)
        torch.cuda.synchronize()
        a, t, s = accepted.cpu().numpy(), toks.cpu().numpy(), stat.cpu().numpy()
        say(f"[accept V=2^22] kind={kind} a={a.tolist()} tokens={t.tolist()} oracle a={ra.tolist()} {rt.tolist()}")
        np.testing.assert_array_equal(s, rs)
        assert a[0] == 2
        if kind == sx.SPEXIS_INPUT_PROBS:
            np.testing.assert_array_equal(a, ra)
            np.testing.assert_array_equal(t, rt)
        else:
            for b in range(B):
                if a[b] != ra[b] or not np.array_equal(t[b], rt[b]):
                    assert borderline(p, q, ids, ua, us, qsl, b, ra[b], rt[b], a[b], t[b]), b


@pytest.mark.parametrize("V", [1, 2, 3])
def test_accept_tiny_vocabularies(V):
    # degenerate rows: with one entry every test passes and every token is 0; with two or three,
    # both input kinds agree with the oracle (probabilities bit for bit)
    rng = np.random.default_rng(40 + V)
    k = np.array([0, 1, 2, 3, 2, 1, 0, 3])
    B, K = len(k), 3
    qsl = np.concatenate([[0], np.cumsum(k + 1)]).astype(np.int32)
    T = int(qsl[-1])
    tl = (rng.standard_normal((T, V)) * 2).astype(np.float32)
    dl = (rng.standard_normal((T - B, V)) * 2).astype(np.float32)
    ids = rng.integers(0, V, T - B).astype(np.int32)
    ua = rng.random(T - B, dtype=np.float32)
    us = rng.random(B, dtype=np.float32)
    p, q = oracle.softmax(tl, 1.0), oracle.softmax(dl, 1.0)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    for kind, tg, dr in ((sx.SPEXIS_INPUT_PROBS, p, q), (sx.SPEXIS_INPUT_LOGITS, tl, dl)):
        accepted = torch.empty(B, dtype=torch.int32, device="cuda")
        toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
        stat = torch.empty(B, dtype=torch.int32, device="cuda")
        sx.spexis_accept(kind, dev(qsl), dev(tg), dev(dr), dev(ids), dev(ua), dev(us), K, accepted, toks, stat, ws,
                         temperature=1.0)
        torch.cuda.synchronize()
        a, t, s = accepted.cpu().numpy(), toks.cpu().numpy(), stat.cpu().numpy()
        np.testing.assert_array_equal(s, rs)
        if V == 1:
            np.testing.assert_array_equal(a, k)
            assert all((t[b, :k[b] + 1] == 0).all() and (t[b, k[b] + 1:] == -1).all() for b in range(B))
        if kind == sx.SPEXIS_INPUT_PROBS:
            np.testing.assert_array_equal(a, ra)
            np.testing.assert_array_equal(t, rt)
        else:
            for b in range(B):
                if a[b] != ra[b] or not np.array_equal(t[b], rt[b]):
                    assert borderline(p, q, ids, ua, us, qsl, b, ra[b], rt[b], a[b], t[b]), b


def test_accept_logits_empty_residual_falls_back_to_target_row():
    # Rejections whose residual is empty in fixed point, with logits.  Sequence 0: identical target
    # and draft rows with the drafted entry at -inf (p(x) = q(x) = 0 rejects), so max(0, p - q)
    # is exactly 0.  Sequence 1: the same, and the draft also drops an entry the target gives
    # e^-35 of its largest probability, so the residual's only weight lies below 2^-40 of max p:
    # at the target row's scale it is 0 and the token comes from p (never that entry).
    V, B, K = 5000, 2, 1
    rng = np.random.default_rng(21)
    qsl = np.array([0, 2, 4], np.int32)
    tl = (rng.standard_normal((4, V)) * 2).astype(np.float32)
    ids = np.array([11, 22], np.int32)
    j = 4321
    for b in range(B):
        tl[qsl[b], ids[b]] = -np.inf
    tl[qsl[1], j] = tl[qsl[1]].max() - 35.0
    dl = np.stack([tl[qsl[0]], tl[qsl[1]]]).copy()
    dl[1, j] = -np.inf
    ua = np.full(B, 0.5, np.float32)
    us = rng.random(B, dtype=np.float32)
    dev = lambda x: torch.as_tensor(x, device="cuda")
    accepted = torch.empty(B, dtype=torch.int32, device="cuda")
    toks = torch.empty((B, K + 1), dtype=torch.int32, device="cuda")
    stat = torch.empty(B, dtype=torch.int32, device="cuda")
    ws = torch.empty(sx.spexis_accept_workspace_size(B, V, K), dtype=torch.uint8, device="cuda")
    sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, dev(qsl), dev(tl), dev(dl), dev(ids), dev(ua), dev(us), K, accepted,
                     toks, stat, ws, temperature=1.0)
    torch.cuda.synchronize()
    a, t, s = accepted.cpu().numpy(), toks.cpu().numpy(), stat.cpu().numpy()
    p, q = oracle.softmax(tl, 1.0), oracle.softmax(dl, 1.0)
    ra, rt, rs, _ = oracle.accept(qsl, p, q, ids, ua, us, max_k=K)
    say(f"[accept empty residual] tokens {t[:, 0].tolist()} oracle {rt[:, 0].tolist()}")
    assert list(a) == [0, 0] and list(ra) == [0, 0] and (s == 0).all() and (rs == 0).all()
    assert t[1, 0] != j and rt[1, 0] != j
    for b in range(B):
        assert t[b, 0] == rt[b, 0] or borderline(p, q, ids, ua, us, qsl, b, ra[b], rt[b], a[b], t[b]), b


# -------------------------------------------------------------------------- boundary

@pytest.mark.parametrize("wid,B", [(2, 16), (1, None)])
def test_verify_step_graph_replays_equal_the_eager_step(wid, B):
    # append + attention + acceptance captured into a HIP graph: every replay, with eager work
    # and synchronisations between them, gives bit for bit the eager step's outputs (workload 2:
    # acceptance in test rounds; workload 1: one round)
    over = {} if B is None else {"batch": B}
    spec, batch, attn, acc = case(wid, seed=3, **over)
    step = VerifyStep(batch, attn, acc)
    step.run()
    torch.cuda.synchronize()
    outs = lambda: [t.clone() for t in (step.out, step.accepted_len, step.out_tokens, step.row_status,
                                        attn.k_pool, attn.v_pool)]
    ref = outs()
    step.capture()
    for i in range(3):
        step.out.zero_()
        step.accepted_len.fill_(-7)
        step.out_tokens.fill_(-7)
        step.row_status.fill_(-7)
        step.attn_ws.fill_(0x5A)
        step.acc_ws.fill_(0x5A)
        torch.cuda.synchronize()
        step.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs(), ref):
            assert torch.equal(a, b), i
        say(f"[verify graph] workload {wid} replay {i}: equal to the eager step")


def test_boundary_errors_on_gpu():
    spec, batch, attn, acc = case(1)
    step = VerifyStep(batch, attn, acc, kv_chunk_tokens=32)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(sx.SpexisError) as e:
        sx.spexis_verify_attention(attn.k_pool, attn.v_pool, batch.num_blocks, spec.num_kv_heads, spec.block_size,
                                   spec.head_dim, step.qsl, step.seq_lens, step.tables, batch.T, batch.max_query_len,
                                   batch.max_seq_len, attn.q, spec.num_q_heads, 0.125, step.out, small,
                                   kv_chunk_tokens=32)
    assert e.value.code == sx.SPEXIS_ERR_WORKSPACE_TOO_SMALL
    with pytest.raises(sx.SpexisError) as e:
        sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, step.qsl, acc.target_logits, acc.draft_logits, acc.draft_ids,
                         acc.u_accept, acc.u_sample, batch.max_k, step.accepted_len, step.out_tokens,
                         step.row_status, step.acc_ws, temperature=0.0)
    assert e.value.code == sx.SPEXIS_ERR_INVALID_ARGUMENT


def test_empty_batches_return_ok_and_touch_nothing():
    # no sequences or no rows: every entry point returns OK without reading or writing a buffer
    # (zero-element tensors pass NULL pointers); the outputs and pools keep their contents
    dev = "cuda"
    i32 = lambda *s: torch.full(s, 77, dtype=torch.int32, device=dev)
    bf = lambda *s: torch.empty(s, dtype=torch.bfloat16, device=dev)
    f32 = lambda *s: torch.full(s, 0.25, dtype=torch.float32, device=dev)
    none8 = torch.empty(0, dtype=torch.uint8, device=dev)
    k_pool = torch.full((4, 2, 16, 64), 1.5, dtype=torch.bfloat16, device=dev)
    v_pool = k_pool.clone()
    qsl0 = torch.zeros(1, dtype=torch.int32, device=dev)
    sx.spexis_append_kv(k_pool, v_pool, 4, 2, 16, 64, qsl0, i32(0), i32(0, 4), 0, 1, bf(0, 2, 64), bf(0, 2, 64))
    sx.spexis_verify_attention(k_pool, v_pool, 4, 2, 16, 64, qsl0, i32(0), i32(0, 4), 0, 1, 16, bf(0, 4, 64), 4,
                               0.125, bf(0, 4, 64), workspace=None)
    V = 100
    for kind in (sx.SPEXIS_INPUT_PROBS, sx.SPEXIS_INPUT_LOGITS):
        sx.spexis_accept(kind, qsl0, f32(0, V), f32(0, V), i32(0), f32(0), f32(0), 2, i32(0), i32(0, 3), i32(0),
                         none8)
    sx.spexis_accept_with_stats(qsl0, f32(0, V), f32(0, V), f32(0, 1, 2), f32(0, 1, 2), i32(0), f32(0), f32(0), 2,
                                i32(0), i32(0, 3), i32(0), none8)
    sx.spexis_softmax_rows(f32(0, V), f32(0, V))
    sx.spexis_sample_tokens(sx.SPEXIS_INPUT_LOGITS, f32(0, V), f32(0), i32(0), i32(0), none8)
    kept_qsl = i32(1)
    sx.spexis_select_drafts(qsl0, f32(0), 0.3, i32(0), kept_qsl, i32(0))
    g = torch.Generator().manual_seed(1)
    w_lm = sx.spexis_pack_weight(torch.randn((V, 256), generator=g).to(torch.bfloat16).cuda())
    w_lin = sx.spexis_pack_weight(torch.randn((64, 256), generator=g).to(torch.bfloat16).cuda())
    sx.spexis_lm_head(bf(0, 256), w_lm, f32(0, 1, 2), logits=f32(0, V))
    sx.spexis_linear(bf(0, 256), w_lin, bf(0, 64))
    torch.cuda.synchronize()
    assert (k_pool == 1.5).all() and (v_pool == 1.5).all()
    assert kept_qsl.item() == 77
    say("[empty] every entry point accepted an empty batch")
