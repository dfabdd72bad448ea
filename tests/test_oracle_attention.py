"""Pins of the oracle's append and attention against what the mathematics fixes.

* dense recomputation with torch's fp64 ``scaled_dot_product_attention`` (a library routine)
  over the same logical K/V equals the paged result (GQA, causal window per query token);
* k = 0 reduces to single-token decode attention;
* closed forms: Q = 0 gives the mean of the visible V rows; constant V rows give that
  constant; a query that sees one key returns that key's V row;
* physical block placement does not matter (bit-identical under a block permutation);
* append writes exactly the new rows at positions L_b..S_b-1 and nothing else.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from tests import layout_ref as lr


def bf16_bits(x: np.ndarray) -> np.ndarray:
    return torch.as_tensor(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def make_case(rng, B, hq, hkv, D, bs, L, k, extra_blocks=3):
    """Random logical K/V per sequence, written into a permuted physical pool (test-side layout)."""
    n = np.asarray(k) + 1
    L = np.asarray(L)
    S = L + n
    nblk = (S + bs - 1) // bs
    num_blocks = int(nblk.sum()) + extra_blocks
    perm = rng.permutation(num_blocks)
    mb = int(nblk.max())
    tables = np.zeros((B, mb), np.int32)
    off = 0
    for b in range(B):
        tables[b, : nblk[b]] = perm[off: off + nblk[b]]
        off += nblk[b]
    qsl = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    pool_k = bf16_bits(rng.standard_normal(num_blocks * hkv * bs * D))
    pool_v = bf16_bits(rng.standard_normal(num_blocks * hkv * bs * D))
    logical_k, logical_v = [], []
    for b in range(B):
        kb = bf16_bits(rng.standard_normal((S[b], hkv, D)))
        vb = bf16_bits(rng.standard_normal((S[b], hkv, D)))
        lr.scatter_seq(pool_k, "k", tables[b], kb, hkv, bs, D)
        lr.scatter_seq(pool_v, "v", tables[b], vb, hkv, bs, D)
        logical_k.append(kb)
        logical_v.append(vb)
    q = bf16_bits(rng.standard_normal((int(qsl[-1]), hq, D)))
    return dict(B=B, hq=hq, hkv=hkv, D=D, bs=bs, L=L, n=n, S=S.astype(np.int32), qsl=qsl, tables=tables,
                num_blocks=num_blocks, pool_k=pool_k, pool_v=pool_v, lk=logical_k, lv=logical_v, q=q)


def run_oracle(c, scale=None, seqs=None):
    scale = 1.0 / math.sqrt(c["D"]) if scale is None else scale
    return oracle.attention(c["pool_k"], c["pool_v"], c["num_blocks"], c["hkv"], c["bs"], c["D"], c["qsl"],
                            c["S"], c["tables"], c["q"], c["hq"], float(np.float32(scale)), seqs=seqs)


def sdpa_reference(c, scale=None):
    """torch fp64 SDPA with an explicit causal mask, per sequence, GQA by head repetition."""
    D, hq, hkv = c["D"], c["hq"], c["hkv"]
    G = hq // hkv
    scale = float(np.float32(1.0 / math.sqrt(D) if scale is None else scale))
    out = np.zeros((int(c["qsl"][-1]), hq, D))
    for b in range(c["B"]):
        n, L, S = int(c["n"][b]), int(c["L"][b]), int(c["S"][b])
        q = torch.as_tensor(bits_to_f64(c["q"][c["qsl"][b]: c["qsl"][b] + n]))      # [n, hq, D]
        k = torch.as_tensor(bits_to_f64(c["lk"][b])).repeat_interleave(G, dim=1)     # [S, hq, D]
        v = torch.as_tensor(bits_to_f64(c["lv"][b])).repeat_interleave(G, dim=1)
        mask = torch.arange(S)[None, :] <= (L + torch.arange(n))[:, None]           # [n, S]
        o = torch.nn.functional.scaled_dot_product_attention(
            q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1), attn_mask=mask, scale=scale)
        out[c["qsl"][b]: c["qsl"][b] + n] = o.transpose(0, 1).numpy()
    return out


@pytest.mark.parametrize("hq,hkv,D,bs", [(8, 2, 64, 16), (4, 4, 128, 32), (7, 1, 64, 32), (6, 3, 128, 16)])
def test_paged_equals_dense_sdpa(hq, hkv, D, bs):
    rng = np.random.default_rng(11 + hq + D + bs)
    B = 5
    c = make_case(rng, B, hq, hkv, D, bs, L=rng.integers(0, 70, B), k=rng.integers(0, 6, B))
    got = run_oracle(c)
    ref = sdpa_reference(c)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_k0_is_single_token_decode():
    rng = np.random.default_rng(5)
    B = 6
    c = make_case(rng, B, 8, 2, 64, 16, L=rng.integers(1, 90, B), k=np.zeros(B, int))
    got = run_oracle(c)
    # decode attention: the one query attends to every cached key and itself, no mask
    G = 4
    for b in range(B):
        S = int(c["S"][b])
        q = bits_to_f64(c["q"][c["qsl"][b]])                       # [hq, D]
        for h in range(8):
            kk = bits_to_f64(c["lk"][b][:, h // G])                 # [S, D]
            vv = bits_to_f64(c["lv"][b][:, h // G])
            s = (kk @ q[h]) * float(np.float32(1 / 8.0))
            w = np.exp(s - s.max())
            ref = (w / w.sum()) @ vv
            np.testing.assert_allclose(got[c["qsl"][b], h], ref, rtol=1e-12, atol=1e-12)
        assert S == c["L"][b] + 1


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(7)
    B = 4
    c = make_case(rng, B, 4, 2, 64, 16, L=rng.integers(0, 40, B), k=np.full(B, 3))
    c["q"][:] = 0
    got = run_oracle(c)
    for b in range(B):
        for j in range(int(c["n"][b])):
            vis = int(c["L"][b]) + j + 1
            for h in range(4):
                ref = bits_to_f64(c["lv"][b][:vis, h // 2]).mean(axis=0)
                np.testing.assert_allclose(got[c["qsl"][b] + j, h], ref, rtol=1e-12, atol=1e-13)


def test_constant_values_give_that_constant():
    rng = np.random.default_rng(8)
    B = 3
    c = make_case(rng, B, 4, 1, 64, 32, L=rng.integers(0, 60, B), k=np.full(B, 2))
    const = bf16_bits(rng.standard_normal(64))
    for b in range(B):
        rows = np.broadcast_to(const, (int(c["S"][b]), 1, 64)).copy()
        lr.scatter_seq(c["pool_v"], "v", c["tables"][b], rows, 1, 32, 64)
    got = run_oracle(c)
    np.testing.assert_allclose(got, np.broadcast_to(bits_to_f64(const), got.shape), rtol=1e-14, atol=0)


def test_single_visible_key_returns_its_value():
    rng = np.random.default_rng(9)
    c = make_case(rng, 3, 8, 2, 128, 16, L=np.zeros(3, int), k=np.array([0, 3, 5]))
    got = run_oracle(c)
    for b in range(3):
        for h in range(8):   # token j = 0 with an empty cache sees only itself
            np.testing.assert_array_equal(got[c["qsl"][b], h], bits_to_f64(c["lv"][b][0, h // 4]))


def test_block_permutation_invariance():
    rng = np.random.default_rng(10)
    B = 4
    c = make_case(rng, B, 8, 2, 64, 16, L=rng.integers(20, 100, B), k=np.full(B, 4))
    base = run_oracle(c)
    # move every physical block to a new id and rewrite the tables accordingly
    nb, hkv, bs, D = c["num_blocks"], 2, 16, 64
    newid = rng.permutation(nb)
    blk_elems = hkv * bs * D
    pk = np.empty_like(c["pool_k"])
    pv = np.empty_like(c["pool_v"])
    for old in range(nb):
        pk[newid[old] * blk_elems:(newid[old] + 1) * blk_elems] = c["pool_k"][old * blk_elems:(old + 1) * blk_elems]
        pv[newid[old] * blk_elems:(newid[old] + 1) * blk_elems] = c["pool_v"][old * blk_elems:(old + 1) * blk_elems]
    c2 = dict(c, pool_k=pk, pool_v=pv, tables=newid[c["tables"]].astype(np.int32))
    moved = run_oracle(c2)
    np.testing.assert_array_equal(base, moved)


def test_subset_rows_match_full_run():
    rng = np.random.default_rng(12)
    B = 5
    c = make_case(rng, B, 8, 2, 64, 16, L=rng.integers(0, 50, B), k=rng.integers(0, 4, B))
    full = run_oracle(c)
    sub = run_oracle(c, seqs=np.array([3, 1]))
    for b in (1, 3):
        s, e = c["qsl"][b], c["qsl"][b + 1]
        np.testing.assert_array_equal(sub[s:e], full[s:e])
    assert np.isnan(sub[c["qsl"][0]:c["qsl"][1]]).all()


@pytest.mark.parametrize("bs,D", [(16, 64), (32, 128)])
def test_append_writes_exactly_the_new_rows(bs, D):
    rng = np.random.default_rng(13 + bs)
    B, hkv = 5, 2
    L = rng.integers(0, 80, B)
    k = rng.integers(0, 8, B)
    c = make_case(rng, B, 4, hkv, D, bs, L=L, k=k)
    T = int(c["qsl"][-1])
    new_k = bf16_bits(rng.standard_normal((T, hkv, D)))
    new_v = bf16_bits(rng.standard_normal((T, hkv, D)))
    pk, pv = c["pool_k"].copy(), c["pool_v"].copy()
    oracle.append_kv(pk, pv, c["num_blocks"], hkv, bs, D, c["qsl"], c["S"], c["tables"], new_k, new_v)
    exp_k, exp_v = c["pool_k"].copy(), c["pool_v"].copy()
    for b in range(B):
        s, e = c["qsl"][b], c["qsl"][b + 1]
        lr.scatter_seq(exp_k, "k", c["tables"][b], new_k[s:e], hkv, bs, D, start=int(c["L"][b]))
        lr.scatter_seq(exp_v, "v", c["tables"][b], new_v[s:e], hkv, bs, D, start=int(c["L"][b]))
        # the cached prefix is untouched
        np.testing.assert_array_equal(lr.gather_seq(pk, "k", c["tables"][b], int(c["L"][b]), hkv, bs, D),
                                      c["lk"][b][: int(c["L"][b])])
    np.testing.assert_array_equal(pk, exp_k)
    np.testing.assert_array_equal(pv, exp_v)


def test_append_rejects_out_of_range_block():
    rng = np.random.default_rng(14)
    c = make_case(rng, 2, 4, 2, 64, 16, L=np.array([5, 5]), k=np.array([2, 2]))
    tables = c["tables"].copy()
    tables[1, 0] = c["num_blocks"] + 4
    with pytest.raises(ValueError):
        oracle.append_kv(c["pool_k"].copy(), c["pool_v"].copy(), c["num_blocks"], 2, 16, 64, c["qsl"], c["S"],
                         tables, np.zeros((6, 2, 64), np.uint16), np.zeros((6, 2, 64), np.uint16))
