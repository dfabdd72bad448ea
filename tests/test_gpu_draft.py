"""The drafting step on the GPU (DraftStep: adapter linear, q/k/v, append, attention, output
projection with residual, LM head, draw) against the oracle, stage by stage.

Each stage's GPU output is compared, element by element, with the oracle's function of that
stage applied to the GPU's own bf16 inputs of the stage (as the chain feeds them), so every
bound is the stage's own:
  * linear layers (x, q, k, v, y): |gpu - oracle| <= 2^-8 |oracle| + 4 K 2^-24 sum_j |x_j W_oj|
    (one bf16 rounding and an fp32 sum of K exact products);
  * append: the pools equal the oracle's append of the GPU's k and v, bit for bit;
  * attention: |gpu - oracle| <= 1e-2 + 1e-2 |oracle|;
  * LM head: |gpu - oracle| <= 2 K 2^-24 sum_j |y_j W_vj| + 1e-6 per logit;
  * draw: the token equals the oracle's exact inverse-CDF draw on the softmax of the GPU's
    logits, or the uniform lies within 1e-5 of the CDF boundary between the two; the confidence
    is within 1e-5 of the oracle's probability of the token.
The first stage is also checked against oracle.draft_step, the adapter's composition.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_34370_amd import workloads as wl
from paper_2609_34370_amd.draft import DraftStep
from paper_2609_34370_amd.step import bf16_to_u16

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def f64(bits):
    return oracle.bf16_value(bits)


def check_linear(name, got_bits, x_bits, w_bits, res_bits=None):
    ref = oracle.linear(x_bits, w_bits, res_bits)
    mag = np.abs(f64(x_bits)) @ np.abs(f64(w_bits)).T
    bound = 2.0 ** -8 * np.abs(ref) + 4 * x_bits.shape[1] * 2.0 ** -24 * mag + 1e-30
    err = np.abs(f64(got_bits) - ref)
    say(f"  {name}: max err/bound {(err / bound).max():.3f}")
    assert (err <= bound).all(), name


@pytest.mark.parametrize("wid,B", [(1, 64), (2, 16)])
def test_draft_step_matches_oracle(wid, B):
    spec = wl.spec_with(wid, batch=B)
    base = wl.make_batch(spec)
    batch = wl.make_batch(spec, ctx_lens=base.ctx_lens, k=np.zeros(B, np.int32))
    cache = wl.make_attention_inputs(spec, batch, device="cuda")
    kp0, vp0 = bf16_to_u16(cache.k_pool).copy(), bf16_to_u16(cache.v_pool).copy()
    ad = wl.make_adapter_inputs(spec, batch, device="cuda")
    say(f"[draft] workload {wid} B={B} d={ad.h.shape[1]} V={spec.vocab}")
    step = DraftStep(batch, cache, ad)
    step.run()
    torch.cuda.synchronize()
    u16 = bf16_to_u16
    hq, hkv, D, T = spec.num_q_heads, spec.num_kv_heads, spec.head_dim, ad.temperature
    w = {n: u16(getattr(ad, n)) for n in ("h", "w_in", "w_q", "w_k", "w_v", "w_o", "w_lm")}
    g = {n: u16(getattr(step, n)).reshape(B, -1) for n in ("x", "q", "k", "v", "o", "y")}
    # the adapter's first stage, also from the oracle's whole composition
    ref = oracle.draft_step(w["h"], w["w_in"], w["w_q"], w["w_k"], w["w_v"], w["w_o"], w["w_lm"], kp0.copy(),
                            vp0.copy(), batch.num_blocks, hkv, hq, spec.block_size, D, batch.seq_lens,
                            batch.block_tables, T, ad.u.cpu().numpy())
    check_linear("x", g["x"], w["h"], w["w_in"])
    assert (np.abs(f64(g["x"]) - f64(ref["x"])) <= 2.0 ** -7 * np.abs(f64(ref["x"])) + 1e-30).all()
    for n in ("q", "k", "v"):
        check_linear(n, g[n], g["x"], w["w_" + n])
    # append of the GPU's k and v: bit for bit
    kp, vp = kp0.copy(), vp0.copy()
    oracle.append_kv(kp, vp, batch.num_blocks, hkv, spec.block_size, D, batch.qsl, batch.seq_lens,
                     batch.block_tables, g["k"].reshape(B, hkv, D), g["v"].reshape(B, hkv, D))
    assert np.array_equal(u16(cache.k_pool), kp) and np.array_equal(u16(cache.v_pool), vp)
    # attention of the GPU's q over those pools
    o_ref = oracle.attention(kp, vp, batch.num_blocks, hkv, spec.block_size, D, batch.qsl, batch.seq_lens,
                             batch.block_tables, g["q"].reshape(B, hq, D), hq, float(np.float32(step.scale)))
    err = np.abs(f64(g["o"]) - o_ref.reshape(B, -1))
    bound = 1e-2 + 1e-2 * np.abs(o_ref.reshape(B, -1))
    say(f"  o: max err/bound {(err / bound).max():.3f}")
    assert (err <= bound).all()
    # output projection with the residual x
    check_linear("y", g["y"], g["o"], w["w_o"], g["x"])
    # LM head on the GPU's y
    lg = step.logits.cpu().numpy()
    lref, _, _ = oracle.lm_head(g["y"], w["w_lm"], T)
    mag = np.abs(f64(g["y"])) @ np.abs(f64(w["w_lm"])).T
    bound = 2 * g["y"].shape[1] * 2.0 ** -24 * mag + 1e-6
    err = np.abs(lg.astype(np.float64) - lref)
    say(f"  logits: max err {err.max():.3e}, max err/bound {(err / bound).max():.3f}")
    assert (err <= bound).all()
    # the draw from the GPU's logits
    p = oracle.softmax(lg, T)
    otok, oprob, ost = oracle.sample(p, ad.u.cpu().numpy())
    tok, conf, st = step.tokens.cpu().numpy(), step.conf.cpu().numpy(), step.status.cpu().numpy()
    assert (st == 0).all() and (ost == 0).all()
    u = ad.u.cpu().numpy().astype(np.float64)
    same = 0
    for b in range(B):
        t, to = int(tok[b]), int(otok[b])
        if t != to:
            cdf = np.cumsum(p[b].astype(np.float64))
            cdf /= cdf[-1]
            assert abs(cdf[min(t, to)] - u[b]) <= 1e-5, (b, t, to)
        same += t == to
        assert abs(float(conf[b]) - float(p[b, t])) <= 1e-5, b
    say(f"  tokens equal to the oracle's draw for {same}/{B}")


def test_draft_step_graph_replays_equal_the_eager_step():
    # the step captured into a HIP graph: every replay, with eager work and synchronisations
    # between them, gives bit for bit the eager step's outputs
    spec = wl.spec_with(2, batch=16)
    base = wl.make_batch(spec)
    batch = wl.make_batch(spec, ctx_lens=base.ctx_lens, k=np.zeros(16, np.int32))
    cache = wl.make_attention_inputs(spec, batch, device="cuda")
    ad = wl.make_adapter_inputs(spec, batch, device="cuda")
    step = DraftStep(batch, cache, ad)
    step.run()
    torch.cuda.synchronize()
    outs = lambda: [t.clone() for t in (step.x, step.o, step.logits, step.stats, step.tokens, step.conf, step.status)]
    ref = outs()
    step.capture()
    for i in range(3):
        for t in (step.x, step.o, step.logits, step.stats, step.conf):
            t.zero_()
        step.tokens.fill_(-7)
        step.status.fill_(-7)
        torch.cuda.synchronize()
        step.replay()
        torch.cuda.synchronize()
        got = outs()
        for a, b in zip(got, ref):
            assert torch.equal(a, b), i
        say(f"[draft graph] replay {i}: equal to the eager step")
