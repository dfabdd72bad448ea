"""Benchmark of the speculative verification step on one MI355X.

A step is one pass of the whole hot path over one synthetic batch already resident in HBM:
spexis_append_kv -> spexis_verify_attention -> spexis_accept (logits mode, temperature as
the workload sets).  Throughput is verified tokens per second: sum_b (a_b + 1) emitted tokens
(accepted drafts plus the resampled or bonus token) over the step time.

Prints ONE JSON line.  Also reports the attention kernel against the HBM roofline (algorithmic
bytes over its event-timed duration) and the CPU oracle timed on the host cores.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 2] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "verified tokens/sec (verify-attn + accept) at 1 GPU; achieved HBM GB/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attention_bytes(batch, spec) -> int:
    """Algorithmic bytes of one verify-attention launch: every cached K and V element once,
    Q in and O out once, and the block-table entries the sequences use."""
    D, hkv, hq = spec.head_dim, spec.num_kv_heads, spec.num_q_heads
    kv = int(batch.seq_lens.astype(np.int64).sum()) * hkv * D * 2 * 2
    qo = batch.T * hq * D * 2 * 2
    tables = int(((batch.seq_lens + spec.block_size - 1) // spec.block_size).sum()) * 4
    return kv + qo + tables


def attention_flops(batch, spec) -> int:
    D, hq = spec.head_dim, spec.num_q_heads
    f = 0
    for b in range(batch.B):
        n, L = int(batch.k[b]) + 1, int(batch.ctx_lens[b])
        f += hq * 4 * D * sum(L + j + 1 for j in range(n))
    return f


def cpu_baseline(spec, batch, attn, acc, min_seconds=10.0, max_reps=40):
    """Time the oracle on the whole step (attention of every sequence, softmax of every target
    and draft row, acceptance) on the host cores; returns the verified tokens/s it reaches."""
    import oracle
    from paper_2609_34370_amd.step import bf16_to_u16

    kp, vp = bf16_to_u16(attn.k_pool).copy(), bf16_to_u16(attn.v_pool).copy()
    q = bf16_to_u16(attn.q)
    nk, nv = bf16_to_u16(attn.new_k), bf16_to_u16(attn.new_v)
    tl, dl = acc.target_logits.cpu().numpy(), acc.draft_logits.cpu().numpy()
    ids, ua, us = acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(), acc.u_sample.cpu().numpy()
    scale = float(np.float32(1.0 / math.sqrt(spec.head_dim)))
    reps, emitted, t_total = 0, 0, 0.0
    while reps < max_reps and (reps == 0 or t_total < min_seconds):
        t0 = time.perf_counter()
        oracle.append_kv(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                         batch.seq_lens, batch.block_tables, nk, nv)
        oracle.attention(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                         batch.seq_lens, batch.block_tables, q, spec.num_q_heads, scale)
        p = oracle.softmax(tl, acc.temperature)
        qq = oracle.softmax(dl, acc.temperature)
        a, _, _, _ = oracle.accept(batch.qsl, p, qq, ids, ua, us, max_k=batch.max_k)
        t_total += time.perf_counter() - t0
        emitted += int((a.astype(np.int64) + 1).sum())
        reps += 1
    return {"value": round(emitted / t_total, 2), "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"the full {spec.name} step ({batch.B} sequences: append, fp64 attention, fp64 softmax of "
                      f"{batch.T}+{batch.T - batch.B} rows, exact acceptance) x{reps}, {t_total:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--kv-chunk", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="first copy BYTES device-to-device 3 times (a known-size kernel for counter calibration)")
    ap.add_argument("--ingest-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic.json from two rocprofv3 --pmc counter_collection.csv files "
                         "(FETCH_SIZE, WRITE_SIZE) of runs with --copy-probe N (pass the same N); needs no GPU")
    ap.add_argument("--component", choices=["step", "lm_head", "select", "lookahead", "draft"], default="step",
                    help="lm_head: time spexis_lm_head and acceptance from its fused statistics at the "
                         "workload's shape instead of the verification step; select: time selective "
                         "speculation and measure the acceptance rate of the kept drafts; lookahead: time "
                         "Algorithm 1's memory estimate; draft: time one drafting step (each prints its own "
                         "JSON line)")
    ap.add_argument("--alpha", type=float, nargs="+", default=[0.15, 0.3])
    args = ap.parse_args()
    if args.component == "lm_head":
        return bench_lm_head(args)
    if args.component == "select":
        return bench_select(args)
    if args.component == "lookahead":
        return bench_lookahead(args)
    if args.component == "draft":
        return bench_draft(args)
    if args.ingest_traffic:
        if args.copy_probe <= 0:
            raise SystemExit("--ingest-traffic needs --copy-probe N: the copy size the counter runs used")
        ingest_traffic(*args.ingest_traffic, workload=args.workload, copy_bytes=args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_34370_amd import spexis as sx
    from paper_2609_34370_amd import workloads as wl
    from paper_2609_34370_amd.step import VerifyStep

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    spec = wl.WORKLOADS[args.workload]
    log(f"[bench] workload {spec.wid} ({spec.name}): generating inputs on the GPU")
    batch = wl.make_batch(spec, seed=args.seed)
    attn = wl.make_attention_inputs(spec, batch, device="cuda", seed=args.seed)
    acc = wl.make_accept_inputs(spec, batch, device="cuda", seed=args.seed)
    torch.cuda.synchronize()
    # host copies for the oracle baseline are taken before the GPU appends (same bytes it saw)
    baseline_inputs = None
    if not args.no_cpu_baseline:
        baseline_inputs = wl.AttentionInputs(attn.k_pool.cpu(), attn.v_pool.cpu(), attn.q.cpu(), attn.new_k.cpu(),
                                             attn.new_v.cpu())
    step = VerifyStep(batch, attn, acc, kv_chunk_tokens=args.kv_chunk, kind=sx.SPEXIS_INPUT_LOGITS)
    stream = torch.cuda.current_stream()
    if args.copy_probe > 0:
        src = torch.empty(args.copy_probe, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()

    K = args.steps
    # Timed region: exactly K whole steps, nothing recorded between the calls.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step.run()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    # Per-phase durations: K more steps with HIP events on the launch stream around each call
    # (an event record idles the stream for a few microseconds, so these steps are not the
    # ones `value` is computed from).
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        ev[i][0].record(stream)
        step.append()
        ev[i][1].record(stream)
        step.attention()
        ev[i][2].record(stream)
        step.accept()
        ev[i][3].record(stream)
    torch.cuda.synchronize()

    a, toks, status = step.accept_outputs()
    emitted = int((a.astype(np.int64) + 1).sum())
    ms_append = float(np.mean([ev[i][0].elapsed_time(ev[i][1]) for i in range(K)]))
    ms_attn = float(np.mean([ev[i][1].elapsed_time(ev[i][2]) for i in range(K)]))
    ms_accept = float(np.mean([ev[i][2].elapsed_time(ev[i][3]) for i in range(K)]))
    ms_step = elapsed * 1e3 / K
    value = emitted / (ms_step * 1e-3)
    abytes = attention_bytes(batch, spec)
    achieved = abytes / (ms_attn * 1e-3) / 1e9
    log(f"[bench] append {ms_append * 1e3:.1f} us  attention {ms_attn * 1e3:.1f} us  accept {ms_accept * 1e3:.1f} us"
        f"  step {ms_step * 1e3:.1f} us  emitted {emitted}/step  accepted mean {a.mean():.3f}  status!=0 "
        f"{int((status != 0).sum())}")
    log(f"[bench] attention {abytes / 1e9:.3f} GB algorithmic -> {achieved:.0f} GB/s "
        f"({achieved / HBM_PEAK_GBS:.1%} of 8 TB/s); {attention_flops(batch, spec) / (ms_attn * 1e-3) / 1e12:.1f} "
        f"TFLOP/s")

    cpu = None
    if baseline_inputs is not None and int(os.environ.get("RANK", "0")) == 0:
        log("[bench] timing the CPU oracle on the host cores")
        cpu = cpu_baseline(spec, batch, baseline_inputs, acc)
        log(f"[bench] oracle: {cpu}")

    traffic = None
    prof = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(prof):
        with open(prof) as f:
            t = json.load(f).get(f"workload{spec.wid}")
        if t and t.get("source_digest") == _kernel_digest():
            traffic = t["bytes_per_launch"]

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": spec.name, "batch": batch.B, "q_heads": spec.num_q_heads,
                   "kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim, "block_size": spec.block_size,
                   "context": list(spec.ctx), "draft_tokens": list(spec.k), "vocab": spec.vocab,
                   "temperature": spec.temperature, "accept_input": "logits", "parallelism": "none"},
        "phases_us": {"append": round(ms_append * 1e3, 2), "verify_attention": round(ms_attn * 1e3, 2),
                      "accept": round(ms_accept * 1e3, 2)},
        "emitted_tokens_per_step": emitted,
        "roofline": {"bound": "hbm", "kernel": "spexis_verify_attention", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": abytes},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


MFMA_BF16_TFLOPS = 2500.0


def bench_lm_head(args):
    """The LM head in front of acceptance (logits = h W^T with fused statistics) at the workload's
    target rows, then acceptance from those statistics against acceptance that computes its own.
    Synthetic bf16 weights; every input is resident in HBM before timing."""
    import torch

    from paper_2609_34370_amd import spexis as sx
    from paper_2609_34370_amd import workloads as wl
    from paper_2609_34370_amd.step import VerifyStep

    spec = wl.WORKLOADS[args.workload]
    batch = wl.make_batch(spec, seed=args.seed)
    attn = wl.make_attention_inputs(spec, batch, device="cuda", seed=args.seed)
    acc = wl.make_accept_inputs(spec, batch, device="cuda", seed=args.seed)
    d, V, T = wl.HIDDEN[spec.wid], spec.vocab, batch.T
    g = torch.Generator(device="cuda").manual_seed(260934370)
    h = torch.randn((T, d), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((V, d), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    tiles = sx.spexis_lm_head_tiles(V)
    logits = torch.empty((T, V), dtype=torch.float32, device="cuda")
    stats = torch.empty((T, tiles, 2), dtype=torch.float32, device="cuda")
    dstats = torch.empty((batch.T - batch.B, tiles, 2), dtype=torch.float32, device="cuda")
    temp = acc.temperature

    def timed(fn, steps, warmup):
        for _ in range(warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / steps   # us

    w = sx.spexis_pack_weight(w)   # once per weight, outside the timed region
    us_lm = timed(lambda: sx.spexis_lm_head(h, w, stats, logits=logits, temperature=temp), args.steps, args.warmup)
    us_lm_stats = timed(lambda: sx.spexis_lm_head(h, w, stats, temperature=temp, vocab=V), args.steps, args.warmup)
    # Acceptance on logits this LM head produced: target rows from h, draft rows from h plus
    # noise (a draft model sharing the head), drafts drawn from the draft rows (input generation,
    # untimed).  Timed: acceptance computing its own statistics, and from the fused ones.
    step = VerifyStep(batch, attn, acc)
    rows_d = torch.as_tensor(np.concatenate([np.arange(batch.qsl[b], batch.qsl[b] + batch.k[b])
                                             for b in range(batch.B)]).astype(np.int64), device="cuda")
    hd = (h.float()[rows_d] + 0.3 * torch.randn((len(rows_d), d), generator=g, device="cuda")).to(torch.bfloat16)
    dlogits = torch.empty((len(rows_d), V), dtype=torch.float32, device="cuda")
    sx.spexis_lm_head(h, w, stats, logits=logits, temperature=temp)
    sx.spexis_lm_head(hd, w, dstats, logits=dlogits, temperature=temp)
    ids = torch.multinomial(torch.softmax(dlogits / temp, dim=1), 1, generator=g).view(-1).to(torch.int32)
    torch.cuda.synchronize()
    run_own = lambda: sx.spexis_accept(sx.SPEXIS_INPUT_LOGITS, step.qsl, logits, dlogits, ids, acc.u_accept,
                                       acc.u_sample, batch.max_k, step.accepted_len, step.out_tokens,
                                       step.row_status, step.acc_ws, temperature=temp)
    run_fused = lambda: sx.spexis_accept_with_stats(step.qsl, logits, dlogits, stats, dstats, ids, acc.u_accept,
                                                    acc.u_sample, batch.max_k, step.accepted_len,
                                                    step.out_tokens, step.row_status, step.acc_ws,
                                                    temperature=temp)
    us_acc = timed(run_own, args.steps, args.warmup)
    a_own = step.accepted_len.cpu().numpy().copy()
    us_acc_stats = timed(run_fused, args.steps, args.warmup)
    a_fused = step.accepted_len.cpu().numpy()
    log(f"[lm_head] accepted mean {a_own.mean():.3f} (own statistics) / {a_fused.mean():.3f} (fused); "
        f"decisions differ on {int((a_own != a_fused).sum())} of {batch.B} sequences")
    wbytes, hbytes, lbytes, sbytes = V * d * 2, T * d * 2, T * V * 4, T * tiles * 8
    flops = 2.0 * T * V * d
    gbs = (wbytes + hbytes + lbytes + sbytes) / (us_lm * 1e-6) / 1e9
    tfl = flops / (us_lm * 1e-6) / 1e12
    line = {
        "component": "spexis_lm_head", "workload": spec.name, "rows": T, "hidden": d, "vocab": V,
        "us": round(us_lm, 2), "us_stats_only": round(us_lm_stats, 2),
        "hbm": {"achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                "bytes": wbytes + hbytes + lbytes + sbytes},
        "mfma": {"achieved": round(tfl, 1), "peak": MFMA_BF16_TFLOPS, "unit": "TFLOP/s",
                 "frac": round(tfl / MFMA_BF16_TFLOPS, 4), "flops": flops},
        "accept_us": round(us_acc, 2), "accept_with_stats_us": round(us_acc_stats, 2),
        "dtype": "bf16", "data": "synthetic",
    }
    log(f"[lm_head] {T}x{d} @ {V}x{d}: {us_lm:.1f} us ({us_lm_stats:.1f} us without logits) -> {gbs:.0f} GB/s "
        f"({gbs / HBM_PEAK_GBS:.1%}), {tfl:.0f} TFLOP/s ({tfl / MFMA_BF16_TFLOPS:.1%}); accept {us_acc:.1f} us, "
        f"with given statistics {us_acc_stats:.1f} us")
    print(json.dumps(line), flush=True)


PIPE_STAGES = 4   # pipeline stages of the Eq. 3-4 model in the select component


def bench_select(args):
    """Selective speculation at the workload's batch: latency of spexis_select_drafts, and the
    speculation accuracy of the drafts it keeps.  Confidences are the draft probabilities of the
    drawn drafts, q_i(x_i), from the workload's synthetic draft rows.  A kept set is a prefix of
    each sequence's drafts and acceptance is sequential, so the kept drafts of sequence b that
    verification accepts number min(a_b, kept_k_b), where a_b is the accepted length over all
    drafts: Theta_alpha = sum_b min(a_b, kept_k_b) / sum_b kept_k_b against Theta = sum a_b / sum k_b."""
    import torch

    from paper_2609_34370_amd import schedule
    from paper_2609_34370_amd import spexis as sx
    from paper_2609_34370_amd import workloads as wl
    from paper_2609_34370_amd.step import VerifyStep

    spec = wl.WORKLOADS[args.workload]
    batch = wl.make_batch(spec, seed=args.seed)
    attn = wl.make_attention_inputs(spec, batch, device="cuda", seed=args.seed)
    acc = wl.make_accept_inputs(spec, batch, device="cuda", seed=args.seed)
    step = VerifyStep(batch, attn, acc, kind=sx.SPEXIS_INPUT_LOGITS)
    step.accept()
    a = step.accept_outputs()[0].astype(np.int64)
    q = torch.softmax(acc.draft_logits / acc.temperature, dim=1)
    conf = q.gather(1, acc.draft_ids.long().view(-1, 1)).view(-1).contiguous()
    B, N = batch.B, batch.T - batch.B
    kept_k = torch.empty(B, dtype=torch.int32, device="cuda")
    kept_qsl = torch.empty(B + 1, dtype=torch.int32, device="cuda")
    keep = torch.empty(max(N, 1), dtype=torch.int32, device="cuda")
    k = batch.k.astype(np.int64)
    theta = float(np.minimum(a, k).sum() / max(k.sum(), 1))

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / args.steps

    rows = []
    for alpha in args.alpha:
        us = timed(lambda: sx.spexis_select_drafts(step.qsl, conf, alpha, kept_k, kept_qsl, keep[:N]))
        kk = kept_k.cpu().numpy().astype(np.int64)
        theta_a = float(np.minimum(a, kk).sum() / max(kk.sum(), 1))
        # Eq. 3-4 with the measured accuracies, for a 4-stage pipeline and this batch
        b_eff0 = schedule.effective_batch(B, 0.0, PIPE_STAGES, theta)
        b_eff = schedule.effective_batch(B, alpha, PIPE_STAGES, theta_a)
        rows.append({"alpha": alpha, "us": round(us, 2), "kept_drafts": int(kk.sum()), "drafts": int(N),
                     "theta": round(theta, 4), "theta_alpha": round(theta_a, 4),
                     "accepted_kept": int(np.minimum(a, kk).sum()), "accepted_all": int(np.minimum(a, k).sum()),
                     "pipeline_stages": PIPE_STAGES,
                     "steady_batch": round(schedule.steady_batch(B, alpha, PIPE_STAGES), 2),
                     "effective_batch": round(b_eff, 2), "effective_batch_no_drop": round(b_eff0, 2)})
        log(f"[select] alpha={alpha}: {us:.1f} us; kept {kk.sum()}/{N} drafts; theta {theta:.4f} -> "
            f"theta_alpha {theta_a:.4f}; accepted {np.minimum(a, kk).sum()}/{np.minimum(a, k).sum()}; "
            f"Eq. 4 effective batch {b_eff0:.1f} -> {b_eff:.1f} (N={PIPE_STAGES})")
    # the largest supported batch: 1024 sequences x 16 drafts
    qsl_max = torch.arange(0, 17 * 1025, 17, dtype=torch.int32, device="cuda")
    conf_max = torch.rand(16384, generator=torch.Generator(device="cuda").manual_seed(1), device="cuda")
    km, kqm, keepm = (torch.empty(1024, dtype=torch.int32, device="cuda"),
                      torch.empty(1025, dtype=torch.int32, device="cuda"),
                      torch.empty(16384, dtype=torch.int32, device="cuda"))
    us_max = timed(lambda: sx.spexis_select_drafts(qsl_max, conf_max, 0.3, km, kqm, keepm))
    log(f"[select] 16384 drafts (1024 x 16): {us_max:.1f} us")
    print(json.dumps({"component": "spexis_select_drafts", "workload": spec.name, "batch": B, "drafts": N,
                      "alphas": rows, "us_16384_drafts": round(us_max, 2), "data": "synthetic"}), flush=True)


def bench_lookahead(args):
    """Algorithm 1's look-ahead memory estimate over 64 iterations for running batches of the
    workload's size and larger (request lengths from the workload's context distribution,
    remaining lengths on the ordinal thresholds, precision 0.83, depth 4, theta 0.7)."""
    import torch

    from paper_2609_34370_amd import spexis as sx
    from paper_2609_34370_amd import workloads as wl

    spec = wl.WORKLOADS[args.workload]
    rows = []
    for n in (spec.batch, 4096, 65536):
        rng = np.random.default_rng(n)
        batch = wl.make_batch(wl.spec_with(spec.wid, batch=min(n, spec.batch)), seed=args.seed)
        ell = torch.as_tensor(np.resize(batch.ctx_lens.astype(np.int64), n), device="cuda")
        tau = torch.as_tensor(rng.choice(np.array([4, 8, 16, 32, 64, 1 << 30], np.int32), n), device="cuda")
        prec = torch.where(tau < (1 << 30), 0.83, 0.0).to(torch.float64)
        mem = torch.empty(64, dtype=torch.float64, device="cuda")
        call = lambda: sx.spexis_lookahead_memory(ell, tau, prec, 4, 0.7, mem)
        for _ in range(args.warmup):
            call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            call()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / args.steps
        m = mem.cpu().numpy()
        rows.append({"requests": n, "us": round(us, 2), "mem_1": round(float(m[0]), 1), "mem_64": round(float(m[63]), 1)})
        log(f"[lookahead] {n} requests: {us:.1f} us per call; estimate {m[0]:.0f} -> {m[63]:.0f} tokens")
    print(json.dumps({"component": "spexis_lookahead_memory", "workload": spec.name, "iters": 64, "pp": 4,
                      "theta": 0.7, "runs": rows, "data": "synthetic"}), flush=True)


def bench_draft(args):
    """One drafting step at the workload's batch (one draft token per sequence): adapter linear
    and q/k/v projections, append and attention over the adapter's paged cache (contexts of the
    workload), output projection with residual, LM head with fused statistics, draft draw.
    Synthetic bf16 weights; inputs resident in HBM.  Per phase: HIP events on the stream."""
    import torch

    from paper_2609_34370_amd import workloads as wl
    from paper_2609_34370_amd.draft import DraftStep

    spec = wl.WORKLOADS[args.workload]
    base = wl.make_batch(spec, seed=args.seed)
    batch = wl.make_batch(spec, seed=args.seed, ctx_lens=base.ctx_lens, k=np.zeros(base.B, np.int32))
    cache = wl.make_attention_inputs(spec, batch, device="cuda", seed=args.seed)
    ad = wl.make_adapter_inputs(spec, batch, device="cuda", seed=args.seed)
    step = DraftStep(batch, cache, ad)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step.run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    # the same step replayed from a HIP graph: no host work between its kernels
    step.capture()
    for _ in range(args.warmup):
        step.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step.replay()
    torch.cuda.synchronize()
    ms_graph = (time.perf_counter() - t0) * 1e3 / args.steps
    phases = (("adapter_in", step.adapter_in), ("attention", step.attention), ("adapter_out", step.adapter_out),
              ("lm_head", step.lm_head), ("sample", step.sample))
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(phases) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        ev[i][0].record(stream)
        for j, (_, fn) in enumerate(phases):
            fn()
            ev[i][j + 1].record(stream)
    torch.cuda.synchronize()
    us = {name: float(np.mean([ev[i][j].elapsed_time(ev[i][j + 1]) for i in range(args.steps)])) * 1e3
          for j, (name, _) in enumerate(phases)}
    B, d, V = batch.B, ad.h.shape[1], spec.vocab
    hq, hkv, D = spec.num_q_heads, spec.num_kv_heads, spec.head_dim
    w_bytes = {"adapter_in": (d * d + (hq + 2 * hkv) * D * d) * 2, "adapter_out": d * hq * D * 2,
               "lm_head": V * d * 2 + B * V * 4}
    kv_bytes = int(batch.seq_lens.astype(np.int64).sum()) * hkv * D * 2 * 2
    total = sum(w_bytes.values()) + kv_bytes
    lm_gbs = w_bytes["lm_head"] / (us["lm_head"] * 1e-6) / 1e9
    at_gbs = kv_bytes / (us["attention"] * 1e-6) / 1e9
    tok = step.tokens.cpu().numpy()
    conf = step.conf.cpu().numpy()
    log(f"[draft] {spec.name}: step {ms * 1e3:.1f} us ({ms_graph * 1e3:.1f} us replayed from a graph); "
        + ", ".join(f"{k} {v:.1f} us" for k, v in us.items()))
    log(f"[draft] LM head {w_bytes['lm_head'] / 1e9:.3f} GB -> {lm_gbs:.0f} GB/s ({lm_gbs / HBM_PEAK_GBS:.1%}); "
        f"attention {kv_bytes / 1e9:.3f} GB -> {at_gbs:.0f} GB/s; whole step {total / 1e9:.3f} GB -> "
        f"{total / (ms * 1e-3) / 1e9:.0f} GB/s; confidence median {np.median(conf):.2e}")
    print(json.dumps({"component": "draft_step", "workload": spec.name, "batch": B, "hidden": d, "vocab": V,
                      "us_per_step": round(ms * 1e3, 2), "us_per_step_graph": round(ms_graph * 1e3, 2),
                      "phases_us": {k: round(v, 2) for k, v in us.items()},
                      "draft_tokens_per_s": round(B / (ms * 1e-3), 1),
                      "draft_tokens_per_s_graph": round(B / (ms_graph * 1e-3), 1),
                      "lm_head": {"bytes": w_bytes["lm_head"], "achieved": round(lm_gbs, 1), "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "frac": round(lm_gbs / HBM_PEAK_GBS, 4)},
                      "attention": {"bytes": kv_bytes, "achieved": round(at_gbs, 1), "unit": "GB/s"},
                      "bytes_per_step": total, "valid_tokens": int((tok >= 0).sum()), "data": "synthetic"}),
          flush=True)


ATTN_KERNELS = ("verify_attn_kernel", "attn_merge_kernel")   # the launches of spexis_verify_attention
COPY_KERNEL = "copyBuffer"


def ingest_traffic(fetch_csv: str, write_csv: str, workload: int, copy_bytes: int) -> None:
    """HBM bytes per spexis_verify_attention call from two counter runs of
    `bench.py --copy-probe N`: each counter's KiB per dispatch, summed over the call's kernels,
    averaged over the dispatches, and scaled by N / (the counter's reading for one copy of N
    bytes), so that a plain copy reads and writes exactly N bytes."""
    import csv

    def per_kernel(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        out = {}
        for r in rows:
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return out

    result = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        k = per_kernel(path, name)
        copies = [v for n, vals in k.items() if COPY_KERNEL in n for v in vals]
        if not copies:
            raise SystemExit(f"{path}: no {COPY_KERNEL} dispatch; run the profile with --copy-probe N")
        probe = max(copies)   # the 3 probe copies are the largest copies of the run
        size = copy_bytes
        factor = size / probe
        attn = sum(float(np.mean(vals)) for n, vals in k.items() if any(a in n for a in ATTN_KERNELS))
        result[name] = {"raw_bytes_per_call": attn, "copy_reading": probe, "copy_bytes": size,
                        "factor": factor, "bytes_per_call": attn * factor}
    total = result["FETCH_SIZE"]["bytes_per_call"] + result["WRITE_SIZE"]["bytes_per_call"]
    prof = os.path.join(ROOT, "profiles", "traffic.json")
    data = json.load(open(prof)) if os.path.exists(prof) else {}
    data[f"workload{workload}"] = {"source_digest": _kernel_digest(), "bytes_per_launch": round(total),
                                   "counters": result, "kernels": list(ATTN_KERNELS)}
    with open(prof, "w") as f:
        json.dump(data, f, indent=1)
        f.write("\n")
    print(json.dumps(data[f"workload{workload}"], indent=1))


def _kernel_digest() -> str:
    """Digest of the sources the attention kernels are built from (their code, the shared device
    helpers, and the header with their parameters and launch constants): a stored traffic figure
    is used only while they are unchanged."""
    import hashlib
    h = hashlib.sha256()
    for name in ("attention.hip", "common.h", "kernels.h"):
        with open(os.path.join(ROOT, "paper_2609_34370_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
