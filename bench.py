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
PHASE_STEPS = 100           # event-timed steps per phase pass (at least; more when --steps is larger)
MFMA_BF16_TFLOPS = 2500.0   # dense bf16 matrix-core peak of the MI355X
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
    and draft row, acceptance) on the host cores; returns (the baseline record, the oracle's
    accepted lengths and tokens).  For the two smallest workloads the oracle is also timed on
    one thread."""
    import oracle
    from paper_2609_34370_amd.step import bf16_to_u16

    kp, vp = bf16_to_u16(attn.k_pool).copy(), bf16_to_u16(attn.v_pool).copy()
    q = bf16_to_u16(attn.q)
    nk, nv = bf16_to_u16(attn.new_k), bf16_to_u16(attn.new_v)
    tl, dl = acc.target_logits.cpu().numpy(), acc.draft_logits.cpu().numpy()
    ids, ua, us = acc.draft_ids.cpu().numpy(), acc.u_accept.cpu().numpy(), acc.u_sample.cpu().numpy()
    scale = float(np.float32(1.0 / math.sqrt(spec.head_dim)))

    def one_step():
        oracle.append_kv(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                         batch.seq_lens, batch.block_tables, nk, nv)
        oracle.attention(kp, vp, batch.num_blocks, spec.num_kv_heads, spec.block_size, spec.head_dim, batch.qsl,
                         batch.seq_lens, batch.block_tables, q, spec.num_q_heads, scale)
        p = oracle.softmax(tl, acc.temperature)
        qq = oracle.softmax(dl, acc.temperature)
        return oracle.accept(batch.qsl, p, qq, ids, ua, us, max_k=batch.max_k)

    def timed(min_s, max_r):
        reps, emitted, t_total, out = 0, 0, 0.0, None
        while reps < max_r and (reps == 0 or t_total < min_s):
            t0 = time.perf_counter()
            out = one_step()
            t_total += time.perf_counter() - t0
            emitted += int((out[0].astype(np.int64) + 1).sum())
            reps += 1
        return emitted / t_total, reps, t_total, out

    threads = oracle.num_threads()
    value, reps, t_total, out = timed(min_seconds, max_reps)
    rec = {"value": round(value, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"the full {spec.name} step ({batch.B} sequences: append, fp64 attention, fp64 softmax of "
                     f"{batch.T}+{batch.T - batch.B} rows, exact acceptance) x{reps}, {t_total:.1f} s",
           "cpu_model": cpu_model()}
    if spec.wid in (1, 2):
        oracle.set_num_threads(1)
        try:
            v1, r1, t1, _ = timed(5.0, 3)
        finally:
            oracle.set_num_threads(threads)
        rec["one_thread"] = {"value": round(v1, 2), "unit": "tokens/s", "reps": r1, "seconds": round(t1, 2)}
    return rec, (out[0], out[1])


def accept_bytes(batch, spec, accepted) -> int:
    """Algorithmic bytes of one logits-mode acceptance: the normalisers of target and draft rows
    0..a_b (test i needs both of row i's), 4V (a_b + 1) + 4V min(a_b + 1, k_b), plus the sampled
    row(s) read again for the fixed-point sums: target and draft row a_b for a residual (8V),
    target row k_b for the bonus token (4V)."""
    V = spec.vocab
    total = 0
    for b in range(batch.B):
        a, k = int(accepted[b]), int(batch.k[b])
        total += 4 * V * (a + 1) + 4 * V * min(a + 1, k)
        total += 8 * V if a < k else 4 * V
    return total


def pct(xs):
    xs = np.asarray(xs, dtype=np.float64)
    return {"mean": round(float(xs.mean()), 2), "median": round(float(np.median(xs)), 2),
            "p10": round(float(np.percentile(xs, 10)), 2), "p90": round(float(np.percentile(xs, 90)), 2)}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _read_probe():
    """The read probes of libspexis_probe.so (coalesced 16-byte loads, strided or in chunks)."""
    import ctypes
    from paper_2609_34370_amd import build as _b
    probe = ctypes.CDLL(_b.PROBE_LIB_PATH)
    probe.spexis_probe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                                               ctypes.c_void_p]
    probe.spexis_probe_stream_read.restype = ctypes.c_int
    probe.spexis_probe_chunk_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int64,
                                              ctypes.c_void_p, ctypes.c_void_p]
    probe.spexis_probe_chunk_read.restype = ctypes.c_int
    return probe


SETTLE_MS = 60.0


def settle(torch, fn, ms=SETTLE_MS):
    """Runs `fn` back to back for `ms` milliseconds before it is timed.  After input generation or
    an idle spell this GPU takes some 40 ms of load to reach its clocks: the first 20 calls of a
    compute-bound kernel ran up to 15% slower than later ones (an LM head at 320 x 4096 @ 128256:
    431 us, then 400, 394, 379, 371, and 368-370 us from then on), while the verification step,
    memory-bound, settled within its warmup and ran slower after a longer sustained load (phase
    times 149 against 145 us of attention after 200 ms of load).  So the component timings settle
    on their own call for this long, and the step bench keeps its W warmup steps only."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < ms * 1e-3:
        for _ in range(4):
            fn()
        torch.cuda.synchronize()


def stream_peaks(torch, nbytes=4 << 30, reps=5):
    """Measured HBM rates on this GPU: the read probes of libspexis_probe.so over a 4 GiB
    buffer (coalesced 16-byte non-temporal loads, grid-strided or in contiguous chunks per
    workgroup; the best pattern, grid and repetition is `read`, each pattern's best is reported
    too) and torch's device copy (bytes read plus bytes written per second)."""
    import ctypes
    probe = _read_probe()
    src = torch.zeros(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    sink = torch.empty(8192 * 256, dtype=torch.int32, device="cuda")
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def best(fn):
        fn()
        t = float("inf")
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t = min(t, e0.elapsed_time(e1) * 1e-3)
        return t

    def read(grid):
        rc = probe.spexis_probe_stream_read(ctypes.c_void_p(src.data_ptr()), nbytes, grid,
                                            ctypes.c_void_p(sink.data_ptr()), s)
        if rc != 0:
            raise RuntimeError(f"stream probe failed: {rc}")

    def chunks(grid, chunk):
        rc = probe.spexis_probe_chunk_read(ctypes.c_void_p(src.data_ptr()), nbytes, grid, chunk,
                                           ctypes.c_void_p(sink.data_ptr()), s)
        if rc != 0:
            raise RuntimeError(f"stream probe failed: {rc}")

    strided = max(nbytes / best(lambda g=g: read(g)) / 1e9 for g in (1024, 2048, 4096, 8192))
    chunked = max(nbytes / best(lambda g=g, c=c: chunks(g, c)) / 1e9
                  for g in (2048, 4096) for c in (64 << 10, 1 << 20))
    out = {"read": round(max(strided, chunked), 1), "read_strided": round(strided, 1),
           "read_chunked": round(chunked, 1), "copy": round(2 * nbytes / best(lambda: dst.copy_(src)) / 1e9, 1)}
    del src, dst, sink
    torch.cuda.empty_cache()
    return out


def clone_step(step_cls, batch, attn, acc, kv_chunk, kind, wl):
    """A VerifyStep over fresh copies of the inputs (same bytes, different HBM addresses)."""
    a2 = wl.AttentionInputs(attn.k_pool.clone(), attn.v_pool.clone(), attn.q.clone(), attn.new_k.clone(),
                            attn.new_v.clone())
    c2 = wl.AcceptInputs(acc.target_logits.clone(), acc.draft_logits.clone(), acc.draft_ids.clone(),
                         acc.u_accept.clone(), acc.u_sample.clone(), acc.temperature)
    return step_cls(batch, a2, c2, kv_chunk_tokens=kv_chunk, kind=kind)


def phase_pass(torch, steps, K, stream, flush=None):
    """Per-phase HIP-event durations (us) of K steps, step i on steps[i % len(steps)]; with
    `flush`, that function runs before every step, outside the events."""
    names = ("append", "verify_attention", "accept")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        st = steps[i % len(steps)]
        if flush is not None:
            flush()
        ev[i][0].record(stream)
        st.append()
        ev[i][1].record(stream)
        st.attention()
        ev[i][2].record(stream)
        st.accept()
        ev[i][3].record(stream)
    torch.cuda.synchronize()
    return {n: [ev[i][j].elapsed_time(ev[i][j + 1]) * 1e3 for i in range(K)] for j, n in enumerate(names)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--kv-chunk", type=int, default=0)
    ap.add_argument("--graph", action="store_true",
                    help="replay each input copy's step from a HIP graph (captured before timing) in the timed "
                         "loops, instead of launching its calls one by one")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="first copy BYTES device-to-device 3 times (a known-size kernel for counter calibration); "
                         "skips the flushed pass and the stream-rate probe, whose copies would be confused with it")
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
    kind = sx.SPEXIS_INPUT_LOGITS
    step = VerifyStep(batch, attn, acc, kv_chunk_tokens=args.kv_chunk, kind=kind)
    # Cold steps: R copies of every input, used in turn, so that between two uses of one copy the
    # other copies' steps stream at least 1 GiB through HBM; neither the 256 MB last-level cache
    # nor the L2s can still hold a step's data.  Warm steps reuse one copy back to back.
    abytes = attention_bytes(batch, spec)
    R = 1 + min(7, max(1, -(-(1 << 30) // abytes)))   # tiny workloads: 8 copies, still far under 1 GiB
    steps = [step] + [clone_step(VerifyStep, batch, attn, acc, args.kv_chunk, kind, wl) for _ in range(R - 1)]
    stream = torch.cuda.current_stream()
    if args.copy_probe > 0:
        src = torch.empty(args.copy_probe, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.graph:
        for st in steps:
            st.capture()
    go = [st.replay if args.graph else st.run for st in steps]
    for i in range(args.warmup):
        go[i % R]()
    torch.cuda.synchronize()

    K = args.steps
    # Timed region (the headline): exactly K whole cold steps, nothing recorded between calls.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        go[i % R]()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # The same K steps warm (one copy of the inputs, back to back), beside the headline.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        go[0]()
    torch.cuda.synchronize()
    elapsed_warm = time.perf_counter() - t0

    # Per-phase durations: max(K, 100) more steps with HIP events on the launch stream around each call
    # (an event record idles the stream for a few microseconds, so these steps are not the ones
    # `value` is computed from): cold as in the timed region, warm, and after a 1 GiB read
    # (a reduction over a scratch buffer: it leaves no dirty lines to write back) before every step.
    KP = max(K, PHASE_STEPS)
    cold = phase_pass(torch, steps, KP, stream)
    warm = phase_pass(torch, [step], KP, stream)
    flushed = None
    if args.copy_probe == 0:
        fa = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        flushed = phase_pass(torch, [step], KP, stream, flush=lambda: fa.sum())
        del fa
        torch.cuda.empty_cache()
    # the read-rate probe (not in counter runs: its copies would be taken for the calibration's)
    peaks = stream_peaks(torch) if args.copy_probe == 0 else None

    a, toks, status = step.accept_outputs()
    # every input copy that ran decided the same (with fewer steps than copies, some never ran)
    for other in steps[1:min(R, max(args.warmup, K))]:
        a2, t2, s2 = other.accept_outputs()
        assert np.array_equal(a, a2) and np.array_equal(toks, t2) and np.array_equal(status, s2)
    emitted = int((a.astype(np.int64) + 1).sum())
    ms_append = float(np.mean(cold["append"])) * 1e-3
    ms_attn = float(np.mean(cold["verify_attention"])) * 1e-3
    ms_accept = float(np.mean(cold["accept"])) * 1e-3
    ms_step = elapsed * 1e3 / K
    ms_step_warm = elapsed_warm * 1e3 / K
    value = emitted / (ms_step * 1e-3)
    achieved = abytes / (ms_attn * 1e-3) / 1e9
    aflops = attention_flops(batch, spec)
    acc_bytes = accept_bytes(batch, spec, a)
    acc_gbs = acc_bytes / (ms_accept * 1e-3) / 1e9
    log(f"[bench] cold: append {ms_append * 1e3:.1f} us  attention {ms_attn * 1e3:.1f} us  accept "
        f"{ms_accept * 1e3:.1f} us  step {ms_step * 1e3:.1f} us (warm {ms_step_warm * 1e3:.1f} us, {R} input copies)"
        f"  emitted {emitted}/step  accepted mean {a.mean():.3f}  status!=0 {int((status != 0).sum())}")
    log(f"[bench] attention {abytes / 1e9:.3f} GB algorithmic -> {achieved:.0f} GB/s "
        f"({achieved / HBM_PEAK_GBS:.1%} of 8 TB/s); {aflops / (ms_attn * 1e-3) / 1e12:.1f} "
        f"TFLOP/s; accept {acc_bytes / 1e9:.3f} GB algorithmic -> {acc_gbs:.0f} GB/s "
        f"({acc_gbs / HBM_PEAK_GBS:.1%}); measured stream rates {peaks}")

    cpu = None
    agreement = None
    if baseline_inputs is not None and int(os.environ.get("RANK", "0")) == 0:
        log("[bench] timing the CPU oracle on the host cores")
        cpu, ref = cpu_baseline(spec, batch, baseline_inputs, acc)
        ra, rt = ref
        same = int(sum(1 for b in range(batch.B) if a[b] == ra[b] and np.array_equal(toks[b], rt[b])))
        agreement = {"sequences": batch.B, "agree": same, "rate": round(same / batch.B, 6),
                     "what": "logits-mode accepted lengths and tokens against the oracle's exact rule on its "
                             "fp64 softmax of the same logits"}
        log(f"[bench] oracle: {cpu}; acceptance agreement {same}/{batch.B}")

    traffic = stored_traffic(spec.wid, "verify_attention")
    acc_traffic = stored_traffic(spec.wid, "accept")
    read_peak = peaks["read"] if peaks else None
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": spec.name, "batch": batch.B, "q_heads": spec.num_q_heads,
                   "kv_heads": spec.num_kv_heads, "head_dim": spec.head_dim, "block_size": spec.block_size,
                   "context": list(spec.ctx), "draft_tokens": list(spec.k), "vocab": spec.vocab,
                   "temperature": spec.temperature, "accept_input": "logits", "parallelism": "none",
                   "launch": "hip_graph" if args.graph else "eager"},
        "protocol": f"cold (headline): {R} copies of the inputs used in turn, {(R - 1) * abytes / 2**30:.2f} GiB "
                    f"of other steps' attention reads between two uses of one copy; warm: one copy back to back; "
                    f"flushed: one copy, a 1 GiB read before each step (phase times only); phase statistics "
                    f"over {KP} event-timed steps per pass",
        "warm": {"value": round(emitted / (ms_step_warm * 1e-3), 1), "ms_per_step": round(ms_step_warm, 4)},
        "phases_us": {"append": round(ms_append * 1e3, 2), "verify_attention": round(ms_attn * 1e3, 2),
                      "accept": round(ms_accept * 1e3, 2)},
        "phase_stats_us": {"cold": {k: pct(v) for k, v in cold.items()},
                           "warm": {k: pct(v) for k, v in warm.items()},
                           "flushed": {k: pct(v) for k, v in flushed.items()} if flushed else None},
        "emitted_tokens_per_step": emitted,
        "query_tokens_per_s": round(batch.T / (ms_step * 1e-3), 1),
        "attention_mfma": {"achieved": round(aflops / (ms_attn * 1e-3) / 1e12, 1), "peak": MFMA_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": round(aflops / (ms_attn * 1e-3) / 1e12 / MFMA_BF16_TFLOPS, 4),
                           "flops": aflops, "what": "the causal products of the real query rows (padding rows of "
                                                    "a 32-row tile not counted)"},
        "roofline": {"bound": "hbm", "kernel": "spexis_verify_attention", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": abytes,
                     "frac_of_measured_read": round(achieved / read_peak, 4) if read_peak else None},
        "roofline_accept": {"bound": "hbm", "kernel": "spexis_accept", "achieved": round(acc_gbs, 1),
                            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(acc_gbs / HBM_PEAK_GBS, 4),
                            "traffic": acc_traffic, "algorithmic_bytes": acc_bytes,
                            "frac_of_measured_read": round(acc_gbs / read_peak, 4) if read_peak else None},
        "stream_peak_gbs": peaks,
        "accept_agreement": agreement,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)



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
        settle(torch, fn)
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

    w_plain = w
    w = sx.spexis_pack_weight(w)   # once per weight, outside the timed region
    us_lm = timed(lambda: sx.spexis_lm_head(h, w, stats, logits=logits, temperature=temp), args.steps, args.warmup)
    us_lm_stats = timed(lambda: sx.spexis_lm_head(h, w, stats, temperature=temp, vocab=V), args.steps, args.warmup)
    # context: torch's bf16 GEMM of the same product (bf16 output, no statistics), both as
    # h W^T and as W h^T (the transposed logits), whose library kernels differ
    us_torch = timed(lambda: torch.nn.functional.linear(h, w_plain), args.steps, args.warmup)
    ht = h.t()
    us_torch_t = timed(lambda: torch.mm(w_plain, ht), args.steps, args.warmup)
    del w_plain, ht
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
    # the LM head also gathering the logits at the drafts, and acceptance from those
    tg = torch.empty(T, dtype=torch.float32, device="cuda")
    dg = torch.empty(len(rows_d), dtype=torch.float32, device="cuda")
    cols = torch.empty(T, dtype=torch.int32, device="cuda")
    sx.spexis_verify_gather_columns(step.qsl, ids, cols)
    us_lm_gather = timed(lambda: sx.spexis_lm_head_gather(h, w, stats, cols, tg, logits=logits, temperature=temp),
                         args.steps, args.warmup)
    sx.spexis_lm_head_gather(hd, w, dstats, ids, dg, logits=dlogits, temperature=temp)
    run_gathered = lambda: sx.spexis_accept_with_stats(step.qsl, logits, dlogits, stats, dstats, ids, acc.u_accept,
                                                       acc.u_sample, batch.max_k, step.accepted_len,
                                                       step.out_tokens, step.row_status, step.acc_ws,
                                                       temperature=temp, target_gathered=tg, draft_gathered=dg)
    us_acc_gathered = timed(run_gathered, args.steps, args.warmup)
    assert np.array_equal(step.accepted_len.cpu().numpy(), a_fused)
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
        "us_with_gathers": round(us_lm_gather, 2), "accept_with_stats_gathered_us": round(us_acc_gathered, 2),
        "torch_bf16_us": {"h_wT": round(us_torch, 2), "w_hT": round(us_torch_t, 2)},
        "protocol": f"each figure: {SETTLE_MS:.0f} ms of the same call, {args.warmup} warmup calls, then the "
                    f"mean of {args.steps} calls",
        "dtype": "bf16", "data": "synthetic",
    }
    log(f"[lm_head] {T}x{d} @ {V}x{d}: {us_lm:.1f} us ({us_lm_stats:.1f} us without logits) -> {gbs:.0f} GB/s "
        f"({gbs / HBM_PEAK_GBS:.1%}), {tfl:.0f} TFLOP/s ({tfl / MFMA_BF16_TFLOPS:.1%}); accept {us_acc:.1f} us, "
        f"with given statistics {us_acc_stats:.1f} us; with the gathers fused: LM head {us_lm_gather:.1f} us, "
        f"accept {us_acc_gathered:.1f} us; torch bf16 GEMM {us_torch:.1f} us (h W^T), {us_torch_t:.1f} us (W h^T)")
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
        settle(torch, fn)
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
        settle(torch, call)
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
    settle(torch, step.run)
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
    settle(torch, step.replay)
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
    settle(torch, step.run)
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


COPY_KERNEL = "copyBuffer"
# per call: (kernel-name fragments of its launches, the launch that runs exactly once per call,
# the sources its kernels are built from)
TRAFFIC_CALLS = {
    "verify_attention": (("verify_attn_kernel", "attn_merge_kernel"), "verify_attn_kernel", ("attention.hip",)),
    "accept": (("accept_",), "accept_search_kernel", ("accept.hip",)),
}


def ingest_traffic(fetch_csv: str, write_csv: str, workload: int, copy_bytes: int) -> None:
    """HBM bytes per spexis_verify_attention and per spexis_accept call from two counter runs of
    `bench.py --copy-probe N`: each counter's KiB per dispatch, summed over the call's launches
    and divided by the number of calls, and scaled by N / (the counter's reading for one copy of
    N bytes), so that a plain copy reads and writes exactly N bytes."""
    import csv

    def per_kernel(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        out = {}
        for r in rows:
            out.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        # the probe: the last three copies before the library's first launch (bench.py makes
        # them after generating and copying the inputs, before the first step)
        first = next((i for i, r in enumerate(rows) if "spexis::" in r["Kernel_Name"]), len(rows))
        copies = [float(r["Counter_Value"]) * 1024.0 for r in rows[:first] if COPY_KERNEL in r["Kernel_Name"]]
        return out, copies[-3:]

    readings = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        k, probe = per_kernel(path, name)
        if len(probe) < 3:
            raise SystemExit(f"{path}: no {COPY_KERNEL} probe dispatches; run the profile with --copy-probe N")
        readings[name] = (k, float(np.median(probe)))
    prof = os.path.join(ROOT, "profiles", "traffic.json")
    data = json.load(open(prof)) if os.path.exists(prof) else {}
    for call, (frags, anchor, sources) in TRAFFIC_CALLS.items():
        result = {}
        for name, (k, probe) in readings.items():
            calls = sum(len(vals) for n, vals in k.items() if anchor in n)
            if calls == 0:
                break
            raw = sum(sum(vals) for n, vals in k.items() if any(f in n for f in frags)) / calls
            factor = copy_bytes / probe
            result[name] = {"raw_bytes_per_call": raw, "copy_reading": probe, "copy_bytes": copy_bytes,
                            "factor": factor, "bytes_per_call": raw * factor, "calls": calls}
        if len(result) < 2:
            continue
        total = result["FETCH_SIZE"]["bytes_per_call"] + result["WRITE_SIZE"]["bytes_per_call"]
        data[f"workload{workload}:{call}"] = {"source_digest": _kernel_digest(sources),
                                              "bytes_per_launch": round(total), "counters": result,
                                              "kernels": list(frags)}
    with open(prof, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps({k: v for k, v in data.items() if k.startswith(f"workload{workload}:")}, indent=1))


def stored_traffic(workload: int, call: str):
    """Calibrated counter bytes per call from profiles/traffic.json, if taken on the current sources."""
    prof = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(prof):
        return None
    with open(prof) as f:
        t = json.load(f).get(f"workload{workload}:{call}")
    if t and t.get("source_digest") == _kernel_digest(TRAFFIC_CALLS[call][2]):
        return t["bytes_per_launch"]
    return None


def _kernel_digest(sources=("attention.hip",)) -> str:
    """Digest of the sources a call's kernels are built from (their code, the shared device
    helpers, and the header with their parameters and launch constants): a stored traffic figure
    is used only while they are unchanged."""
    import hashlib
    h = hashlib.sha256()
    for name in tuple(sources) + ("common.h", "kernels.h"):
        with open(os.path.join(ROOT, "paper_2609_34370_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
