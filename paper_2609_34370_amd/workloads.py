"""Seeded synthetic inputs for the speculative verification step.

This module is the only code shared by the oracle side and the HIP side of the tests and
the benchmark.  It draws inputs -- sequence lengths, draft counts, block tables, Q/K/V,
logits, draft tokens and uniforms -- and holds none of the verification arithmetic
(no attention, no softmax, no acceptance test, no sampling rule).

The five workloads stand in for the serving traffic of the paper's evaluation (SpecBench,
LMSYS-Chat, ShareGPT and UltraChat, Sec. 7), none of which is available here.  They take
the head shapes of Llama-3-8B/70B and Qwen3 models, serving-like context distributions and
draft/target disagreement spanning the acceptance rates of Table 3 (0.46-0.84) and beyond.

Recipe (every draw is seeded; ``seed = 260934370 + workload id`` unless overridden):
  * metadata (context lengths L_b, draft counts k_b, the physical-block permutation,
    uniforms) comes from numpy ``Philox`` streams spawned from ``SeedSequence(seed)``;
  * bulk tensors (pool, Q, new K/V, logits, Gumbel noise for drafting) come from a
    ``torch.Generator`` on the target device seeded with ``seed + stream``; host copies
    are taken from whatever was drawn, so the oracle and the GPU see identical bytes;
  * Q, K and V are N(0,1) rounded to bf16 (round to nearest even);
  * target logits are N(0, sigma_t) in fp32; draft logits = target + N(0, sigma_b);
  * draft token x_i is drawn from softmax(draft_i / T) by the Gumbel-max trick
    (argmax of draft_i / T + Gumbel noise) -- this stands in for the draft model's own
    sampler, which the verification step receives as an input;
  * uniforms are ``Generator(Philox).random(dtype=float32)``: multiples of 2^-24 in [0,1).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

BASE_SEED = 260934370

# stream indices of SeedSequence(seed).spawn(12) / torch seeds seed + stream
_S_CTX, _S_K, _S_PERM, _S_Q, _S_POOL, _S_NEWKV, _S_TGT, _S_NOISE, _S_SIGMA, _S_DRAFT, _S_UACC, _S_USMP = range(12)


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    wid: int
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    ctx: tuple            # ("uniform", lo, hi) | ("lognormal", median, sigma, lo, hi)
    k: tuple              # ("fixed", k) | ("uniform", lo, hi)
    vocab: int
    target_std: float
    draft_noise: tuple    # ("fixed", s) | ("uniform", lo, hi)
    temperature: float = 1.0
    pool_fill: float = 1.0  # fraction of the physical pool the sequences occupy


WORKLOADS = {
    1: WorkloadSpec(1, "tiny", 4, 8, 2, 64, 16, ("uniform", 32, 256), ("fixed", 4), 1024,
                    2.0, ("fixed", 0.5)),
    2: WorkloadSpec(2, "llama3-8b-layer", 64, 32, 8, 128, 16, ("uniform", 1024, 4096),
                    ("fixed", 4), 128256, 3.0, ("fixed", 1.0)),
    3: WorkloadSpec(3, "long-context", 256, 64, 8, 128, 16, ("lognormal", 2048, 0.7, 128, 16384),
                    ("fixed", 5), 128256, 3.0, ("fixed", 1.0), pool_fill=0.9),
    4: WorkloadSpec(4, "ragged-selective", 128, 32, 8, 128, 16, ("uniform", 256, 8192),
                    ("uniform", 0, 8), 32000, 3.0, ("uniform", 0.1, 3.0)),
    5: WorkloadSpec(5, "acceptance-stress", 512, 28, 4, 128, 32, ("uniform", 512, 2048),
                    ("fixed", 8), 152064, 4.0, ("fixed", 2.0), temperature=0.7),
}


def spec_with(wid: int, **overrides) -> WorkloadSpec:
    """A workload spec with some fields replaced (smaller batches, other shapes...)."""
    return dataclasses.replace(WORKLOADS[wid], **overrides)


@dataclasses.dataclass
class Batch:
    """Metadata of one verification step (host numpy + device copies)."""
    spec: WorkloadSpec
    ctx_lens: np.ndarray        # [B] int32, L_b: tokens cached before the step
    k: np.ndarray               # [B] int32, drafts per sequence
    qsl: np.ndarray             # [B+1] int32, query_start_loc
    seq_lens: np.ndarray        # [B] int32, S_b = L_b + k_b + 1
    block_tables: np.ndarray    # [B, max_blocks] int32
    num_blocks: int

    @property
    def B(self) -> int:
        return int(self.ctx_lens.shape[0])

    @property
    def T(self) -> int:
        return int(self.qsl[-1])

    @property
    def max_query_len(self) -> int:
        return int((self.k + 1).max())

    @property
    def max_k(self) -> int:
        return int(self.k.max())

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max())


def _streams(seed: int):
    return [np.random.Generator(np.random.Philox(s)) for s in np.random.SeedSequence(seed).spawn(12)]


def _draw_ctx(spec: WorkloadSpec, rng: np.random.Generator, B: int) -> np.ndarray:
    kind = spec.ctx[0]
    if kind == "uniform":
        lo, hi = spec.ctx[1], spec.ctx[2]
        return rng.integers(lo, hi + 1, size=B).astype(np.int32)
    if kind == "lognormal":
        median, sigma, lo, hi = spec.ctx[1:]
        x = np.exp(rng.normal(math.log(median), sigma, size=B))
        return np.clip(np.rint(x), lo, hi).astype(np.int32)
    if kind == "fixed":
        return np.full(B, spec.ctx[1], dtype=np.int32)
    raise ValueError(kind)


def _draw_k(spec: WorkloadSpec, rng: np.random.Generator, B: int) -> np.ndarray:
    if spec.k[0] == "fixed":
        return np.full(B, spec.k[1], dtype=np.int32)
    lo, hi = spec.k[1], spec.k[2]
    return rng.integers(lo, hi + 1, size=B).astype(np.int32)


def make_batch(spec: WorkloadSpec, seed: Optional[int] = None, ctx_lens=None, k=None) -> Batch:
    """Sequence lengths, draft counts and randomly permuted block tables."""
    seed = BASE_SEED + spec.wid if seed is None else seed
    st = _streams(seed)
    B = spec.batch
    L = np.asarray(ctx_lens, dtype=np.int32) if ctx_lens is not None else _draw_ctx(spec, st[_S_CTX], B)
    kk = np.asarray(k, dtype=np.int32) if k is not None else _draw_k(spec, st[_S_K], B)
    assert L.shape == (B,) and kk.shape == (B,)
    n = kk + 1
    qsl = np.zeros(B + 1, dtype=np.int32)
    qsl[1:] = np.cumsum(n)
    S = (L + n).astype(np.int32)
    bs = spec.block_size
    nblk = (S + bs - 1) // bs
    used = int(nblk.sum())
    num_blocks = max(used, int(math.ceil(used / spec.pool_fill)))
    perm = st[_S_PERM].permutation(num_blocks).astype(np.int32)
    max_blocks = int(nblk.max())
    # entries past a sequence's last block are never read; they hold a valid id (0)
    tables = np.zeros((B, max_blocks), dtype=np.int32)
    off = 0
    for b in range(B):
        tables[b, : nblk[b]] = perm[off: off + nblk[b]]
        off += nblk[b]
    return Batch(spec, L, kk, qsl, S, tables, num_blocks)


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _randn_bf16(shape, gen, device, chunk=1 << 26) -> torch.Tensor:
    """N(0,1) rounded to bf16, drawn in slices to bound the fp32 temporaries."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    for s in range(0, flat.numel(), chunk):
        e = min(flat.numel(), s + chunk)
        flat[s:e] = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
    return out


@dataclasses.dataclass
class AttentionInputs:
    k_pool: torch.Tensor   # [num_blocks * Hkv * bs * D] bf16 (flat; layout is the library's)
    v_pool: torch.Tensor
    q: torch.Tensor        # [T, Hq, D] bf16
    new_k: torch.Tensor    # [T, Hkv, D] bf16
    new_v: torch.Tensor


def make_attention_inputs(spec: WorkloadSpec, batch: Batch, device="cpu", seed: Optional[int] = None) -> AttentionInputs:
    seed = BASE_SEED + spec.wid if seed is None else seed
    hkv, D, bs = spec.num_kv_heads, spec.head_dim, spec.block_size
    pool_elems = batch.num_blocks * hkv * bs * D
    gp = _gen(device, seed + _S_POOL)
    k_pool = _randn_bf16((pool_elems,), gp, device)
    v_pool = _randn_bf16((pool_elems,), gp, device)
    q = _randn_bf16((batch.T, spec.num_q_heads, D), _gen(device, seed + _S_Q), device)
    gn = _gen(device, seed + _S_NEWKV)
    new_k = _randn_bf16((batch.T, hkv, D), gn, device)
    new_v = _randn_bf16((batch.T, hkv, D), gn, device)
    return AttentionInputs(k_pool, v_pool, q, new_k, new_v)


@dataclasses.dataclass
class AcceptInputs:
    target_logits: torch.Tensor  # [T, V] fp32; row qsl[b]+i is target position i of b
    draft_logits: torch.Tensor   # [T-B, V] fp32; row qsl[b]-b+i is draft position i of b
    draft_ids: torch.Tensor      # [T-B] int32
    u_accept: torch.Tensor       # [T-B] fp32 in [0,1)
    u_sample: torch.Tensor       # [B] fp32 in [0,1)
    temperature: float


def draft_row_index(batch: Batch) -> np.ndarray:
    """For every draft row r (0..T-B), the target row holding the same position."""
    rows = []
    for b in range(batch.B):
        rows.extend(range(int(batch.qsl[b]), int(batch.qsl[b]) + int(batch.k[b])))
    return np.asarray(rows, dtype=np.int64)


def make_accept_inputs(spec: WorkloadSpec, batch: Batch, device="cpu", seed: Optional[int] = None,
                       row_chunk: int = 256) -> AcceptInputs:
    seed = BASE_SEED + spec.wid if seed is None else seed
    st = _streams(seed)
    V, T, B = spec.vocab, batch.T, batch.B
    nd = T - B
    target = torch.empty((T, V), dtype=torch.float32, device=device)
    gt = _gen(device, seed + _S_TGT)
    for s in range(0, T, row_chunk):
        e = min(T, s + row_chunk)
        target[s:e] = torch.randn((e - s, V), generator=gt, device=device) * spec.target_std
    # per-sequence draft-noise std
    if spec.draft_noise[0] == "fixed":
        sig = np.full(B, spec.draft_noise[1], dtype=np.float32)
    else:
        sig = st[_S_SIGMA].uniform(spec.draft_noise[1], spec.draft_noise[2], size=B).astype(np.float32)
    src = draft_row_index(batch)
    sig_rows = np.repeat(sig, batch.k).astype(np.float32)
    draft = torch.empty((nd, V), dtype=torch.float32, device=device)
    ids = torch.empty((nd,), dtype=torch.int32, device=device)
    gn = _gen(device, seed + _S_NOISE)
    gd = _gen(device, seed + _S_DRAFT)
    inv_t = 1.0 / spec.temperature
    for s in range(0, nd, row_chunk):
        e = min(nd, s + row_chunk)
        rows = torch.as_tensor(src[s:e], device=device)
        sr = torch.as_tensor(sig_rows[s:e], device=device).unsqueeze(1)
        draft[s:e] = target.index_select(0, rows) + torch.randn((e - s, V), generator=gn, device=device) * sr
        # Gumbel-max draw of the draft token from softmax(draft / T)
        u = torch.rand((e - s, V), generator=gd, device=device, dtype=torch.float64).clamp_(min=1e-300)
        gumbel = -torch.log(-torch.log(u))
        ids[s:e] = torch.argmax(draft[s:e].double() * inv_t + gumbel, dim=1).to(torch.int32)
    u_acc = st[_S_UACC].random(nd, dtype=np.float32)
    u_smp = st[_S_USMP].random(B, dtype=np.float32)
    return AcceptInputs(target, draft, ids, torch.as_tensor(u_acc, device=device),
                        torch.as_tensor(u_smp, device=device), float(spec.temperature))


def subset_batch(batch: Batch, seqs) -> tuple:
    """Metadata of a subset of sequences, with row maps into the full tensors.

    Returns (sub_batch, target_rows, draft_rows): the sub-batch's query/target rows are
    ``target_rows`` of the full batch, its draft rows ``draft_rows``.
    """
    seqs = np.asarray(seqs, dtype=np.int64)
    L, kk = batch.ctx_lens[seqs], batch.k[seqs]
    n = kk + 1
    qsl = np.zeros(len(seqs) + 1, dtype=np.int32)
    qsl[1:] = np.cumsum(n)
    trows = np.concatenate([np.arange(batch.qsl[b], batch.qsl[b + 1]) for b in seqs]).astype(np.int64)
    drows = np.concatenate([np.arange(batch.qsl[b] - b, batch.qsl[b] - b + batch.k[b]) for b in seqs]).astype(np.int64) \
        if kk.sum() > 0 else np.zeros(0, dtype=np.int64)
    sub = Batch(batch.spec, L.astype(np.int32), kk.astype(np.int32), qsl, batch.seq_lens[seqs].astype(np.int32),
                batch.block_tables[seqs], batch.num_blocks)
    return sub, trows, drows


# hidden size of the model behind each workload (equal to Hq * D for all of them)
HIDDEN = {1: 512, 2: 4096, 3: 4096, 4: 4096, 5: 3584}


@dataclasses.dataclass
class AdapterInputs:
    """Synthetic weights and inputs of one drafting step (the adapter: a linear layer, an
    attention layer with q/k/v and output projections, then the LM head)."""
    h: torch.Tensor        # [B, d] bf16 exit hidden states
    w_in: torch.Tensor     # [d, d] bf16
    w_q: torch.Tensor      # [Hq*D, d]
    w_k: torch.Tensor      # [Hkv*D, d]
    w_v: torch.Tensor      # [Hkv*D, d]
    w_o: torch.Tensor      # [d, Hq*D]
    w_lm: torch.Tensor     # [V, d]
    u: torch.Tensor        # [B] fp32 uniforms of the draft draw
    temperature: float


def make_adapter_inputs(spec: WorkloadSpec, batch: Batch, device="cpu", seed: Optional[int] = None) -> AdapterInputs:
    """N(0, 1) exit states; every weight N(0, 1/fan_in) (activations stay O(1)) except the LM
    head, N(0, 4/d) (logits of standard deviation about 2)."""
    seed = BASE_SEED + 100 + spec.wid if seed is None else seed
    d, hq, hkv, D = HIDDEN[spec.wid], spec.num_q_heads, spec.num_kv_heads, spec.head_dim
    g = _gen(device, seed)

    def w(rows, cols, std):
        return (torch.randn((rows, cols), generator=g, device=device) * std).to(torch.bfloat16)

    h = torch.randn((batch.B, d), generator=g, device=device).to(torch.bfloat16)
    w_in = w(d, d, d ** -0.5)
    w_q = w(hq * D, d, d ** -0.5)
    w_k = w(hkv * D, d, d ** -0.5)
    w_v = w(hkv * D, d, d ** -0.5)
    w_o = w(d, hq * D, (hq * D) ** -0.5)
    w_lm = torch.empty((spec.vocab, d), dtype=torch.bfloat16, device=device)
    for r in range(0, spec.vocab, 16384):   # in chunks: the fp32 draw of the whole head is large
        e = min(spec.vocab, r + 16384)
        w_lm[r:e] = (torch.randn((e - r, d), generator=g, device=device) * (2.0 / d ** 0.5)).to(torch.bfloat16)
    u = torch.rand(batch.B, generator=g, device=device)
    return AdapterInputs(h, w_in, w_q, w_k, w_v, w_o, w_lm, u, spec.temperature)
