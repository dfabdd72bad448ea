"""One drafting step on the GPU: the adapter forward and the draft draw.

The adapter follows the paper's description (Implementation: a linear layer and an attention
layer, followed by the LM head, after Kangaroo): from the exit hidden states h of the batch,
    x = h W_in^T
    q, k, v = x W_q^T, x W_k^T, x W_v^T        (k, v appended to the adapter's paged cache)
    o = attention(q, cache)                     (one query token per sequence: the k = 0 case)
    y = o W_o^T + x
    logits = y W_lm^T                           (with the fused softmax statistics)
    draft token ~ softmax(logits / T), with its probability q(x) as the confidence
Every step is one libspexis call on one stream (q, k and v together: one call over their stacked
weights); the adapter's KV cache uses the library's paged layout and the sequences' block tables.
"""
from __future__ import annotations

import math

import torch

from . import spexis as sx
from .workloads import AdapterInputs, AttentionInputs, Batch


class DraftStep:
    def __init__(self, batch: Batch, cache: AttentionInputs, ad: AdapterInputs, device="cuda"):
        spec = batch.spec
        assert int(batch.k.max()) == 0, "a drafting step has one query token per sequence"
        self.batch, self.spec, self.cache, self.ad = batch, spec, cache, ad
        # the projections read packed weights (laid out once, as at model load)
        self.w_in, self.w_o, self.w_lm = (sx.spexis_pack_weight(w) for w in (ad.w_in, ad.w_o, ad.w_lm))
        self.w_qkv = sx.spexis_pack_weight(torch.cat([ad.w_q, ad.w_k, ad.w_v], dim=0))
        dev = torch.device(device)
        B, d = ad.h.shape
        hq, hkv, D = spec.num_q_heads, spec.num_kv_heads, spec.head_dim
        self.d, self.hq, self.hkv, self.D = d, hq, hkv, D
        self.qsl = torch.as_tensor(batch.qsl, device=dev)
        self.seq_lens = torch.as_tensor(batch.seq_lens, device=dev)
        self.tables = torch.as_tensor(batch.block_tables, device=dev)
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.x = torch.empty((B, d), **bf)
        self.q = torch.empty((B, hq, D), **bf)
        self.k = torch.empty((B, hkv, D), **bf)
        self.v = torch.empty((B, hkv, D), **bf)
        self.o = torch.empty((B, hq, D), **bf)
        self.y = torch.empty((B, d), **bf)
        V = ad.w_lm.shape[0]
        self.logits = torch.empty((B, V), dtype=torch.float32, device=dev)
        self.stats = torch.empty((B, sx.spexis_lm_head_tiles(V), 2), dtype=torch.float32, device=dev)
        self.tokens = torch.empty(B, dtype=torch.int32, device=dev)
        self.conf = torch.empty(B, dtype=torch.float32, device=dev)
        self.status = torch.empty(B, dtype=torch.int32, device=dev)
        lin = max([sx.spexis_linear_workspace_size(B, n, kk) for n, kk in ((d, d), (d, hq * D))] +
                  [sx.spexis_linear_split_workspace_size(B, (hq + 2 * hkv) * D, d)])
        self.lin_ws = torch.empty(max(lin, 16), dtype=torch.uint8, device=dev)
        aw = sx.spexis_verify_attention_workspace_size(B, hq, hkv, D, 1, batch.max_seq_len, 0)
        self.attn_ws = torch.empty(max(aw, 16), dtype=torch.uint8, device=dev)
        self.smp_ws = torch.empty(sx.spexis_sample_workspace_size(B, V), dtype=torch.uint8, device=dev)
        self.scale = 1.0 / math.sqrt(D)

    def adapter_in(self, stream=None):
        a, B = self.ad, self.batch.B
        sx.spexis_linear(a.h, self.w_in, self.x, workspace=self.lin_ws, stream=stream)
        sx.spexis_linear_split(self.x, self.w_qkv, [self.q.view(B, -1), self.k.view(B, -1), self.v.view(B, -1)],
                               self.lin_ws, stream=stream)

    def attention(self, stream=None):
        s, b, c = self.spec, self.batch, self.cache
        sx.spexis_append_kv(c.k_pool, c.v_pool, b.num_blocks, s.num_kv_heads, s.block_size, s.head_dim, self.qsl,
                            self.seq_lens, self.tables, b.T, 1, self.k, self.v, stream=stream)
        sx.spexis_verify_attention(c.k_pool, c.v_pool, b.num_blocks, s.num_kv_heads, s.block_size, s.head_dim,
                                   self.qsl, self.seq_lens, self.tables, b.T, 1, b.max_seq_len, self.q,
                                   s.num_q_heads, self.scale, self.o, self.attn_ws, stream=stream)

    def adapter_out(self, stream=None):
        B = self.batch.B
        sx.spexis_linear(self.o.view(B, -1), self.w_o, self.y, residual=self.x, workspace=self.lin_ws,
                         stream=stream)

    def lm_head(self, stream=None):
        sx.spexis_lm_head(self.y, self.w_lm, self.stats, logits=self.logits, temperature=self.ad.temperature,
                          stream=stream)

    def sample(self, stream=None):
        sx.spexis_sample_tokens(sx.SPEXIS_INPUT_LOGITS, self.logits, self.ad.u, self.tokens, self.status,
                                self.smp_ws, token_prob=self.conf, stats=self.stats,
                                temperature=self.ad.temperature, stream=stream)

    def run(self, stream=None):
        self.adapter_in(stream)
        self.attention(stream)
        self.adapter_out(stream)
        self.lm_head(stream)
        self.sample(stream)

    def capture(self, warmup: int = 1):
        """Records run() into a HIP graph (torch.cuda.CUDAGraph); replay() then launches the whole
        step at once, with no host work between its kernels.  Every buffer the step touches is
        allocated in __init__ and the library calls neither allocate nor set memory, so the graph
        holds only the step's kernel launches.  Like run(), a replay reads the current contents of
        the input buffers (h, the cache, the uniforms); the sizes are those of this batch."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(warmup):
                self.run()
        torch.cuda.current_stream().wait_stream(side)
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.run()
        return self.graph

    def replay(self):
        self.graph.replay()
