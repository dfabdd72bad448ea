"""One verification step on the GPU: append -> verify attention -> accept.

Holds the device buffers of a batch (metadata, pools, outputs, workspaces sized once from the
library's queries) and calls the three entry points of libspexis in order on one stream.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np
import torch

from . import spexis as sx
from .workloads import AcceptInputs, AttentionInputs, Batch


class VerifyStep:
    def __init__(self, batch: Batch, attn: AttentionInputs, acc: Optional[AcceptInputs], kv_chunk_tokens: int = 0,
                 kind: int = sx.SPEXIS_INPUT_LOGITS, device="cuda"):
        spec = batch.spec
        self.batch, self.spec, self.kind = batch, spec, kind
        self.kv_chunk_tokens = kv_chunk_tokens
        dev = torch.device(device)
        self.qsl = torch.as_tensor(batch.qsl, device=dev)
        self.seq_lens = torch.as_tensor(batch.seq_lens, device=dev)
        self.tables = torch.as_tensor(batch.block_tables, device=dev)
        self.attn = attn
        self.out = torch.empty_like(attn.q)
        self.scale = 1.0 / math.sqrt(spec.head_dim)
        ws = sx.spexis_verify_attention_workspace_size(batch.B, spec.num_q_heads, spec.num_kv_heads, spec.head_dim,
                                                      batch.max_query_len, batch.max_seq_len, kv_chunk_tokens)
        self.attn_ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=dev)
        self.acc = acc
        self.max_k = batch.max_k
        if acc is not None:
            aw = sx.spexis_accept_workspace_size(batch.B, spec.vocab, self.max_k)
            self.acc_ws = torch.empty(aw, dtype=torch.uint8, device=dev)
            self.accepted_len = torch.empty(batch.B, dtype=torch.int32, device=dev)
            self.out_tokens = torch.empty((batch.B, self.max_k + 1), dtype=torch.int32, device=dev)
            self.row_status = torch.empty(batch.B, dtype=torch.int32, device=dev)

    def append(self, stream=None):
        s, b = self.spec, self.batch
        sx.spexis_append_kv(self.attn.k_pool, self.attn.v_pool, b.num_blocks, s.num_kv_heads, s.block_size,
                            s.head_dim, self.qsl, self.seq_lens, self.tables, b.T, b.max_query_len,
                            self.attn.new_k, self.attn.new_v, stream=stream)

    def attention(self, stream=None):
        s, b = self.spec, self.batch
        sx.spexis_verify_attention(self.attn.k_pool, self.attn.v_pool, b.num_blocks, s.num_kv_heads, s.block_size,
                                   s.head_dim, self.qsl, self.seq_lens, self.tables, b.T, b.max_query_len,
                                   b.max_seq_len, self.attn.q, s.num_q_heads, self.scale, self.out, self.attn_ws,
                                   kv_chunk_tokens=self.kv_chunk_tokens, stream=stream)

    def accept(self, target=None, draft=None, kind=None, stream=None, seq_lens_inout=None):
        a = self.acc
        kind = self.kind if kind is None else kind
        target = a.target_logits if target is None else target
        draft = a.draft_logits if draft is None else draft
        sx.spexis_accept(kind, self.qsl, target, draft, a.draft_ids, a.u_accept, a.u_sample, self.max_k,
                         self.accepted_len, self.out_tokens, self.row_status, self.acc_ws,
                         temperature=a.temperature, seq_lens_inout=seq_lens_inout, stream=stream)

    def run(self, stream=None):
        self.append(stream)
        self.attention(stream)
        if self.acc is not None:
            self.accept(stream=stream)

    def capture(self, warmup: int = 1):
        """Records run() into a HIP graph (torch.cuda.CUDAGraph); replay() then launches the whole
        step at once.  Every buffer is allocated in __init__ and the library calls neither
        allocate nor set memory (the acceptance counters are cleared by its first kernel), so the
        graph holds only the step's kernel launches.  A replay reads the current contents of the
        input buffers; the sizes are those of this batch."""
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

    def accept_outputs(self):
        return (self.accepted_len.cpu().numpy(), self.out_tokens.cpu().numpy(), self.row_status.cpu().numpy())


def bf16_to_u16(t: torch.Tensor) -> np.ndarray:
    """Host uint16 view of a bf16 tensor's bits (for the oracle)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
