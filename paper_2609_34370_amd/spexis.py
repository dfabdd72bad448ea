"""Python binding of libspexis: the C entry points under the same names, taking torch tensors.

Argument marshalling only -- every step runs in the HIP kernels of libspexis.so.  Tensors must
live on the GPU (torch's ``cuda`` device on ROCm); the calls are asynchronous on the given
stream (default: torch's current stream).  There is no CPU fallback: without the built
library every call raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libspexis.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "spexis.h")

SPEXIS_OK = 0
SPEXIS_ERR_INVALID_ARGUMENT = -1
SPEXIS_ERR_UNSUPPORTED = -2
SPEXIS_ERR_WORKSPACE_TOO_SMALL = -3
SPEXIS_ERR_HIP = -4
SPEXIS_INPUT_PROBS = 0
SPEXIS_INPUT_LOGITS = 1
SPEXIS_ROW_OK, SPEXIS_ROW_EMPTY, SPEXIS_ROW_BAD_VALUE, SPEXIS_ROW_BAD_TOKEN, SPEXIS_ROW_INTERNAL = 0, 1, 2, 3, 4


class SpexisError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


_lib = None


def header_functions() -> list:
    """Names of the functions include/spexis.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(spexis_\w+)\s*\(", text, re.M)))


def lib():
    """The loaded libspexis.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(the HIP path has no fallback)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    L.spexis_version.argtypes, L.spexis_version.restype = [], ctypes.c_int
    L.spexis_last_error.argtypes, L.spexis_last_error.restype = [], ctypes.c_char_p
    L.spexis_append_kv.argtypes = [P, P, i32, i32, i32, i32, i32, P, P, P, i32, i32, i32, P, P, P]
    L.spexis_append_kv.restype = ctypes.c_int
    L.spexis_verify_attention_workspace_size.argtypes = [i32, i32, i32, i32, i32, i32, i32]
    L.spexis_verify_attention_workspace_size.restype = sz
    L.spexis_verify_attention.argtypes = [P, P, i32, i32, i32, i32, i32, P, P, P, i32, i32, i32, i32, P, i32, f32,
                                          P, i32, P, sz, P]
    L.spexis_verify_attention.restype = ctypes.c_int
    L.spexis_softmax_rows.argtypes = [P, P, i64, i32, f32, P]
    L.spexis_softmax_rows.restype = ctypes.c_int
    L.spexis_accept_workspace_size.argtypes = [i32, i32, i32]
    L.spexis_accept_workspace_size.restype = sz
    L.spexis_accept.argtypes = [i32, i32, i32, i32, f32, i32, P, P, P, P, P, P, P, P, P, P, P, sz, P]
    L.spexis_accept.restype = ctypes.c_int
    L.spexis_accept_noalloc.argtypes = [i32, i32, i32, i32, f32, i32, P, P, P, P, P, P, P, P, P, P, P]
    L.spexis_accept_noalloc.restype = ctypes.c_int
    L.spexis_lm_head.argtypes = [P, P, i32, i32, i32, f32, P, P, P]
    L.spexis_lm_head.restype = ctypes.c_int
    L.spexis_lm_head_tiles.argtypes, L.spexis_lm_head_tiles.restype = [i32], i32
    L.spexis_lm_head_stats_size.argtypes, L.spexis_lm_head_stats_size.restype = [i32, i32], sz
    L.spexis_accept_with_stats.argtypes = [i32, i32, i32, f32, i32, P, P, P, P, P, i32, P, P, P, P, P, P, P, P, P,
                                           P, sz, P]
    L.spexis_lm_head_gather.argtypes = [P, P, i32, i32, i32, f32, P, P, P, P, P]
    L.spexis_lm_head_gather.restype = ctypes.c_int
    L.spexis_verify_gather_columns.argtypes = [i32, i32, P, P, P, P]
    L.spexis_verify_gather_columns.restype = ctypes.c_int
    L.spexis_accept_with_stats.restype = ctypes.c_int
    L.spexis_select_drafts.argtypes = [i32, i32, P, P, f32, P, P, P, P]
    L.spexis_select_drafts.restype = ctypes.c_int
    L.spexis_sample_tokens.argtypes = [i32, i32, i32, f32, P, P, i32, P, P, P, P, P, sz, P]
    L.spexis_sample_tokens.restype = ctypes.c_int
    L.spexis_sample_workspace_size.argtypes = [i32, i32]
    L.spexis_sample_workspace_size.restype = sz
    L.spexis_pack_weight.argtypes = [P, i32, i32, P, P]
    L.spexis_pack_weight.restype = ctypes.c_int
    L.spexis_packed_weight_size.argtypes = [i32, i32]
    L.spexis_packed_weight_size.restype = sz
    L.spexis_linear.argtypes = [P, P, P, i32, i32, i32, P, P, sz, P]
    L.spexis_linear.restype = ctypes.c_int
    L.spexis_linear_workspace_size.argtypes = [i32, i32, i32]
    L.spexis_linear_workspace_size.restype = sz
    L.spexis_linear_split.argtypes = [P, P, i32, i32, i32, ctypes.POINTER(i32), ctypes.POINTER(P), P, sz, P]
    L.spexis_linear_split.restype = ctypes.c_int
    L.spexis_linear_split_workspace_size.argtypes = [i32, i32, i32]
    L.spexis_linear_split_workspace_size.restype = sz
    L.spexis_lookahead_memory.argtypes = [i32, P, P, P, i32, ctypes.c_double, i32, P, P, P, P, P]
    L.spexis_lookahead_memory.restype = ctypes.c_int
    _lib = L
    return L


def _check(rc: int) -> None:
    if rc != SPEXIS_OK:
        raise SpexisError(rc, lib().spexis_last_error().decode())


def _ptr(t: Optional[torch.Tensor], dtype=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"expected {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def spexis_version() -> int:
    return int(lib().spexis_version())


def spexis_append_kv(k_cache, v_cache, num_blocks, num_kv_heads, block_size, head_dim, query_start_loc, seq_lens,
                     block_tables, total_tokens, max_query_len, new_k, new_v, stream=None) -> None:
    _check(lib().spexis_append_kv(
        _ptr(k_cache, torch.bfloat16), _ptr(v_cache, torch.bfloat16), num_blocks, num_kv_heads, block_size,
        head_dim, query_start_loc.shape[0] - 1, _ptr(query_start_loc, torch.int32), _ptr(seq_lens, torch.int32),
        _ptr(block_tables, torch.int32), block_tables.shape[1], total_tokens, max_query_len,
        _ptr(new_k, torch.bfloat16), _ptr(new_v, torch.bfloat16), _stream(stream)))


def spexis_verify_attention_workspace_size(num_seqs, num_q_heads, num_kv_heads, head_dim, max_query_len, max_seq_len,
                                           kv_chunk_tokens=0) -> int:
    return int(lib().spexis_verify_attention_workspace_size(num_seqs, num_q_heads, num_kv_heads, head_dim,
                                                            max_query_len, max_seq_len, kv_chunk_tokens))


def spexis_verify_attention(k_cache, v_cache, num_blocks, num_kv_heads, block_size, head_dim, query_start_loc,
                            seq_lens, block_tables, total_tokens, max_query_len, max_seq_len, q, num_q_heads, scale,
                            out, workspace=None, kv_chunk_tokens=0, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spexis_verify_attention(
        _ptr(k_cache, torch.bfloat16), _ptr(v_cache, torch.bfloat16), num_blocks, num_kv_heads, block_size,
        head_dim, query_start_loc.shape[0] - 1, _ptr(query_start_loc, torch.int32), _ptr(seq_lens, torch.int32),
        _ptr(block_tables, torch.int32), block_tables.shape[1], total_tokens, max_query_len, max_seq_len,
        _ptr(q, torch.bfloat16), num_q_heads, ctypes.c_float(scale), _ptr(out, torch.bfloat16), kv_chunk_tokens,
        _ptr(workspace), ws_bytes, _stream(stream)))


def spexis_softmax_rows(logits, probs, temperature=1.0, stream=None) -> None:
    rows, vocab = logits.shape
    _check(lib().spexis_softmax_rows(_ptr(logits, torch.float32), _ptr(probs, torch.float32), rows, vocab,
                                     ctypes.c_float(temperature), _stream(stream)))


def spexis_accept_workspace_size(num_seqs, vocab, max_k) -> int:
    return int(lib().spexis_accept_workspace_size(num_seqs, vocab, max_k))


def spexis_accept(kind, query_start_loc, target, draft, draft_ids, u_accept, u_sample, max_k, accepted_len,
                  out_tokens, row_status, workspace, temperature=1.0, seq_lens_inout=None, stream=None) -> None:
    num_seqs = query_start_loc.shape[0] - 1
    total_tokens, vocab = target.shape
    ws_bytes = workspace.numel() * workspace.element_size()
    nd = total_tokens - num_seqs
    _check(lib().spexis_accept(
        kind, num_seqs, vocab, max_k, ctypes.c_float(temperature), total_tokens, _ptr(query_start_loc, torch.int32),
        _ptr(target, torch.float32), _ptr(draft, torch.float32) if nd > 0 else None,
        _ptr(draft_ids, torch.int32) if nd > 0 else None, _ptr(u_accept, torch.float32) if nd > 0 else None,
        _ptr(u_sample, torch.float32), _ptr(accepted_len, torch.int32), _ptr(out_tokens, torch.int32),
        _ptr(row_status, torch.int32), _ptr(seq_lens_inout, torch.int32), _ptr(workspace), ws_bytes,
        _stream(stream)))


SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES = 16 << 20


def spexis_accept_noalloc(kind, query_start_loc, target, draft, draft_ids, u_accept, u_sample, max_k, accepted_len,
                          out_tokens, row_status, temperature=1.0, seq_lens_inout=None, stream=None) -> None:
    """spexis_accept working in the library's static scratch array (no workspace argument)."""
    num_seqs = query_start_loc.shape[0] - 1
    total_tokens, vocab = target.shape
    nd = total_tokens - num_seqs
    _check(lib().spexis_accept_noalloc(
        kind, num_seqs, vocab, max_k, ctypes.c_float(temperature), total_tokens, _ptr(query_start_loc, torch.int32),
        _ptr(target, torch.float32), _ptr(draft, torch.float32) if nd > 0 else None,
        _ptr(draft_ids, torch.int32) if nd > 0 else None, _ptr(u_accept, torch.float32) if nd > 0 else None,
        _ptr(u_sample, torch.float32), _ptr(accepted_len, torch.int32), _ptr(out_tokens, torch.int32),
        _ptr(row_status, torch.int32), _ptr(seq_lens_inout, torch.int32), _stream(stream)))


def spexis_lm_head_tiles(vocab: int) -> int:
    return int(lib().spexis_lm_head_tiles(vocab))


def spexis_lm_head_stats_size(rows: int, vocab: int) -> int:
    return int(lib().spexis_lm_head_stats_size(rows, vocab))


def spexis_lm_head(hidden, weight, stats, logits=None, temperature=1.0, vocab=None, stream=None) -> None:
    """weight: packed by spexis_pack_weight; vocab defaults to the stats / logits shape."""
    rows, hidden_dim = hidden.shape
    if vocab is None:
        vocab = logits.shape[1] if logits is not None else None
    if vocab is None:
        raise ValueError("vocab is needed when logits is None")
    assert weight.numel() * 2 == spexis_packed_weight_size(vocab, hidden_dim), "weight must be packed"
    _check(lib().spexis_lm_head(_ptr(hidden, torch.bfloat16), _ptr(weight, torch.bfloat16), rows, vocab, hidden_dim,
                                ctypes.c_float(temperature), _ptr(logits, torch.float32),
                                _ptr(stats, torch.float32), _stream(stream)))


def spexis_lm_head_gather(hidden, weight, stats, gather_cols, gathered, logits=None, temperature=1.0, vocab=None,
                          stream=None) -> None:
    """spexis_lm_head that also writes gathered[m] = logits[m][gather_cols[m]] (for columns in
    [0, V))."""
    rows, hidden_dim = hidden.shape
    if vocab is None:
        vocab = logits.shape[1] if logits is not None else None
    if vocab is None:
        raise ValueError("vocab is needed when logits is None")
    assert weight.numel() * 2 == spexis_packed_weight_size(vocab, hidden_dim), "weight must be packed"
    _check(lib().spexis_lm_head_gather(
        _ptr(hidden, torch.bfloat16), _ptr(weight, torch.bfloat16), rows, vocab, hidden_dim,
        ctypes.c_float(temperature), _ptr(logits, torch.float32), _ptr(stats, torch.float32),
        _ptr(gather_cols, torch.int32), _ptr(gathered, torch.float32), _stream(stream)))


def spexis_verify_gather_columns(query_start_loc, draft_ids, cols, stream=None) -> None:
    """cols[qsl[b]+i] = the draft id row qsl[b]+i verifies (i < k_b), -1 for bonus rows."""
    num_seqs = query_start_loc.shape[0] - 1
    total = cols.shape[0]
    _check(lib().spexis_verify_gather_columns(num_seqs, total, _ptr(query_start_loc, torch.int32),
                                              _ptr(draft_ids, torch.int32) if draft_ids.numel() else None,
                                              _ptr(cols, torch.int32), _stream(stream)))


def spexis_accept_with_stats(query_start_loc, target_logits, draft_logits, target_stats, draft_stats, draft_ids,
                             u_accept, u_sample, max_k, accepted_len, out_tokens, row_status, workspace,
                             temperature=1.0, seq_lens_inout=None, target_gathered=None, draft_gathered=None,
                             stream=None) -> None:
    num_seqs = query_start_loc.shape[0] - 1
    total_tokens, vocab = target_logits.shape
    tiles = target_stats.shape[1]
    nd = total_tokens - num_seqs
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().spexis_accept_with_stats(
        num_seqs, vocab, max_k, ctypes.c_float(temperature), total_tokens, _ptr(query_start_loc, torch.int32),
        _ptr(target_logits, torch.float32), _ptr(draft_logits, torch.float32) if nd > 0 else None,
        _ptr(target_stats, torch.float32), _ptr(draft_stats, torch.float32) if nd > 0 else None, tiles,
        _ptr(draft_ids, torch.int32) if nd > 0 else None, _ptr(u_accept, torch.float32) if nd > 0 else None,
        _ptr(u_sample, torch.float32), _ptr(target_gathered, torch.float32), _ptr(draft_gathered, torch.float32),
        _ptr(accepted_len, torch.int32), _ptr(out_tokens, torch.int32),
        _ptr(row_status, torch.int32), _ptr(seq_lens_inout, torch.int32), _ptr(workspace), ws_bytes,
        _stream(stream)))


def spexis_select_drafts(query_start_loc, draft_conf, alpha, kept_k, kept_query_start_loc, keep,
                         stream=None) -> None:
    num_seqs = query_start_loc.shape[0] - 1
    n = draft_conf.shape[0]
    _check(lib().spexis_select_drafts(
        num_seqs, num_seqs + n, _ptr(query_start_loc, torch.int32), _ptr(draft_conf, torch.float32) if n else None,
        ctypes.c_float(alpha), _ptr(kept_k, torch.int32), _ptr(kept_query_start_loc, torch.int32),
        _ptr(keep, torch.int32) if n else None, _stream(stream)))


def spexis_lookahead_memory(cur_len, remaining, precision, pp, theta, mem, e_gen=None, e_nfin=None, e_lfin=None,
                            stream=None) -> None:
    """Algorithm 1's look-ahead memory estimate for len(mem) iterations (fp64 outputs)."""
    n = cur_len.shape[0]
    opt = lambda t: _ptr(t, torch.float64) if t is not None else None
    _check(lib().spexis_lookahead_memory(
        n, _ptr(cur_len, torch.int64) if n else None, _ptr(remaining, torch.int32) if n else None,
        _ptr(precision, torch.float64) if n else None, pp, ctypes.c_double(theta), mem.shape[0],
        _ptr(mem, torch.float64), opt(e_gen), opt(e_nfin), opt(e_lfin), _stream(stream)))


def spexis_linear_workspace_size(rows: int, out_features: int, in_features: int) -> int:
    return int(lib().spexis_linear_workspace_size(rows, out_features, in_features))


def spexis_linear(x, weight, y, residual=None, workspace=None, stream=None) -> None:
    """y = bf16(x weight^T (+ residual)) for bf16 x [rows, in] and a packed weight [out, in]
    (spexis_pack_weight); out is y's width."""
    rows, n_in = x.shape
    n_out = y.shape[1]
    assert weight.numel() * 2 == spexis_packed_weight_size(n_out, n_in), "weight must be packed"
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().spexis_linear(_ptr(x, torch.bfloat16), _ptr(weight, torch.bfloat16),
                               _ptr(residual, torch.bfloat16) if residual is not None else None, rows, n_out, n_in,
                               _ptr(y, torch.bfloat16), _ptr(workspace) if workspace is not None else None, ws_bytes,
                               _stream(stream)))


def spexis_linear_split_workspace_size(rows: int, total_out_features: int, in_features: int) -> int:
    return int(lib().spexis_linear_split_workspace_size(rows, total_out_features, in_features))


def spexis_linear_split(x, weight, outputs, workspace, stream=None) -> None:
    """outputs[i] = bf16(x W_i^T) for bf16 x [rows, in] and the packed stack of the weights W_i
    (spexis_pack_weight of their rows stacked in output order); W_i's height is outputs[i]'s
    width."""
    rows, n_in = x.shape
    widths = [int(o.shape[1]) for o in outputs]
    assert all(int(o.shape[0]) == rows for o in outputs)
    assert weight.numel() * 2 == spexis_packed_weight_size(sum(widths), n_in), "weight must be packed"
    m = len(widths)
    w_arr = (ctypes.c_int32 * m)(*widths)
    o_arr = (ctypes.c_void_p * m)(*[_ptr(o, torch.bfloat16).value for o in outputs])
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().spexis_linear_split(_ptr(x, torch.bfloat16), _ptr(weight, torch.bfloat16), rows, n_in, m, w_arr,
                                     o_arr, _ptr(workspace), ws_bytes, _stream(stream)))


def spexis_sample_workspace_size(rows: int, vocab: int) -> int:
    return int(lib().spexis_sample_workspace_size(rows, vocab))


def spexis_sample_tokens(kind, inputs, u, tokens, row_status, workspace, token_prob=None, stats=None,
                         temperature=1.0, stream=None) -> None:
    """One token per row of `inputs` [rows, V] (logits or probabilities), with its probability."""
    rows, V = inputs.shape
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().spexis_sample_tokens(
        kind, rows, V, ctypes.c_float(temperature), _ptr(inputs, torch.float32),
        _ptr(stats, torch.float32) if stats is not None else None, stats.shape[1] if stats is not None else 0,
        _ptr(u, torch.float32), _ptr(tokens, torch.int32),
        _ptr(token_prob, torch.float32) if token_prob is not None else None, _ptr(row_status, torch.int32),
        _ptr(workspace), ws_bytes, _stream(stream)))


def spexis_packed_weight_size(rows: int, cols: int) -> int:
    return int(lib().spexis_packed_weight_size(rows, cols))


def spexis_pack_weight(weight, stream=None) -> torch.Tensor:
    """The packed layout of a bf16 weight [rows, cols] (a new flat bf16 tensor), for
    spexis_lm_head and spexis_linear; allocated here, once per weight."""
    rows, cols = weight.shape
    n = spexis_packed_weight_size(rows, cols)
    if n == 0:
        raise SpexisError(SPEXIS_ERR_UNSUPPORTED, f"cannot pack a [{rows}, {cols}] weight")
    out = torch.empty(n // 2, dtype=torch.bfloat16, device=weight.device)
    _check(lib().spexis_pack_weight(_ptr(weight, torch.bfloat16), rows, cols, _ptr(out, torch.bfloat16),
                                    _stream(stream)))
    return out
