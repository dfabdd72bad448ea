"""CPU oracle of the speculative verification step -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and its Python
binding) never does, and shares no code with it: ``spexis_oracle.c`` restates the cache
layout, the fp64 attention, the fp64 softmax and the exact-arithmetic acceptance rule from
their definitions (see the header of that file for the passages each function follows).

Everything here takes and returns numpy arrays on the host.  bf16 tensors are passed as
their uint16 bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "spexis_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libspexis_oracle.so")

# row_status codes of the acceptance rule
OK, EMPTY_ROW, BAD_ROW, BAD_TOKEN = 0, 1, 2, 3


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (plain C11 + OpenMP, no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                               "-Wall", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        L.oracle_append_kv.argtypes = [P, P, i32, i32, i32, i32, i32, P, P, P, i32, P, P]
        L.oracle_append_kv.restype = ctypes.c_int
        L.oracle_attention.argtypes = [P, P, i32, i32, i32, i32, i32, P, P, P, i32, P, i32, f32, P, i32, P]
        L.oracle_attention.restype = ctypes.c_int
        L.oracle_softmax.argtypes = [P, i64, i32, f32, P]
        L.oracle_lm_head.argtypes = [P, P, i64, i32, i32, f32, P, P, P]
        L.oracle_select_drafts.argtypes = [i32, P, P, f32, P, P, P]
        L.oracle_select_drafts.restype = ctypes.c_int
        L.oracle_linear.argtypes = [P, P, P, i64, i32, i32, P]
        L.oracle_lookahead.argtypes = [i32, P, P, P, i32, ctypes.c_double, i32, P, P, P, P]
        L.oracle_lookahead.restype = ctypes.c_int
        L.oracle_softmax.restype = None
        L.oracle_accept.argtypes = [i32, i32, i32, P, P, P, P, P, P, P, P, P, P]
        L.oracle_accept.restype = None
        L.oracle_set_num_threads.argtypes = [ctypes.c_int]
        L.oracle_set_num_threads.restype = None
        L.oracle_num_threads.argtypes = []
        L.oracle_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _c(a: np.ndarray, dtype) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on."""
    lib().oracle_set_num_threads(int(n))


def append_kv(k_pool: np.ndarray, v_pool: np.ndarray, num_blocks: int, num_kv_heads: int, block_size: int,
              head_dim: int, qsl, seq_lens, block_tables, new_k: np.ndarray, new_v: np.ndarray) -> None:
    """Write new K/V rows [T, Hkv, D] (uint16 bf16 bits) into the pools, in place."""
    assert k_pool.dtype == np.uint16 and v_pool.dtype == np.uint16
    assert k_pool.flags.c_contiguous and v_pool.flags.c_contiguous
    qsl, seq_lens = _c(qsl, np.int32), _c(seq_lens, np.int32)
    bt = _c(block_tables, np.int32)
    nk, nv = _c(new_k, np.uint16), _c(new_v, np.uint16)
    B = len(seq_lens)
    rc = lib().oracle_append_kv(_p(k_pool), _p(v_pool), num_blocks, num_kv_heads, block_size, head_dim, B,
                                _p(qsl), _p(seq_lens), _p(bt), bt.shape[1], _p(nk), _p(nv))
    if rc != 0:
        raise ValueError("oracle_append_kv: index out of range")


def attention(k_pool: np.ndarray, v_pool: np.ndarray, num_blocks: int, num_kv_heads: int, block_size: int,
              head_dim: int, qsl, seq_lens, block_tables, q: np.ndarray, num_q_heads: int, scale: float,
              seqs=None, out: np.ndarray = None) -> np.ndarray:
    """fp64 attention output [T, Hq, D]; only rows of ``seqs`` (default: all) are computed."""
    qsl, seq_lens = _c(qsl, np.int32), _c(seq_lens, np.int32)
    bt = _c(block_tables, np.int32)
    qq = _c(q, np.uint16)
    B = len(seq_lens)
    T = int(qsl[-1])
    seqs = _c(np.arange(B) if seqs is None else seqs, np.int32)
    if out is None:
        out = np.full((T, num_q_heads, head_dim), np.nan, dtype=np.float64)
    assert out.dtype == np.float64 and out.flags.c_contiguous
    rc = lib().oracle_attention(_p(k_pool), _p(v_pool), num_blocks, num_kv_heads, block_size, head_dim, B,
                                _p(qsl), _p(seq_lens), _p(bt), bt.shape[1], _p(qq), num_q_heads,
                                ctypes.c_float(scale), _p(seqs), len(seqs), _p(out))
    if rc != 0:
        raise ValueError("oracle_attention: bad arguments or index out of range")
    return out


def softmax(logits: np.ndarray, temperature: float = 1.0) -> np.ndarray:
    """fp32 probabilities of fp32 logits [rows, V], computed in fp64."""
    x = _c(logits, np.float32)
    rows, V = x.shape
    out = np.empty_like(x)
    lib().oracle_softmax(_p(x), rows, V, ctypes.c_float(temperature), _p(out))
    return out


def lm_head(h: np.ndarray, W: np.ndarray, temperature: float = 1.0, want_logits: bool = True):
    """fp64 logits h W^T of bf16 bit arrays h [rows, d], W [V, d], and each row's softmax
    statistics at `temperature`: (logits or None, mx [rows], z [rows]) with
    mx = max(logits) / T and z = sum(exp(logits / T - mx))."""
    hh = _c(h, np.uint16)
    ww = _c(W, np.uint16)
    rows, d = hh.shape
    V, d2 = ww.shape
    assert d == d2
    logits = np.empty((rows, V), np.float64) if want_logits else None
    mx = np.empty(rows, np.float64)
    z = np.empty(rows, np.float64)
    lib().oracle_lm_head(_p(hh), _p(ww), rows, V, d, ctypes.c_float(temperature),
                         _p(logits) if want_logits else None, _p(mx), _p(z))
    return logits, mx, z


def select_drafts(qsl, conf, alpha: float):
    """Selective speculation: (kept_k [B], kept_qsl [B+1], keep [N]) for draft confidences conf [N]
    of the batch qsl (drafts of sequence b at qsl[b]-b ..)."""
    qsl = _c(qsl, np.int32)
    B = len(qsl) - 1
    N = int(qsl[-1]) - B
    cf = _c(conf, np.float32) if N > 0 else np.zeros(1, np.float32)
    kept_k = np.empty(B, np.int32)
    kept_qsl = np.empty(B + 1, np.int32)
    keep = np.empty(max(N, 1), np.int32)
    rc = lib().oracle_select_drafts(B, _p(qsl), _p(cf), ctypes.c_float(alpha), _p(kept_k), _p(kept_qsl), _p(keep))
    if rc != 0:
        raise ValueError("oracle_select_drafts: bad arguments")
    return kept_k, kept_qsl, keep[:N]


def linear(x: np.ndarray, W: np.ndarray, residual=None):
    """fp64 y = x W^T (+ residual) of bf16 bit arrays x [rows, in], W [out, in], residual [rows, out]."""
    xx = _c(x, np.uint16)
    ww = _c(W, np.uint16)
    rows, n_in = xx.shape
    n_out, n_in2 = ww.shape
    assert n_in == n_in2
    rr = _c(residual, np.uint16) if residual is not None else None
    if rr is not None:
        assert rr.shape == (rows, n_out)
    y = np.empty((rows, n_out), np.float64)
    lib().oracle_linear(_p(xx), _p(ww), _p(rr) if rr is not None else None, rows, n_out, n_in, _p(y))
    return y


def to_bf16(x) -> np.ndarray:
    """Bits of the bf16 nearest to each value (ties to even), through fp32."""
    f = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = f + np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_value(bits) -> np.ndarray:
    """fp64 values of bf16 bit patterns."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def sample(probs: np.ndarray, u):
    """One token per fp32 probability row by the exact inverse CDF of acceptance with no drafts,
    and its probability: (tokens [R], token_prob [R], row_status [R])."""
    pr = _c(probs, np.float32)
    R, V = pr.shape
    qsl = np.arange(R + 1, dtype=np.int32)
    _, toks, status, _ = accept(qsl, pr, np.zeros((0, V), np.float32), np.zeros(0, np.int32), np.zeros(0, np.float32),
                                u, max_k=0)
    tok = toks[:, 0].copy()
    prob = np.where(tok >= 0, pr[np.arange(R), np.maximum(tok, 0)], np.float32(0)).astype(np.float32)
    return tok, prob, status


def draft_step(h, w_in, w_q, w_k, w_v, w_o, w_lm, k_pool, v_pool, num_blocks, num_kv_heads, num_q_heads,
               block_size, head_dim, seq_lens, block_tables, temperature, u):
    """The drafting adapter's forward and the draft draw for one query token per sequence, in
    the adapter's order (a linear layer, an attention layer, the LM head), every intermediate
    rounded to bf16 as the tensors that hold it; the pools are updated in place.  All weights
    and states are bf16 bit arrays.  Returns a dict of the intermediates and (tokens, conf,
    status)."""
    B = len(seq_lens)
    qsl = np.arange(B + 1, dtype=np.int32)
    x = to_bf16(linear(h, w_in))
    q = to_bf16(linear(x, w_q))
    k = to_bf16(linear(x, w_k))
    v = to_bf16(linear(x, w_v))
    append_kv(k_pool, v_pool, num_blocks, num_kv_heads, block_size, head_dim, qsl, seq_lens, block_tables,
              k.reshape(B, num_kv_heads, head_dim), v.reshape(B, num_kv_heads, head_dim))
    o = attention(k_pool, v_pool, num_blocks, num_kv_heads, block_size, head_dim, qsl, seq_lens, block_tables,
                  q.reshape(B, num_q_heads, head_dim), num_q_heads, 1.0 / np.sqrt(head_dim))
    o = to_bf16(o.reshape(B, num_q_heads * head_dim))
    y = to_bf16(linear(o, w_o, x))
    logits, _, _ = lm_head(y, w_lm, temperature)
    p = softmax(logits.astype(np.float32), temperature)
    tok, conf, status = sample(p, u)
    return dict(x=x, q=q, k=k, v=v, o=o, y=y, logits=logits, probs=p, tokens=tok, conf=conf, status=status)


def batch_recurrence(B: float, alpha: float, N: int, steps: int = 20000) -> float:
    """B_t of the selective-speculation recurrence B_{t+1} = alpha B_{t+1-N} + (1 - alpha) B_t
    (Sec. 5, Eq. 3) iterated from B_0 = B with no earlier history (B_t = 0 for t < 0)."""
    hist = [0.0] * (N - 1) + [float(B)]   # B_{t-N+1} .. B_t
    for _ in range(steps):
        nxt = alpha * hist[-N] + (1.0 - alpha) * hist[-1] if N > 1 else hist[-1]
        hist.append(nxt)
        hist.pop(0)
    return hist[-1]


def lookahead(cur_len, remaining, precision, pp: int, theta: float, iters: int = 64):
    """Algorithm 1: (mem, e_gen, e_nfin, e_lfin), each fp64 [iters], for the running requests'
    current lengths, predicted remaining lengths and prediction precisions."""
    n = len(cur_len)
    cl = _c(cur_len, np.int64) if n else np.zeros(1, np.int64)
    rm = _c(remaining, np.int32) if n else np.zeros(1, np.int32)
    pr = _c(precision, np.float64) if n else np.zeros(1, np.float64)
    out = [np.empty(iters, np.float64) for _ in range(4)]
    rc = lib().oracle_lookahead(n, _p(cl), _p(rm), _p(pr), pp, ctypes.c_double(theta), iters, *[_p(o) for o in out])
    if rc != 0:
        raise ValueError("oracle_lookahead: bad arguments")
    return tuple(out)


def accept(qsl, target: np.ndarray, draft: np.ndarray, draft_ids, u_accept, u_sample, max_k: int = None,
           seq_lens=None):
    """Acceptance on fp32 probability rows.

    Returns (accepted_len [B], out_tokens [B, max_k+1], row_status [B], new_seq_lens or None).
    """
    qsl = _c(qsl, np.int32)
    B = len(qsl) - 1
    tg = _c(target, np.float32)
    V = tg.shape[1]
    nd = int(qsl[-1]) - B
    dr = _c(draft, np.float32).reshape(nd, V) if nd > 0 else np.zeros((1, V), np.float32)
    ids = _c(draft_ids, np.int32) if nd > 0 else np.zeros(1, np.int32)
    ua = _c(u_accept, np.float32) if nd > 0 else np.zeros(1, np.float32)
    us = _c(u_sample, np.float32)
    if max_k is None:
        max_k = int((np.diff(qsl) - 1).max())
    acc = np.empty(B, np.int32)
    toks = np.empty((B, max_k + 1), np.int32)
    status = np.empty(B, np.int32)
    sl = _c(seq_lens, np.int32).copy() if seq_lens is not None else None
    lib().oracle_accept(B, V, max_k, _p(qsl), _p(tg), _p(dr), _p(ids), _p(ua), _p(us), _p(acc), _p(toks),
                        _p(status), _p(sl) if sl is not None else None)
    return acc, toks, status, sl
