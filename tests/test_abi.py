"""The C-ABI library loads, exports every function include/spexis.h declares, and rejects
bad scalar arguments on the host with the documented codes (no GPU needed: validation
returns before any device call)."""
import ctypes
import math
import os
import subprocess

import pytest
import torch

from paper_2609_34370_amd import spexis as sx

pytestmark = pytest.mark.skipif(not os.path.exists(sx.LIB_PATH), reason="libspexis.so not built")

# Never dereferenced: every call that passes FAKE fails host validation before any launch.
# As a second guard these calls only run where no GPU is visible.
FAKE = ctypes.c_void_p(256)
no_gpu = pytest.mark.skipif(torch.cuda.is_available(), reason="fake-pointer validation runs only without a GPU")


def test_every_header_function_is_exported():
    declared = sx.header_functions()
    assert {"spexis_append_kv", "spexis_verify_attention", "spexis_accept"} <= set(declared)
    out = subprocess.run(["nm", "-D", "--defined-only", sx.LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    missing = [f for f in declared if f not in exported]
    assert not missing, missing
    L = sx.lib()
    for f in declared:
        assert hasattr(L, f)


@no_gpu
def test_version_and_last_error():
    assert sx.spexis_version() == 100
    L = sx.lib()
    assert L.spexis_append_kv(None, None, 1, 1, 16, 64, 1, None, None, None, 1, 1, 1, None, None, None) == \
        sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert b"null pointer" in L.spexis_last_error()


def attn(**kw):
    a = dict(k=FAKE, v=FAKE, nb=10, hkv=2, bs=16, d=64, B=2, qsl=FAKE, sl=FAKE, bt=FAKE, mb=4, T=4, mq=2, ms=40,
             q=FAKE, hq=8, scale=0.125, out=ctypes.c_void_p(512), chunk=0, ws=None, wsb=0)
    a.update(kw)
    return sx.lib().spexis_verify_attention(a["k"], a["v"], a["nb"], a["hkv"], a["bs"], a["d"], a["B"], a["qsl"],
                                            a["sl"], a["bt"], a["mb"], a["T"], a["mq"], a["ms"], a["q"], a["hq"],
                                            ctypes.c_float(a["scale"]), a["out"], a["chunk"], a["ws"], a["wsb"],
                                            None)


@no_gpu
def test_attention_validation():
    assert attn(hq=7) == sx.SPEXIS_ERR_INVALID_ARGUMENT          # Hq not a multiple of Hkv
    assert attn(d=96) == sx.SPEXIS_ERR_UNSUPPORTED
    assert attn(bs=8) == sx.SPEXIS_ERR_UNSUPPORTED
    assert attn(hq=66, hkv=2, mq=3) == sx.SPEXIS_ERR_UNSUPPORTED  # G = 33, 99 rows
    assert attn(out=FAKE) == sx.SPEXIS_ERR_INVALID_ARGUMENT       # out aliases q
    assert attn(scale=float("nan")) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert attn(ms=4000, chunk=32) == sx.SPEXIS_ERR_WORKSPACE_TOO_SMALL
    assert b"workspace" in sx.lib().spexis_last_error()


def test_workspace_queries():
    # attention: one header and two partial slots per wave; each KV head's tiles are cut into
    # shares (the even split: about 1024 waves in all, at least 2 tiles a share, shares in pairs
    # and a grid of a multiple of 8 and of 2 hkv waves within 1024; a fixed share size: enough
    # shares for the largest possible stream), one wave per (share, head)
    def expect(B, hq, hkv, D, mq, max_s, chunk):
        rows = (hq // hkv) * mq
        slot = -(-rows * (D + 2) // 16) * 16
        tiles = B * -(-max_s // 32)
        per = -(-chunk // 32) if chunk else 2
        shares = max(-(-tiles // per), 1)
        step = 4
        if not chunk:
            shares = min(shares, max(1, 1024 // hkv))
            L = math.lcm(8, 2 * hkv)
            s2 = shares - shares % 2
            while s2 > 2 and -(-(s2 * hkv) // L) * L > 1024:
                s2 -= 2
            if shares >= 2 and -(-(s2 * hkv) // L) * L <= 1024:
                shares, step = s2, L
        waves = -(-(shares * hkv) // step) * step
        return waves * (2 * slot * 4 + 8 * 4)
    for args in [(4, 8, 2, 64, 5, 256, 0), (64, 32, 8, 128, 5, 4100, 0), (64, 32, 8, 128, 5, 4100, 100),
                 (1, 8, 8, 128, 1, 1, 0), (3, 64, 8, 128, 8, 16384, 4096), (5, 24, 3, 128, 4, 3000, 0),
                 (7, 12, 12, 64, 2, 700, 0), (2, 40, 5, 128, 3, 33, 0), (64, 300, 300, 64, 1, 4100, 0)]:
        n = sx.spexis_verify_attention_workspace_size(*args)
        assert n == expect(*args) and n % 64 == 0, args
    assert sx.spexis_verify_attention_workspace_size(64, 32, 8, 128, 5, 1 << 20, 0) <= 1024 * (2 * 2608 * 4 + 32)
    assert sx.spexis_verify_attention_workspace_size(0, 32, 8, 128, 5, 4100, 0) == 0
    assert sx.spexis_accept_workspace_size(64, 128256, 4) > 64 * 32 * 8


def acc(**kw):
    a = dict(kind=1, B=2, V=100, mk=2, t=1.0, T=6, qsl=FAKE, tg=FAKE, dr=FAKE, ids=FAKE, ua=FAKE, us=FAKE,
             al=FAKE, ot=FAKE, rs=FAKE, sl=None, ws=FAKE, wsb=1 << 20)
    a.update(kw)
    return sx.lib().spexis_accept(a["kind"], a["B"], a["V"], a["mk"], ctypes.c_float(a["t"]), a["T"], a["qsl"],
                                  a["tg"], a["dr"], a["ids"], a["ua"], a["us"], a["al"], a["ot"], a["rs"], a["sl"],
                                  a["ws"], a["wsb"], None)


@no_gpu
def test_accept_validation():
    assert acc(kind=5) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc(t=0.0) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc(t=-1.0) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc(dr=None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc(mk=33) == sx.SPEXIS_ERR_UNSUPPORTED
    assert acc(V=(1 << 22) + 1) == sx.SPEXIS_ERR_UNSUPPORTED
    assert acc(wsb=16) == sx.SPEXIS_ERR_WORKSPACE_TOO_SMALL
    assert acc(T=1) == sx.SPEXIS_ERR_INVALID_ARGUMENT            # fewer rows than sequences


def acc_noalloc(**kw):
    a = dict(kind=1, B=2, V=100, mk=2, t=1.0, T=6, qsl=FAKE, tg=FAKE, dr=FAKE, ids=FAKE, ua=FAKE, us=FAKE,
             al=FAKE, ot=FAKE, rs=FAKE, sl=None)
    a.update(kw)
    return sx.lib().spexis_accept_noalloc(a["kind"], a["B"], a["V"], a["mk"], ctypes.c_float(a["t"]), a["T"],
                                          a["qsl"], a["tg"], a["dr"], a["ids"], a["ua"], a["us"], a["al"], a["ot"],
                                          a["rs"], a["sl"], None)


@no_gpu
def test_accept_noalloc_validation():
    # the same host checks as spexis_accept, and a problem beyond the static scratch array is
    # rejected before the array is ever looked up
    assert acc_noalloc(kind=5) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc_noalloc(t=0.0) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc_noalloc(dr=None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert acc_noalloc(mk=33) == sx.SPEXIS_ERR_UNSUPPORTED
    B, V, K = 512, 1 << 18, 32
    assert sx.spexis_accept_workspace_size(B, V, K) > sx.SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES
    assert acc_noalloc(B=B, V=V, mk=K, T=B * (K + 1)) == sx.SPEXIS_ERR_UNSUPPORTED
    assert b"scratch" in sx.lib().spexis_last_error()
    assert acc_noalloc(B=0, T=0, qsl=None, tg=None, dr=None, ids=None, ua=None, us=None, al=None, ot=None,
                       rs=None) == sx.SPEXIS_OK


@no_gpu
def test_lm_head_gather_validation():
    L = sx.lib()
    # a NULL gathered output or column array, and a hidden size the projection does not take
    assert L.spexis_lm_head_gather(FAKE, FAKE, 8, 1000, 256, ctypes.c_float(1.0), None, FAKE, FAKE, None,
                                   None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_lm_head_gather(FAKE, FAKE, 8, 1000, 256, ctypes.c_float(1.0), None, FAKE, None, FAKE,
                                   None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_lm_head_gather(FAKE, FAKE, 8, 1000, 300, ctypes.c_float(1.0), None, FAKE, FAKE, FAKE,
                                   None) == sx.SPEXIS_ERR_UNSUPPORTED
    assert L.spexis_verify_gather_columns(3, 2, FAKE, FAKE, FAKE, None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_verify_gather_columns(3, 7, None, FAKE, FAKE, None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_verify_gather_columns(0, 0, None, None, None, None) == sx.SPEXIS_OK
    # acceptance takes both gathered arrays or neither
    a = [2, 100, 2, ctypes.c_float(1.0), 6, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, FAKE, FAKE]
    assert L.spexis_accept_with_stats(*a, FAKE, None, FAKE, FAKE, FAKE, None, FAKE, 1 << 20, None) == \
        sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert b"gathered" in L.spexis_last_error()


@no_gpu
def test_softmax_validation():
    L = sx.lib()
    assert L.spexis_softmax_rows(FAKE, FAKE, 4, 10, ctypes.c_float(0.0), None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_softmax_rows(FAKE, FAKE, -1, 10, ctypes.c_float(1.0), None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert L.spexis_softmax_rows(None, FAKE, 4, 10, ctypes.c_float(1.0), None) == sx.SPEXIS_ERR_INVALID_ARGUMENT


@no_gpu
def test_append_validation():
    L = sx.lib()
    assert L.spexis_append_kv(FAKE, FAKE, 10, 2, 8, 64, 2, FAKE, FAKE, FAKE, 4, 4, 2, FAKE, FAKE, None) == \
        sx.SPEXIS_ERR_UNSUPPORTED
    assert L.spexis_append_kv(FAKE, FAKE, 0, 2, 16, 64, 2, FAKE, FAKE, FAKE, 4, 4, 2, FAKE, FAKE, None) == \
        sx.SPEXIS_ERR_INVALID_ARGUMENT
    # nothing to do: no launch, success
    assert L.spexis_append_kv(FAKE, FAKE, 10, 2, 16, 64, 0, FAKE, FAKE, FAKE, 4, 0, 2, FAKE, FAKE, None) == sx.SPEXIS_OK


def split(widths, rows=4, n_in=256, outs=None, ws=FAKE, wsb=1 << 30, x=FAKE, w=FAKE):
    m = len(widths)
    w_arr = (ctypes.c_int32 * max(m, 1))(*widths)
    o_arr = (ctypes.c_void_p * max(m, 1))(*([256 * (i + 4) for i in range(m)] if outs is None else outs))
    return sx.lib().spexis_linear_split(x, w, rows, n_in, m, w_arr, o_arr, ws, wsb, None)


@no_gpu
def test_linear_split_validation():
    assert split([]) == sx.SPEXIS_ERR_INVALID_ARGUMENT                      # no outputs
    assert split([8, 8, 8, 8, 8]) == sx.SPEXIS_ERR_INVALID_ARGUMENT         # more than four
    assert split([8, 0]) == sx.SPEXIS_ERR_INVALID_ARGUMENT                  # empty output
    assert split([8, 6]) == sx.SPEXIS_ERR_UNSUPPORTED                       # width not a multiple of 4
    assert split([8], n_in=320) == sx.SPEXIS_ERR_UNSUPPORTED                # in_features % 256
    assert split([8], rows=-1) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert split([8], rows=0, x=None, w=None, outs=[None], ws=None, wsb=0) == sx.SPEXIS_OK   # no work
    assert split([8], x=None) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert split([8, 8], outs=[512, None]) == sx.SPEXIS_ERR_INVALID_ARGUMENT
    assert split([4096, 1024, 1024], rows=64, n_in=4096, wsb=100) == sx.SPEXIS_ERR_WORKSPACE_TOO_SMALL
    assert b"workspace" in sx.lib().spexis_last_error()


def test_linear_split_workspace_query():
    # the fp32 products of every K-split part pass through the workspace, also without a split
    for rows, n, k in [(64, 6144, 4096), (5, 116, 256), (300, 320, 512), (1, 4, 256)]:
        got = sx.spexis_linear_split_workspace_size(rows, n, k)
        plain = sx.spexis_linear_workspace_size(rows, n, k)
        assert got == (plain if plain > 0 else rows * n * 4), (rows, n, k)
    assert sx.spexis_linear_split_workspace_size(0, 64, 256) == 0
    assert sx.spexis_linear_split_workspace_size(4, 64, 300) == 0

