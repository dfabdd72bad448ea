"""The test suite's own reading of the paged-cache layout documented in include/spexis.h.

    K pool: bf16 [num_blocks][Hkv][D/8][bs][8]
    V pool: bf16 [num_blocks][Hkv][D][bs], slot index stored with bits 2 and 3 swapped

Written with numpy fancy indexing, independently of the oracle's C loops and of the HIP
kernels, so that a layout mistake in either shows up as a disagreement with this file.
"""
import numpy as np


def swap23(slot):
    slot = np.asarray(slot)
    return (slot & ~12) | (((slot >> 2) & 1) << 3) | (((slot >> 3) & 1) << 2)


def k_offsets(blk, h, slot, d, hkv, bs, D):
    return (((blk * hkv + h) * (D // 8) + d // 8) * bs + slot) * 8 + d % 8


def v_offsets(blk, h, slot, d, hkv, bs, D):
    return ((blk * hkv + h) * D + d) * bs + swap23(slot)


def token_blocks(block_table_row, S, bs):
    t = np.arange(S)
    return block_table_row[t // bs], t % bs


def gather_seq(pool, which, block_table_row, S, hkv, bs, D):
    """Logical rows [S, Hkv, D] of one sequence read out of a flat pool."""
    blk, slot = token_blocks(block_table_row, S, bs)
    h = np.arange(hkv)
    d = np.arange(D)
    B_, H_, D_ = np.meshgrid(np.arange(S), h, d, indexing="ij")
    f = k_offsets if which == "k" else v_offsets
    off = f(blk[B_], H_, slot[B_], D_, hkv, bs, D)
    return pool[off]


def scatter_seq(pool, which, block_table_row, rows, hkv, bs, D, start=0):
    """Write logical rows [n, Hkv, D] at positions start..start+n of one sequence."""
    n = rows.shape[0]
    t = np.arange(start, start + n)
    blk, slot = block_table_row[t // bs], t % bs
    T_, H_, D_ = np.meshgrid(np.arange(n), np.arange(hkv), np.arange(D), indexing="ij")
    f = k_offsets if which == "k" else v_offsets
    off = f(blk[T_], H_, slot[T_], D_, hkv, bs, D)
    pool[off] = rows
