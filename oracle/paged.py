"""Read a request's logical keys/values out of the library's documented paged
cache layout (test infrastructure only).

Layout (block = 16 tokens): K pool [blocks][Hkv][16][hd], V pool
[blocks][Hkv][hd][16]; token t of a request lives in block
block_table_row[t // 16], slot t % 16.
"""
from __future__ import annotations

import numpy as np

BLOCK = 16


def depage(k_pool: np.ndarray, v_pool: np.ndarray, table_row: np.ndarray, n: int):
    """Keys and values of tokens 0..n-1 as float64 arrays [n, Hkv, hd]."""
    Hkv, hd = k_pool.shape[1], k_pool.shape[3]
    K = np.zeros((n, Hkv, hd))
    V = np.zeros((n, Hkv, hd))
    for t in range(n):
        b, slot = int(table_row[t // BLOCK]), t % BLOCK
        K[t] = k_pool[b, :, slot, :]
        V[t] = v_pool[b, :, :, slot]
    return K, V


def depage_blocks(k_blocks: np.ndarray, v_blocks: np.ndarray, n: int):
    """Same, for the request's blocks already gathered in table order
    (k_blocks [nb][Hkv][16][hd], v_blocks [nb][Hkv][hd][16])."""
    nb, Hkv, hd = k_blocks.shape[0], k_blocks.shape[1], k_blocks.shape[3]
    K = k_blocks.transpose(0, 2, 1, 3).reshape(nb * BLOCK, Hkv, hd)[:n]
    V = v_blocks.transpose(0, 3, 1, 2).reshape(nb * BLOCK, Hkv, hd)[:n]
    return np.asarray(K, np.float64), np.asarray(V, np.float64)
