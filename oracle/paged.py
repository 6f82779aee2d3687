"""Read a request's logical keys/values out of the library's documented paged
cache layout (test infrastructure only).

Layout (block = 16 tokens): K and V pools are [blocks][Hkv][16 * hd]; inside
the tile of a (block, head), token slot t and dimension h sit at
    K: ((h // 32) * 64 + ((h % 32) // 8) * 16 + t) * 8 + h % 8
    V: (((h // 32) * 64 + (t // 4) * 16 + h % 16) * 2 + (h // 16) % 2) * 4 + t % 4
Token t of a request lives in block block_table_row[t // 16], slot t % 16.
"""
from __future__ import annotations

import numpy as np

BLOCK = 16


def tile_index(hd: int):
    """Offsets of (slot, dim) in a K tile and a V tile, each [16, hd]."""
    t = np.arange(BLOCK)[:, None]
    h = np.arange(hd)[None, :]
    k = ((h // 32) * 64 + ((h % 32) // 8) * 16 + t) * 8 + h % 8
    v = (((h // 32) * 64 + (t // 4) * 16 + h % 16) * 2 + (h // 16) % 2) * 4 + t % 4
    return k, v


def depage_blocks(k_blocks: np.ndarray, v_blocks: np.ndarray, n: int):
    """Keys and values of tokens 0..n-1 as float64 [n, Hkv, hd], from the
    request's blocks gathered in table order (k_blocks, v_blocks:
    [nb][Hkv][16 * hd])."""
    nb, Hkv, tile = k_blocks.shape
    hd = tile // BLOCK
    ki, vi = tile_index(hd)
    K = k_blocks[:, :, ki]          # [nb, Hkv, 16, hd]
    V = v_blocks[:, :, vi]
    K = K.transpose(0, 2, 1, 3).reshape(nb * BLOCK, Hkv, hd)[:n]
    V = V.transpose(0, 2, 1, 3).reshape(nb * BLOCK, Hkv, hd)[:n]
    return np.asarray(K, np.float64), np.asarray(V, np.float64)
