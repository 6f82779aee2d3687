"""Device tensors of a workload (inputs only; no layer arithmetic).

Weights and cache pools are generated directly on the target device with the
counter-based generator, so full-size layers appear in HBM in milliseconds
with exactly the bits the CPU generator gives.
"""
from __future__ import annotations

import numpy as np
import torch

from . import Batch, LayerShape, hidden_states, kv_pool, layer_weights


def layer_tensors(shape: LayerShape, tag: str, layer: int, num_blocks: int,
                  device="cuda") -> dict:
    """Weights of one layer plus its K and V pools, all on `device`."""
    t = layer_weights(shape, tag, layer, device=device)
    t["k_cache"] = kv_pool(shape, tag, layer, num_blocks, "k", device=device)
    t["v_cache"] = kv_pool(shape, tag, layer, num_blocks, "v", device=device)
    return t


def batch_tensors(b: Batch, device="cuda") -> dict:
    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)
    return {
        "row_idx": i32(b.row_idx),
        "positions": i32(b.positions),
        "seq_starts": None if b.seq_starts is None else i32(b.seq_starts),
        "block_table": i32(b.block_table),
        "ctx_lens": i32(b.ctx_lens),
    }


def hidden_tensor(shape: LayerShape, tag: str, rows: int, device="cuda") -> torch.Tensor:
    return hidden_states(shape, tag, rows, device=device)
