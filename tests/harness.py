"""Glue shared by the GPU tests and smoke(): build a replica on the GPU from a
workload, run the oracle on chosen rows, compare.

Oracle inputs come from the counter-based generator, never from memory the
library writes:
  * prior cache tokens are always regenerated on the CPU, block by block
    (``W.kv_pool(..., blocks=...)``), so a kernel that overwrote an earlier
    token's slot cannot feed that value to the oracle too;
  * weights are generated on the CPU (``source="cpu"``) or, for the largest
    layers, copied from the weight tensors the same generator produced on the
    GPU (``source="device"``); the library only reads weights, and
    test_generator_is_identical_on_cpu_and_gpu shows the two are bit-identical.
"""
from __future__ import annotations

import math
import time

import numpy as np
import torch

import oracle
import paper_2607_04181_amd as coco
import workloads as W
from oracle.paged import depage_blocks
from workloads import device as WD

# Layer-output bound from the task: max relative error 2e-2, read normwise
# per output tensor: max|gpu - oracle| / max|oracle|.
TOL = 2e-2


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def to64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)


def normwise_err(got, ref) -> float:
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64).reshape(ref.shape)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def elementwise_err(got, ref) -> float:
    """max_i |got_i - ref_i| / max(|ref_i|, rms(ref)): an elementwise relative
    error whose denominator never drops below the tensor's rms (reported next
    to the normwise bound, not bound itself)."""
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64).reshape(ref.shape)
    rms = float(np.sqrt(np.mean(ref * ref))) if ref.size else 0.0
    den = np.maximum(np.abs(ref), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(got - ref) / den)) if ref.size else 0.0


class Replica:
    """Weights, caches and a library handle for a workload's layer(s)."""

    def __init__(self, shape: W.LayerShape, tag: str, n_layers: int, num_blocks: int,
                 max_rows: int, max_seqs: int, max_blocks: int, layers=None):
        self.shape, self.tag, self.n_layers = shape, tag, n_layers
        self.layers = layers if layers is not None else [
            WD.layer_tensors(shape, tag, l, num_blocks) for l in range(n_layers)]
        self.cfg = coco.make_config(shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                                    shape.head_dim, shape.d_ffn, n_layers, shape.dtype, max_rows,
                                    max_seqs, max_blocks, shape.rope_theta, shape.rms_eps)
        self.h = coco.coco_layer_init(self.cfg, self.layers)

    @classmethod
    def for_batch(cls, shape, tag, n_layers, batch: W.Batch, max_rows=None, max_seqs=None):
        return cls(shape, tag, n_layers, batch.num_blocks, max_rows or batch.n_rows,
                   max_seqs or batch.n_seqs, batch.block_table.shape[1])

    def forward(self, layer, hidden, bt: dict, stream=None):
        coco.coco_layer_forward(self.h, layer, hidden, bt["row_idx"], bt["positions"],
                                bt["seq_starts"], bt["block_table"], bt["ctx_lens"], stream)

    def span(self, first, n, hidden, bt: dict, stream=None):
        coco.coco_layer_span_forward(self.h, first, n, hidden, bt["row_idx"], bt["positions"],
                                     bt["seq_starts"], bt["block_table"], bt["ctx_lens"], stream)

    def workspace(self, which, rows, cols, dtype):
        out = torch.empty(rows, cols, dtype=dtype, device="cuda")
        coco.coco_layer_workspace(self.h, which, out)
        torch.cuda.synchronize()
        return out


def oracle_weights(shape, tag, layer, source="cpu", dev_layer=None) -> dict:
    if source == "device":
        t = {k: dev_layer[k] for k in shape.weight_shapes()}
    else:
        t = W.layer_weights(shape, tag, layer)
    return {k: to64(v) for k, v in t.items()}


def oracle_cache(shape, tag, layer, batch: W.Batch, seqs, num_blocks) -> oracle.KVCache:
    """Logical caches of call-sequences `seqs`: the prior tokens regenerated on
    the CPU from the pool's generator stream (never read back from the GPU
    pools, which the library writes), room up to ctx_lens for the tokens the
    call appends."""
    Ks, Vs = [], []
    Hkv, hd = shape.n_kv_heads, shape.head_dim
    for s in seqs:
        prior, ctx = int(batch.prior_lens[s]), int(batch.ctx_lens[s])
        nb = -(-prior // W.BLOCK_SIZE)
        blocks = batch.block_table[s, :nb]
        kb = to64(W.kv_pool(shape, tag, layer, num_blocks, "k", blocks=blocks))
        vb = to64(W.kv_pool(shape, tag, layer, num_blocks, "v", blocks=blocks))
        K = np.zeros((ctx, Hkv, hd))
        V = np.zeros((ctx, Hkv, hd))
        if prior:
            K[:prior], V[:prior] = depage_blocks(kb, vb, prior)
        Ks.append(K)
        Vs.append(V)
    return oracle.KVCache(Ks, Vs)


def oracle_decode_rows(shape, tag, layer, batch: W.Batch, call_rows, hidden64, source="cpu",
                       dev_layer=None, w64=None, record=False):
    """Oracle output rows (in call-row order) of a decode batch's call rows."""
    sub = batch.select(call_rows)
    w64 = w64 if w64 is not None else oracle_weights(shape, tag, layer, source, dev_layer)
    cache = oracle_cache(shape, tag, layer, sub, range(sub.n_seqs), batch.num_blocks)
    out, rec = oracle.layer_forward(w64, shape, hidden64, sub.row_idx, sub.positions, None,
                                    sub.ctx_lens, cache, record=record)
    return out[sub.row_idx], rec, cache


def oracle_prefill_seqs(shape, tag, layer, batch: W.Batch, seqs, hidden64, source="cpu",
                        dev_layer=None, w64=None, record=False):
    sub = batch.select_seqs(seqs)
    w64 = w64 if w64 is not None else oracle_weights(shape, tag, layer, source, dev_layer)
    cache = oracle_cache(shape, tag, layer, sub, range(sub.n_seqs), batch.num_blocks)
    out, rec = oracle.layer_forward(w64, shape, hidden64, sub.row_idx, sub.positions,
                                    sub.seq_starts, sub.ctx_lens, cache, record=record)
    return out[sub.row_idx], rec, cache, sub


def gpu_cache_tokens(layer_t: dict, batch: W.Batch, s: int, t0: int, t1: int):
    """Keys/values of tokens t0..t1-1 of call-sequence s, read back from the
    GPU pools, as float64 [n, Hkv, hd]."""
    b0, b1 = t0 // W.BLOCK_SIZE, (t1 - 1) // W.BLOCK_SIZE + 1
    idx = torch.from_numpy(batch.block_table[s, b0:b1].astype(np.int64)).cuda()
    kb = to64(layer_t["k_cache"].index_select(0, idx))
    vb = to64(layer_t["v_cache"].index_select(0, idx))
    K, V = depage_blocks(kb, vb, (b1 - b0) * W.BLOCK_SIZE)
    off = t0 - b0 * W.BLOCK_SIZE
    return K[off:off + t1 - t0], V[off:off + t1 - t0]


def small_bf16_shape(d=512, hq=8, hkv=2, ffn=768, theta=1e4, eps=1e-5):
    return W.LayerShape(d, hq, hkv, 128, ffn, theta, eps, "bf16")


def ragged_decode_batch(seed, priors, max_ctx, hidden_rows=None, row_idx=None):
    rng = np.random.default_rng(seed)
    return W.decode_batch(rng, np.asarray(priors), max_ctx, hidden_rows=hidden_rows,
                          row_idx=row_idx)


def ragged_prefill_batch(seed, priors, lens, max_ctx, hidden_rows=None):
    """Prefill of len_s new tokens after prior_s cached ones, rows shuffled
    into a hidden buffer of hidden_rows rows."""
    rng = np.random.default_rng(seed)
    priors = np.asarray(priors, np.int64)
    lens = np.asarray(lens, np.int64)
    life = priors + lens
    table, nblk = W._assign_blocks(rng, life, -(-max_ctx // W.BLOCK_SIZE))
    M = int(lens.sum())
    hr = hidden_rows or M
    rows = rng.permutation(hr)[:M].astype(np.int32)
    pos = np.concatenate([np.arange(p, p + n) for p, n in zip(priors, lens)]).astype(np.int32)
    starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return W.Batch(hr, rows, pos, starts, priors.astype(np.int32), life.astype(np.int32), table,
                   nblk)


def bf16_round64(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (via float32), as the hidden buffer holds."""
    t = torch.from_numpy(np.asarray(x, np.float64)).to(torch.float32)
    return t.to(torch.bfloat16).to(torch.float32).double().numpy()


def expected_attention_flops(batch: W.Batch, shape) -> float:
    return 4.0 * shape.n_q_heads * shape.head_dim * float(np.sum(batch.positions + 1))


def isclose_report(name, got, ref, tol=TOL):
    e = normwise_err(got, ref)
    log(f"{name}: normwise err {e:.3e} (bound {tol:g}), elementwise (rms floor) "
        f"{elementwise_err(got, ref):.3e}")
    return e


def pool_blocks_of_new_tokens(batch: W.Batch) -> np.ndarray:
    """Physical blocks that hold the tokens a call appends (positions
    prior_lens .. ctx_lens - 1 of each of its sequences)."""
    out = set()
    for s in range(batch.n_seqs):
        p0, p1 = int(batch.prior_lens[s]), int(batch.ctx_lens[s])
        if p1 > p0:
            out.update(int(b) for b in batch.block_table[s, p0 // W.BLOCK_SIZE:
                                                         (p1 - 1) // W.BLOCK_SIZE + 1])
    return np.array(sorted(out), np.int64)


class PoolSnapshot:
    """Saved contents of chosen physical blocks of a layer's pools, to put the
    cache back into its state before a call (so a later call that skipped or
    misplaced its append cannot pass on the bytes an earlier call wrote)."""

    def __init__(self, layer_t: dict, blocks: np.ndarray):
        self.layer_t = layer_t
        self.idx = torch.from_numpy(np.asarray(blocks, np.int64)).cuda()
        self.saved = {k: layer_t[k][self.idx].clone() for k in ("k_cache", "v_cache")}

    def restore(self):
        for k, v in self.saved.items():
            self.layer_t[k][self.idx] = v
        torch.cuda.synchronize()


__all__ = ["Replica", "oracle_weights", "oracle_cache", "oracle_decode_rows",
           "oracle_prefill_seqs", "normwise_err", "elementwise_err", "to64", "TOL", "log",
           "math", "PoolSnapshot", "pool_blocks_of_new_tokens"]
