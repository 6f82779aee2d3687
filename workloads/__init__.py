"""Seeded synthetic workloads for the layer-replica hot path.

This module holds only input generation: layer shapes, seeded weights, hidden
states, KV-cache contents, context-length draws, block tables and row subsets.
It contains none of the layer's arithmetic. Both the oracle-side tests and the
GPU-side tests/bench draw their inputs from here, so the two sides see the same
bits.

Large tensors come from a counter-based generator written with torch integer
ops (``normal``). The same code runs on the CPU and on the GPU and gives
bit-identical values on both, so a full-size tensor can be produced on the GPU
in milliseconds while the CPU side regenerates only the slice it needs (any
element range can be produced on its own).

Small per-batch arrays (context lengths, permutations, the Zipf row subset)
come from ``numpy.random.default_rng(SeedSequence(20260000 + config_id))``.

Paper context: a "hot" replica runs a span of consecutive decoder layers on its
sub-batch of in-flight requests (Sec. 3.1, replication mechanism); the workloads
below give that replica its share at the shapes of Llama/Qwen-style layers.
The paper's own datasets (the Alpaca 1k/64 ablation inputs, LongBench prompts,
the Alibaba and Azure traces of Sec. 6.1) are not available; the lognormal
context-length draws and the Zipf-skewed row subset stand in for them.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional

import numpy as np
import torch

BLOCK_SIZE = 16

# ----------------------------------------------------------------------------
# Layer shapes
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class LayerShape:
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    rope_theta: float
    rms_eps: float
    dtype: str  # "bf16" or "f32"
    block_size: int = BLOCK_SIZE

    @property
    def qkv_width(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    def weight_shapes(self) -> dict:
        d, hd, F = self.d_model, self.head_dim, self.d_ffn
        return {
            "w_qkv": (self.qkv_width, d),
            "w_o": (d, self.n_q_heads * hd),
            "w_gate_up": (2 * F, d),
            "w_down": (d, F),
            "gamma_attn": (d,),
            "gamma_mlp": (d,),
        }

    def param_count(self) -> int:
        return sum(math.prod(s) for s in self.weight_shapes().values())

    def kv_bytes_per_token(self) -> int:
        return 2 * self.n_kv_heads * self.head_dim * self.elem_bytes


TINY = LayerShape(256, 4, 2, 64, 688, 1.0e4, 1e-6, "f32")
LLAMA8B = LayerShape(4096, 32, 8, 128, 14336, 5.0e5, 1e-5, "bf16")
QWEN32B = LayerShape(5120, 40, 8, 128, 27648, 1.0e6, 1e-6, "bf16")
LLAMA70B = LayerShape(8192, 64, 8, 128, 28672, 5.0e5, 1e-5, "bf16")

# ----------------------------------------------------------------------------
# Counter-based generator (SplitMix64 finalizer, Irwin-Hall normal)
# ----------------------------------------------------------------------------

_MASK64 = (1 << 64) - 1
_GOLDEN = 0x9E3779B97F4A7C15
_MIX1 = 0xBF58476D1CE4E5B9
_MIX2 = 0x94D049BB133111EB
# Irwin-Hall sum of 8 uniform 16-bit integers: mean 8*65535/2, variance
# 8*(65536^2-1)/12. Standardised and scaled by sigma with one float32 multiply.
_IH_TERMS = 8
_IH_CENTER = _IH_TERMS * 65535 // 2
_IH_STD = math.sqrt(_IH_TERMS * (65536.0 ** 2 - 1.0) / 12.0)
_CHUNK_CPU = 1 << 18   # keeps the int64 temporaries cache-resident
_CHUNK_GPU = 1 << 25


def _s64(x: int) -> int:
    x &= _MASK64
    return x - (1 << 64) if x >= (1 << 63) else x


def _lsr(z: torch.Tensor, k: int) -> torch.Tensor:
    """Logical right shift of int64 lanes (torch's >> is arithmetic)."""
    return (z >> k) & ((1 << (64 - k)) - 1)


def _mix64(z: torch.Tensor) -> torch.Tensor:
    z = (z ^ _lsr(z, 30)) * _s64(_MIX1)
    z = (z ^ _lsr(z, 27)) * _s64(_MIX2)
    return z ^ _lsr(z, 31)


def stream_key(*parts) -> int:
    """Stable 64-bit key for a named tensor stream (e.g. ("c2", "w_qkv", 0))."""
    h = hashlib.blake2b("/".join(str(p) for p in parts).encode(), digest_size=8)
    return _s64(int.from_bytes(h.digest(), "little"))


def _bf16_rne(x: torch.Tensor) -> torch.Tensor:
    """Round float32 lanes to bfloat16, nearest-even, with integer ops only."""
    u = x.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    r = torch.where(r >= 32768, r - 65536, r).to(torch.int16)
    return r.view(torch.bfloat16)


def normal(key: int, numel: int, sigma: float, mean: float = 0.0, *,
           dtype: torch.dtype = torch.bfloat16, device="cpu",
           start: int = 0) -> torch.Tensor:
    """Elements ``start .. start+numel`` of the stream ``key``.

    Element e is built from two SplitMix64 outputs at counters
    ``key + (2e+j)*golden`` (j = 0, 1): their eight 16-bit fields are summed
    (Irwin-Hall, within 4.9 sigma of the mean), standardised, multiplied by
    sigma in float32, shifted by ``mean`` in float32 and, for bf16, rounded to
    nearest-even. Every step is exact integer work or a single correctly
    rounded float32 operation, so CPU and GPU give identical bits.
    """
    out = torch.empty(numel, dtype=dtype, device=device)
    scale = torch.tensor(sigma / _IH_STD, dtype=torch.float32, device=device)
    shift = torch.tensor(mean, dtype=torch.float32, device=device)
    gold = _s64(_GOLDEN)
    chunk = _CHUNK_CPU if out.device.type == "cpu" else _CHUNK_GPU
    for c0 in range(0, numel, chunk):
        n = min(chunk, numel - c0)
        e = torch.arange(start + c0, start + c0 + n, dtype=torch.int64, device=device)
        acc = None
        for j in range(2):
            h = _mix64(e * _s64(2 * gold) + _s64(key + j * gold))
            s = (h & 0xFFFF) + (_lsr(h, 16) & 0xFFFF) + (_lsr(h, 32) & 0xFFFF) + _lsr(h, 48)
            acc = s if acc is None else acc + s
        x = (acc - _IH_CENTER).to(torch.float32) * scale
        if mean != 0.0:
            x = x + shift
        out[c0:c0 + n] = _bf16_rne(x) if dtype == torch.bfloat16 else x
    return out


# ----------------------------------------------------------------------------
# Weights, hidden states, KV pools
# ----------------------------------------------------------------------------

WEIGHT_SIGMA = 0.02
GAMMA_SIGMA = 0.1


def layer_weights(shape: LayerShape, tag: str, layer: int, device="cpu") -> dict:
    """Weights of one decoder layer in nn.Linear layout ([out, in], row-major).

    w_qkv rows: the Hq query heads, then the Hkv key heads, then the Hkv value
    heads, each head_dim rows. w_gate_up rows: the F gate rows, then the F up
    rows. Matmul weights ~N(0, 0.02); RMSNorm gains 1 + N(0, 0.1).
    """
    out = {}
    for name, shp in shape.weight_shapes().items():
        numel = math.prod(shp)
        if name.startswith("gamma"):
            t = normal(stream_key(tag, name, layer), numel, GAMMA_SIGMA, 1.0,
                       dtype=shape.torch_dtype, device=device)
        else:
            t = normal(stream_key(tag, name, layer), numel, WEIGHT_SIGMA,
                       dtype=shape.torch_dtype, device=device)
        out[name] = t.view(*shp)
    return out


def weight_rows(shape: LayerShape, tag: str, layer: int, name: str, r0: int, r1: int,
                device="cpu") -> torch.Tensor:
    """Rows r0..r1 of one weight matrix, generated on their own."""
    rows, cols = shape.weight_shapes()[name]
    t = normal(stream_key(tag, name, layer), (r1 - r0) * cols, WEIGHT_SIGMA,
               dtype=shape.torch_dtype, device=device, start=r0 * cols)
    return t.view(r1 - r0, cols)


def hidden_states(shape: LayerShape, tag: str, rows: int, device="cpu") -> torch.Tensor:
    """The full-batch hidden buffer [rows, d] ~N(0, 1)."""
    return normal(stream_key(tag, "hidden"), rows * shape.d_model, 1.0,
                  dtype=shape.torch_dtype, device=device).view(rows, shape.d_model)


def kv_pool_shapes(shape: LayerShape, num_blocks: int):
    """Paged cache pools: K and V are [blocks, Hkv, block * hd] (one tile per
    block and key/value head; the order inside a tile is the library's)."""
    bs, h, hd = shape.block_size, shape.n_kv_heads, shape.head_dim
    return (num_blocks, h, bs * hd), (num_blocks, h, bs * hd)


def kv_pool(shape: LayerShape, tag: str, layer: int, num_blocks: int, which: str,
            device="cpu", blocks: Optional[np.ndarray] = None) -> torch.Tensor:
    """Random N(0,1) contents of a layer's K or V pool (taken as post-RoPE K).

    With ``blocks`` given, only those physical blocks are generated (same
    values as in the full pool), stacked in the order given.
    """
    kshape, vshape = kv_pool_shapes(shape, num_blocks)
    shp = kshape if which == "k" else vshape
    per_block = math.prod(shp[1:])
    key = stream_key(tag, "kv_" + which, layer)
    if blocks is None:
        return normal(key, num_blocks * per_block, 1.0, dtype=shape.torch_dtype,
                      device=device).view(*shp)
    parts = [normal(key, per_block, 1.0, dtype=shape.torch_dtype, device=device,
                    start=int(b) * per_block) for b in blocks]
    if not parts:
        return torch.empty((0,) + shp[1:], dtype=shape.torch_dtype, device=device)
    return torch.stack(parts).view(len(parts), *shp[1:])


# ----------------------------------------------------------------------------
# Batches
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class Batch:
    """One call's batch, with every array in the call's own row/sequence order.

    Rows i = 0..M-1 are the call rows; ``row_idx[i]`` is the hidden-buffer row.
    Sequences s = 0..S-1 own the call rows ``seq_starts[s]..seq_starts[s+1]``
    (decode: row i is sequence i and ``seq_starts`` is None).
    ``prior_lens[s]`` tokens are cached before the call; ``ctx_lens[s]`` after
    it. ``positions[i]`` is the absolute position of row i's token.
    """
    hidden_rows: int
    row_idx: np.ndarray
    positions: np.ndarray
    seq_starts: Optional[np.ndarray]
    prior_lens: np.ndarray
    ctx_lens: np.ndarray
    block_table: np.ndarray
    num_blocks: int

    @property
    def n_rows(self) -> int:
        return int(self.row_idx.shape[0])

    @property
    def n_seqs(self) -> int:
        return int(self.ctx_lens.shape[0])

    @property
    def is_decode(self) -> bool:
        return self.seq_starts is None

    def rows_of_seq(self, s: int) -> np.ndarray:
        if self.seq_starts is None:
            return np.array([s])
        return np.arange(self.seq_starts[s], self.seq_starts[s + 1])

    def select(self, call_rows) -> "Batch":
        """Decode sub-batch made of the given call rows (a replica's share)."""
        assert self.is_decode
        r = np.asarray(call_rows, dtype=np.int64)
        return Batch(self.hidden_rows, self.row_idx[r].copy(), self.positions[r].copy(),
                     None, self.prior_lens[r].copy(), self.ctx_lens[r].copy(),
                     self.block_table[r].copy(), self.num_blocks)

    def select_seqs(self, seqs) -> "Batch":
        """Prefill sub-batch made of whole sequences (request-aligned)."""
        assert not self.is_decode
        seqs = np.asarray(seqs, dtype=np.int64)
        rows = np.concatenate([self.rows_of_seq(int(s)) for s in seqs]) if len(seqs) else \
            np.zeros(0, np.int64)
        lens = np.array([self.seq_starts[s + 1] - self.seq_starts[s] for s in seqs], np.int64)
        starts = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        return Batch(self.hidden_rows, self.row_idx[rows].copy(), self.positions[rows].copy(),
                     starts, self.prior_lens[seqs].copy(), self.ctx_lens[seqs].copy(),
                     self.block_table[seqs].copy(), self.num_blocks)


def _assign_blocks(rng, lens_total: np.ndarray, max_blocks: int, spare: int = 0):
    need = -(-lens_total // BLOCK_SIZE)
    num_blocks = int(need.sum()) + spare
    perm = rng.permutation(num_blocks).astype(np.int32)
    table = np.full((len(lens_total), max_blocks), -1, np.int32)
    off = 0
    for s, n in enumerate(need):
        table[s, :n] = perm[off:off + n]
        off += n
    return table, num_blocks


def _lognormal_ctx(rng, n, mu, sigma, lo, hi):
    x = rng.lognormal(mean=mu, sigma=sigma, size=n)
    return np.clip(np.floor(x), lo, hi).astype(np.int64)


def decode_batch(rng, prior: np.ndarray, max_ctx: int, hidden_rows=None, row_idx=None) -> Batch:
    prior = np.asarray(prior, np.int64)
    n = len(prior)
    ctx = prior + 1
    max_blocks = -(-max_ctx // BLOCK_SIZE)
    table, nblk = _assign_blocks(rng, ctx, max_blocks)
    rows = np.arange(n, dtype=np.int32) if row_idx is None else np.asarray(row_idx, np.int32)
    return Batch(hidden_rows or n, rows, prior.astype(np.int32), None,
                 prior.astype(np.int32), ctx.astype(np.int32), table, nblk)


def zipf_subset(rng, population: int, k: int, s: float) -> np.ndarray:
    """k distinct indices from [0, population): ranks from a seeded
    permutation, weights rank^-s, weighted sampling without replacement,
    drawn order kept."""
    order = rng.permutation(population)
    w = np.empty(population)
    w[order] = np.arange(1, population + 1, dtype=np.float64) ** (-s)
    return rng.choice(population, size=k, replace=False, p=w / w.sum()).astype(np.int32)


@dataclasses.dataclass
class Workload:
    name: str
    tag: str
    shape: LayerShape
    n_layers: int
    batch: Batch
    description: str
    full_batch: Optional[Batch] = None  # C3: the whole 256-row batch
    decode_after: Optional[Batch] = None  # C4: the decode step on the same cache


def _rng(cid: int):
    return np.random.default_rng(np.random.SeedSequence(20260000 + cid))


def c1_tiny() -> Workload:
    rng = _rng(1)
    prior = rng.integers(1, 65, size=8)
    full = decode_batch(rng, prior, max_ctx=65, hidden_rows=8)
    sub = full.select([1, 3, 4, 6])
    return Workload("c1_tiny_f32", "c1", TINY, 1, sub,
                    "tiny fp32 layer, decode rows {1,3,4,6} of 8, ctx U[1,64]", full_batch=full)


def c2_llama8b_decode(batch: int = 64) -> Workload:
    rng = _rng(2)
    prior = _lognormal_ctx(rng, batch, math.log(1024), 0.8, 16, 8192)
    b = decode_batch(rng, prior, max_ctx=8193)
    return Workload("llama8b_decode_b64", "c2", LLAMA8B, 1, b,
                    "Llama-3-8B-shaped layer, bf16 decode, batch 64, ctx lognormal(ln1024,0.8)")


def c3_llama8b_skewed() -> Workload:
    rng = _rng(3)
    prior = _lognormal_ctx(rng, 256, math.log(2048), 1.0, 16, 16384)
    full = decode_batch(rng, prior, max_ctx=16385)
    subset = zipf_subset(rng, 256, 96, 1.1)
    return Workload("llama8b_skewed_96of256", "c3", LLAMA8B, 1, full.select(subset),
                    "8B-shaped layer, Zipf(1.1) subset of 96 of 256 in-flight rows",
                    full_batch=full)


def c4_qwen32b() -> Workload:
    rng = _rng(4)
    chunk = 512
    pre_prior = np.array([0, 512, 1024, 4096], np.int64)
    dec_prior_rest = _lognormal_ctx(rng, 124, math.log(1024), 0.8, 16, 8192)
    # Lifetime lengths: prefill requests grow by the chunk and one decode token.
    life = np.concatenate([pre_prior + chunk + 1, dec_prior_rest + 1])
    max_ctx = 8193
    table, nblk = _assign_blocks(rng, life, -(-max_ctx // BLOCK_SIZE))
    rows = np.arange(4 * chunk, dtype=np.int32)
    positions = np.concatenate([np.arange(p, p + chunk) for p in pre_prior]).astype(np.int32)
    starts = (np.arange(5) * chunk).astype(np.int32)
    prefill = Batch(4 * chunk, rows, positions, starts, pre_prior.astype(np.int32),
                    (pre_prior + chunk).astype(np.int32), table[:4].copy(), nblk)
    dprior = np.concatenate([pre_prior + chunk, dec_prior_rest])
    decode = Batch(128, np.arange(128, dtype=np.int32), dprior.astype(np.int32), None,
                   dprior.astype(np.int32), (dprior + 1).astype(np.int32), table.copy(), nblk)
    return Workload("qwen32b_prefill2048", "c4", QWEN32B, 1, prefill,
                    "Qwen-32B-shaped layer, chunked prefill of 4x512 tokens over ctx "
                    "{0,512,1024,4096}, then batch-128 decode", decode_after=decode)


def c5_llama70b_span(batch: int = 128) -> Workload:
    rng = _rng(5)
    prior = _lognormal_ctx(rng, batch, math.log(4096), 0.7, 64, 32768)
    b = decode_batch(rng, prior, max_ctx=32769)
    return Workload("llama70b_span8_b128", "c5", LLAMA70B, 8, b,
                    "70B-shaped span of 8 layers, decode batch 128, ctx lognormal(ln4096,0.7)")


ALL = {
    "c1": c1_tiny,
    "c2": c2_llama8b_decode,
    "c3": c3_llama8b_skewed,
    "c4": c4_qwen32b,
    "c5": c5_llama70b_span,
}


def even_partition(n: int, parts: int) -> list:
    """Split 0..n-1 into `parts` consecutive groups of ceil/floor(n/parts)
    (heaviest first), as the uneven sub-batches of the heterogeneous model."""
    base, extra = divmod(n, parts)
    out, off = [], 0
    for p in range(parts):
        k = base + (1 if p < extra else 0)
        out.append(np.arange(off, off + k))
        off += k
    return out
