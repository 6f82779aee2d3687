"""Full-size configurations, in the launch configuration bench.py times.

The GPU runs the whole batch; the oracle recomputes sampled output rows one
by one (decode rows are independent; prefill checks whole requests), and
properties that hold at any size (split-batch bit identity of output rows and
appended cache bytes) are checked on the whole batch, each split run starting
from the cache state before the first run. Prior cache tokens reach the
oracle regenerated on the CPU; weights of the largest layers as host copies
of the tensors the counter-based generator produced on the GPU (the library
only reads them; test_generator_is_identical_on_cpu_and_gpu shows these are
the bits the CPU generator gives).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from harness import (TOL, PoolSnapshot, Replica, elementwise_err, gpu_cache_tokens, log,
                     normwise_err, oracle_cache, oracle_decode_rows, oracle_prefill_seqs,
                     oracle_weights, pool_blocks_of_new_tokens, to64)
from workloads import device as WD

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def sample_rows(b: W.Batch, k: int, seed: int = 0):
    """Call rows with the shortest and the longest context plus k-2 seeded
    others."""
    ctx = b.ctx_lens
    rows = {int(np.argmin(ctx)), int(np.argmax(ctx))}
    rng = np.random.default_rng(seed)
    for r in rng.permutation(b.n_rows):
        if len(rows) >= k:
            break
        rows.add(int(r))
    return sorted(rows)


def check(name, got, ref, x):
    e = normwise_err(got, ref)
    ed = normwise_err(got - x, ref - x)
    log(f"{name}: output err {e:.2e}, branch err {ed:.2e}, elementwise (rms floor) "
        f"{elementwise_err(got, ref):.2e}")
    assert e < TOL and ed < TOL, (name, e, ed)


def _kv_new_tokens(layer_t, b: W.Batch, seqs):
    out = []
    for s in seqs:
        K, V = gpu_cache_tokens(layer_t, b, s, int(b.prior_lens[s]), int(b.ctx_lens[s]))
        out.append((K, V))
    return out


def _same_kv(a, b):
    return all(np.array_equal(k1, k2) and np.array_equal(v1, v2)
               for (k1, v1), (k2, v2) in zip(a, b))


def test_generator_is_identical_on_cpu_and_gpu():
    shape = W.LLAMA8B
    dev = W.layer_weights(shape, "c2", 0, device="cuda")
    for name in ("w_qkv", "w_down", "gamma_attn"):
        n = 4096
        cpu = W.normal(W.stream_key("c2", name, 0), n, 0.1 if name.startswith("gamma") else 0.02,
                       1.0 if name.startswith("gamma") else 0.0, start=0)
        assert torch.equal(cpu.view(torch.int16), dev[name].reshape(-1)[:n].cpu().view(torch.int16))
    rows = W.weight_rows(shape, "c2", 0, "w_gate_up", 1000, 1003)
    assert torch.equal(rows.view(torch.int16), dev["w_gate_up"][1000:1003].cpu().view(torch.int16))
    blocks = np.array([7, 0, 999])
    kc = W.kv_pool(shape, "c2", 0, 1000, "k", blocks=blocks)
    kg = W.kv_pool(shape, "c2", 0, 1000, "k", device="cuda")[torch.from_numpy(blocks).cuda()]
    assert torch.equal(kc.view(torch.int16), kg.cpu().view(torch.int16))


def test_c2_llama8b_decode_batch64_sampled_rows():
    wl = W.c2_llama8b_decode()
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    rows = sample_rows(b, 6)
    ref, _, cache = oracle_decode_rows(shape, wl.tag, 0, b, rows, h0, source="cpu")
    got = to64(hidden)[b.row_idx[rows]]
    check("c2 sampled rows", got, ref, h0[b.row_idx[rows]])
    for j, r in enumerate(rows):
        p = int(b.positions[r])
        K, V = gpu_cache_tokens(rep.layers[0], b, r, p, p + 1)
        assert normwise_err(K[0], cache.K[j][p]) < TOL and normwise_err(V[0], cache.V[j][p]) < TOL


def test_llama8b_decode_300_rows_matches_oracle_and_splits():
    """300 decode rows of the 8B layer: the gate/up and down projections
    (7- and 8-wave plans) take the row-split GEMM in two passes (256 rows,
    then 44), QKV and O three 128-row passes. Sampled rows of both passes
    against the oracle; the whole batch bit-identical to a 200/100 split
    (one row-split pass, then the 128-row kernel)."""
    wl = W.c2_llama8b_decode(300)
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_new_tokens(rep.layers[0], b, range(b.n_seqs))
    snap.restore()
    split = hidden.clone()
    for part in (np.arange(0, 200), np.arange(200, 300)):
        rep.forward(0, split, WD.batch_tensors(b.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    assert _same_kv(_kv_new_tokens(rep.layers[0], b, range(b.n_seqs)), kv_whole)
    rows = sorted(set(sample_rows(b, 3, seed=5)) | {130, 255, 256, 299})
    ref, _, _ = oracle_decode_rows(shape, wl.tag, 0, b, rows, h0, source="device",
                                   dev_layer=rep.layers[0])
    check("300-row decode sampled rows", to64(whole)[b.row_idx[rows]], ref,
          h0[b.row_idx[rows]])


def test_llama8b_decode_129_rows_across_gemm_row_limits():
    """129 decode rows of the 8B layer split at the decode GEMMs' row limits:
    the whole batch (gate/up and down: one 256-row pass of the row-split
    GEMM, mostly past M), 65 rows (down: a 128-row pass of it), 64 rows
    (the 64-row kernel) give identical bits; sampled rows against the
    oracle."""
    wl = W.c2_llama8b_decode(129)
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_new_tokens(rep.layers[0], b, range(b.n_seqs))
    snap.restore()
    split = hidden.clone()
    for part in (np.arange(0, 65), np.arange(65, 129)):
        rep.forward(0, split, WD.batch_tensors(b.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    assert _same_kv(_kv_new_tokens(rep.layers[0], b, range(b.n_seqs)), kv_whole)
    rows = sorted(set(sample_rows(b, 2, seed=7)) | {0, 64, 128})
    ref, _, _ = oracle_decode_rows(shape, wl.tag, 0, b, rows, h0, source="device",
                                   dev_layer=rep.layers[0])
    check("129-row decode sampled rows", to64(whole)[b.row_idx[rows]], ref,
          h0[b.row_idx[rows]])


def test_qwen32b_decode_192_rows_row_split_gate_up():
    """192 decode rows of the 32B layer: its 8-wave gate/up plan takes the
    row-split GEMM's 256-row pass with the SwiGLU epilogue; two 96-row
    halves (its 128-row pass) give identical bits, and sampled rows match
    the oracle."""
    shape = W.QWEN32B
    rng = np.random.default_rng(192)
    prior = np.clip(np.exp(rng.normal(np.log(1024), 0.8, 192)).astype(np.int64), 16, 4096)
    b = W.decode_batch(rng, prior, max_ctx=4097)
    tag = "c4x"
    rep = Replica.for_batch(shape, tag, 1, b)
    hidden = WD.hidden_tensor(shape, tag, b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_new_tokens(rep.layers[0], b, range(b.n_seqs))
    snap.restore()
    halves = hidden.clone()
    for part in (np.arange(0, 96), np.arange(96, 192)):
        rep.forward(0, halves, WD.batch_tensors(b.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(halves.view(torch.int16), whole.view(torch.int16))
    assert _same_kv(_kv_new_tokens(rep.layers[0], b, range(b.n_seqs)), kv_whole)
    rows = sorted(set(sample_rows(b, 2, seed=9)) | {0, 191})
    ref, _, _ = oracle_decode_rows(shape, tag, 0, b, rows, h0, source="device",
                                   dev_layer=rep.layers[0])
    check("32B 192-row decode sampled rows", to64(whole)[b.row_idx[rows]], ref,
          h0[b.row_idx[rows]])


def test_c3_skewed_split_is_bit_identical_and_matches_oracle():
    """The hot replica's Zipf share (96 of 256 rows), the whole 256-row
    batch, and the share cut into uneven sub-batches of the heterogeneous
    model (v = 5: 20, 19, 19, 19, 19) give identical rows and cache bytes."""
    wl = W.c3_llama8b_skewed()
    full, sub, shape = wl.full_batch, wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, full, max_rows=full.n_rows, max_seqs=full.n_seqs)
    hidden = WD.hidden_tensor(shape, wl.tag, full.hidden_rows)
    h0 = to64(hidden)
    # Blocks holding the new tokens of all 256 requests, restored between runs.
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(full))
    restore = snap.restore

    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(full))
    torch.cuda.synchronize()
    kv_whole = _kv_new_tokens(rep.layers[0], sub, range(sub.n_seqs))
    rows = sub.row_idx.astype(np.int64)

    restore()
    share = hidden.clone()
    rep.forward(0, share, WD.batch_tensors(sub))
    torch.cuda.synchronize()
    assert torch.equal(share[rows].view(torch.int16), whole[rows].view(torch.int16))
    others = np.setdiff1d(np.arange(full.hidden_rows), rows)
    assert torch.equal(share[others].view(torch.int16), hidden[others].view(torch.int16))
    for (k1, v1), (k2, v2) in zip(_kv_new_tokens(rep.layers[0], sub, range(sub.n_seqs)), kv_whole):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)

    restore()
    parts = hidden.clone()
    for p in W.even_partition(sub.n_rows, 5):
        rep.forward(0, parts, WD.batch_tensors(sub.select(p)))
    torch.cuda.synchronize()
    assert torch.equal(parts[rows].view(torch.int16), whole[rows].view(torch.int16))
    for (k1, v1), (k2, v2) in zip(_kv_new_tokens(rep.layers[0], sub, range(sub.n_seqs)), kv_whole):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)

    sample = sample_rows(sub, 4, seed=3)
    ref, _, _ = oracle_decode_rows(shape, wl.tag, 0, sub, sample, h0, source="device",
                                   dev_layer=rep.layers[0])
    check("c3 sampled rows", to64(share)[rows[sample]], ref, h0[rows[sample]])


def test_c4_qwen32b_prefill_then_decode():
    """The 32B chunked prefill (4 x 512 tokens after {0, 512, 1024, 4096}
    cached), then the batch-128 decode on the same cache.
      * prefill: a request-aligned split, run from the cache state before the
        whole batch, gives the whole batch's output rows and appended cache
        bytes; every request's rows and appended keys/values against the
        oracle;
      * decode: two 64-row halves, run from the cache state before the whole
        batch, give its bits; the four prefilled requests (keys from the
        oracle's own prefill) and sampled decode-only requests against the
        oracle."""
    wl = W.c4_qwen32b()
    pre, dec, shape = wl.batch, wl.decode_after, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, pre, max_rows=pre.n_rows, max_seqs=dec.n_seqs)
    w64 = oracle_weights(shape, wl.tag, 0, "device", rep.layers[0])
    hidden = WD.hidden_tensor(shape, wl.tag, pre.hidden_rows)
    h0 = to64(hidden)
    lay = rep.layers[0]
    snap = PoolSnapshot(lay, pool_blocks_of_new_tokens(pre))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(pre))
    torch.cuda.synchronize()
    kv_whole = _kv_new_tokens(lay, pre, range(pre.n_seqs))
    snap.restore()
    split = hidden.clone()
    for seqs in ([2, 0], [3, 1]):
        rep.forward(0, split, WD.batch_tensors(pre.select_seqs(seqs)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    assert _same_kv(_kv_new_tokens(lay, pre, range(pre.n_seqs)), kv_whole)
    got = to64(whole)
    caches = []
    for s in range(pre.n_seqs):
        ref, _, cache, sub = oracle_prefill_seqs(shape, wl.tag, 0, pre, [s], h0, w64=w64)
        rows = sub.row_idx.astype(np.int64)
        check(f"c4 prefill request {s} (prior {int(pre.prior_lens[s])})", got[rows], ref, h0[rows])
        t0, t1 = int(pre.prior_lens[s]), int(pre.ctx_lens[s])
        K, V = kv_whole[s]
        assert normwise_err(K, cache.K[0][t0:t1]) < TOL and normwise_err(V, cache.V[0][t0:t1]) < TOL
        caches.append(cache)
        log(f"c4 prefill request {s}: appended keys/values match the oracle")

    # Batch-128 decode on the same cache.
    dh = WD.hidden_tensor(shape, wl.tag + "dec", dec.hidden_rows)
    d0 = to64(dh)
    dsnap = PoolSnapshot(lay, pool_blocks_of_new_tokens(dec))
    rep.forward(0, dh, WD.batch_tensors(dec))
    torch.cuda.synchronize()
    kv_dec = _kv_new_tokens(lay, dec, range(dec.n_seqs))
    dsnap.restore()
    # Two 64-row halves (the 64-row GEMM kernels) give the bits of the whole
    # batch (the 8-wave gate/up plan's 128-row pass of the row-split kernel).
    halves = WD.hidden_tensor(shape, wl.tag + "dec", dec.hidden_rows)
    for part in (np.arange(0, 64), np.arange(64, 128)):
        rep.forward(0, halves, WD.batch_tensors(dec.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(halves.view(torch.int16), dh.view(torch.int16))
    assert _same_kv(_kv_new_tokens(lay, dec, range(dec.n_seqs)), kv_dec)
    got = to64(dh)
    sample = [0, 1, 2, 3] + [s + 4 for s in sample_rows(dec.select(range(4, 128)), 3, seed=4)]
    for r in sample:
        sb = dec.select([r])
        if r < pre.n_seqs:
            # Prefilled request: its keys/values up to the prefill's end from the
            # oracle's own prefill of it.
            ctx = int(sb.ctx_lens[0])
            K = np.zeros((ctx, shape.n_kv_heads, shape.head_dim))
            V = np.zeros_like(K)
            n = int(pre.ctx_lens[r])
            K[:n], V[:n] = caches[r].K[0][:n], caches[r].V[0][:n]
            c = oracle.KVCache([K], [V])
        else:
            c = oracle_cache(shape, wl.tag, 0, sb, [0], dec.num_blocks)
        out, _ = oracle.layer_forward(w64, shape, d0, sb.row_idx, sb.positions, None,
                                      sb.ctx_lens, c)
        check(f"c4 decode row {r}", got[sb.row_idx], out[sb.row_idx], d0[sb.row_idx])


def test_c5_llama70b_span8_sampled_rows():
    wl = W.c5_llama70b_span()
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, wl.n_layers, b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)
    h0 = to64(hidden)
    rep.span(0, wl.n_layers, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    rows = sample_rows(b, 3, seed=5)
    sub = b.select(rows)
    x = h0.copy()
    for l in range(wl.n_layers):
        w64 = oracle_weights(shape, wl.tag, l, "device", rep.layers[l])
        c = oracle_cache(shape, wl.tag, l, sub, range(sub.n_seqs), b.num_blocks)
        x, _ = oracle.layer_forward(w64, shape, x, sub.row_idx, sub.positions, None,
                                    sub.ctx_lens, c)
        del w64
        log(f"c5 oracle layer {l} done")
    got = to64(hidden)[sub.row_idx]
    check("c5 span sampled rows", got, x[sub.row_idx], h0[sub.row_idx])
