"""GPU parity of the HIP layer against the fp64 oracle, and the bit-exact
properties of the path (all through the C ABI).

Sizes here finish in seconds on the oracle yet span several GEMM tiles,
several split-KV partitions (256 tokens) and ragged tails. Full-size configs
are in test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import paper_2607_04181_amd as coco
import workloads as W
from harness import (TOL, PoolSnapshot, Replica, elementwise_err, gpu_cache_tokens, log,
                     normwise_err, oracle_decode_rows, oracle_prefill_seqs,
                     pool_blocks_of_new_tokens, ragged_decode_batch, ragged_prefill_batch,
                     small_bf16_shape, to64)
from workloads import device as WD

pytestmark = pytest.mark.gpu

# Context lengths hitting block (16) and partition (256) edges; 0 prior = the
# token attends only to itself.
DECODE_PRIORS = [0, 1, 14, 15, 16, 17, 100, 254, 255, 256, 511, 600, 1000, 3, 2047]
# The branch y - x is computed from bf16 operands; its normwise error is
# bounded by the same 2e-2.
DELTA_TOL = 2e-2


def _small_decode(seed=0, shape=None, priors=DECODE_PRIORS, hidden_rows=24):
    shape = shape or small_bf16_shape()
    rng = np.random.default_rng(seed)
    rows = rng.permutation(hidden_rows)[:len(priors)]
    b = ragged_decode_batch(seed, priors, max_ctx=2049, hidden_rows=hidden_rows, row_idx=rows)
    return shape, b


def _check_rows(name, got, ref, x):
    e = normwise_err(got, ref)
    ed = normwise_err(got - x, ref - x)
    log(f"{name}: output err {e:.2e}, branch err {ed:.2e}, elementwise (rms floor) "
        f"{elementwise_err(got, ref):.2e}")
    assert e < TOL, f"{name}: output error {e} exceeds {TOL}"
    assert ed < DELTA_TOL, f"{name}: branch error {ed} exceeds {DELTA_TOL}"


def test_c1_tiny_f32_layer_matches_oracle():
    wl = W.c1_tiny()
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, "c1", 1, b, max_rows=8, max_seqs=8)
    hidden = WD.hidden_tensor(shape, "c1", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, rec, cache = oracle_decode_rows(shape, "c1", 0, b, range(b.n_rows), h0, record=True)
    got = to64(hidden)
    _check_rows("c1", got[b.row_idx], ref, h0[b.row_idx])
    # fp32 path: far inside the bound.
    assert normwise_err(got[b.row_idx] - h0[b.row_idx], ref - h0[b.row_idx]) < 1e-4
    others = sorted(set(range(b.hidden_rows)) - set(b.row_idx.tolist()))
    assert np.array_equal(got[others], h0[others])
    for s in range(b.n_seqs):
        p = int(b.positions[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, p, p + 1)
        assert normwise_err(K[0], cache.K[s][p]) < 1e-4
        assert normwise_err(V[0], cache.V[s][p]) < 1e-4


def test_small_bf16_decode_matches_oracle_with_intermediates():
    shape, b = _small_decode(1)
    rep = Replica.for_batch(shape, "s1", 1, b)
    hidden = WD.hidden_tensor(shape, "s1", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, rec, cache = oracle_decode_rows(shape, "s1", 0, b, range(b.n_rows), h0, record=True)
    got = to64(hidden)
    M, d, qd, F = b.n_rows, shape.d_model, shape.n_q_heads * 128, shape.d_ffn
    bf = torch.bfloat16
    # bf16 decode folds the gather and RMSNorm_1 into the QKV projection, so
    # h is never materialised; q depends on it and is checked instead.
    inter = {
        "q": (coco.COCO_WS_Q, qd, bf), "o": (coco.COCO_WS_O, qd, bf),
        "x1": (coco.COCO_WS_X1, d, torch.float32), "h2": (coco.COCO_WS_H2, d, bf),
        "a": (coco.COCO_WS_U, F, bf)}
    errs = {}
    for name, (which, cols, dt) in inter.items():
        errs[name] = normwise_err(to64(rep.workspace(which, M, cols, dt)), rec[name])
    log("intermediate errors: " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    for k, v in errs.items():
        assert v < TOL, f"intermediate {k}: {v}"
    _check_rows("small decode", got[b.row_idx], ref, h0[b.row_idx])
    others = sorted(set(range(b.hidden_rows)) - set(b.row_idx.tolist()))
    assert np.array_equal(got[others], h0[others])
    for s in range(b.n_seqs):
        p = int(b.positions[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, p, p + 1)
        assert normwise_err(K[0], cache.K[s][p]) < TOL
        assert normwise_err(V[0], cache.V[s][p]) < TOL


def test_small_bf16_prefill_matches_oracle():
    shape = small_bf16_shape()
    b = ragged_prefill_batch(2, priors=[0, 3, 16, 300, 40], lens=[1, 15, 64, 100, 77],
                             max_ctx=512, hidden_rows=300)
    rep = Replica.for_batch(shape, "s2", 1, b)
    hidden = WD.hidden_tensor(shape, "s2", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, rec, cache, sub = oracle_prefill_seqs(shape, "s2", 0, b, range(b.n_seqs), h0,
                                               record=True)
    got = to64(hidden)
    e_o = normwise_err(to64(rep.workspace(coco.COCO_WS_O, b.n_rows, shape.n_q_heads * 128,
                                          torch.bfloat16)), rec["o"])
    log(f"prefill attention output err {e_o:.2e}")
    assert e_o < TOL
    _check_rows("small prefill", got[b.row_idx], ref, h0[b.row_idx])
    for s in range(b.n_seqs):
        t0, t1 = int(b.prior_lens[s]), int(b.ctx_lens[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, t0, t1)
        assert normwise_err(K, cache.K[s][t0:t1]) < TOL
        assert normwise_err(V, cache.V[s][t0:t1]) < TOL


def test_prefill_attention_key_set_edges_match_oracle():
    """The prefill attention splits every 128-key stage between two sets of
    waves (keys 0-63 and 64-127 of the stage) and merges their softmax states
    per row. Chunks here put rows on both sides of those edges: rows whose
    second-set keys are all masked (positions 50-63 of a 16-row group that
    reaches 64), single rows at keys 63/64/65 and 127/128/129, and groups that
    end inside the second set. Every row of the attention output is checked
    against the oracle on its own."""
    shape = small_bf16_shape()
    priors = [50, 63, 64, 65, 112, 127, 128, 129, 0, 190]
    lens = [30, 1, 1, 1, 40, 1, 1, 1, 140, 70]
    b = ragged_prefill_batch(21, priors=priors, lens=lens, max_ctx=512, hidden_rows=300)
    rep = Replica.for_batch(shape, "s21", 1, b)
    hidden = WD.hidden_tensor(shape, "s21", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, rec, _, _ = oracle_prefill_seqs(shape, "s21", 0, b, range(b.n_seqs), h0, record=True)
    o = to64(rep.workspace(coco.COCO_WS_O, b.n_rows, shape.n_q_heads * 128, torch.bfloat16))
    ro = np.asarray(rec["o"], np.float64).reshape(o.shape)
    per_row = [normwise_err(o[i], ro[i]) for i in range(b.n_rows)]
    worst = int(np.argmax(per_row))
    log(f"key-set edges: attention output err {normwise_err(o, ro):.2e}, worst row {worst} "
        f"(position {int(b.positions[worst])}) {per_row[worst]:.2e}")
    assert np.all(np.isfinite(o))
    assert max(per_row) < TOL
    _check_rows("key-set edges", to64(hidden)[b.row_idx], ref, h0[b.row_idx])


def _kv_snapshot(rep, b):
    out = []
    for s in range(b.n_seqs):
        p0, p1 = int(b.prior_lens[s]), int(b.ctx_lens[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, p0, p1)
        out.append((K, V))
    return out


def test_decode_split_batch_is_bit_identical():
    """Any partition of a decode batch into replica shares gives the same
    output rows and cache bytes as the whole batch (uneven shares too). Each
    partition runs from the cache state before the whole batch, so a share
    that skipped or misplaced its append would read the old slot and fail."""
    shape, b = _small_decode(3)
    bt = WD.batch_tensors(b)
    rep = Replica.for_batch(shape, "s3", 1, b)
    hidden = WD.hidden_tensor(shape, "s3", b.hidden_rows)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, bt)
    torch.cuda.synchronize()
    kv_whole = _kv_snapshot(rep, b)
    for parts in (W.even_partition(b.n_rows, 2), W.even_partition(b.n_rows, 5),
                  [np.array([i]) for i in range(b.n_rows)]):
        snap.restore()
        split = hidden.clone()
        for p in parts:
            sub = b.select(p)
            rep.forward(0, split, WD.batch_tensors(sub))
        torch.cuda.synchronize()
        assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
        kv = _kv_snapshot(rep, b)
        for (k1, v1), (k2, v2) in zip(kv, kv_whole):
            assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


def test_decode_of_many_sequences_matches_oracle_and_splits():
    """300 decode sequences with lengths on block and partition edges, each
    length 25 times (the attention's work list is built over 64 sequences at a
    time and orders the partial partitions by size, ties included): every row
    against the oracle, the whole batch bit-identical to two uneven halves."""
    shape = small_bf16_shape()
    edges = [0, 1, 15, 254, 255, 256, 257, 510, 511, 512, 700, 16]
    priors = [edges[i % len(edges)] for i in range(300)]
    b = ragged_decode_batch(9, priors, max_ctx=1025, hidden_rows=320,
                            row_idx=np.random.default_rng(9).permutation(320)[:300])
    rep = Replica.for_batch(shape, "s9", 1, b)
    hidden = WD.hidden_tensor(shape, "s9", b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_snapshot(rep, b)
    rows = list(range(300))
    ref, _, _ = oracle_decode_rows(shape, "s9", 0, b, rows, h0)
    got = to64(whole)[b.row_idx[rows]]
    _check_rows("300-sequence decode", got, ref, h0[b.row_idx[rows]])
    snap.restore()
    split = hidden.clone()
    for part in (np.arange(0, 97), np.arange(97, 300)):
        rep.forward(0, split, WD.batch_tensors(b.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    for (k1, v1), (k2, v2) in zip(_kv_snapshot(rep, b), kv_whole):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


def test_decode_of_short_sequences_only_matches_oracle_and_splits():
    """Every sequence shorter than one 256-key partition, so the attention's
    work list holds partial partitions only (sorted by size, with ties and
    single-key sequences): every row against the oracle, the batch bit-identical
    to two uneven halves."""
    shape = small_bf16_shape()
    priors = [0, 3, 100, 254, 17, 100, 0, 200, 63, 64, 3, 150] * 6
    b = ragged_decode_batch(19, priors, max_ctx=256, hidden_rows=80,
                            row_idx=np.random.default_rng(19).permutation(80)[:len(priors)])
    rep = Replica.for_batch(shape, "s19", 1, b)
    hidden = WD.hidden_tensor(shape, "s19", b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    rows = list(range(b.n_rows))
    ref, _, _ = oracle_decode_rows(shape, "s19", 0, b, rows, h0)
    _check_rows("short-sequence decode", to64(whole)[b.row_idx], ref, h0[b.row_idx])
    snap.restore()
    split = hidden.clone()
    for part in (np.arange(0, 29), np.arange(29, b.n_rows)):
        rep.forward(0, split, WD.batch_tensors(b.select(part)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))


def test_prefill_request_aligned_split_is_bit_identical():
    """Request-aligned shares of a prefill batch, run from the cache state
    before the whole batch, give its output rows and appended cache bytes."""
    shape = small_bf16_shape()
    b = ragged_prefill_batch(4, priors=[0, 5, 30, 200], lens=[70, 1, 33, 64], max_ctx=512,
                             hidden_rows=200)
    rep = Replica.for_batch(shape, "s4", 1, b)
    hidden = WD.hidden_tensor(shape, "s4", b.hidden_rows)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_snapshot(rep, b)
    snap.restore()
    split = hidden.clone()
    for seqs in ([2, 0], [3], [1]):
        rep.forward(0, split, WD.batch_tensors(b.select_seqs(seqs)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    for (k1, v1), (k2, v2) in zip(_kv_snapshot(rep, b), kv_whole):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


# Gate/up plans at d = 640, F = 3456 (36 column tiles of 96 outputs): (priors,
# lengths, request-aligned shares, request checked against the oracle). The
# whole batch takes the persistent kernel (row tiles dividing 32): 2048 rows
# (8 row tiles, up to two column tiles per workgroup) and 4096 rows (16 row
# tiles, up to three); the shares of 900 rows (persistent, one tile each),
# 1148, 1500 and 2596 rows (5, 6 and 11 row tiles) take the one-tile kernel.
GATE_UP_PLANS = [
    ([0, 100, 37], [900, 248, 900], ([0], [1, 2]), 1),
    ([0, 64, 5], [1500, 300, 2296], ([0], [1, 2]), 1),
]


@pytest.mark.parametrize("priors,lens,shares,req", GATE_UP_PLANS)
def test_prefill_gate_up_plans_agree_bit_exactly_and_match_oracle(priors, lens, shares, req):
    """The persistent gate/up GEMM, where a workgroup takes its row tile
    through several column tiles with the load ring running across them,
    against request-aligned shares on the one-tile kernel: rows and appended
    cache bytes bit-identical; a request's rows and cache against the
    oracle."""
    shape = small_bf16_shape(d=640, hq=5, hkv=1, ffn=3456)
    b = ragged_prefill_batch(31, priors=priors, lens=lens, max_ctx=2560,
                             hidden_rows=sum(lens) + 52)
    rep = Replica.for_batch(shape, "s31", 1, b)
    hidden = WD.hidden_tensor(shape, "s31", b.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(b))
    torch.cuda.synchronize()
    kv_whole = _kv_snapshot(rep, b)
    ref, _, cache, sub = oracle_prefill_seqs(shape, "s31", 0, b, [req], h0)
    _check_rows(f"gate/up plans, {sum(lens)} rows, request {req}", to64(whole)[sub.row_idx], ref,
                h0[sub.row_idx])
    t0, t1 = int(b.prior_lens[req]), int(b.ctx_lens[req])
    K, V = gpu_cache_tokens(rep.layers[0], b, req, t0, t1)
    assert normwise_err(K, cache.K[0][t0:t1]) < TOL
    assert normwise_err(V, cache.V[0][t0:t1]) < TOL
    snap.restore()
    split = hidden.clone()
    for seqs in shares:
        rep.forward(0, split, WD.batch_tensors(b.select_seqs(seqs)))
    torch.cuda.synchronize()
    assert torch.equal(split.view(torch.int16), whole.view(torch.int16))
    for (k1, v1), (k2, v2) in zip(_kv_snapshot(rep, b), kv_whole):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2)


def test_prefill_gate_up_single_row_tile_matches_oracle():
    """One request of 200 rows at d = 640, F = 3456: a single row tile, so the
    persistent gate/up GEMM gives each of 36 workgroups one column tile and
    the other 220 leave at once."""
    shape = small_bf16_shape(d=640, hq=5, hkv=1, ffn=3456)
    b = ragged_prefill_batch(32, priors=[40], lens=[200], max_ctx=256, hidden_rows=230)
    rep = Replica.for_batch(shape, "s32", 1, b)
    hidden = WD.hidden_tensor(shape, "s32", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, cache, _ = oracle_prefill_seqs(shape, "s32", 0, b, [0], h0)
    _check_rows("gate/up, one row tile", to64(hidden)[b.row_idx], ref, h0[b.row_idx])
    untouched = np.setdiff1d(np.arange(b.hidden_rows), b.row_idx)
    assert torch.equal(hidden[untouched].view(torch.int16), WD.hidden_tensor(
        shape, "s32", b.hidden_rows)[untouched].view(torch.int16))


def test_zero_output_projections_give_identity_bit_exactly():
    """With W_o = W_d = 0 the layer returns its input rows: pins gather ->
    residual -> scatter bit for bit."""
    shape, b = _small_decode(5)
    # The library copies the weights at init, so they are zeroed before it.
    layers = [WD.layer_tensors(shape, "s5", 0, b.num_blocks)]
    layers[0]["w_o"].zero_()
    layers[0]["w_down"].zero_()
    rep = Replica(shape, "s5", 1, b.num_blocks, b.n_rows, b.n_seqs, b.block_table.shape[1],
                  layers=layers)
    hidden = WD.hidden_tensor(shape, "s5", b.hidden_rows)
    h0 = hidden.clone()
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    assert torch.equal(hidden.view(torch.int16), h0.view(torch.int16))


def test_block_permutation_gives_bit_identical_output():
    shape, b = _small_decode(6)
    rep = Replica.for_batch(shape, "s6", 1, b)
    hidden = WD.hidden_tensor(shape, "s6", b.hidden_rows)
    out1 = hidden.clone()
    pools = {k: rep.layers[0][k].clone() for k in ("k_cache", "v_cache")}
    rep.forward(0, out1, WD.batch_tensors(b))
    torch.cuda.synchronize()
    # Move every physical block to a new place and rewrite the table.
    perm = np.random.default_rng(0).permutation(b.num_blocks)
    for k in ("k_cache", "v_cache"):
        moved = torch.empty_like(pools[k])
        moved[torch.from_numpy(perm).cuda()] = pools[k]
        rep.layers[0][k].copy_(moved)
    b2 = W.Batch(b.hidden_rows, b.row_idx, b.positions, None, b.prior_lens, b.ctx_lens,
                 np.where(b.block_table >= 0, perm[np.maximum(b.block_table, 0)], -1)
                 .astype(np.int32), b.num_blocks)
    out2 = hidden.clone()
    rep.forward(0, out2, WD.batch_tensors(b2))
    torch.cuda.synchronize()
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))


def test_span_equals_successive_layers_bit_exactly():
    shape, b = _small_decode(7, priors=[5, 300, 17, 0, 900])
    L = 3
    rep = Replica.for_batch(shape, "s7", L, b)
    pools0 = [{k: t[k].clone() for k in ("k_cache", "v_cache")} for t in rep.layers]
    hidden = WD.hidden_tensor(shape, "s7", b.hidden_rows)
    bt = WD.batch_tensors(b)
    a = hidden.clone()
    rep.span(0, L, a, bt)
    torch.cuda.synchronize()
    for t, p in zip(rep.layers, pools0):
        for k in p:
            t[k].copy_(p[k])
    c = hidden.clone()
    for l in range(L):
        rep.forward(l, c, bt)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), c.view(torch.int16))


def test_prefill_span_equals_successive_layers_bit_exactly():
    """A prefill span reuses the per-row cache slots its first layer computes;
    every layer's output rows and appended cache bytes equal those of one-layer
    calls."""
    shape = small_bf16_shape()
    b = ragged_prefill_batch(12, priors=[0, 21, 300, 7], lens=[40, 3, 90, 33], max_ctx=512,
                             hidden_rows=200)
    L = 3
    rep = Replica.for_batch(shape, "s10", L, b)
    pools0 = [{k: t[k].clone() for k in ("k_cache", "v_cache")} for t in rep.layers]
    hidden = WD.hidden_tensor(shape, "s10", b.hidden_rows)
    bt = WD.batch_tensors(b)
    a = hidden.clone()
    rep.span(0, L, a, bt)
    torch.cuda.synchronize()
    pools_span = [{k: t[k].clone() for k in ("k_cache", "v_cache")} for t in rep.layers]
    for t, p in zip(rep.layers, pools0):
        for k in p:
            t[k].copy_(p[k])
    c = hidden.clone()
    for l in range(L):
        rep.forward(l, c, bt)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), c.view(torch.int16))
    for t, p in zip(rep.layers, pools_span):
        for k in p:
            assert torch.equal(t[k].view(torch.int16), p[k].view(torch.int16)), k


@pytest.mark.parametrize("hq", [5, 3])
def test_prefill_with_an_odd_head_count_matches_oracle(hq):
    """One KV head with five (three) query heads and d = 384: the QKV width
    of 7 (5) heads takes the narrow-tile QKV GEMM with 224-column (160-column)
    tiles of whole rotation pairs, split unevenly between the two waves of a
    row quarter, and d takes the narrow O and down GEMMs with three
    128-column tiles."""
    shape = small_bf16_shape(d=384, hq=hq, hkv=1, ffn=768)
    b = ragged_prefill_batch(13, priors=[0, 50, 17], lens=[30, 70, 16], max_ctx=256,
                             hidden_rows=150)
    rep = Replica.for_batch(shape, "s11", 1, b)
    hidden = WD.hidden_tensor(shape, "s11", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, cache, _ = oracle_prefill_seqs(shape, "s11", 0, b, range(b.n_seqs), h0)
    _check_rows("odd-head prefill", to64(hidden)[b.row_idx], ref, h0[b.row_idx])
    for s in range(b.n_seqs):
        t0, t1 = int(b.prior_lens[s]), int(b.ctx_lens[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, t0, t1)
        assert normwise_err(K, cache.K[s][t0:t1]) < TOL
        assert normwise_err(V, cache.V[s][t0:t1]) < TOL


def test_prefill_without_fused_projections_matches_oracle():
    """d = 4224 (33 x 128) and nine query heads with one KV head (11 heads):
    no prefill GEMM plan fuses the QKV projection (1408 columns) or the O and
    down projections, so the projections write fp32 partials, the separate
    QKV epilogue applies RoPE and the cache append, the separate residual +
    RMSNorm_2 kernel and the residual + scatter kernel run, and the gate/up
    GEMM's SwiGLU epilogue takes RMSNorm_2's output as it is."""
    shape = small_bf16_shape(d=4224, hq=9, hkv=1, ffn=768)
    b = ragged_prefill_batch(17, priors=[0, 33], lens=[40, 25], max_ctx=128, hidden_rows=90)
    rep = Replica.for_batch(shape, "s17", 1, b)
    hidden = WD.hidden_tensor(shape, "s17", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, cache, _ = oracle_prefill_seqs(shape, "s17", 0, b, range(b.n_seqs), h0)
    _check_rows("unfused prefill", to64(hidden)[b.row_idx], ref, h0[b.row_idx])
    for s in range(b.n_seqs):
        t0, t1 = int(b.prior_lens[s]), int(b.ctx_lens[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, t0, t1)
        assert normwise_err(K, cache.K[s][t0:t1]) < TOL
        assert normwise_err(V, cache.V[s][t0:t1]) < TOL


def test_prefill_at_high_positions_matches_oracle():
    """A chunk at positions near 30,000: far rows of the prefill RoPE table and
    the cache slots of a long sequence, against the oracle (its 30,000 prior
    tokens regenerated on the CPU)."""
    shape = small_bf16_shape()
    b = ragged_prefill_batch(14, priors=[30000, 5], lens=[40, 20], max_ctx=32768,
                             hidden_rows=80)
    rep = Replica.for_batch(shape, "s12", 1, b)
    hidden = WD.hidden_tensor(shape, "s12", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, cache, _ = oracle_prefill_seqs(shape, "s12", 0, b, range(b.n_seqs), h0)
    _check_rows("high-position prefill", to64(hidden)[b.row_idx], ref, h0[b.row_idx])
    for s in range(b.n_seqs):
        t0, t1 = int(b.prior_lens[s]), int(b.ctx_lens[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, t0, t1)
        assert normwise_err(K, cache.K[s][t0:t1]) < TOL
        assert normwise_err(V, cache.V[s][t0:t1]) < TOL


def test_empty_call_is_a_no_op():
    shape, b = _small_decode(8)
    rep = Replica.for_batch(shape, "s8", 1, b)
    hidden = WD.hidden_tensor(shape, "s8", b.hidden_rows)
    h0 = hidden.clone()
    bt = WD.batch_tensors(b.select([]))
    rep.forward(0, hidden, bt)
    torch.cuda.synchronize()
    assert torch.equal(hidden.view(torch.int16), h0.view(torch.int16))


def test_kv_append_is_a_bit_copy():
    shape = small_bf16_shape()
    b = ragged_decode_batch(9, [10, 40, 0], max_ctx=256)
    rep = Replica.for_batch(shape, "s9", 1, b)
    n = 20
    g = torch.Generator(device="cuda").manual_seed(0)
    k = torch.randn(n, shape.n_kv_heads, 128, device="cuda", generator=g).to(torch.bfloat16)
    v = torch.randn(n, shape.n_kv_heads, 128, device="cuda", generator=g).to(torch.bfloat16)
    seq = np.array([0] * 8 + [1] * 7 + [2] * 5, np.int32)
    pos = np.concatenate([np.arange(3, 11), np.arange(30, 37), np.arange(0, 5)]).astype(np.int32)
    coco.coco_kv_append(rep.h, 0, k, v, torch.from_numpy(seq).cuda(), torch.from_numpy(pos).cuda(),
                        WD.batch_tensors(b)["block_table"])
    torch.cuda.synchronize()
    kh, vh = to64(k), to64(v)
    for t in range(n):
        K, V = gpu_cache_tokens(rep.layers[0], b, int(seq[t]), int(pos[t]), int(pos[t]) + 1)
        assert np.array_equal(K[0], kh[t]) and np.array_equal(V[0], vh[t])


def test_abi_rejects_bad_arguments_and_stays_usable():
    shape, b = _small_decode(10)
    rep = Replica.for_batch(shape, "s10", 1, b)
    hidden = WD.hidden_tensor(shape, "s10", b.hidden_rows)
    bt = WD.batch_tensors(b)
    with pytest.raises(coco.CocoError) as e:
        coco.coco_layer_forward(rep.h, 1, hidden, bt["row_idx"], bt["positions"], None,
                                bt["block_table"], bt["ctx_lens"])
    assert e.value.code == -1
    big = WD.batch_tensors(W.decode_batch(np.random.default_rng(0), np.ones(b.n_rows + 1, int),
                                          2049, hidden_rows=b.hidden_rows + 1))
    with pytest.raises(coco.CocoError):
        coco.coco_layer_forward(rep.h, 0, hidden, big["row_idx"], big["positions"], None,
                                big["block_table"], big["ctx_lens"])
    # Validation mode: duplicate rows, out-of-range positions, bad blocks.
    coco.coco_layer_set_validate(rep.h, True)
    dup = dict(bt)
    ri = b.row_idx.copy()
    ri[1] = ri[0]
    dup["row_idx"] = torch.from_numpy(ri).cuda()
    with pytest.raises(coco.CocoError, match="duplicate"):
        rep.forward(0, hidden, dup)
    badpos = dict(bt)
    badpos["positions"] = bt["positions"] + 1
    with pytest.raises(coco.CocoError, match="positions"):
        rep.forward(0, hidden, badpos)
    badbt = dict(bt)
    t = b.block_table.copy()
    t[0, 0] = b.num_blocks + 5
    badbt["block_table"] = torch.from_numpy(t).cuda()
    with pytest.raises(coco.CocoError, match="block_table"):
        rep.forward(0, hidden, badbt)
    # The handle still works after rejected calls.
    h0 = hidden.clone()
    rep.forward(0, hidden, bt)
    torch.cuda.synchronize()
    assert not torch.equal(hidden, h0)


def test_init_rejects_unsupported_shapes():
    bad = coco.make_config(512, 8, 2, 64, 768, 1, "bf16", 8, 8, 4, 1e4, 1e-5)
    t = WD.layer_tensors(small_bf16_shape(), "x", 0, 4)
    with pytest.raises(coco.CocoError, match="head_dim"):
        coco.coco_layer_init(bad, [t])


def test_single_request_decode_with_a_full_block_table_matches_oracle():
    """Degenerate and maximal cases in one call: a batch of one request whose
    context fills its block table exactly (ctx = max_blocks * 16 = 1024), so
    the last partition and the last block end at the table's edge."""
    shape = small_bf16_shape()
    b = ragged_decode_batch(8, [1023], max_ctx=1024, hidden_rows=5, row_idx=np.array([3]))
    assert int(b.ctx_lens[0]) == b.block_table.shape[1] * W.BLOCK_SIZE
    rep = Replica.for_batch(shape, "s8", 1, b)
    hidden = WD.hidden_tensor(shape, "s8", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, _ = oracle_decode_rows(shape, "s8", 0, b, range(b.n_rows), h0)
    got = to64(hidden)
    y, x = got[b.row_idx], h0[b.row_idx]
    e = normwise_err(y, ref)
    assert e < TOL, e
    # One row: the branch y - x is ~15x smaller than y itself, so the bf16
    # rounding of the stored output (half an ulp, 2^-9 |y|) alone is several
    # percent of the branch. The branch bound is widened by exactly that
    # rounding budget.
    ed = normwise_err(y - x, ref - x)
    budget = 2.0 ** -8 * np.max(np.abs(ref)) / np.max(np.abs(ref - x))
    log(f"single full-table decode: output err {e:.2e}, branch err {ed:.2e} (rounding budget {budget:.2e})")
    assert ed < DELTA_TOL + budget, (ed, budget)
    others = sorted(set(range(b.hidden_rows)) - set(b.row_idx.tolist()))
    assert np.array_equal(got[others], h0[others])


def test_one_token_prefill_chunks_match_oracle_and_split():
    """The smallest prefill chunks: each request brings one token (one at
    position 0, so it attends only to itself). The rows match the oracle, and
    one request called alone gives the bits it gets inside the batch."""
    shape = small_bf16_shape()
    priors = [0, 17, 300]
    p = ragged_prefill_batch(9, priors=priors, lens=[1, 1, 1], max_ctx=512, hidden_rows=6)
    rep = Replica.for_batch(shape, "s9", 1, p)
    hidden = WD.hidden_tensor(shape, "s9", p.hidden_rows)
    h0 = to64(hidden)
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(p))
    whole = hidden.clone()
    rep.forward(0, whole, WD.batch_tensors(p))
    torch.cuda.synchronize()
    ref, _, _, _ = oracle_prefill_seqs(shape, "s9", 0, p, range(p.n_seqs), h0)
    _check_rows("one-token prefill", to64(whole)[p.row_idx], ref, h0[p.row_idx])
    snap.restore()
    alone = hidden.clone()
    rep.forward(0, alone, WD.batch_tensors(p.select_seqs([1])))
    torch.cuda.synchronize()
    r = int(p.row_idx[1])
    assert torch.equal(alone[r].view(torch.int16), whole[r].view(torch.int16))


def test_decode_row_before_the_cached_end_attends_up_to_its_position():
    """A decode row whose position lies before its sequence's cached end
    (positions[i] < ctx_lens[i] - 1, e.g. a rewound request) rewrites the slot
    of its position and attends keys 0 .. position only: the cached tokens past
    it are not read. Lengths cross block and 256-token partition edges (600
    cached, attending 301 keys; 256 cached, attending 256), a row at position 0
    attends only itself. Against the oracle, which takes
    min(ctx_lens, position + 1) keys."""
    shape = small_bf16_shape()
    priors = np.array([600, 256, 17, 1000, 40, 300], np.int64)
    back = np.array([300, 1, 17, 0, 24, 44], np.int64)   # position = prior - back
    base = ragged_decode_batch(21, priors, max_ctx=1025, hidden_rows=10,
                               row_idx=np.random.default_rng(21).permutation(10)[:6])
    b = W.Batch(base.hidden_rows, base.row_idx, (priors - back).astype(np.int32), None,
                base.prior_lens, base.ctx_lens, base.block_table, base.num_blocks)
    assert int(np.sum(b.positions < b.ctx_lens - 1)) == 5
    rep = Replica.for_batch(shape, "s21", 1, b)
    coco.coco_layer_set_validate(rep.h, True)  # the rows are valid input
    hidden = WD.hidden_tensor(shape, "s21", b.hidden_rows)
    h0 = to64(hidden)
    rep.forward(0, hidden, WD.batch_tensors(b))
    torch.cuda.synchronize()
    ref, _, cache = oracle_decode_rows(shape, "s21", 0, b, range(b.n_rows), h0)
    _check_rows("decode before the cached end", to64(hidden)[b.row_idx], ref, h0[b.row_idx])
    for s in range(b.n_seqs):
        p = int(b.positions[s])
        K, V = gpu_cache_tokens(rep.layers[0], b, s, p, p + 1)
        assert normwise_err(K[0], cache.K[s][p]) < TOL and normwise_err(V[0], cache.V[s][p]) < TOL
