"""HIP-graph capture and replay of the forward entry points.

The forward calls only enqueue kernels on the caller's stream: no allocation,
no synchronisation, no memset, fixed workspace addresses (Sec. 5.2, graph
execution compatibility). So a captured span replays the same kernels on the
same buffers. Each graph is replayed several times, with the program's own
eager work and synchronisations in between, and every replay is compared bit
for bit with the eager result (output rows and written cache bytes).
"""
import numpy as np
import pytest
import torch

import workloads as W
from harness import (PoolSnapshot, Replica, log, pool_blocks_of_new_tokens, ragged_decode_batch,
                     ragged_prefill_batch, small_bf16_shape)
from workloads import device as WD

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _pools(rep):
    return [{k: t[k].clone() for k in ("k_cache", "v_cache")} for t in rep.layers]


def _same_pools(rep, pools):
    return all(torch.equal(t[k].view(torch.int16), p[k].view(torch.int16))
               for t, p in zip(rep.layers, pools) for k in p)


def _capture(fn):
    """Capture fn() on a side stream after one eager warm-up there."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def _restore(rep, pools):
    for t, p in zip(rep.layers, pools):
        for k in p:
            t[k].copy_(p[k])


def _replay_and_check(g, static_hidden, hidden, ref, rep, ref_pools, eager_noise, init_pools):
    for r in range(REPLAYS):
        static_hidden.copy_(hidden)   # eager input reset between replays
        eager_noise()                 # unrelated eager work on the same buffers' device
        _restore(rep, init_pools)     # the cache as before the eager run: every
        torch.cuda.synchronize()      # appended byte must come from the replay
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(static_hidden.view(torch.int16), ref.view(torch.int16)), r
        assert _same_pools(rep, ref_pools), r
        log(f"replay {r}: bit-identical to eager")


def test_graph_replay_of_decode_span_is_bit_identical():
    shape = small_bf16_shape()
    b = ragged_decode_batch(11, [0, 17, 255, 256, 700, 3, 1500], max_ctx=2049, hidden_rows=20,
                            row_idx=np.random.default_rng(11).permutation(20)[:7])
    L = 3
    rep = Replica.for_batch(shape, "g1", L, b)
    bt = WD.batch_tensors(b)
    hidden = WD.hidden_tensor(shape, "g1", b.hidden_rows)
    init_pools = _pools(rep)

    ref = hidden.clone()
    rep.span(0, L, ref, bt)
    torch.cuda.synchronize()
    ref_pools = _pools(rep)

    static_hidden = hidden.clone()
    g = _capture(lambda: rep.span(0, L, static_hidden, bt))
    scratch = torch.empty(1 << 20, device="cuda")

    def noise():
        scratch.normal_()
        torch.mm(scratch[:4096].view(64, 64), scratch[4096:8192].view(64, 64))

    _replay_and_check(g, static_hidden, hidden, ref, rep, ref_pools, noise, init_pools)


def test_graph_replay_of_prefill_is_bit_identical():
    shape = small_bf16_shape()
    b = ragged_prefill_batch(12, priors=[0, 40, 300], lens=[65, 1, 130], max_ctx=512,
                             hidden_rows=220)
    rep = Replica.for_batch(shape, "g2", 1, b)
    bt = WD.batch_tensors(b)
    hidden = WD.hidden_tensor(shape, "g2", b.hidden_rows)
    init_pools = _pools(rep)

    ref = hidden.clone()
    rep.forward(0, ref, bt)
    torch.cuda.synchronize()
    ref_pools = _pools(rep)

    static_hidden = hidden.clone()
    g = _capture(lambda: rep.forward(0, static_hidden, bt))
    other = hidden.clone()

    def noise():  # an eager forward of the same layer between replays
        other.copy_(hidden)
        rep.forward(0, other, bt)

    _replay_and_check(g, static_hidden, hidden, ref, rep, ref_pools, noise, init_pools)


@pytest.mark.slow
def test_graph_replay_of_llama8b_decode_step_is_bit_identical():
    """The bench configuration: batch-64 decode of the 8B-shaped layer."""
    wl = W.c2_llama8b_decode()
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, b)
    bt = WD.batch_tensors(b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)

    # Only the new tokens' blocks change; compare those, and put them back
    # into their state before the eager run ahead of every replay.
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    idx = snap.idx
    ref = hidden.clone()
    rep.forward(0, ref, bt)
    torch.cuda.synchronize()
    ref_kv = [rep.layers[0][k][idx].clone() for k in ("k_cache", "v_cache")]

    static_hidden = hidden.clone()
    g = _capture(lambda: rep.forward(0, static_hidden, bt))
    for r in range(REPLAYS):
        static_hidden.copy_(hidden)
        snap.restore()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(static_hidden.view(torch.int16), ref.view(torch.int16)), r
        for t, k in zip(ref_kv, ("k_cache", "v_cache")):
            assert torch.equal(rep.layers[0][k][idx].view(torch.int16), t.view(torch.int16)), r
    log("8B decode step: graph replays bit-identical to eager")
