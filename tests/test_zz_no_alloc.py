"""The no-alloc entry point (per-call buffers in the library's static scratch
array) against coco_layer_forward: two calls in a row, the second with a
smaller batch, each bit-identical to the regular entry point on the same
inputs and cache state (output rows and appended cache bytes); a call whose
buffers exceed the array is refused before any work."""
import numpy as np
import pytest
import torch

import paper_2607_04181_amd as coco
import workloads as W
from harness import (PoolSnapshot, Replica, gpu_cache_tokens, log, pool_blocks_of_new_tokens,
                     ragged_decode_batch, ragged_prefill_batch, small_bf16_shape)
from workloads import device as WD

pytestmark = pytest.mark.gpu


def _kv(rep, b):
    return [gpu_cache_tokens(rep.layers[0], b, s, int(b.prior_lens[s]), int(b.ctx_lens[s]))
            for s in range(b.n_seqs)]


def _same(rep, b, hidden, tag):
    """Regular and no-alloc forward of batch b from one cache state."""
    snap = PoolSnapshot(rep.layers[0], pool_blocks_of_new_tokens(b))
    bt = WD.batch_tensors(b)
    ref = hidden.clone()
    coco.coco_layer_forward(rep.h, 0, ref, bt["row_idx"], bt["positions"], bt["seq_starts"],
                            bt["block_table"], bt["ctx_lens"])
    torch.cuda.synchronize()
    kv_ref = _kv(rep, b)
    snap.restore()
    got = hidden.clone()
    coco.coco_layer_forward_noalloc(rep.h, 0, got, bt["row_idx"], bt["positions"],
                                    bt["seq_starts"], bt["block_table"], bt["ctx_lens"])
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), tag
    for (k1, v1), (k2, v2) in zip(_kv(rep, b), kv_ref):
        assert np.array_equal(k1, k2) and np.array_equal(v1, v2), tag
    log(f"no-alloc {tag}: {b.n_rows} rows bit-identical to coco_layer_forward")


def test_noalloc_decode_matches_the_regular_entry_point_twice():
    shape = small_bf16_shape()
    priors = [0, 15, 255, 256, 700, 1000, 3, 2047, 16, 511, 40, 90]
    b1 = ragged_decode_batch(31, priors, max_ctx=2049, hidden_rows=16,
                             row_idx=np.random.default_rng(31).permutation(16)[:12])
    rep = Replica.for_batch(shape, "na1", 1, b1)
    hidden = WD.hidden_tensor(shape, "na1", b1.hidden_rows)
    _same(rep, b1, hidden, "first call")
    # Second call: a smaller share of the same batch (the array keeps the
    # first call's contents).
    _same(rep, b1.select([7, 2, 10, 0, 5]), hidden, "second, smaller call")


def test_noalloc_prefill_matches_the_regular_entry_point_twice():
    shape = small_bf16_shape()
    b = ragged_prefill_batch(32, priors=[0, 40, 300], lens=[65, 1, 130], max_ctx=512,
                             hidden_rows=220)
    rep = Replica.for_batch(shape, "na2", 1, b)
    hidden = WD.hidden_tensor(shape, "na2", b.hidden_rows)
    _same(rep, b, hidden, "first prefill call")
    _same(rep, b.select_seqs([1, 0]), hidden, "second, smaller prefill call")


def test_noalloc_refuses_a_call_beyond_its_array():
    # The 32B-shaped 2048-token prefill needs far more than the 64 MiB array;
    # refused on the host, nothing enqueued.
    wl = W.c4_qwen32b()
    b, shape = wl.batch, wl.shape
    rep = Replica.for_batch(shape, wl.tag, 1, b)
    hidden = WD.hidden_tensor(shape, wl.tag, b.hidden_rows)
    h0 = hidden.clone()
    bt = WD.batch_tensors(b)
    with pytest.raises(coco.CocoError, match="scratch") as e:
        coco.coco_layer_forward_noalloc(rep.h, 0, hidden, bt["row_idx"], bt["positions"],
                                        bt["seq_starts"], bt["block_table"], bt["ctx_lens"])
    assert e.value.code == -1  # COCO_EINVAL
    torch.cuda.synchronize()
    assert torch.equal(hidden.view(torch.int16), h0.view(torch.int16))
