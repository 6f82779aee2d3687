"""Input generators: determinism, sub-range regeneration, bf16 rounding and
the shapes/distributions each workload promises (CPU only)."""
import json
import math
import os

import numpy as np
import pytest
import torch

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_generator_is_deterministic_and_sub_ranges_match():
    k = W.stream_key("t", 1)
    a = W.normal(k, 300_000, 1.0)
    b = W.normal(k, 300_000, 1.0)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    part = W.normal(k, 5000, 1.0, start=123_456)
    assert torch.equal(part.view(torch.int16), a[123_456:128_456].view(torch.int16))
    other = W.normal(W.stream_key("t", 2), 1000, 1.0)
    assert not torch.equal(other, a[:1000])


def test_generator_moments_and_range():
    x = W.normal(W.stream_key("m"), 1_000_000, 0.02, dtype=torch.float32).double()
    assert abs(x.mean().item()) < 1e-4
    assert abs(x.std().item() / 0.02 - 1) < 5e-3
    assert x.abs().max().item() <= 0.02 * 4.9
    g = W.normal(W.stream_key("g"), 100_000, 0.1, 1.0, dtype=torch.float32).double()
    assert abs(g.mean().item() - 1) < 2e-3 and abs(g.std().item() - 0.1) < 2e-3


def test_bf16_rounding_is_nearest_even():
    f = torch.randn(200_000, generator=torch.Generator().manual_seed(0)) * 7
    f[:4] = torch.tensor([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0])
    mine = W._bf16_rne(f).view(torch.int16)
    assert torch.equal(mine, f.to(torch.bfloat16).view(torch.int16))
    # Ties: 1 + 2^-8 rounds down to 1 (even), 1 + 3*2^-8 rounds up.
    assert W._bf16_rne(f[:2]).float().tolist() == [1.0, 1.0 + 2 ** -6]


def test_weights_have_linear_layout_and_sizes():
    w = W.layer_weights(W.TINY, "c1", 0)
    assert w["w_qkv"].shape == (8 * 64, 256) and w["w_qkv"].dtype == torch.float32
    assert w["w_gate_up"].shape == (2 * 688, 256) and w["w_down"].shape == (256, 688)
    rows = W.weight_rows(W.TINY, "c1", 0, "w_down", 10, 20)
    assert torch.equal(rows, w["w_down"][10:20])
    assert W.LLAMA8B.param_count() == 218_112_000


def test_kv_pool_block_subset_matches_full_pool():
    full = W.kv_pool(W.TINY, "c1", 0, 21, "v")
    sub = W.kv_pool(W.TINY, "c1", 0, 21, "v", blocks=np.array([5, 0, 20]))
    assert torch.equal(sub, full[[5, 0, 20]])
    assert full.shape == (21, 2, 16 * 64)


@pytest.mark.parametrize("cid", sorted(W.ALL))
def test_workload_batches_are_consistent(cid):
    wl = W.ALL[cid]()
    for b in [wl.batch] + [x for x in (wl.full_batch, wl.decode_after) if x is not None]:
        assert len(set(b.row_idx.tolist())) == b.n_rows
        assert b.row_idx.max() < b.hidden_rows
        used = b.block_table[b.block_table >= 0]
        assert used.max() < b.num_blocks
        for s in range(b.n_seqs):
            need = -(-int(b.ctx_lens[s]) // 16)
            assert (b.block_table[s, :need] >= 0).all()
            rows = b.rows_of_seq(s)
            assert list(b.positions[rows]) == list(range(b.prior_lens[s], b.ctx_lens[s]))
    # Physical blocks are never shared between requests.
    b = wl.full_batch or wl.decode_after or wl.batch
    used = b.block_table[b.block_table >= 0]
    assert len(np.unique(used)) == len(used)


def test_workload_distributions():
    c2 = W.c2_llama8b_decode().batch
    assert c2.n_rows == 64 and 16 <= c2.prior_lens.min() and c2.prior_lens.max() <= 8192
    c3 = W.c3_llama8b_skewed()
    assert c3.batch.n_rows == 96 and c3.full_batch.n_rows == 256
    c4 = W.c4_qwen32b()
    assert c4.batch.n_rows == 2048 and list(c4.batch.prior_lens) == [0, 512, 1024, 4096]
    assert c4.decode_after.n_rows == 128
    assert list(c4.decode_after.prior_lens[:4]) == [512, 1024, 1536, 4608]
    c1 = W.c1_tiny()
    assert list(c1.batch.row_idx) == [1, 3, 4, 6] and c1.batch.hidden_rows == 8


def test_even_partition_matches_paper_examples():
    with open(os.path.join(GOLDEN, "split_examples.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        parts = W.even_partition(c["bs"], c["v"])
        assert [len(p) for p in parts] == c["sizes"]
        assert max(len(p) for p in parts) == math.ceil(c["bs"] / c["v"])
        assert np.array_equal(np.concatenate(parts), np.arange(c["bs"]))


def test_depager_matches_the_documented_tile_formula():
    """The oracle-side de-pager against explicit loops over the layout."""
    from oracle.paged import depage_blocks
    rng = np.random.default_rng(0)
    for hd in (64, 128):
        nb, Hkv = 3, 2
        K = rng.normal(size=(nb * 16, Hkv, hd))
        V = rng.normal(size=(nb * 16, Hkv, hd))
        kb = np.zeros((nb, Hkv, 16 * hd))
        vb = np.zeros((nb, Hkv, 16 * hd))
        for tok in range(nb * 16):
            b, t = divmod(tok, 16)
            for g in range(Hkv):
                for h in range(hd):
                    kb[b, g, ((h // 32) * 64 + ((h % 32) // 8) * 16 + t) * 8 + h % 8] = K[tok, g, h]
                    vb[b, g, (((h // 32) * 64 + (t // 4) * 16 + h % 16) * 2 + (h // 16) % 2) * 4
                       + t % 4] = V[tok, g, h]
        K2, V2 = depage_blocks(kb, vb, nb * 16 - 5)
        assert np.array_equal(K2, K[:nb * 16 - 5]) and np.array_equal(V2, V[:nb * 16 - 5])
        # Each tile formula is a permutation of the tile.
        from oracle.paged import tile_index
        ki, vi = tile_index(hd)
        assert sorted(ki.ravel()) == list(range(16 * hd)) == sorted(vi.ravel())
