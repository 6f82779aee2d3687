"""Pins of the float64 oracle against things other than itself (CPU only).

Each part of the layer is checked against a closed form, an invariant, a torch
library routine evaluated in float64, or the independent brute-force layer in
brute.py. ``test_planted_mistakes_are_caught`` plants plausible mistakes in the
oracle and checks that these pins fail on them.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import brute
import oracle
from oracle import layer as OL

TINY = SimpleNamespace(d_model=12, n_q_heads=4, n_kv_heads=2, head_dim=4, d_ffn=10,
                       rope_theta=100.0, rms_eps=1e-6)


def tiny_weights(cfg, seed):
    rng = np.random.default_rng(seed)
    d, hd, F = cfg.d_model, cfg.head_dim, cfg.d_ffn
    qkv = (cfg.n_q_heads + 2 * cfg.n_kv_heads) * hd
    return {
        "w_qkv": rng.normal(0, 0.3, (qkv, d)),
        "w_o": rng.normal(0, 0.3, (d, cfg.n_q_heads * hd)),
        "w_gate_up": rng.normal(0, 0.3, (2 * F, d)),
        "w_down": rng.normal(0, 0.3, (d, F)),
        "gamma_attn": 1 + rng.normal(0, 0.1, d),
        "gamma_mlp": 1 + rng.normal(0, 0.1, d),
    }


def tiny_case(cfg, seed, prefill=False):
    """A 6-row hidden buffer, 3 requests with random cached context."""
    rng = np.random.default_rng(seed + 100)
    hidden = rng.normal(0, 1, (6, cfg.d_model))
    cap = 12
    K = [rng.normal(0, 1, (cap, cfg.n_kv_heads, cfg.head_dim)) for _ in range(3)]
    V = [rng.normal(0, 1, (cap, cfg.n_kv_heads, cfg.head_dim)) for _ in range(3)]
    if not prefill:
        prior = np.array([3, 0, 7])
        row_idx = np.array([4, 0, 2])
        positions = prior.copy()
        seq_starts = None
        ctx = prior + 1
    else:
        prior = np.array([2, 0, 5])
        lens = np.array([2, 3, 1])
        row_idx = np.array([5, 1, 3, 0, 2, 4])
        positions = np.concatenate([np.arange(p, p + n) for p, n in zip(prior, lens)])
        seq_starts = np.concatenate([[0], np.cumsum(lens)])
        ctx = prior + lens
    return hidden, row_idx, positions, seq_starts, ctx, K, V


def seq_of(n_rows, seq_starts):
    if seq_starts is None:
        return list(range(n_rows))
    out = []
    for s in range(len(seq_starts) - 1):
        out += [s] * int(seq_starts[s + 1] - seq_starts[s])
    return out


def run_brute(w, cfg, hidden, row_idx, positions, seq_starts, ctx, K, V):
    wl = {k: v.tolist() for k, v in w.items()}
    Kl = [k.tolist() for k in K]
    Vl = [v.tolist() for v in V]
    out = brute.layer(wl, cfg, hidden.tolist(), [int(r) for r in row_idx],
                      [int(p) for p in positions], seq_of(len(row_idx), seq_starts),
                      [int(c) for c in ctx], Kl, Vl)
    return np.array(out), [np.array(k) for k in Kl], [np.array(v) for v in Vl]


# ---------------------------------------------------------------- RMSNorm

def test_rmsnorm_constant_vector_closed_form():
    c, eps = 1.7, 1e-6
    g = np.linspace(0.5, 1.5, 16)
    got = oracle.rms_norm(np.full(16, c), g, eps)
    np.testing.assert_allclose(got, c / math.sqrt(c * c + eps) * g, rtol=1e-15)


def test_rmsnorm_matches_torch_float64():
    rng = np.random.default_rng(0)
    x = rng.normal(0, 2, (5, 33))
    g = rng.normal(1, 0.1, 33)
    ref = Fn.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.rms_norm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------------- RoPE

def test_rope_is_identity_at_position_zero():
    u = np.random.default_rng(1).normal(size=(3, 8))
    assert np.array_equal(oracle.rope(u, 0, 1e4), u)


def test_rope_single_pair_closed_form():
    # hd = 2: one pair, angle = pos * theta^0 = pos radians.
    got = oracle.rope(np.array([1.0, 0.0]), 1, 1e4)
    np.testing.assert_allclose(got, [math.cos(1.0), math.sin(1.0)], rtol=1e-15)
    got = oracle.rope(np.array([0.0, 1.0]), 2, 1e4)
    np.testing.assert_allclose(got, [-math.sin(2.0), math.cos(2.0)], rtol=1e-15)


def test_rope_matches_complex_rotation():
    rng = np.random.default_rng(2)
    hd, theta = 16, 5e5
    u = rng.normal(size=(4, hd))
    for pos in (1, 7, 1234, 32767):
        z = (u[:, :hd // 2] + 1j * u[:, hd // 2:]) * np.exp(
            1j * pos * np.power(theta, -np.arange(0, hd, 2) / hd))
        np.testing.assert_allclose(oracle.rope(u, pos, theta),
                                   np.concatenate([z.real, z.imag], axis=1),
                                   rtol=1e-12, atol=1e-12)


def test_rope_preserves_pair_norms_and_relative_logits():
    rng = np.random.default_rng(3)
    hd, theta = 8, 1e4
    q, k = rng.normal(size=hd), rng.normal(size=hd)
    r = oracle.rope(q, 37, theta)
    np.testing.assert_allclose(r[:4] ** 2 + r[4:] ** 2, q[:4] ** 2 + q[4:] ** 2, rtol=1e-12)
    base = oracle.rope(q, 10, theta) @ oracle.rope(k, 3, theta)
    for delta in (1, 100, 4000):
        shifted = oracle.rope(q, 10 + delta, theta) @ oracle.rope(k, 3 + delta, theta)
        assert abs(shifted - base) < 1e-9


# ---------------------------------------------------------------- SiLU

def test_silu_matches_torch_float64():
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(oracle.silu(z), Fn.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-14, atol=1e-300)
    assert oracle.silu(np.array([0.0]))[0] == 0.0


# ---------------------------------------------------------------- attention

def test_attend_single_key_returns_value():
    rng = np.random.default_rng(4)
    v = rng.normal(size=(1, 8))
    np.testing.assert_array_equal(oracle.attend(rng.normal(size=8), rng.normal(size=(1, 8)), v),
                                  v[0])


def test_attend_equal_keys_give_mean_value():
    rng = np.random.default_rng(5)
    k = np.tile(rng.normal(size=8), (6, 1))
    V = rng.normal(size=(6, 8))
    np.testing.assert_allclose(oracle.attend(rng.normal(size=8), k, V), V.mean(0), rtol=1e-13)


def test_attend_matches_torch_sdpa_gqa():
    rng = np.random.default_rng(6)
    Hq, Hkv, hd, n = 8, 2, 16, 37
    q = rng.normal(size=(Hq, hd))
    K = rng.normal(size=(n, Hkv, hd))
    V = rng.normal(size=(n, Hkv, hd))
    ref = Fn.scaled_dot_product_attention(
        torch.from_numpy(q)[None, :, None, :], torch.from_numpy(K).permute(1, 0, 2)[None],
        torch.from_numpy(V).permute(1, 0, 2)[None], enable_gqa=True)[0, :, 0].numpy()
    got = np.stack([oracle.attend(q[h], K[:, h // (Hq // Hkv)], V[:, h // (Hq // Hkv)])
                    for h in range(Hq)])
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- whole layer

@pytest.mark.parametrize("prefill", [False, True])
@pytest.mark.parametrize("seed", [0, 1])
def test_layer_matches_brute_force(prefill, seed):
    cfg = TINY
    w = tiny_weights(cfg, seed)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, seed, prefill)
    cache = oracle.KVCache(K, V)
    got, _ = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx, cache)
    ref, Kb, Vb = run_brute(w, cfg, hidden, row_idx, pos, starts, ctx, K, V)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)
    for s in range(3):
        np.testing.assert_allclose(cache.K[s], Kb[s], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(cache.V[s], Vb[s], rtol=1e-12, atol=1e-12)


def test_layer_attention_matches_torch_sdpa_with_causal_mask():
    cfg = TINY
    w = tiny_weights(cfg, 3)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 3, prefill=True)
    cache = oracle.KVCache(K, V)
    _, rec = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx, cache, record=True)
    Hq, Hkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    so = seq_of(len(row_idx), starts)
    for s in range(3):
        rows = [i for i in range(len(row_idx)) if so[i] == s]
        n = int(ctx[s])
        q = torch.from_numpy(rec["q"][rows]).permute(1, 0, 2)[None]
        k = torch.from_numpy(cache.K[s][:n]).permute(1, 0, 2)[None]
        v = torch.from_numpy(cache.V[s][:n]).permute(1, 0, 2)[None]
        mask = torch.tensor([[t <= pos[i] for t in range(n)] for i in rows])
        ref = Fn.scaled_dot_product_attention(q, k, v, attn_mask=mask, enable_gqa=True)
        ref = ref[0].permute(1, 0, 2).reshape(len(rows), Hq * hd).numpy()
        np.testing.assert_allclose(rec["o"][rows], ref, rtol=1e-12, atol=1e-12)


def test_zero_output_projections_pass_rows_through():
    cfg = TINY
    w = tiny_weights(cfg, 4)
    w["w_o"][:] = 0.0
    w["w_down"][:] = 0.0
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 4)
    got, _ = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx,
                                  oracle.KVCache(K, V))
    assert np.array_equal(got, hidden)


def test_rows_outside_the_subset_are_untouched():
    cfg = TINY
    w = tiny_weights(cfg, 5)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 5)
    got, _ = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx,
                                  oracle.KVCache(K, V))
    others = sorted(set(range(6)) - set(row_idx.tolist()))
    assert np.array_equal(got[others], hidden[others])


def test_prefill_rows_equal_successive_decodes():
    cfg = TINY
    w = tiny_weights(cfg, 6)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 6, prefill=True)
    pre, _ = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx,
                                  oracle.KVCache(K, V))
    cache = oracle.KVCache(K, V)
    so = seq_of(len(row_idx), starts)
    for i in range(len(row_idx)):  # rows of a request are in position order
        s = so[i]
        out, _ = oracle.layer_forward(w, cfg, hidden, [row_idx[i]], [pos[i]], [0, 1],
                                      [pos[i] + 1], _SingleSeq(cache, s))
        np.testing.assert_allclose(out[row_idx[i]], pre[row_idx[i]], rtol=1e-11, atol=1e-11)


class _SingleSeq:
    """View of one request of a KVCache as a one-request cache."""

    def __init__(self, cache, s):
        self.K = [cache.K[s]]
        self.V = [cache.V[s]]


def test_split_batch_equals_whole_batch():
    cfg = TINY
    w = tiny_weights(cfg, 7)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 7)
    whole, _ = oracle.layer_forward(w, cfg, hidden, row_idx, pos, starts, ctx,
                                    oracle.KVCache(K, V))
    cache = oracle.KVCache(K, V)
    out = hidden.copy()
    for part in ([0, 2], [1]):
        sub = _Sub(cache, part)
        out, _ = oracle.layer_forward(w, cfg, out, row_idx[part], pos[part], None, ctx[part], sub)
    np.testing.assert_allclose(out, whole, rtol=1e-12, atol=1e-12)


class _Sub:
    def __init__(self, cache, seqs):
        self.K = [cache.K[s] for s in seqs]
        self.V = [cache.V[s] for s in seqs]


def test_span_is_layer_after_layer():
    cfg = TINY
    ws = [tiny_weights(cfg, 10 + i) for i in range(3)]
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg, 8)
    caches = [oracle.KVCache(K, V) for _ in ws]
    got = oracle.span_forward(ws, cfg, hidden, row_idx, pos, starts, ctx, caches)
    h = hidden
    for w in ws:
        h, _ = oracle.layer_forward(w, cfg, h, row_idx, pos, starts, ctx, oracle.KVCache(K, V))
    np.testing.assert_allclose(got, h, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- planted mistakes

def _pins_pass():
    """Run the pins that a planted mistake should break; True if all pass."""
    try:
        test_rope_matches_complex_rotation()
        test_attend_matches_torch_sdpa_gqa()
        for prefill in (False, True):
            test_layer_matches_brute_force(prefill, 0)
        test_layer_attention_matches_torch_sdpa_with_causal_mask()
    except AssertionError:
        return False
    return True


MUTATIONS = {
    "rope sign flipped": ("rope", lambda orig: lambda u, p, t: orig(u, -p, t)),
    "rope halves swapped": ("rope", lambda orig: lambda u, p, t: orig(u[..., ::-1], p, t)[..., ::-1]),
    "rms without eps": ("rms_norm", lambda orig: lambda x, g, e: orig(x, g, 0.0) * (1 + 1e-3)),
    "rms mean over wrong axis": ("rms_norm", lambda orig: lambda x, g, e: (
        np.asarray(x) / np.sqrt(np.mean(np.asarray(x) ** 2, axis=0, keepdims=True) + e) * g)),
    "silu as sigmoid": ("silu", lambda orig: lambda z: 1.0 / (1.0 + np.exp(-np.asarray(z)))),
    "attention scale dropped": ("attend", lambda orig: lambda q, K, V: orig(q * math.sqrt(q.shape[-1]), K, V)),
    "attention misses last key": ("attend", lambda orig: lambda q, K, V: orig(q, K[:-1], V[:-1]) if len(K) > 1 else orig(q, K, V)),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, make = MUTATIONS[name]
    orig = getattr(OL, attr)
    bad = make(orig)
    monkeypatch.setattr(OL, attr, bad)
    monkeypatch.setattr(oracle, attr, bad)
    assert not _pins_pass(), f"planted mistake '{name}' went unnoticed"


def test_planted_gqa_mapping_mistake_is_caught(monkeypatch):
    # Interleaved instead of contiguous head groups.
    src = OL.layer_forward

    def bad_layer(w, cfg, *a, **k):
        w2 = dict(w)
        Hq, hd = cfg.n_q_heads, cfg.head_dim
        G = Hq // cfg.n_kv_heads
        perm = [(h % G) * cfg.n_kv_heads + h // G for h in range(Hq)]
        q = w["w_qkv"][:Hq * hd].reshape(Hq, hd, -1)[perm].reshape(Hq * hd, -1)
        w2["w_qkv"] = np.concatenate([q, w["w_qkv"][Hq * hd:]])
        wo = w["w_o"].reshape(w["w_o"].shape[0], Hq, hd)[:, perm].reshape(w["w_o"].shape[0], -1)
        w2["w_o"] = wo
        return src(w2, cfg, *a, **k)

    monkeypatch.setattr(OL, "layer_forward", bad_layer)
    monkeypatch.setattr(oracle, "layer_forward", bad_layer)
    assert not _pins_pass()


def test_planted_transposed_weight_is_caught(monkeypatch):
    src = OL.layer_forward
    cfg_sq = SimpleNamespace(**{**vars(TINY), "d_model": 16})  # W_o square: 16 x 16

    def bad_layer(w, cfg, *a, **k):
        w2 = dict(w)
        w2["w_o"] = np.ascontiguousarray(w["w_o"].T) if w["w_o"].shape[0] == w["w_o"].shape[1] \
            else w["w_o"]
        return src(w2, cfg, *a, **k)

    monkeypatch.setattr(OL, "layer_forward", bad_layer)
    monkeypatch.setattr(oracle, "layer_forward", bad_layer)
    w = tiny_weights(cfg_sq, 0)
    hidden, row_idx, pos, starts, ctx, K, V = tiny_case(cfg_sq, 0)
    got, _ = oracle.layer_forward(w, cfg_sq, hidden, row_idx, pos, starts, ctx,
                                  oracle.KVCache(K, V))
    ref, _, _ = run_brute(w, cfg_sq, hidden, row_idx, pos, starts, ctx, K, V)
    assert not np.allclose(got, ref, rtol=1e-6, atol=1e-6)
