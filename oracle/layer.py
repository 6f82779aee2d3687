"""Plain float64 decoder layer, row by row. Test infrastructure only.

Notation: d model width, Hq query heads, Hkv key/value heads, hd head size,
F SwiGLU width, G = Hq / Hkv query heads per key/value head.

Readings where the paper is silent (it names only "Transformer layers" with a
SwiGLU MLP, Sec. 3 and Sec. 4.2):
  * pre-norm block, no biases, no QK-norm;
  * rotary embedding in the rotate-half form, angle p * theta^(-2j/hd);
  * query head h reads key/value head floor(h / G);
  * the cache holds rotated keys and raw values; a token's own key/value are
    appended before attention, so every token attends to itself and to all
    earlier positions of its request (Sec. 3.1: each replica appends new
    key/value entries to its own cache partition).
"""
from __future__ import annotations

import math

import numpy as np


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gamma over the last axis.

    Pinned by: constant-vector closed form; torch.nn.functional.rms_norm in
    float64; brute force.
    """
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, np.float64)


def rope(u: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate every head vector of u (shape [..., hd]) to absolute position pos.

    For j < hd/2, with a = pos * theta^(-2j/hd):
      u'[j]        = u[j] cos a - u[j + hd/2] sin a
      u'[j + hd/2] = u[j + hd/2] cos a + u[j] sin a
    Pinned by: identity at position 0; the equivalent complex rotation
    (u[j] + i u[j+hd/2]) * exp(i a); pair norms preserved; logits depend only
    on relative position; brute force.
    """
    u = np.asarray(u, np.float64)
    hd = u.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    a = float(pos) * theta ** (-2.0 * j / hd)
    c, s = np.cos(a), np.sin(a)
    lo, hi = u[..., :half], u[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    """z * sigmoid(z). Pinned by torch.nn.functional.silu in float64."""
    z = np.asarray(z, np.float64)
    return z / (1.0 + np.exp(-z))


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Softmax attention of one query vector over n keys.

    q [hd], K [n, hd], V [n, hd] -> sum_t w_t V[t] with
    w = softmax(K q / sqrt(hd)).
    Pinned by: one key gives V[0]; equal keys give mean(V); weights sum to
    one; torch scaled_dot_product_attention in float64; brute force.
    """
    hd = q.shape[-1]
    z = K @ q / math.sqrt(hd)
    w = np.exp(z - z.max())
    w = w / w.sum()
    return w @ V


class KVCache:
    """Logical per-request key/value store: K[s], V[s] of shape [cap, Hkv, hd].

    Position t of request s lives at K[s][t]; the paged physical layout is the
    GPU library's business and is not modelled here.
    """

    def __init__(self, keys: list, values: list):
        self.K = [np.asarray(k, np.float64).copy() for k in keys]
        self.V = [np.asarray(v, np.float64).copy() for v in values]

    def copy(self) -> "KVCache":
        return KVCache(self.K, self.V)


def _row_seq(n_rows: int, seq_starts) -> np.ndarray:
    if seq_starts is None:
        return np.arange(n_rows)
    out = np.empty(n_rows, np.int64)
    for s in range(len(seq_starts) - 1):
        out[seq_starts[s]:seq_starts[s + 1]] = s
    return out


def layer_forward(w: dict, cfg, hidden: np.ndarray, row_idx, positions, seq_starts,
                  ctx_lens, cache: KVCache, record: bool = False):
    """One decoder layer applied to the call rows ``row_idx`` of ``hidden``.

    Arguments follow the library's call: row i of the call reads hidden row
    row_idx[i], belongs to request s(i) (s(i) = i in decode, else given by
    seq_starts) and holds the token at absolute position positions[i];
    ctx_lens[s] is request s's cached length once this call's tokens are in.

    Returns (new_hidden, intermediates or None). ``cache`` is updated in place
    with the rotated keys and raw values of the call's tokens. Rows not in
    row_idx are returned unchanged. Weights are float64 arrays in nn.Linear
    layout ([out, in]).

    Parity: pinned piecewise (see the functions above) and as a whole by a
    brute-force layer on tiny shapes; end-to-end values on random inputs have
    no published fixture, so beyond those pins they rest on this definition.
    """
    d, Hq, Hkv, hd, F = cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ffn
    G = Hq // Hkv
    row_idx = np.asarray(row_idx, np.int64)
    positions = np.asarray(positions, np.int64)
    ctx_lens = np.asarray(ctx_lens, np.int64)
    M = len(row_idx)
    seq_of = _row_seq(M, seq_starts)

    # Segment-boundary gather of the sub-batch rows (Sec. 3.1).
    x = np.asarray(hidden, np.float64)[row_idx]
    h = rms_norm(x, w["gamma_attn"], cfg.rms_eps)
    qkv = h @ np.asarray(w["w_qkv"], np.float64).T
    q = qkv[:, :Hq * hd].reshape(M, Hq, hd)
    k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(M, Hkv, hd)
    v = qkv[:, (Hq + Hkv) * hd:].reshape(M, Hkv, hd)
    q_rot = np.stack([rope(q[i], positions[i], cfg.rope_theta) for i in range(M)]) if M else q
    k_rot = np.stack([rope(k[i], positions[i], cfg.rope_theta) for i in range(M)]) if M else k

    # Local append into the replica's own cache partition (Sec. 3.1).
    for i in range(M):
        s, p = seq_of[i], positions[i]
        cache.K[s][p] = k_rot[i]
        cache.V[s][p] = v[i]

    # Attention of every query head over its request's keys 0..p.
    o = np.zeros((M, Hq, hd))
    for i in range(M):
        s, p = seq_of[i], positions[i]
        n = min(int(ctx_lens[s]), int(p) + 1)
        for hq in range(Hq):
            g = hq // G
            o[i, hq] = attend(q_rot[i, hq], cache.K[s][:n, g], cache.V[s][:n, g])

    x1 = x + o.reshape(M, Hq * hd) @ np.asarray(w["w_o"], np.float64).T
    h2 = rms_norm(x1, w["gamma_mlp"], cfg.rms_eps)
    gu = h2 @ np.asarray(w["w_gate_up"], np.float64).T
    a = silu(gu[:, :F]) * gu[:, F:]
    y = x1 + a @ np.asarray(w["w_down"], np.float64).T

    # Segment-boundary scatter back into the full-batch buffer (Sec. 3.1).
    out = np.array(hidden, np.float64, copy=True)
    out[row_idx] = y
    rec = None
    if record:
        rec = dict(x=x, h=h, q=q_rot, k=k_rot, v=v, o=o.reshape(M, Hq * hd), x1=x1,
                   h2=h2, a=a, y=y)
    return out, rec


def span_forward(weights: list, cfg, hidden, row_idx, positions, seq_starts, ctx_lens,
                 caches: list, round_between=None):
    """Consecutive layers as one replicated unit (Sec. 3.1): gather once, run
    every layer on the resident rows, scatter once.

    ``round_between`` (optional callable) is applied to the rows after every
    layer, e.g. to model a bf16 hidden state kept between layers; the oracle
    itself never rounds. Returns the new hidden buffer.
    """
    row_idx = np.asarray(row_idx, np.int64)
    M = len(row_idx)
    rows = np.asarray(hidden, np.float64)[row_idx]
    local = np.arange(M)
    for li, w in enumerate(weights):
        out, _ = layer_forward(w, cfg, rows, local, positions, seq_starts, ctx_lens,
                               caches[li])
        rows = out if round_between is None else round_between(out)
    result = np.array(hidden, np.float64, copy=True)
    result[row_idx] = rows
    return result
