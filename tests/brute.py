"""Brute-force decoder layer in plain Python (lists and the math module).

An independent second writing of the layer for tiny shapes, used only to pin
the float64 oracle. It shares nothing with the oracle: every sum is an explicit
loop and the rotary embedding is written as a complex rotation.
"""
import cmath
import math


def matvec(W, x):
    """W is a list of rows (nn.Linear layout [out][in])."""
    return [sum(W[r][c] * x[c] for c in range(len(x))) for r in range(len(W))]


def rmsnorm(x, g, eps):
    ms = sum(v * v for v in x) / len(x)
    inv = 1.0 / math.sqrt(ms + eps)
    return [x[i] * inv * g[i] for i in range(len(x))]


def rotate(u, pos, theta):
    hd = len(u)
    half = hd // 2
    out = [0.0] * hd
    for j in range(half):
        z = complex(u[j], u[j + half]) * cmath.exp(1j * pos * theta ** (-2.0 * j / hd))
        out[j], out[j + half] = z.real, z.imag
    return out


def softmax_attend(q, keys, vals):
    hd = len(q)
    z = [sum(q[c] * k[c] for c in range(hd)) / math.sqrt(hd) for k in keys]
    m = max(z)
    e = [math.exp(t - m) for t in z]
    tot = sum(e)
    return [sum(e[t] * vals[t][c] for t in range(len(keys))) / tot for c in range(hd)]


def layer(w, cfg, hidden, row_idx, positions, seq_of, ctx_lens, K, V):
    """hidden: list of rows; K[s][t][g] / V[s][t][g]: lists (mutated)."""
    d, Hq, Hkv, hd, F = cfg.d_model, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ffn
    G = Hq // Hkv
    Wqkv, Wo, Wgu, Wd = w["w_qkv"], w["w_o"], w["w_gate_up"], w["w_down"]
    xs, qs = [], []
    for i, r in enumerate(row_idx):
        x = list(hidden[r])
        h = rmsnorm(x, w["gamma_attn"], cfg.rms_eps)
        qkv = matvec(Wqkv, h)
        q = [rotate(qkv[a * hd:(a + 1) * hd], positions[i], cfg.rope_theta) for a in range(Hq)]
        k = [rotate(qkv[(Hq + a) * hd:(Hq + a + 1) * hd], positions[i], cfg.rope_theta)
             for a in range(Hkv)]
        v = [qkv[(Hq + Hkv + a) * hd:(Hq + Hkv + a + 1) * hd] for a in range(Hkv)]
        K[seq_of[i]][positions[i]] = k
        V[seq_of[i]][positions[i]] = v
        xs.append(x)
        qs.append(q)
    out = [list(r) for r in hidden]
    for i, r in enumerate(row_idx):
        s, p = seq_of[i], positions[i]
        n = min(ctx_lens[s], p + 1)
        o = []
        for a in range(Hq):
            g = a // G
            o += softmax_attend(qs[i][a], [K[s][t][g] for t in range(n)],
                                [V[s][t][g] for t in range(n)])
        x1 = [xs[i][c] + t for c, t in enumerate(matvec(Wo, o))]
        h2 = rmsnorm(x1, w["gamma_mlp"], cfg.rms_eps)
        gu = matvec(Wgu, h2)
        act = [gu[j] / (1.0 + math.exp(-gu[j])) * gu[F + j] for j in range(F)]
        y = [x1[c] + t for c, t in enumerate(matvec(Wd, act))]
        out[r] = y
    return out
