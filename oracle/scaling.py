"""Speedup and cost model of layer-wise replication, plain float64 Python.
TEST INFRASTRUCTURE ONLY (see the package docstring).

Written from Sec. 4.2 (cost and speedup modelling, heterogeneous
generalisation) and the scaling algorithm of Sec. 4.4:

* split_sizes:     sub-batch sizes when bs rows are divided over v devices.
* cost_mem/comp:   Eq. (cost_mem) and Eq. (cost_com), per device.
* comm_time:       T(P), boundary scatter + gather of the offloaded rows.
* work, speedup:   W(N, P) and S(N, P) (Eq. speedup_simple).
* speedup_ab:      the alpha/beta form (Eq. speedup_final).
* span_vector, work_vec, comm_vec, speedup_vec: the per-layer vector form
                   W(v), T(v), S(v).
* distance, scale_candidates: the L1 transition distance and the candidate
                   ranking of the unified scaling algorithm.

Readings (where the paper is silent or inconsistent):
* T(P) and T(v) are printed without bytes per element; `elem_bytes` makes it
  explicit (2 for bf16). T(v) is printed without the sequence length l; the
  same factor as in T(P) is applied.
* A transition of v is an index l with v[l] != v[l+1], taking v[L] = 1 after
  the last layer (rows return to the host); its volume uses v[l] as printed,
  so only the exit of a replicated span moves rows, and the factor 2 covers
  both directions.
* split_sizes gives ceil(bs/v) to the first bs mod v devices and floor(bs/v)
  to the rest (heaviest first); this is the paper's "heaviest device gets
  ceil, the others floor" whenever bs mod v <= 1 and keeps the total bs.
* Device k of layer l's set is device k of one global list (device 0 is the
  host): layer l runs on devices 0 .. v[l]-1.
* Cost(N, P), the resource count of the scaling algorithm, is the number of
  replica devices P - 1 (extending N at fixed P costs none, as in the paper's
  N=10 -> 20 example).
* Candidates are ranked by distance, then by larger speedup, then smaller P,
  then smaller N (the paper leaves ties open).
"""
from __future__ import annotations

import math


def split_sizes(bs: int, v: int) -> list:
    """Rows per device when a batch of bs rows is split over v devices
    (Sec. 3.1: 15 -> 8 + 7; Sec. 4.2: heaviest ceil(bs/v), others floor)."""
    if bs < 0 or v < 1:
        raise ValueError("bs >= 0 and v >= 1 required")
    base, extra = divmod(bs, v)
    return [base + 1 if k < extra else base for k in range(v)]


def cost_mem(N: int, P: int, bs: float, l: float, d_hidden: float, kappa: float = 2.0) -> float:
    """Per-device memory of a replica set (Eq. cost_mem): N layers of 12 d^2
    weights plus the device's activation share bs/P * l * d, kappa bytes each."""
    return N * kappa * (12.0 * d_hidden * d_hidden + bs / P * l * d_hidden)


def cost_comp(N: int, P: int, bs: float, l: float, d_hidden: float) -> float:
    """Per-device compute of a replica set (Eq. cost_com): N/P * 24 bs l d^2."""
    return N / P * 24.0 * bs * l * d_hidden * d_hidden


def comm_time(bs: float, P: int, l: float, d_hidden: float, bandwidth: float,
              elem_bytes: float = 2.0) -> float:
    """T(P): the (P-1)/P share of the batch leaves and returns once per
    forward (factor 2), l tokens of d_hidden elements each, at bandwidth B."""
    return 2.0 * (bs / P * (P - 1) * l * d_hidden * elem_bytes) / bandwidth


def work(L: int, N: int, P: int, t_comp: float) -> float:
    """W(N, P): L-N layers on the host, N layers at P-fold parallelism."""
    return (L - N) * t_comp + N * t_comp / P


def speedup(L: int, N: int, P: int, t_comp: float, t_comm: float = 0.0) -> float:
    """S(N, P) = L t / (W(N, P) + T(P)) (Eq. speedup_simple)."""
    return L * t_comp / (work(L, N, P, t_comp) + t_comm)


def speedup_ab(alpha: float, beta: float, P: int) -> float:
    """S = 1 / (1 - alpha + alpha/P + beta) (Eq. speedup_final)."""
    return 1.0 / (1.0 - alpha + alpha / P + beta)


def span_vector(L: int, first: int, N: int, P: int) -> list:
    """Per-layer parallelism: P on layers first .. first+N-1, 1 elsewhere."""
    if not (0 <= first and N >= 0 and first + N <= L):
        raise ValueError("span outside the model")
    return [P if first <= i < first + N else 1 for i in range(L)]


def work_vec(v, bs: int, t_dev) -> float:
    """W(v) = sum_l max_{k in D(l)} t_k * ceil(bs / v_l) / bs, with D(l) the
    first v_l devices."""
    total = 0.0
    for vl in v:
        slowest = max(t_dev[k] for k in range(vl))
        total += slowest * math.ceil(bs / vl) / bs
    return total


def comm_vec(v, bs: int, l: float, d_hidden: float, b_min: float,
             elem_bytes: float = 2.0) -> float:
    """T(v) = sum over transitions of 2 ceil(bs (v_l - 1)/v_l) l d / B_min."""
    total = 0.0
    L = len(v)
    for i in range(L):
        nxt = v[i + 1] if i + 1 < L else 1
        if v[i] != nxt:
            rows = math.ceil(bs * (v[i] - 1) / v[i])
            total += 2.0 * rows * l * d_hidden * elem_bytes / b_min
    return total


def speedup_vec(v, bs: int, l: float, d_hidden: float, t_dev, bandwidths,
                elem_bytes: float = 2.0) -> float:
    """S(v) = sum_l t_host / (W(v) + T(v)), B_min the slowest link."""
    b_min = min(bandwidths)
    return len(v) * t_dev[0] / (work_vec(v, bs, t_dev) +
                                comm_vec(v, bs, l, d_hidden, b_min, elem_bytes))


def distance(v_a, v_b) -> int:
    """Transition distance: the L1 norm of the difference of two vectors."""
    return sum(abs(a - b) for a, b in zip(v_a, v_b))


def scale_candidates(L: int, first: int, P_max: int, N_cur: int, P_cur: int,
                     latency_over_slo: float, t_comp: float, bs: float, l: float,
                     d_hidden: float, bandwidth: float, cold_devices: int,
                     elem_bytes: float = 2.0):
    """The unified scaling step for one instance: the required speedup
    S(cur) * latency/SLO, the (N, P) spans that reach it ranked by distance
    from the current vector, and the first one whose extra devices fit.

    Returns (alpha_req, ranked, chosen): ranked is a list of
    (N, P, S, distance), chosen the first affordable (N, P) or None. P = 1
    (no replication) is the single candidate (0, 1)."""
    def s_of(N, P):
        t = comm_time(bs, P, l, d_hidden, bandwidth, elem_bytes) if N > 0 else 0.0
        return speedup(L, N, P, t_comp, t)

    cur_v = span_vector(L, first, N_cur, P_cur)
    alpha_req = s_of(N_cur, P_cur) * latency_over_slo
    cands = [(0, 1)] + [(N, P) for P in range(2, P_max + 1) for N in range(1, L - first + 1)]
    ranked = []
    for N, P in cands:
        s = s_of(N, P)
        if s >= alpha_req:
            ranked.append((N, P, s, distance(cur_v, span_vector(L, first, N, P))))
    ranked.sort(key=lambda c: (c[3], -c[2], c[1], c[0]))
    chosen = None
    for N, P, _, _ in ranked:
        delta = (P - 1) - (P_cur - 1)
        if delta <= 0 or cold_devices >= delta:
            chosen = (N, P)
            break
    return alpha_req, ranked, chosen
