"""Pins of the speedup/cost model oracle (oracle/scaling.py), CPU only.

The paper prints a few values of the model (Sec. 4.1: N = 20, P = 2 on a
60-layer model approaches a 1.2x speedup; Sec. 4.2: with bs = 1 no split can
speed anything up; Sec. 3.1: 15 rows split 8 + 7; Sec. 4.4: extending a span
from 10 to 20 layers at P = 2 needs no extra device). Beyond those, the two
forms of the model are checked against each other and against the classical
Amdahl formula they extend, and the cost formulas against explicit counts.
Planted mistakes show the pins catch plausible slips.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import scaling as OS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "split_examples.json")


def test_n20_p2_on_60_layers_approaches_1_2():
    # Sec. 4.1: "N = 20 and P = 2 ... a speedup approaching 120%" (no comm).
    assert math.isclose(OS.speedup(60, 20, 2, 1.0, 0.0), 1.2, rel_tol=0, abs_tol=1e-15)
    # and with a small boundary cost it stays below
    assert OS.speedup(60, 20, 2, 1.0, 0.05) < 1.2


def test_speedup_reduces_to_amdahl_without_communication():
    # Sec. 4.2 builds S(N, P) on S(a, p) = 1 / ((1 - a) + a/p).
    rng = np.random.default_rng(0)
    for _ in range(200):
        L = int(rng.integers(1, 129))
        N = int(rng.integers(0, L + 1))
        P = int(rng.integers(1, 9))
        t = float(rng.uniform(1e-4, 1.0))
        a = N / L
        amdahl = 1.0 / ((1.0 - a) + a / P)
        assert math.isclose(OS.speedup(L, N, P, t, 0.0), amdahl, rel_tol=1e-13)


def test_simple_and_alpha_beta_forms_agree():
    rng = np.random.default_rng(1)
    for _ in range(200):
        L = int(rng.integers(1, 129))
        N = int(rng.integers(0, L + 1))
        P = int(rng.integers(1, 9))
        t = float(rng.uniform(1e-4, 1.0))
        T = float(rng.uniform(0.0, 3.0)) * t
        s1 = OS.speedup(L, N, P, t, T)
        s2 = OS.speedup_ab(N / L, T / (L * t), P)
        assert math.isclose(s1, s2, rel_tol=1e-12)


def test_split_sizes_match_the_papers_examples():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        assert OS.split_sizes(c["bs"], c["v"]) == c["sizes"], c
    # Heaviest gets ceil, the sum is kept, sizes differ by at most one.
    for bs in range(0, 70):
        for v in range(1, 9):
            s = OS.split_sizes(bs, v)
            assert sum(s) == bs and max(s) == -(-bs // v) and max(s) - min(s) <= 1


def test_batch_of_one_cannot_be_sped_up():
    # Sec. 4.2: with bs = 1 and v > 1, ceil(1/P) = 1, so no vector helps.
    rng = np.random.default_rng(2)
    for _ in range(100):
        L = int(rng.integers(1, 40))
        v = [int(x) for x in rng.integers(1, 5, L)]
        s = OS.speedup_vec(v, 1, 1.0, 4096, [1e-3] * 4, [1.5e11] * 4)
        assert s <= 1.0 + 1e-15


def test_vector_form_reduces_to_the_span_form():
    # One replicated span on a homogeneous cluster with bs a multiple of P:
    # W(v) = W(N, P) and T(v) = T(P).
    rng = np.random.default_rng(3)
    for _ in range(200):
        L = int(rng.integers(1, 80))
        N = int(rng.integers(1, L + 1))
        first = int(rng.integers(0, L - N + 1))
        P = int(rng.integers(2, 9))
        bs = P * int(rng.integers(1, 40))
        t = float(rng.uniform(1e-4, 1e-2))
        d, l, B = 4096, 1, 1.53e11
        v = OS.span_vector(L, first, N, P)
        assert math.isclose(OS.work_vec(v, bs, [t] * P), OS.work(L, N, P, t), rel_tol=1e-12)
        assert math.isclose(OS.comm_vec(v, bs, l, d, B), OS.comm_time(bs, P, l, d, B),
                            rel_tol=1e-12)
        T = OS.comm_time(bs, P, l, d, B)
        assert math.isclose(OS.speedup_vec(v, bs, l, d, [t] * P, [B] * P),
                            OS.speedup(L, N, P, t, T), rel_tol=1e-12)


def test_comm_time_counts_the_offloaded_rows_both_ways():
    # One row of d bf16 elements out and back: 2 * d * 2 bytes at B.
    assert OS.comm_time(2, 2, 1, 4096, 1.0) == 2 * 4096 * 2
    assert OS.comm_time(64, 1, 1, 4096, 1.5e11) == 0.0
    assert OS.comm_time(96, 4, 1, 8192, 1.0) == 2 * 72 * 8192 * 2


def test_costs_match_explicit_counts():
    # A SwiGLU-free 12 d^2 block (the model's count): 4 d^2 attention + 8 d^2
    # MLP weights; 2 flops per weight per token.
    d, bs, l, N, P = 256, 12, 3, 5, 4
    weights = 4 * d * d + 8 * d * d
    assert OS.cost_comp(N, P, bs, l, d) == N / P * 2 * weights * bs * l
    assert OS.cost_mem(N, P, bs, l, d, 2.0) == N * (2 * weights + 2 * (bs / P) * l * d)


def test_extending_the_span_is_a_cheap_transition():
    # Sec. 4.4: N = 10 -> 20 at P = 2 copies 10 adjacent layers and needs no
    # extra device.
    L = 60
    a, b = OS.span_vector(L, 0, 10, 2), OS.span_vector(L, 0, 20, 2)
    assert OS.distance(a, b) == 10
    # a different P over the same span moves every layer
    assert OS.distance(a, OS.span_vector(L, 0, 10, 3)) == 10
    assert OS.distance(a, OS.span_vector(L, 0, 20, 4)) == 10 * 2 + 10 * 3


def test_scaling_example_as_the_model_gives_it():
    """Sec. 4.4's example (N=10, P=2 at 1.3x the SLO) names N=20, P=2, but
    the model as printed gives S(20, 2) = 1.2 < S(10, 2) * 1.3 = 1.418 at
    L = 60; the nearest spans that reach 1.418 are N = 36 at P = 2. The
    oracle follows the equations; the discrepancy is recorded as a reading."""
    L = 60
    alpha, ranked, chosen = OS.scale_candidates(L, 0, 4, 10, 2, 1.3, t_comp=1.0, bs=64, l=1,
                                                d_hidden=5120, bandwidth=1e30, cold_devices=0)
    assert math.isclose(alpha, 1.3 / (1 - 10 / 60 + 10 / 120), rel_tol=1e-12)
    assert OS.speedup(L, 20, 2, 1.0, 0.0) < alpha
    assert chosen == (36, 2) and ranked[0][:2] == (36, 2) and ranked[0][3] == 26
    # P = 3 and 4 reach it with fewer layers but a larger distance.
    first_p3 = next(c for c in ranked if c[1] == 3)
    assert first_p3[:2] == (27, 3) and first_p3[3] == 10 * 1 + 17 * 2


def test_scale_down_and_device_limits():
    L = 64
    # Latency well under the SLO: the nearest span meeting the lower target.
    alpha, ranked, chosen = OS.scale_candidates(L, 0, 4, 32, 4, 0.7, t_comp=1.0, bs=64, l=1,
                                                d_hidden=5120, bandwidth=1e30, cold_devices=0)
    assert all(c[2] >= alpha for c in ranked)
    assert chosen is not None and chosen[1] <= 4
    # No cold device: a candidate needing more devices than now is skipped.
    alpha, ranked, chosen = OS.scale_candidates(L, 0, 4, 16, 2, 2.0, t_comp=1.0, bs=64, l=1,
                                                d_hidden=5120, bandwidth=1e30, cold_devices=0)
    assert chosen is None or chosen[1] <= 2


def test_search_space_size():
    # Sec. 4.3/4.4 quote L x P_max = 256 entries for L = 64, P_max = 4; the
    # enumerated (N, P) pairs with 2 <= P <= P_max number L x (P_max - 1).
    L, P_max = 64, 4
    pairs = [(N, P) for P in range(2, P_max + 1) for N in range(1, L + 1)]
    assert len(pairs) == 192


# ---------------------------------------------------------------- planted mistakes

def _pins_pass() -> bool:
    try:
        for f in (test_n20_p2_on_60_layers_approaches_1_2,
                  test_speedup_reduces_to_amdahl_without_communication,
                  test_split_sizes_match_the_papers_examples,
                  test_batch_of_one_cannot_be_sped_up,
                  test_vector_form_reduces_to_the_span_form,
                  test_comm_time_counts_the_offloaded_rows_both_ways,
                  test_costs_match_explicit_counts,
                  test_extending_the_span_is_a_cheap_transition):
            f()
    except AssertionError:
        return False
    return True


PLANTED = {
    "replicated layers multiplied by P": ("work", lambda L, N, P, t: (L - N) * t + N * t * P),
    "replicated layers not removed from the host": ("work", lambda L, N, P, t: L * t + N * t / P),
    "floor for every device": ("split_sizes", lambda bs, v: [bs // v] * v),
    "one-way transfer": ("comm_time",
                         lambda bs, P, l, d, B, e=2.0: (bs / P * (P - 1) * l * d * e) / B),
    "ceil dropped in W(v)": ("work_vec",
                             lambda v, bs, t: sum(max(t[k] for k in range(x)) / x for x in v)),
    "distance counts changed layers only": ("distance",
                                            lambda a, b: sum(1 for x, y in zip(a, b) if x != y)),
}


@pytest.mark.parametrize("name", sorted(PLANTED))
def test_planted_scaling_mistakes_are_caught(name, monkeypatch):
    attr, bad = PLANTED[name]
    assert _pins_pass()
    monkeypatch.setattr(OS, attr, bad)
    assert not _pins_pass(), f"planted mistake '{name}' went unnoticed"
