"""The library's speedup/cost model (include/coco_scaling.h, host code in
libcoco.so) against the oracle (oracle/scaling.py). CPU only: these entry
points are plain arithmetic and need no GPU.

Both sides evaluate the same formulas in the same operation order in double
precision, so results must agree to the last bit; the candidate rankings and
choices must be identical.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import scaling as OS

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2607_04181_amd", "libcoco.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libcoco.so not built")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "split_examples.json")


@pytest.fixture(scope="module")
def coco():
    import paper_2607_04181_amd as c
    return c


def _models(seed, n):
    rng = np.random.default_rng(seed)
    for _ in range(n):
        yield dict(L=int(rng.integers(1, 129)), bs=int(rng.integers(1, 513)),
                   l=int(rng.choice([1, 1, 7, 512, 2048])),
                   d=int(rng.choice([256, 4096, 5120, 8192])),
                   e=float(rng.choice([2.0, 4.0])), t=float(rng.uniform(1e-5, 5e-3)),
                   B=float(rng.uniform(1e10, 9e11)))


def _lib_model(coco, p):
    return coco.make_scale_model(p["L"], p["bs"], p["l"], p["d"], p["e"], p["t"], p["B"])


def test_split_batch_matches_golden_and_oracle(coco):
    for c in json.load(open(GOLDEN))["cases"]:
        assert coco.coco_split_batch(c["bs"], c["v"]) == c["sizes"]
    for bs in range(0, 300, 7):
        for v in range(1, 12):
            assert coco.coco_split_batch(bs, v) == OS.split_sizes(bs, v)


def test_span_model_bit_identical(coco):
    rng = np.random.default_rng(5)
    for p in _models(1, 300):
        m = _lib_model(coco, p)
        for _ in range(4):
            N = int(rng.integers(0, p["L"] + 1))
            P = int(rng.integers(1, 9))
            T = OS.comm_time(p["bs"], P, p["l"], p["d"], p["B"], p["e"])
            assert coco.coco_comm_time(m, P) == T
            ref = OS.speedup(p["L"], N, P, p["t"], T if N > 0 else 0.0)
            assert coco.coco_speedup(m, N, P) == ref
            assert coco.coco_cost_mem(m, N, P) == OS.cost_mem(N, P, p["bs"], p["l"], p["d"], p["e"])
            assert coco.coco_cost_comp(m, N, P) == OS.cost_comp(N, P, p["bs"], p["l"], p["d"])


def test_vector_model_matches_oracle(coco):
    rng = np.random.default_rng(6)
    for p in _models(2, 200):
        n_dev = int(rng.integers(1, 9))
        v = [int(x) for x in rng.integers(1, n_dev + 1, p["L"])]
        t_dev = [float(x) for x in rng.uniform(0.5, 2.0, n_dev) * p["t"]]
        bw = [float(x) for x in rng.uniform(0.5, 1.5, n_dev) * p["B"]]
        got = coco.coco_speedup_vec(_lib_model(coco, p), v, t_dev, bw)
        ref = OS.speedup_vec(v, p["bs"], p["l"], p["d"], t_dev, bw, p["e"])
        # Same terms in the same order; ceil of an exact integer ratio on both.
        assert math.isclose(got, ref, rel_tol=1e-14), (got, ref)


def test_scale_candidates_identical(coco):
    rng = np.random.default_rng(7)
    for p in _models(3, 60):
        L = p["L"]
        first = int(rng.integers(0, L))
        p_max = int(rng.integers(1, 6))
        p_cur = int(rng.integers(1, p_max + 1))
        n_cur = int(rng.integers(0, L - first + 1))
        ratio = float(rng.uniform(0.5, 2.0))
        cold = int(rng.integers(0, 4))
        m = _lib_model(coco, p)
        a1, r1, c1 = coco.coco_scale_candidates(m, first, p_max, n_cur, p_cur, ratio, cold)
        a2, r2, c2 = OS.scale_candidates(L, first, p_max, n_cur, p_cur, ratio, p["t"], p["bs"],
                                         p["l"], p["d"], p["B"], cold, p["e"])
        assert a1 == a2
        assert [c[:2] + (c[3],) for c in r1] == [c[:2] + (c[3],) for c in r2]
        assert [c[2] for c in r1] == [c[2] for c in r2]
        assert c1 == c2


def test_invalid_arguments(coco):
    m = coco.make_scale_model(60, 64, 1, 5120, 2.0, 1e-3, 1.5e11)
    assert math.isnan(coco.coco_speedup(m, 61, 2)) and math.isnan(coco.coco_speedup(m, 5, 0))
    with pytest.raises(coco.CocoError):
        coco.coco_split_batch(-1, 2)
    with pytest.raises(coco.CocoError):
        coco.coco_scale_candidates(m, 60, 4, 0, 1, 1.2, 0)  # first past the last layer
