"""MetaKV's configuration choice (Section 2.3): the library's selector against the oracle's on
random candidate sets with many ties, and hand-made cases that follow the text step by step
(budget filter, FP16 first, least compressed setting per method, accuracy among the rest,
violation score when nothing fits); the constrained success rate (Section 3.1) on a worked
example."""
import os

import numpy as np
import pytest

from oracle.selector import constrained_success_rate, select


@pytest.fixture(scope="module")
def L():
    from paper_2609_07966_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_07966_amd import build
        build.build()
    _lib.lib()
    return _lib


def _c(method, level, lat, mem, p):
    return {"method": method, "level": level, "latency": lat, "memory": mem, "p_correct": p}


def _lib_select(L, cands, l_max, m_max):
    return L.mkv_select_config([(c["method"], c["level"], c["latency"], c["memory"], c["p_correct"])
                                for c in cands], l_max, m_max)


# the paper's ten configurations: (method, level within the method)
GRID = [("fp16", 0), ("kvq", 0), ("kvq", 1), ("kvq", 2), ("h2o", 0), ("h2o", 1), ("h2o", 2),
        ("rocket", 0), ("rocket", 1), ("rocket", 2)]


def test_library_selector_equals_oracle(L):
    r = np.random.default_rng(5)
    for trial in range(3000):
        n = int(r.integers(1, 11))
        rows = [GRID[int(i)] for i in r.integers(0, len(GRID), n)]
        # coarse values so that equal latencies, memories, accuracies and violations occur often
        cands = [_c(m, lv, float(r.integers(1, 6)), float(r.integers(1, 6)), float(r.integers(0, 4)) / 4)
                 for m, lv in rows]
        l_max, m_max = float(r.integers(1, 6)), float(r.integers(1, 6))
        assert _lib_select(L, cands, l_max, m_max) == select(cands, l_max, m_max), (cands, l_max, m_max)


def test_steps_of_the_choice(L):
    fp16 = _c("fp16", 0, 2.0, 34.0, 0.60)
    kvq4, kvq2 = _c("kvq", 0, 20.0, 12.0, 0.63), _c("kvq", 2, 19.0, 6.0, 0.54)
    h60, h20 = _c("h2o", 0, 2.5, 19.0, 0.63), _c("h2o", 2, 2.7, 6.0, 0.51)
    rk8 = _c("rocket", 0, 3.6, 31.0, 0.46)
    cands = [kvq4, kvq2, h60, h20, rk8, fp16]
    for sel in (select, lambda c, a, b: _lib_select(L, c, a, b)):
        # FP16 fits: taken although other candidates are rated more accurate
        assert sel(cands, 50.0, 80.0) == (5, False)
        # FP16 over the memory budget: least compressed passing setting per method (KVQ4, H2O-60,
        # RocketKV-8x), then the highest predicted accuracy (KVQ4 0.63 = H2O-60 0.63: the first)
        assert sel(cands, 50.0, 33.0) == (0, False)
        # a latency budget that only H2O and RocketKV meet: H2O-60 over RocketKV-8x
        assert sel(cands, 5.0, 33.0) == (2, False)
        # memory budget of 10: KVQ2 and H2O-20 pass; one per method, the more accurate KVQ2
        assert sel(cands, 50.0, 10.0) == (1, False)
        # and with the latency budget too only H2O-20 is left
        assert sel(cands, 5.0, 10.0) == (3, False)
        # nothing fits: smallest L/Lmax + M/Mmax (H2O-20: 2.7/1 + 6/1)
        assert sel(cands, 1.0, 1.0) == (3, True)
    # equal violations: the higher predicted accuracy
    tie = [_c("kvq", 2, 2.0, 4.0, 0.5), _c("h2o", 2, 4.0, 2.0, 0.7)]
    assert select(tie, 1.0, 1.0) == (1, True) and _lib_select(L, tie, 1.0, 1.0) == (1, True)


def test_constrained_success_rate_worked_example():
    correct = [True, True, False, True, True]
    lat = [1.0, 3.0, 1.0, 2.0, 2.0]
    mem = [5.0, 5.0, 5.0, 9.0, 6.0]
    # prompt 0 and 4 succeed within (2, 8); 1 is too slow, 2 wrong, 3 over the memory budget
    assert constrained_success_rate(correct, lat, mem, 2.0, 8.0) == 2 / 5
    assert constrained_success_rate(correct, lat, mem, 10.0, 10.0) == 4 / 5


def test_rejects_bad_arguments(L):
    with pytest.raises(L.MkvError):
        L.mkv_select_config([], 1.0, 1.0)
    with pytest.raises(L.MkvError):
        L.mkv_select_config([("fp16", 0, 1.0, 1.0, 0.5)], 0.0, 1.0)
