"""Setup-phase bookkeeping (Algorithm 1, Phases 1-3) without a GPU: S_tau aggregation
against the oracle's module average, the receiver rule, the Phase 2 check and the
Phase 3 table (the paper's default allocation, Appendix rank table)."""
import os

import numpy as np
import pytest

from oracle import moara_oracle as O
from tests.conftest import golden

M = pytest.importorskip("paper_2609_15037_amd.moara")
P = pytest.importorskip("paper_2609_15037_amd.profiling")

Q, K, V, OO, GATE, UP, DOWN = range(7)


def test_profiling_steps_are_multiples_of_the_stride_up_to_n_p():
    p = P.AlignmentProfile([Q], stride=50, n_p=200)
    assert [t for t in range(0, 400) if p.due(t)] == [50, 100, 150, 200]
    with pytest.raises(ValueError):
        P.AlignmentProfile([Q], stride=0, n_p=10)


def test_s_tau_is_the_mean_over_steps_and_instances():
    rng = np.random.default_rng(3)
    modules = [Q, K, V, OO, GATE, UP, DOWN] * 3          # three layers
    p = P.AlignmentProfile(modules, stride=10, n_p=100)
    samples = []
    for t in (10, 20, 30, 40):
        s = rng.uniform(0.3, 1.0, len(modules))
        s[rng.integers(0, len(modules))] = np.nan          # an inactive matrix this step
        p.add(s, t)
        samples += [(m, v) for m, v in zip(modules, s) if not np.isnan(v)]
    ref = O.module_alignment(samples)
    got = p.s_tau()
    assert set(got) == set(ref)
    for tau in ref:
        assert got[tau] == pytest.approx(ref[tau], rel=1e-12)
    assert p.steps == [10, 20, 30, 40]
    with pytest.raises(ValueError):
        p.add(np.zeros(3))


def _profile(scores):
    modules = list(scores)
    p = P.AlignmentProfile(modules, stride=1, n_p=1)
    p.add([scores[m] for m in modules], 1)
    return p


def test_receiver_is_the_clearly_lowest_module():
    # the ordering the paper reports: down lowest by a wide margin, k and q next
    p = _profile({Q: 0.93, K: 0.90, V: 0.98, OO: 0.98, GATE: 0.95, UP: 0.95, DOWN: 0.78})
    assert p.ranking()[0] == (DOWN, pytest.approx(0.78))
    assert p.receivers() == [DOWN]
    assert p.validate([Q, K], [DOWN]) == (True, "ok")
    ok, why = p.validate([Q, K], [K])
    assert not ok and "overlap" in why
    ok, why = p.validate([Q, V], [GATE])
    assert not ok and "lowest" in why
    # no clear receiver when the two lowest are within the margin
    assert _profile({Q: 0.90, DOWN: 0.88, V: 0.97}).receivers(margin=0.05) == []
    ok, why = _profile({Q: 0.9, DOWN: 0.8}).validate([K], [DOWN])
    assert not ok and "without alignment samples" in why


def test_allocation_is_the_papers_default_table():
    if not os.path.exists(M.LIB_PATH):
        pytest.skip("libmoara.so not built")
    gd = golden("rank_allocations.json")
    got = P.allocate(256, range(7), [Q, K], [DOWN])       # delta_r = r_base / 2
    assert got[:7] == gd["ours_r256"]
    assert sum(got[:7]) == 7 * 256
