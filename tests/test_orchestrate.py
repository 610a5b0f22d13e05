"""Host-side DSI pieces (paper_2405_14105_amd/orchestrate.py): lookahead
selection (Equation 1) and the latency simulations of non-SI, SI and DSI,
pinned by the paper's worked examples (Section 3.1 "Lookahead" and the MP
vs SP example, Section 4, Appendix F), Proposition 1 and Theorems 1-2."""
import math

import numpy as np
import pytest

from paper_2405_14105_amd.orchestrate import (Acceptance, expected, lookahead_min, offline_speedups,
                                              prop1_bound, servers_needed, simulate_dsi,
                                              simulate_nonsi, simulate_si)


class Pattern:
    """Deterministic acceptance: iteration i accepts counts[i % len] drafts."""

    def __init__(self, counts):
        self.counts, self.i = counts, 0

    def __call__(self, n):
        c = self.counts[self.i % len(self.counts)]
        self.i += 1
        return np.arange(n) < c


def test_lookahead_worked_examples():
    # a 5 % drafter with SP = 4 needs lookahead 5, and at most 1 + 4 = 5 units
    assert lookahead_min(1.0, 0.05, 4) == 5
    assert 1 + servers_needed(1.0, 0.05, 5) == 5
    # seven GPUs, MP = 2 -> SP = 3; drafter 5 % (ratio 20): lookahead 7
    assert lookahead_min(20.0, 1.0, 3) == 7
    assert lookahead_min(1.0, 0.05, 3) == 7
    # a 10 % drafter with lookahead 2 runs on 5 target GPUs + 1 drafter GPU
    assert servers_needed(1.0, 0.1, 2) == 5
    # minimality: one less violates Equation 1
    for t, d, sp in [(1.0, 0.05, 4), (20.0, 1.0, 3), (1.0, 0.14, 8), (1.0, 0.3, 2)]:
        L = lookahead_min(t, d, sp)
        assert math.ceil(t / (L * d) - 1e-12) <= sp
        assert L == 1 or math.ceil(t / ((L - 1) * d) - 1e-12) > sp


def test_mp_vs_sp_example_arithmetic():
    # acceptance 80 %, lookahead 2: a^2 of the target forwards hidden, 36 % left,
    # so model parallelism must speed the target up 1 / 0.36 = 2.78x to match
    a = 0.8
    assert math.isclose(1 - a ** 2, 0.36)
    assert round(1 / (1 - a ** 2), 2) == 2.78


def test_si_worked_example():
    # 100 tokens, 1.5 accepted drafts per iteration on average, lookahead 5,
    # drafter 6 ms, target 30 ms: 40 target and 200 drafter forwards, 2400 ms,
    # 1.25x faster than non-SI's 3000 ms
    t = simulate_si(30.0, 6.0, 5, 100, Pattern([1, 2]))
    assert t == 2400.0
    assert simulate_nonsi(30.0, 100) == 3000.0
    assert simulate_nonsi(30.0, 100) / t == 1.25


@pytest.mark.parametrize("t1,p", [(0.1, 0.8), (0.3, 0.5), (0.05, 0.95), (0.5, 0.1), (0.2, 0.0)])
def test_proposition1_bound(t1, p):
    N, runs = 120, 3000
    rng = np.random.default_rng(1)
    vals = [simulate_dsi(1.0, t1, 1, 64, N, Acceptance(p, rng)).time for _ in range(runs)]
    mean, sem = float(np.mean(vals)), float(np.std(vals) / np.sqrt(runs))
    assert mean <= prop1_bound(t1, 1.0, p, N) + 4 * sem + 1e-9


def test_dsi_extremes():
    # every draft rejected: one target forward per token (non-SI)
    tr = simulate_dsi(1.0, 0.2, 3, 8, 50, Acceptance(0.0, np.random.default_rng(0)))
    assert tr.time == 50.0 and tr.tokens == 50
    # every draft accepted, lookahead 1: all target latency hidden but one forward
    tr = simulate_dsi(1.0, 0.2, 1, 16, 50, Acceptance(1.0, np.random.default_rng(0)))
    assert math.isclose(tr.time, 49 * 0.2 + 1.0)


@pytest.mark.parametrize("f,a,L", [(0.05, 0.9, 3), (0.2, 0.6, 2), (0.5, 0.3, 1), (0.1, 0.99, 10)])
def test_theorem1_never_slower_than_nonsi(f, a, L):
    rng = np.random.default_rng(2)
    sp = servers_needed(1.0, f, L)
    for _ in range(300):
        tr = simulate_dsi(1.0, f, L, sp, 64, Acceptance(a, rng))
        assert tr.time <= simulate_nonsi(1.0, 64) + 1e-9
        assert tr.tokens == 64


@pytest.mark.parametrize("f,a,L", [(0.05, 0.9, 3), (0.2, 0.6, 2), (0.5, 0.3, 1), (0.1, 0.99, 5)])
def test_theorem2_not_slower_than_si_in_expectation(f, a, L):
    sp = servers_needed(1.0, f, L)
    si = expected(simulate_si, 2000, 3, target_latency=1.0, drafter_latency=f, lookahead=L, N=64, rate=a)
    dsi = expected(simulate_dsi, 2000, 3, target_latency=1.0, drafter_latency=f, lookahead=L, sp=sp,
                   N=64, rate=a)
    assert dsi <= si * 1.001


def test_equation1_means_no_waiting():
    rng = np.random.default_rng(4)
    for f, sp in [(0.05, 4), (0.1, 3), (0.2, 2)]:
        L = lookahead_min(1.0, f, sp)
        waits = [simulate_dsi(1.0, f, L, sp, 80, Acceptance(0.9, rng)).waited for _ in range(100)]
        assert max(waits) == 0.0
        if L > 1:   # a smaller lookahead needs more servers than SP: tasks wait
            waits = [simulate_dsi(1.0, f, L - 1, sp, 80, Acceptance(0.95, rng)).waited
                     for _ in range(100)]
            assert max(waits) > 0.0


def test_offline_speedup_grid():
    """The ablation methodology: DSI is at least as fast as SI and non-SI over
    a grid of drafter latencies and acceptance rates (Theorems 1-2)."""
    over_si, over_nonsi = offline_speedups([0.05, 0.2, 0.6], [0.0, 0.5, 0.9], N=60, runs=20)
    assert np.all(over_si >= 0.97) and np.all(over_nonsi >= 0.999)
    # acceptance 0.9 with a fast drafter: a large speedup over non-SI
    assert over_nonsi[0, 2] > 3.0
