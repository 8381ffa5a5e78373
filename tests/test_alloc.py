"""Bit allocation (eq. mckp, Appendix "Allocators"): the oracle's walks pinned against exhaustive
search, and the library's host routine (jab_allocate) against the oracle, bit for bit; the
sensitivity table of eq. omega (jab_omega) against the oracle's, bit for bit.

Host code only: no GPU."""
import random

import numpy as np
import pytest

from oracle import allocate as al
from oracle import reference as ref
from paper_2609_34866_amd import jab

PAPER_WIDTHS = [2, 3, 4, 8, 16]                  # Method: B = {2, 3, 4, 8, 16}


def _instance(r, n, widths, equal_params=False, convex=False):
    """Omega_i(b) decreasing in b (more bits, less damage), e.g. Tr(H) ||Q_b(W) - W||^2 ~ 4^-b."""
    om = []
    for _ in range(n):
        tr = r.uniform(0.1, 10.0)
        if convex:
            om.append([tr * 4.0 ** (-w) for w in widths])
        else:
            om.append([tr * 4.0 ** (-w) * r.uniform(0.5, 2.0) for w in widths])
    params = [1.0] * n if equal_params else [r.choice([1.0, 4.0, 16.0, 58.7]) for _ in range(n)]
    return om, params


def _cost(choice, widths, params):
    return sum(params[i] * widths[j] for i, j in enumerate(choice))


@pytest.mark.parametrize("method", [al.GREEDY, al.PARETO])
def test_walks_are_feasible_and_never_beat_the_optimum(method):
    r = random.Random(7)
    checked = 0
    for _ in range(300):
        n = r.randint(1, 6)
        om, params = _instance(r, n, PAPER_WIDTHS)
        budget = r.uniform(2.2, 12.0)
        floor = r.choice([0, 3])
        try:
            opt = al.exhaustive(om, PAPER_WIDTHS, params, budget, floor)
        except ValueError:
            with pytest.raises(ValueError):
                al.allocate(om, PAPER_WIDTHS, params, budget, floor, method)
            continue
        ch, obj = al.allocate(om, PAPER_WIDTHS, params, budget, floor, method)
        assert _cost(ch, PAPER_WIDTHS, params) <= budget * sum(params) * (1 + 1e-12)
        assert all(PAPER_WIDTHS[j] >= floor for j in ch)
        assert obj >= opt[1] - 1e-15 * abs(opt[1])
        assert abs(obj - sum(om[i][j] for i, j in enumerate(ch))) <= 1e-15 * abs(obj)
        checked += 1
    assert checked > 200


def test_greedy_is_optimal_with_equal_step_costs_and_convex_scores():
    """Equally spaced widths and equal parameter counts make every downgrade cost the same; with
    each unit's Omega convex in b, taking the cheapest downgrade each time is optimal (exchange
    argument), so the greedy walk must reach the exhaustive optimum."""
    widths = [2, 3, 4, 5, 6]
    r = random.Random(11)
    for _ in range(200):
        n = r.randint(1, 6)
        om, params = _instance(r, n, widths, equal_params=True, convex=True)
        k = r.randint(0, n * (len(widths) - 1))      # number of one-step downgrades the budget forces
        budget = (n * widths[-1] - k) / n
        opt = al.exhaustive(om, widths, params, budget)
        ch, obj = al.allocate(om, widths, params, budget)
        assert abs(obj - opt[1]) <= 1e-12 * abs(opt[1]), (om, budget, ch, opt)


def test_pareto_drops_dominated_widths():
    """A width whose Omega is not below every lower width's can never be chosen by the Pareto walk
    (a cheaper width is at least as good); greedy may pass through it."""
    om = [[1.0, 0.5, 0.7, 0.1, 0.05]]              # b = 4 is dominated by b = 3
    for budget in (2.0, 3.0, 4.0, 6.0, 8.0, 16.0):
        ch, _ = al.allocate(om, PAPER_WIDTHS, [1.0], budget, 0, al.PARETO)
        assert PAPER_WIDTHS[ch[0]] != 4
    assert al.allocate(om, PAPER_WIDTHS, [1.0], 4.0, 0, al.PARETO)[0] == [1]
    assert al.allocate(om, PAPER_WIDTHS, [1.0], 4.0, 0, al.GREEDY)[0] == [2]


def test_floor_and_leftover_upgrades():
    # two units, budget 5.5 bits per parameter, P = (1, 3): all-16 costs 64 > 22
    om = [[8.0, 4.0, 2.0, 0.5, 0.1], [9.0, 3.0, 1.0, 0.2, 0.01]]
    ch, _ = al.allocate(om, PAPER_WIDTHS, [1.0, 3.0], 5.5, 3)
    assert all(PAPER_WIDTHS[j] >= 3 for j in ch)
    assert _cost(ch, PAPER_WIDTHS, [1.0, 3.0]) <= 22.0
    with pytest.raises(ValueError):
        al.allocate(om, PAPER_WIDTHS, [1.0, 3.0], 2.5, 3)    # 3-bit floor costs 12 > 10


# ----------------------------------------------------------------------------- library parity
@pytest.mark.parametrize("method", [jab.ALLOC_GREEDY, jab.ALLOC_PARETO])
def test_library_matches_oracle_bitwise(method):
    r = random.Random(3)
    for t in range(300):
        n = r.randint(1, 40)
        widths = PAPER_WIDTHS if t % 2 == 0 else [2, 3, 4, 5, 6, 8]
        om, params = _instance(r, n, widths)
        budget = r.uniform(2.5, 14.0)
        floor = r.choice([0, 0, 3])
        try:
            want = al.allocate(om, widths, params, budget, floor, method)
        except ValueError:
            with pytest.raises(jab.JabError):
                jab.allocate(om, widths, params, budget, floor, method)
            continue
        got = jab.allocate(om, widths, params, budget, floor, method)
        assert got[0] == want[0]
        assert got[1] == want[1]


def test_library_full_model_scale():
    """224 units (32 layers x 7 modules of Mistral-7B, parameter counts by module) at the paper's
    budgets, both walks, against the oracle."""
    sizes = [16.8, 4.2, 4.2, 16.8, 58.7, 58.7, 58.7]  # q, k, v, o, gate, up, down (millions)
    params = [sizes[m] for _ in range(32) for m in range(7)]
    r = random.Random(5)
    om = [[r.uniform(0.5, 5.0) * 4.0 ** (-w) for w in PAPER_WIDTHS] for _ in params]
    for budget in (3.0, 3.5, 4.0, 4.5, 6.0):
        for method in (jab.ALLOC_GREEDY, jab.ALLOC_PARETO):
            for floor in (0, 3):
                got = jab.allocate(om, PAPER_WIDTHS, params, budget, floor, method)
                want = al.allocate(om, PAPER_WIDTHS, params, budget, floor, method)
                assert got == (want[0], want[1])
                assert _cost(got[0], PAPER_WIDTHS, params) <= budget * sum(params) * (1 + 1e-12)


def test_library_rejects_bad_arguments():
    with pytest.raises(jab.JabError):
        jab.allocate([[1.0, 0.5]], [4, 2], [1.0], 3.0)          # widths not ascending
    with pytest.raises(jab.JabError):
        jab.allocate([[1.0, 0.5]], [2, 4], [0.0], 3.0)          # zero parameter count
    with pytest.raises(jab.JabError):
        jab.allocate([[1.0, float("nan")]], [2, 4], [1.0], 3.0)
    with pytest.raises(jab.JabError):
        jab.allocate([[1.0, 0.5]], [2, 4], [1.0], 3.0, min_bits=8)   # nothing above the floor


@pytest.mark.parametrize("trace", [jab.TRACE_BLOCK, jab.TRACE_UNIT])
@pytest.mark.parametrize("criterion", [jab.OMEGA_C1, jab.OMEGA_C2])
def test_omega_library_matches_oracle_bitwise(trace, criterion):
    """eq. omega's table from curvature terms and weight errors: the library and the oracle sum the
    probes in the same order, so the tables agree bit for bit."""
    r = np.random.default_rng(7 + 2 * trace + criterion)
    curv = r.normal(1.0, 0.5, (5, 9, 7))
    werr = np.abs(r.normal(0.0, 1.0, (5, 4, 3, 2)))
    werr[:, -1] = 0.0                                   # a width kept in float
    got = jab.omega(curv, werr, trace, criterion).numpy()
    want = ref.omega_table(curv, werr, trace, criterion)
    assert got.shape == (15, 4) and np.array_equal(got, want)
    assert np.all(got[:, -1] == 0.0)


def test_omega_rejects_bad_arguments():
    curv, werr = np.ones((2, 3, 7)), np.ones((2, 4, 3, 2))
    with pytest.raises(jab.JabError):
        jab.omega(curv, werr, trace=2)
    with pytest.raises(jab.JabError):
        jab.omega(curv, werr, criterion=5)
    with pytest.raises(jab.JabError):
        jab.omega(curv, np.ones((3, 4, 3, 2)))            # layer counts differ
    bad = curv.copy()
    bad[1, 2, 3] = np.inf
    with pytest.raises(jab.JabError):
        jab.omega(bad, werr)
    L = jab.lib()
    with pytest.raises(jab.JabError):
        jab._check(L.jab_omega(2, 3, None, 4, werr.ctypes.data, 0, 0, werr.ctypes.data))
    with pytest.raises(jab.JabError):
        jab._check(L.jab_omega(2, 0, curv.ctypes.data, 4, werr.ctypes.data, 0, 0, werr.ctypes.data))
