"""Bit allocation by the multiple-choice knapsack of eq. mckp, in plain Python.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Each unit i (a weight matrix) picks a width b_i from the candidate set to

    minimise  sum_i Omega_i(b_i)   subject to   sum_i c_i(b_i) <= B * sum_i P_i,

with the parameter-weighted cost c_i(b) = P_i * b and B the budget in bits per parameter
(Method, eq. mckp; Section "A parameter-weighted budget", eq. pwbudget), optionally with the
floor b_i >= b_min (Section "A 3-Bit Floor").  The two heuristics of the Appendix "Allocators":

* greedy: every unit starts at its highest width; while the budget is exceeded, apply the
  downgrade (a unit to its next lower width) with the smallest Delta Omega / Delta c; then
  spend the leftover budget on upgrades (a unit to its next higher width) with the largest
  -Delta Omega / Delta c, as long as one fits and lowers the objective;
* pareto: the same walk restricted to each unit's Pareto-efficient (cost, Omega) points, a
  width being kept only if its Omega is strictly below that of every lower width.

Readings where the paper is silent (shared with the library): ties go to the lowest unit index;
the spent budget is the sum of the units' costs in unit order, recomputed after every move; the
budget admits costs up to a relative 1e-12 above B * sum_i P_i (so a budget equal to the cost of
the floor is met despite rounding); an upgrade fits when spent + Delta c is within it; a budget
below the all-lowest assignment is an error.  ``exhaustive`` enumerates every assignment and serves the pins.
"""
from itertools import product
from typing import List, Sequence, Tuple

GREEDY, PARETO = 0, 1


def _ladders(omega, widths, min_bits, method) -> List[List[int]]:
    """Per unit, the width indices the walk may use, ascending."""
    allowed = [j for j in range(len(widths)) if widths[j] >= min_bits]
    if not allowed:
        raise ValueError("no candidate width at or above the floor")
    if method == GREEDY:
        return [list(allowed) for _ in omega]
    out = []
    for om in omega:
        keep, best = [], None
        for j in allowed:
            if best is None or om[j] < best:
                keep.append(j)
                best = om[j]
        out.append(keep)
    return out


def _spent(choice, widths, params) -> float:
    s = 0.0
    for i, j in enumerate(choice):
        s += params[i] * widths[j]
    return s


def allocate(omega: Sequence[Sequence[float]], widths: Sequence[int], params: Sequence[float], budget_bits: float,
             min_bits: int = 0, method: int = GREEDY) -> Tuple[List[int], float]:
    """-> (width index per unit, objective sum_i Omega_i(b_i) summed in unit order)."""
    n = len(omega)
    ladders = _ladders(omega, widths, min_bits, method)
    total = 0.0
    for p in params:
        total += p
    cap = budget_bits * total * (1.0 + 1e-12)
    pos = [len(l) - 1 for l in ladders]                 # position on each unit's ladder
    choice = [ladders[i][pos[i]] for i in range(n)]
    spent = _spent(choice, widths, params)
    while spent > cap:
        best, best_r = None, None
        for i in range(n):
            if pos[i] == 0:
                continue
            j, j2 = choice[i], ladders[i][pos[i] - 1]
            r = (omega[i][j2] - omega[i][j]) / (params[i] * widths[j] - params[i] * widths[j2])
            if best is None or r < best_r:
                best, best_r = i, r
        if best is None:
            raise ValueError("budget below the lowest widths")
        pos[best] -= 1
        choice[best] = ladders[best][pos[best]]
        spent = _spent(choice, widths, params)
    while True:
        best, best_r = None, None
        for i in range(n):
            if pos[i] == len(ladders[i]) - 1:
                continue
            j, j2 = choice[i], ladders[i][pos[i] + 1]
            dc = params[i] * widths[j2] - params[i] * widths[j]
            if spent + dc > cap:
                continue
            r = (omega[i][j] - omega[i][j2]) / dc
            if best is None or r > best_r:
                best, best_r = i, r
        if best is None or not best_r > 0.0:
            break
        pos[best] += 1
        choice[best] = ladders[best][pos[best]]
        spent = _spent(choice, widths, params)
    obj = 0.0
    for i, j in enumerate(choice):
        obj += omega[i][j]
    return choice, obj


def exhaustive(omega, widths, params, budget_bits, min_bits=0) -> Tuple[List[int], float]:
    """The optimum of eq. mckp by enumeration (tiny instances only)."""
    allowed = [j for j in range(len(widths)) if widths[j] >= min_bits]
    total = 0.0
    for p in params:
        total += p
    cap = budget_bits * total * (1.0 + 1e-12)
    best, best_obj = None, None
    for choice in product(allowed, repeat=len(omega)):
        if _spent(choice, widths, params) > cap:
            continue
        obj = 0.0
        for i, j in enumerate(choice):
            obj += omega[i][j]
        if best_obj is None or obj < best_obj:
            best, best_obj = list(choice), obj
    if best is None:
        raise ValueError("budget below the lowest widths")
    return best, best_obj
