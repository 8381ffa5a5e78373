// alloc.cpp -- bit allocation by the multiple-choice knapsack of eq. mckp (host code).
//
// Paper: Method, eq. mckp: min sum_i Omega_i(b_i) s.t. sum_i c_i(b_i) <= budget, with the
// parameter-weighted cost c_i(b) = P_i b and budget B sum_i P_i (Section "A parameter-weighted
// budget", eq. pwbudget), an optional floor b_i >= b_min (Section "A 3-Bit Floor"), solved by
// the two heuristics of the Appendix "Allocators":
//  * greedy: every unit starts at its highest width; while the budget is exceeded, the downgrade
//    (a unit to its next lower width) with the smallest Delta Omega / Delta c; then, with the
//    budget met, upgrades (a unit to its next higher width) with the largest -Delta Omega /
//    Delta c while one fits and lowers the objective;
//  * pareto: the same walk on each unit's Pareto-efficient (cost, Omega) points (a width is kept
//    only if its Omega is strictly below that of every lower width).
// Ties go to the lowest unit index; the spent budget is the sum of the units' costs in unit
// order, recomputed after every move; the budget admits costs up to a relative 1e-12 above
// B sum_i P_i; an upgrade fits when spent + Delta c is within it.
#include <cmath>
#include <string>
#include <vector>

#include "jab.h"

namespace jab {
std::string &last_error_ref();
}

namespace {

double spent_of(const std::vector<int> &choice, const int32_t *widths, const double *params) {
    double s = 0.0;
    for (size_t i = 0; i < choice.size(); ++i) s += params[i] * widths[choice[i]];
    return s;
}

jab_status err(const char *msg) {
    jab::last_error_ref() = msg;
    return JAB_E_INVALID;
}

}  // namespace

extern "C" jab_status jab_allocate(int32_t n_units, int32_t n_widths, const int32_t *widths, const double *omega,
                                   const double *params, double budget_bits, int32_t min_bits, int32_t method,
                                   int32_t *choice_out, double *objective) {
    if (n_units < 1 || n_widths < 1 || n_widths > 64) return err("jab_allocate: need n_units >= 1 and 1..64 widths");
    if (!widths || !omega || !params || !choice_out) return err("jab_allocate: NULL argument");
    if (method != JAB_ALLOC_GREEDY && method != JAB_ALLOC_PARETO) return err("jab_allocate: unknown method");
    for (int j = 0; j < n_widths; ++j)
        if (widths[j] < 1 || (j > 0 && widths[j] <= widths[j - 1]))
            return err("jab_allocate: widths must be positive and strictly ascending");
    for (int i = 0; i < n_units; ++i) {
        if (!(params[i] > 0.0) || !std::isfinite(params[i])) return err("jab_allocate: parameter counts must be > 0");
        for (int j = 0; j < n_widths; ++j)
            if (!std::isfinite(omega[(size_t)i * n_widths + j])) return err("jab_allocate: Omega must be finite");
    }
    if (!std::isfinite(budget_bits)) return err("jab_allocate: budget must be finite");
    std::vector<int> allowed;
    for (int j = 0; j < n_widths; ++j)
        if (widths[j] >= min_bits) allowed.push_back(j);
    if (allowed.empty()) return err("jab_allocate: no candidate width at or above the floor");

    // per-unit ladders of usable widths, ascending
    std::vector<std::vector<int>> ladder(n_units);
    for (int i = 0; i < n_units; ++i) {
        const double *om = omega + (size_t)i * n_widths;
        if (method == JAB_ALLOC_GREEDY) {
            ladder[i] = allowed;
        } else {
            bool have = false;
            double best = 0.0;
            for (int j : allowed)
                if (!have || om[j] < best) {
                    ladder[i].push_back(j);
                    best = om[j];
                    have = true;
                }
        }
    }
    double total = 0.0;
    for (int i = 0; i < n_units; ++i) total += params[i];
    const double cap = budget_bits * total * (1.0 + 1e-12);   // costs equal to the budget pass despite rounding
    std::vector<int> pos(n_units), choice(n_units);
    for (int i = 0; i < n_units; ++i) {
        pos[i] = (int)ladder[i].size() - 1;
        choice[i] = ladder[i][pos[i]];
    }
    auto om = [&](int i, int j) { return omega[(size_t)i * n_widths + j]; };
    double spent = spent_of(choice, widths, params);
    while (spent > cap) {
        int best = -1;
        double best_r = 0.0;
        for (int i = 0; i < n_units; ++i) {
            if (pos[i] == 0) continue;
            const int j = choice[i], j2 = ladder[i][pos[i] - 1];
            const double r = (om(i, j2) - om(i, j)) / (params[i] * widths[j] - params[i] * widths[j2]);
            if (best < 0 || r < best_r) {
                best = i;
                best_r = r;
            }
        }
        if (best < 0) return err("jab_allocate: budget below the lowest widths");
        choice[best] = ladder[best][--pos[best]];
        spent = spent_of(choice, widths, params);
    }
    for (;;) {
        int best = -1;
        double best_r = 0.0;
        for (int i = 0; i < n_units; ++i) {
            if (pos[i] == (int)ladder[i].size() - 1) continue;
            const int j = choice[i], j2 = ladder[i][pos[i] + 1];
            const double dc = params[i] * widths[j2] - params[i] * widths[j];
            if (spent + dc > cap) continue;
            const double r = (om(i, j) - om(i, j2)) / dc;
            if (best < 0 || r > best_r) {
                best = i;
                best_r = r;
            }
        }
        if (best < 0 || !(best_r > 0.0)) break;
        choice[best] = ladder[best][++pos[best]];
        spent = spent_of(choice, widths, params);
    }
    double obj = 0.0;
    for (int i = 0; i < n_units; ++i) {
        obj += om(i, choice[i]);
        choice_out[i] = choice[i];
    }
    if (objective) *objective = obj;
    return JAB_OK;
}

// The sensitivity table of eq. omega: C1 = Tr_i ||Q_b(W_i) - W_i||^2, C2 = (L - l) C1, with the
// trace the mean of the block's pooled Hutchinson terms or of the unit's partition terms.
extern "C" jab_status jab_omega(int32_t n_layers, int32_t n_probes, const double *curv, int32_t n_widths,
                                const double *werr, int32_t trace, int32_t criterion, double *omega) {
    if (n_layers < 1 || n_probes < 1 || n_widths < 1) return err("jab_omega: need n_layers, n_probes, n_widths >= 1");
    if (!curv || !werr || !omega) return err("jab_omega: NULL argument");
    if (trace != JAB_TRACE_BLOCK && trace != JAB_TRACE_UNIT) return err("jab_omega: unknown trace");
    if (criterion != JAB_OMEGA_C1 && criterion != JAB_OMEGA_C2) return err("jab_omega: unknown criterion");
    const size_t n_curv = (size_t)n_layers * n_probes * 7, n_werr = (size_t)n_layers * n_widths * 6;
    for (size_t i = 0; i < n_curv; ++i)
        if (!std::isfinite(curv[i])) return err("jab_omega: curvature terms must be finite");
    for (size_t i = 0; i < n_werr; ++i)
        if (!std::isfinite(werr[i])) return err("jab_omega: weight errors must be finite");
    constexpr int kPooled = 3;                         // column of v^T H v in a probe's seven forms
    for (int l = 0; l < n_layers; ++l) {
        const double *cl = curv + (size_t)l * n_probes * 7;
        const double depth = criterion == JAB_OMEGA_C2 ? (double)(n_layers - l) : 1.0;
        for (int m = 0; m < 3; ++m) {
            const int col = trace == JAB_TRACE_BLOCK ? kPooled : m;
            double acc = 0.0;
            for (int p = 0; p < n_probes; ++p) acc += cl[(size_t)p * 7 + col];
            const double tr = acc / n_probes;
            for (int k = 0; k < n_widths; ++k) {
                const double e2 = werr[(((size_t)l * n_widths + k) * 3 + m) * 2];
                omega[((size_t)l * 3 + m) * n_widths + k] = depth * (tr * e2);
            }
        }
    }
    return JAB_OK;
}
