"""Pins of the adaptive-frequency oracle (paper Sec. 4.5, Algorithm 1):
closed forms of the Poisson terms, exact identities of the coverage model,
and the optimiser against a linear-programming solver and a brute-force
grid search on the exact (non-linearised) failure probability."""
import itertools
import math

import numpy as np
import pytest
from scipy.optimize import linprog

from oracle import freq as F

LAM_PAPER = 15e-25      # errors per flop per type (13..20 per 1e25 flops, Sec. 5)


def lam(x):
    return {e: x for e in F.TYPES}


def sections(costs=(100.0, 60.0, 25.0), model="GPT-2"):
    return F.layer_sections(8, 1024, 768, 12, True, model,
                            {"AS": costs[0], "CL": costs[1], "O": costs[2]})


@pytest.mark.parametrize("mu", [1e-9, 1e-3, 0.7, 5.0, 20.0])
def test_poisson_terms_are_a_distribution(mu):
    ks = range(0, 120)
    p = [F.poisson(k, mu) for k in ks]
    assert math.isclose(sum(p), 1.0, rel_tol=1e-12)
    assert math.isclose(sum(k * q for k, q in zip(ks, p)), mu, rel_tol=1e-10)
    assert math.isclose(sum((k - mu) ** 2 * q for k, q in zip(ks, p)), mu, rel_tol=1e-9)


@pytest.mark.parametrize("mu", [1e-14, 1e-9, 1e-4, 0.3, 0.6, 4.0])
def test_two_or_more_errors_matches_the_positive_series(mu):
    direct = sum(F.poisson(k, mu) for k in range(2, 80))  # positive terms only
    assert math.isclose(F.p_two_or_more(mu), direct, rel_tol=1e-12)


def test_r_free_and_r_single_closed_forms():
    secs = sections()
    for x in (LAM_PAPER, 1e-12):
        L = lam(x)
        for s in secs:
            mu = sum(L[e] * op.flops for op in s.ops for e in F.TYPES)
            assert math.isclose(F.r_free(s, L), math.exp(-mu), rel_tol=1e-14)
            for j, op in enumerate(s.ops):
                for e in F.TYPES:
                    assert math.isclose(F.r_single(s, L, j, e), L[e] * op.flops * math.exp(-mu),
                                        rel_tol=1e-13)


def test_coverage_identities():
    """U = 1 - FC; U is linear in f; with ABFT always on only >= 2 errors
    fail; the drop from off to on is the harmful-single mass."""
    L = lam(2e-12)  # moderate means, where FC is not within rounding of 1
    for s in sections():
        for f in (0.0, 0.3, 1.0):
            assert math.isclose(F.unsafe_section(s, L, f) + F.fc_section(s, L, f), 1.0,
                                rel_tol=1e-14)
        u0, u1, uh = (F.unsafe_section(s, L, f) for f in (0.0, 1.0, 0.5))
        assert math.isclose(uh, 0.5 * (u0 + u1), rel_tol=1e-13)
        mu = F.mean_errors(s, L)
        assert math.isclose(u1, 1.0 - math.exp(-mu) * (1.0 + mu), rel_tol=1e-10)
        harm = sum(L[e] * op.flops * op.p[e] for op in s.ops for e in F.TYPES) * math.exp(-mu)
        assert math.isclose(u0 - u1, harm, rel_tol=1e-12)
        assert math.isclose(F.fce(s, L), harm / s.cost, rel_tol=1e-12)
    fr = [0.2, 0.5, 0.9]
    prod = np.prod([F.fc_section(s, L, f) for s, f in zip(sections(), fr)])
    assert math.isclose(F.unsafe_att(sections(), L, fr), 1.0 - prod, rel_tol=1e-9)


def test_at_the_paper_error_rate_no_check_is_needed():
    """13-20 errors per 1e25 flops and a target of one failure per 1e11
    executions: the unprotected layer already meets it at the GPT-2 shape,
    so every frequency is 0 (the paper's low-rate end of its sweep)."""
    secs = sections()
    for x in (13e-25, 20e-25):
        L = lam(x)
        assert F.unsafe_att(secs, L, [0, 0, 0]) < 1e-11
        assert F.optimize(secs, L, 1e-11) == [0.0, 0.0, 0.0]


def test_unreachable_target_turns_everything_on():
    secs = sections()
    L = lam(1e-12)
    floor = F.unsafe_att(secs, L, [1, 1, 1])
    assert F.optimize(secs, L, floor * 0.5) == [1.0, 1.0, 1.0]


def linear_optimum(secs, L, target):
    g = [F.harmful_single(s, L) for s in secs]
    deficit = F.unsafe_att(secs, L, [0] * len(secs)) - target
    # constraint scaled to order one (the solver's tolerances are absolute)
    res = linprog([s.cost for s in secs], A_ub=[[-x / deficit for x in g]], b_ub=[-1.0],
                  bounds=[(0, 1)] * len(secs), method="highs")
    assert res.success
    return res.fun


@pytest.mark.parametrize("x,costs", [(1e-21, (100.0, 60.0, 25.0)), (3e-21, (100.0, 60.0, 25.0)),
                                     (1e-21, (20.0, 80.0, 40.0)), (6e-21, (50.0, 50.0, 50.0))])
def test_greedy_is_the_linear_optimum_and_beats_brute_force(x, costs):
    secs = sections(costs)
    L = lam(x)
    u0, u1 = F.unsafe_att(secs, L, [0] * 3), F.unsafe_att(secs, L, [1] * 3)
    target = u1 + 0.35 * (u0 - u1)
    f = F.optimize(secs, L, target)
    cost = sum(fi * s.cost for fi, s in zip(f, secs))
    assert math.isclose(cost, linear_optimum(secs, L, target), rel_tol=1e-9)
    # at most one section is checked part of the time (fractional knapsack)
    assert sum(1 for fi in f if 0.0 < fi < 1.0) <= 1
    # the exact (product) failure probability meets the target
    assert F.unsafe_att(secs, L, f) <= target * (1 + 1e-9)
    # no grid point that meets the target is cheaper
    grid = np.linspace(0.0, 1.0, 26)
    best = math.inf
    for fs in itertools.product(grid, repeat=3):
        if F.unsafe_att(secs, L, fs) <= target:
            best = min(best, sum(a * s.cost for a, s in zip(fs, secs)))
    assert cost <= best + 1e-9


def test_greedy_takes_sections_in_efficiency_order():
    secs = sections((100.0, 60.0, 25.0))
    L = lam(1e-21)
    eff = [F.fce(s, L) for s in secs]
    order = sorted(range(3), key=lambda i: -eff[i])
    u0, u1 = F.unsafe_att(secs, L, [0] * 3), F.unsafe_att(secs, L, [1] * 3)
    for frac in (0.9, 0.6, 0.3, 0.05):
        f = F.optimize(secs, L, u1 + frac * (u0 - u1))
        ranked = [f[i] for i in order]
        assert all(a >= b for a, b in zip(ranked, ranked[1:]))


@pytest.mark.parametrize("f", [0.0, 1.0, 0.5, 0.25, 1 / 3, 0.71])
def test_schedule_realises_the_frequency(f):
    n = 600
    on = [F.schedule(f, k) for k in range(n)]
    assert sum(on) == math.floor(n * f + 1e-9)
    if f == 0.5:
        assert on[:4] == [False, True, False, True]


def test_table4_transcription_spot_values():
    """Values read off Table 4 (Sec. 3.3)."""
    assert F.table4_p("GPT-2", "AS") == {"INF": 0.569, "NaN": 0.547, "nINF": 0.005}
    assert F.table4_p("Bert", "Q")["nINF"] == 0.459
    assert F.table4_p("Neo", "K")["INF"] == 0.856
    assert F.table4_p("Roberta", "CL")["nINF"] == 0.004
    assert F.table4_p("GPT-2", "O") == {"INF": 1.0, "NaN": 1.0, "nINF": 1.0}


@pytest.mark.parametrize("free", ["AS", "CL", "O"])
def test_a_free_section_is_always_checked_and_the_target_is_met(free):
    """A section whose check costs nothing adds coverage at no cost: it is
    checked every step, and the paid sections then close what is left of
    the deficit (GPT-2-shape layer, one section made free)."""
    costs = {"AS": 100.0, "CL": 60.0, "O": 25.0}
    costs[free] = 0.0
    secs = F.layer_sections(8, 1024, 768, 12, True, "GPT-2", costs)
    L = {e: 1e-21 for e in F.TYPES}
    u0, u1 = F.unsafe_att(secs, L, [0] * 3), F.unsafe_att(secs, L, [1] * 3)
    for target in (u1 + 0.3 * (u0 - u1), u1 + 0.9 * (u0 - u1), u1 + 0.05 * (u0 - u1)):
        f = F.optimize(secs, L, target)
        assert f[[s.name for s in secs].index(free)] == 1.0
        assert F.unsafe_att(secs, L, f) <= target * (1 + 1e-9)
        # no cheaper schedule on a grid of the paid sections meets the target
        cost = sum(fi * s.cost for fi, s in zip(f, secs))
        grid = np.linspace(0.0, 1.0, 21)
        for a in grid:
            for b in grid:
                g = [1.0] * 3
                paid = [i for i, s in enumerate(secs) if s.cost > 0]
                g[paid[0]], g[paid[1]] = a, b
                if F.unsafe_att(secs, L, g) <= target:
                    assert sum(gi * s.cost for gi, s in zip(g, secs)) >= cost * (1 - 0.06)
