"""Pins of the oracle's speedup-bin forecast head to facts other than itself (CPU only).

Table 3's printed edges and representatives, the worked forecasts of Section 3.6 and
Appendix A, closed forms of the expected speedup and of Pr[g >= x], a Monte Carlo draw
from the log-uniform within-bin reading, and brute force for the top-k selection.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import forecast as of
from oracle import select as osel
from paper_2605_31464_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
E = of.HALF_OCTAVE_EDGES


def golden():
    with open(os.path.join(GOLDEN, "speedup_bins.json")) as f:
        return json.load(f)


def rand_p(n, nb=8, seed=0):
    """Seeded forecasts renormalised in float64, so rows sum to 1 to rounding."""
    p = synth.bin_forecasts(n, nb, seed=seed).astype(np.float64)
    return p / p.sum(axis=1, keepdims=True)


# ---------------------------------------------------------------- Table 3
def test_edges_are_the_printed_edges():
    assert np.round(E, 2).tolist() == golden()["table3"]["printed_edges"]


def test_geometric_centres_are_the_printed_values():
    g = golden()["table3"]
    centres = [round(math.sqrt(E[b - 1] * E[b]), 2) for b in range(1, 7)]
    assert centres == g["printed_interior_values"]
    # The printed (rounded) edges do not reproduce them: bin 3 would centre on 0.60.
    pe = g["printed_edges"]
    assert round(math.sqrt(pe[1] * pe[2]), 2) != g["printed_interior_values"][1]


def test_bin_values_layout():
    m = of.table3_bin_values(0.1, 6.0)
    assert m.tolist() == [0.1, *golden()["table3"]["printed_interior_values"], 6.0]
    assert np.all(np.diff(m) > 0)


# ---------------------------------------------------------------- expected speedup
def test_one_hot_forecast_scores_its_bin_value():
    m = of.table3_bin_values(0.12, 7.5)
    s = of.expected_speedup(np.eye(8), m)
    assert np.array_equal(s, m)


def test_constant_bin_values_give_the_constant():
    p = rand_p(50, seed=1)
    assert np.allclose(of.expected_speedup(p, np.full(8, 1.7)), 1.7, atol=1e-15, rtol=0)


def test_uniform_forecast_scores_the_mean_value():
    m = of.table3_bin_values(0.2, 5.0)
    assert of.expected_speedup(np.full((1, 8), 1 / 8), m)[0] == pytest.approx(m.mean(), abs=1e-15)


def test_expected_speedup_is_linear_in_p():
    m = of.table3_bin_values(0.2, 5.0)
    p, q = rand_p(20, seed=2), rand_p(20, seed=3)
    a = 0.3
    lhs = of.expected_speedup(a * p + (1 - a) * q, m)
    rhs = a * of.expected_speedup(p, m) + (1 - a) * of.expected_speedup(q, m)
    assert np.allclose(lhs, rhs, atol=1e-14, rtol=0)


def test_moving_mass_to_a_faster_bin_raises_the_score():
    m = of.table3_bin_values(0.2, 5.0)
    p = rand_p(1, seed=4)
    base = of.expected_speedup(p, m)[0]
    for b in range(7):
        q = p.copy()
        d = q[0, b] / 2
        q[0, b] -= d
        q[0, b + 1] += d
        assert of.expected_speedup(q, m)[0] == pytest.approx(base + d * (m[b + 1] - m[b]),
                                                             abs=1e-14)


def test_sampled_bins_average_to_the_expected_speedup():
    rng = np.random.default_rng(5)
    m = of.table3_bin_values(0.2, 5.0)
    p = rand_p(1, seed=6)[0]
    n = 400_000
    draws = m[rng.choice(8, size=n, p=p)]
    sd = draws.std() / math.sqrt(n)
    assert abs(draws.mean() - of.expected_speedup(p[None], m)[0]) < 5 * sd


# ---------------------------------------------------------------- discovery score
def test_section_3_6_example():
    g = golden()["discovery_example"]
    p = np.zeros((1, 8))
    p[0, 6] = p[0, 7] = g["mass_at_or_above"] / 2
    p[0, :6] = (1 - g["mass_at_or_above"]) / 6
    s = of.discovery_score(p, E, g["cutoff"])
    assert s[0] == pytest.approx(g["mass_at_or_above"], abs=1e-15)
    s32 = s.astype(np.float32)
    assert osel.select_threshold(s32, g["tau_accepting"])[1].tolist() == [0]
    assert osel.select_threshold(s32, g["tau_rejecting"])[1].tolist() == []


def test_appendix_a_forecast():
    g = golden()["appendix_a_forecast"]
    rest = 1 - g["mass_bins_6_to_8"] - g["p_bin5"]
    p = np.array([[rest / 4] * 4 + [g["p_bin5"], (g["mass_bins_6_to_8"] - g["p_bin8"]) / 2,
                                    (g["mass_bins_6_to_8"] - g["p_bin8"]) / 2, g["p_bin8"]]])
    assert p.sum() == pytest.approx(1.0, abs=1e-15)
    assert int(np.argmax(p[0])) + 1 == g["predicted_bin"]
    # Speedup above 1.41 (the edge 2^(1/2)) carries exactly the stated mass.
    assert of.discovery_score(p, E, math.sqrt(2.0))[0] == pytest.approx(g["mass_bins_6_to_8"],
                                                                         abs=1e-15)


def test_cutoffs_on_edges_sum_whole_bins():
    p = rand_p(30, seed=7)
    for j, x in enumerate(E):
        # x = E[j] is the upper edge of bin j: bins j + 1 .. 7 lie wholly at or above it.
        assert np.allclose(of.discovery_score(p, E, x), p[:, j + 1:].sum(axis=1),
                           atol=1e-15, rtol=0)


def test_extreme_cutoffs():
    p = rand_p(30, seed=8)
    assert np.allclose(of.discovery_score(p, E, E[0]), 1 - p[:, 0], atol=1e-15, rtol=0)
    assert np.allclose(of.discovery_score(p, E, E[-1]), p[:, 7], atol=1e-15, rtol=0)
    for bad in (E[0] * 0.99, E[-1] * 1.01, 0.0, -1.0):
        with pytest.raises(ValueError):
            of.discovery_score(p, E, bad)


def test_geometric_centre_splits_its_bin_in_half():
    p = rand_p(10, seed=9)
    for b in range(1, 7):
        x = math.sqrt(E[b - 1] * E[b])
        want = p[:, b + 1:].sum(axis=1) + p[:, b] / 2
        assert np.allclose(of.discovery_score(p, E, x), want, atol=1e-14, rtol=0)


def test_score_falls_monotonically_and_continuously_with_the_cutoff():
    p = rand_p(5, seed=10)
    xs = np.exp(np.linspace(math.log(E[0]), math.log(E[-1]), 2001))
    s = np.stack([of.discovery_score(p, E, x) for x in xs])
    assert np.all(np.diff(s, axis=0) <= 1e-15)
    for x in E[1:-1]:
        lo = of.discovery_score(p, E, x * (1 - 1e-9))
        hi = of.discovery_score(p, E, x * (1 + 1e-9))
        assert np.allclose(lo, hi, atol=1e-8, rtol=0)


def test_log_uniform_draws_match_the_discovery_score():
    rng = np.random.default_rng(11)
    p = rand_p(1, seed=12)[0]
    n = 400_000
    b = rng.choice(8, size=n, p=p)
    g = np.empty(n)
    g[b == 0] = E[0] / 2
    g[b == 7] = E[-1] * 2
    inner = (b > 0) & (b < 7)
    lo, hi = np.log(E[b[inner] - 1]), np.log(E[b[inner]])
    g[inner] = np.exp(lo + (hi - lo) * rng.random(inner.sum()))
    for x in (0.3, 0.6, 1.25, 1.5, 2.0, 3.0):
        emp = float(np.mean(g >= x))
        want = of.discovery_score(p[None], E, x)[0]
        assert abs(emp - want) < 5 * math.sqrt(want * (1 - want) / n) + 1e-12


# ---------------------------------------------------------------- top-k by S_hat
def brute_top(score, k):
    """k rounds of picking the highest remaining score (NaN lowest, lowest index on ties)."""
    s = [(-math.inf if math.isnan(float(v)) else float(v)) for v in np.asarray(score, np.float32)]
    left, chosen = list(range(len(s))), []
    for _ in range(min(k, len(s))):
        best = left[0]
        for i in left[1:]:
            if s[i] > s[best]:
                best = i
        chosen.append(best)
        left.remove(best)
    return sorted(chosen)


def test_top_score_matches_brute_force_with_ties_and_nan():
    pool = [0.5, 0.5, 1.2, -0.0, 0.0, float("nan"), 3.0]
    for n in range(1, 7):
        for combo in itertools.permutations(pool, n):
            for k in range(0, n + 2):
                top, rest = of.select_top_score(np.array(combo, np.float32), k)
                assert top.tolist() == brute_top(combo, k)
                assert sorted(top.tolist() + rest.tolist()) == list(range(n))


def test_top_score_is_budget_select_of_the_negated_score():
    rng = np.random.default_rng(13)
    s = np.round(rng.normal(size=200), 1).astype(np.float32)  # many ties
    for k in (0, 1, 17, 50, 199, 200, 250):
        top, rest = of.select_top_score(s, k)
        d, a = osel.select_budget(-s, k)
        assert top.tolist() == d.tolist() and rest.tolist() == a.tolist()


def test_search_measures_the_best_quarter():
    # Section 3.5: four times as many candidates, the quarter ranked highest is measured.
    m = of.table3_bin_values(0.2, 5.0)
    p = rand_p(4 * 24, seed=14)
    s = of.expected_speedup(p, m).astype(np.float32)
    top, rest = of.select_top_score(s, 24)
    assert len(top) == 24 and len(rest) == 72
    assert s[top].min() >= s[rest].max()


def test_negative_k_is_an_error():
    with pytest.raises(ValueError):
        of.select_top_score(np.zeros(3, np.float32), -1)
