"""Pins of the oracle's forecast-quality measures to closed forms and hand-computed cases
(CPU only): Table 3's bin ranges, Brier and CRPS extremes (including CRPS's distance
awareness and the 1/7 of eight bins), the rewards' ranges, hand-worked ECE buckets,
speedup recovered under perfect and reversed rankings, and the forecast error."""
import math

import numpy as np
import pytest

from oracle import evaluate as ev
from oracle import forecast as of
from paper_2605_31464_amd import synth

E = of.HALF_OCTAVE_EDGES
M = of.table3_bin_values(0.17, 5.6)


def onehot(b, nb=8):
    p = np.zeros((1, nb))
    p[0, b] = 1.0
    return p


def test_measured_bins_follow_table3_ranges():
    # (speedup, 0-based bin): bins close on the right, 2^(1/2) and 2^(-1/2) are exact edges
    cases = [(0.01, 0), (0.25, 0), (0.2500001, 1), (0.5, 1), (0.6, 2), (2 ** -0.5, 2),
             (0.71, 3), (1.0, 3), (1.0001, 4), (1.41, 4), (1.42, 5), (2.0, 5), (2.5, 6),
             (4.0, 6), (4.01, 7), (100.0, 7)]
    S = np.array([c[0] for c in cases])
    assert ev.measured_bin(S, E).tolist() == [c[1] for c in cases]


def test_predicted_bin_is_the_first_argmax():
    p = np.array([[0.1, 0.4, 0.4, 0.1], [0.25, 0.25, 0.25, 0.25], [0, 0, 0.2, 0.8]])
    assert ev.predicted_bin(p).tolist() == [1, 0, 3]


def test_brier_extremes_and_uniform():
    for nb in (2, 5, 8):
        for b in range(nb):
            assert ev.brier(onehot(b, nb), [b])[0] == 0.0
            assert ev.brier(onehot(b, nb), [(b + 1) % nb])[0] == 1.0
        u = np.full((1, nb), 1.0 / nb)
        assert ev.brier(u, [0])[0] == pytest.approx(0.5 * (1 - 1.0 / nb), abs=1e-15)


def test_crps_is_distance_aware():
    for nb in (2, 5, 8):
        for a in range(nb):
            for y in range(nb):
                assert ev.crps(onehot(a, nb), [y])[0] == pytest.approx(abs(a - y) / (nb - 1),
                                                                       abs=1e-15)
    # eight bins, one bin off: the 1/7 of Section 2.2
    assert ev.crps(onehot(3), [4])[0] == pytest.approx(1 / 7, abs=1e-15)


def test_crps_of_a_uniform_forecast():
    nb, y = 8, 3
    want = sum(((k + 1) / nb - (y <= k)) ** 2 for k in range(nb - 1)) / (nb - 1)
    assert ev.crps(np.full((1, nb), 1 / nb), [y])[0] == pytest.approx(want, abs=1e-15)


def test_reward_ranges():
    p = onehot(5)
    out = ev.evaluate(p, np.array([1.8]), M, E, budgets=(0.5,))  # 1.8 lies in bin 5 (0-based)
    assert out["bin"].tolist() == [5]
    assert out["reward_brier"] == 2.0 and out["reward_crps"] == 2.0
    far = ev.evaluate(onehot(0), np.array([10.0]), M, E, budgets=(0.5,))
    assert far["reward_crps"] == pytest.approx(0.0, abs=1e-15)  # wrong and maximally far
    assert far["reward_brier"] == 0.0


def test_ece_hand_cases():
    q = np.array([0.95, 0.95, 0.15, 0.15], np.float32)
    c = np.array([1, 0, 0, 0])
    # bucket 9: acc 0.5, conf 0.95; bucket 1: acc 0, conf 0.15; each holds half
    assert ev.ece(q, c) == pytest.approx(0.5 * 0.45 + 0.5 * 0.15, abs=1e-7)
    assert ev.ece(np.ones(7, np.float32), np.zeros(7)) == 1.0
    assert ev.ece(np.ones(7, np.float32), np.ones(7)) == 0.0
    # calibrated buckets: 10 predictions at 0.7 of which 7 correct
    assert ev.ece(np.full(10, 0.7, np.float32), np.array([1] * 7 + [0] * 3)) == \
        pytest.approx(0.0, abs=1e-7)


def test_ece_bucket_edges():
    # q = 1 joins the last bucket; 0.1 in float32 times 10 reaches bucket 1
    q = np.array([1.0, 0.1, 0.0999], np.float32)
    c = np.array([1, 1, 1])
    want = (1 / 3) * abs(1 - 1.0) + (1 / 3) * abs(1 - float(np.float32(0.1))) \
        + (1 / 3) * abs(1 - float(np.float32(0.0999)))
    assert ev.ece(q, c) == pytest.approx(want, abs=1e-7)


def test_budget_counts():
    assert ev.budget_count(0.01, 480) == 4
    assert ev.budget_count(0.25, 480) == 120
    assert ev.budget_count(0.01, 10) == 1
    assert ev.budget_count(0.5, 3) == 1


def test_speedup_recovered_perfect_and_reversed():
    n = 200
    S = np.arange(1, n + 1, dtype=np.float64)
    rec, per = ev.speedup_recovered(S.astype(np.float32), S)
    assert rec == 100.0 and per == [100.0] * 5
    rec, per = ev.speedup_recovered(-S.astype(np.float32), S)
    # the k_c worst candidates are measured: best of them is k_c
    assert per == pytest.approx([100 * ev.budget_count(c, n) / n for c in ev.PAPER_BUDGETS])
    assert rec == pytest.approx(np.mean([1, 5, 10, 25, 50]))


def test_forecast_error_closed_form():
    p = np.vstack([onehot(2), onehot(6)])
    S = np.array([M[2], M[6] + 0.5])
    out = ev.evaluate(p, S, M, E, budgets=(0.5,))
    assert out["forecast_error"] == pytest.approx(0.25, abs=1e-15)


def test_accuracy_counts_matches():
    rng = np.random.default_rng(3)
    p = synth.bin_forecasts(300, 8, seed=4).astype(np.float64)
    S = np.exp(rng.normal(0, 1, 300))
    out = ev.evaluate(p, S, M, E)
    brute = np.mean([int(np.argmax(p[i]) == sum(S[i] > e for e in E)) for i in range(300)])
    assert out["accuracy"] == brute
