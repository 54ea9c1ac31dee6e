"""Forecast quality against measured speedups (test infrastructure, see package doc).

Given forecasts p_i over speedup bins and each candidate's measured speedup S_i, this
module computes the quantities the paper trains and evaluates with:

* the measured bin y_i of S_i (Table 3: bin b covers (edge_{b-1}, edge_b]);
* the correctness reward 1[y_hat_i = y_i] (Section 2.2);
* the Brier score 1/2 sum_b (p_b - 1[b = y])^2 and the reward r_corr + 1 - Brier
  (Section 2.2);
* the CRPS 1/(B-1) sum_{k<B} (F_k - 1[y <= k])^2 over the cumulative forecast F_k and the
  reward r_corr + 1 - CRPS (Section 2.2; B = 8 gives the printed 1/7);
* the expected calibration error over ten equal-width confidence buckets (Section 3.1);
* the forecast error, the mean |m_{y_hat} - S| (Section 3.1);
* speedup recovered, the best measured speedup among the top c% by expected speedup as a
  percentage of the best overall, averaged over the budgets (Section 3.1).

Readings where the paper is silent:

* Bins of a measured speedup use the exact half-octave edges of oracle.forecast; a speedup
  on an edge belongs to the lower bin (Table 3 closes the bins on the right).
* ECE buckets: bucket m holds confidences q with floor(10 q) = m (m = 9 also takes q = 1),
  with 10 q formed in float32; empty buckets add nothing.
* Top c% for speedup recovered: k_c = max(1, floor(c N)) candidates (the budget is not
  exceeded, and at least one candidate is measured), ranked as oracle.forecast's
  select_top_score (score descending, ties by ascending index).
* The predicted bin y_hat is the first argmax of p (as for the verdict read-out).

Parity status: pinned by ``tests/test_oracle_evaluate_pins.py`` (closed forms, brute force).
"""
from __future__ import annotations

import math

import numpy as np

from . import forecast as fc

PAPER_BUDGETS = (0.01, 0.05, 0.10, 0.25, 0.50)  # Section 3.1


def measured_bin(S, edges) -> np.ndarray:
    """0-based bin index of each speedup: the number of edges strictly below it."""
    S = np.asarray(S, np.float64)
    e = np.asarray(edges, np.float64)
    out = np.zeros(S.shape, np.int64)
    for j in range(e.size):
        out += (S > e[j]).astype(np.int64)
    return out


def predicted_bin(p) -> np.ndarray:
    p = np.asarray(p, np.float64)
    out = np.zeros(p.shape[0], np.int64)
    for i in range(p.shape[0]):
        best = 0
        for b in range(1, p.shape[1]):
            if p[i, b] > p[i, best]:
                best = b
        out[i] = best
    return out


def brier(p, y) -> np.ndarray:
    p = np.asarray(p, np.float64)
    out = np.zeros(p.shape[0])
    for b in range(p.shape[1]):
        out += (p[:, b] - (np.asarray(y) == b)) ** 2
    return 0.5 * out


def crps(p, y) -> np.ndarray:
    p = np.asarray(p, np.float64)
    nb = p.shape[1]
    if nb < 2:
        return np.zeros(p.shape[0])
    y = np.asarray(y)
    out = np.zeros(p.shape[0])
    F = np.zeros(p.shape[0])
    for k in range(nb - 1):
        F = F + p[:, k]
        out += (F - (y <= k)) ** 2
    return out / (nb - 1)


def ece(confidence, correct, n_buckets: int = 10) -> float:
    q = np.asarray(confidence, np.float32)
    c = np.asarray(correct, np.float64)
    n = len(q)
    bucket = np.minimum(np.floor(q * np.float32(n_buckets)).astype(np.int64), n_buckets - 1)
    total = 0.0
    for m in range(n_buckets):
        sel = bucket == m
        if sel.any():
            total += sel.sum() / n * abs(c[sel].mean() - q[sel].astype(np.float64).mean())
    return total


def budget_count(c: float, n: int) -> int:
    return max(1, int(math.floor(c * n)))


def speedup_recovered(score, S, budgets=PAPER_BUDGETS):
    """(mean over budgets, per-budget list) in percent."""
    S = np.asarray(S, np.float64)
    best = S.max()
    per = []
    for c in budgets:
        top, _ = fc.select_top_score(np.asarray(score, np.float32), budget_count(c, len(S)))
        per.append(100.0 * S[top].max() / best)
    return float(np.mean(per)), per


def evaluate(p, S, m, edges, budgets=PAPER_BUDGETS) -> dict:
    """All of the above for one batch; the expected speedup is rounded to float32 before
    ranking, as the device computes it in float32."""
    p = np.asarray(p, np.float64)
    y = measured_bin(S, edges)
    yh = predicted_bin(p)
    corr = (yh == y).astype(np.float64)
    br, cr = brier(p, y), crps(p, y)
    q = p.max(axis=1)
    shat = fc.expected_speedup(p, m)
    rec, per = speedup_recovered(shat.astype(np.float32), S, budgets)
    return {"bin": y, "correct": corr, "brier": br, "crps": cr,
            "accuracy": corr.mean(), "brier_mean": br.mean(), "crps_mean": cr.mean(),
            "reward_brier": (corr + 1 - br).mean(), "reward_crps": (corr + 1 - cr).mean(),
            "ece": ece(q.astype(np.float32), corr),
            "forecast_error": float(np.mean(np.abs(np.asarray(m)[yh] - np.asarray(S, np.float64)))),
            "recovered": rec, "recovered_at": per}
