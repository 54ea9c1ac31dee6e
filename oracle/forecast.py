"""The paper's speedup-bin forecast head (test infrastructure, see package doc).

The forecast target is the speedup S = T_ref / T of a candidate, in eight ordinal bins
on a logarithmic scale (Section 2.1, Forecasting Relative Performance; Table 3).  From a
forecast distribution p over the bins this module computes:

* the expected-speedup score S_hat = sum_b p_b * m_b, with m_b the representative
  speedup of bin b (Section 3.1, Speedup recovered; Table 3);
* the discovery score s = Pr[g >= x] for a speedup cutoff x (Section 3.6);
* the top-k candidates by S_hat, the set a search measures on the device when it ranks
  candidates by expected speedup and measures only the best quarter (Section 3.5), or
  the top c% (Section 3.1).

Readings where the paper is silent:

* Bin edges.  Table 3 prints the edges 0.25, 0.5, 0.71, 1.0, 1.41, 2.0, 4.0 and calls the
  bins half-octave.  They are read as the exact powers 2^-2, 2^-1, 2^-1/2, 1, 2^1/2, 2, 4:
  the printed interior representatives are the geometric centres of these exact bins
  rounded to two decimals (with 0.71 as an edge the third would round to 0.60, not 0.59).
* Bin values.  Interior m_b are the printed Table 3 values; the two open bins have
  empirical means, which are parameters (m_1, m_8).
* Within-bin distribution.  Pr[g >= x] needs the mass of bin b above x when x falls
  inside the bin.  It is read as log-uniform over (lo_b, hi_b]: the fraction above x is
  (ln hi_b - ln x) / (ln hi_b - ln lo_b).  This is the reading under which the table's
  geometric centres are the bins' medians.  The open bins lie wholly on one side of any
  cutoff in [lowest edge, highest edge]; cutoffs outside that range are rejected.  At a
  cutoff equal to an edge no interpolation happens (x = 2: s = p_7 + p_8).
* Top-k order.  Score descending, a NaN score ranks as -inf, ties by ascending index;
  -0.0 equals +0.0; k is clamped to [0, N] and a negative k is an error.  Both index
  lists are returned ascending and together partition range(N).

Parity status: every function is pinned by ``tests/test_oracle_forecast_pins.py``.
"""
from __future__ import annotations

import math

import numpy as np

# Exact half-octave edges of the eight bins (Table 3), lowest first.
HALF_OCTAVE_EDGES = np.array([2.0 ** e for e in (-2.0, -1.0, -0.5, 0.0, 0.5, 1.0, 2.0)])

# Printed representatives of bins 2..7 (Table 3).
TABLE3_INTERIOR_VALUES = (0.35, 0.59, 0.84, 1.19, 1.68, 2.83)


def table3_bin_values(m_first: float, m_last: float) -> np.ndarray:
    """m_1..m_8 with the two open-bin means supplied by the caller (Table 3)."""
    return np.array([m_first, *TABLE3_INTERIOR_VALUES, m_last], dtype=np.float64)


def expected_speedup(p, m) -> np.ndarray:
    """S_hat_i = sum_b p_{i,b} m_b for every row of p (Section 3.1)."""
    p = np.asarray(p, np.float64)
    m = np.asarray(m, np.float64)
    if p.ndim != 2 or p.shape[1] != m.shape[0]:
        raise ValueError("p must be [N, n_bins] with n_bins = len(m)")
    out = np.zeros(p.shape[0])
    for b in range(m.shape[0]):
        out += p[:, b] * m[b]
    return out


def fraction_at_or_above(edges, x: float) -> np.ndarray:
    """Share of each bin's probability mass on speedups >= x, bins (-inf, e_0],
    (e_0, e_1], ..., (e_last, inf), log-uniform inside the interior bins."""
    e = np.asarray(edges, np.float64)
    if e.ndim != 1 or e.size < 1 or not np.all(e > 0) or not np.all(np.diff(e) > 0):
        raise ValueError("edges must be positive and strictly increasing")
    if not (e[0] <= x <= e[-1]):
        raise ValueError("cutoff outside [lowest edge, highest edge]")
    n_bins = e.size + 1
    frac = np.zeros(n_bins)
    frac[0] = 0.0          # (-inf, e_0]: below any cutoff >= e_0
    frac[-1] = 1.0         # (e_last, inf): above any cutoff <= e_last
    for b in range(1, n_bins - 1):
        lo, hi = e[b - 1], e[b]
        if x <= lo:
            frac[b] = 1.0
        elif x >= hi:
            frac[b] = 0.0
        else:
            frac[b] = (math.log(hi) - math.log(x)) / (math.log(hi) - math.log(lo))
    return frac


def discovery_score(p, edges, x: float) -> np.ndarray:
    """s_i = Pr[g >= x] under forecast p_i (Section 3.6)."""
    p = np.asarray(p, np.float64)
    frac = fraction_at_or_above(edges, x)
    if p.ndim != 2 or p.shape[1] != frac.size:
        raise ValueError("p must be [N, len(edges) + 1]")
    out = np.zeros(p.shape[0])
    for b in range(frac.size):
        out += p[:, b] * frac[b]
    return out


def select_top_score(score, k: int):
    """Indices of the min(k, N) highest scores (measured on the device) and the rest,
    both ascending (Sections 3.1 and 3.5)."""
    if k < 0:
        raise ValueError("k must be >= 0")
    s = np.asarray(score, np.float32)
    n = len(s)
    k = min(k, n)

    def key(i):
        v = float(s[i])
        return (-(-math.inf if math.isnan(v) else v), i)

    order = sorted(range(n), key=key)
    chosen = set(order[:k])
    top = [i for i in range(n) if i in chosen]
    rest = [i for i in range(n) if i not in chosen]
    return np.array(top, np.int32), np.array(rest, np.int32)
