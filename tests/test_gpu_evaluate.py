"""GPU parity of the forecast-quality evaluator against the float64 oracle on the same
seeded forecasts and measured speedups.

Bars: measured bins bit-exact; per-candidate Brier and CRPS within (n_bins + 2) 2^-24
(float32 sums of at most n_bins terms each below 1); summary means within 1e-6 (float64
sums of those float32 terms); ECE within 1e-6; speedup recovered exact (max over the same
candidates) when no other candidate's expected speedup lies within float32 rounding of the
budget's k-th, and otherwise between the extreme resolutions of those near-ties.
"""
import numpy as np
import pytest
import torch

from oracle import evaluate as ev
from oracle import forecast as of
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
E8 = of.HALF_OCTAVE_EDGES
M8 = of.table3_bin_values(0.17, 5.6)


def speedups(n, seed, edges):
    rng = np.random.default_rng(seed)
    S = np.exp(rng.normal(0.0, 1.0, n)).astype(np.float32)
    if n >= 16:  # some exactly on the edges (as float32)
        S[rng.integers(0, n, len(edges))] = np.asarray(edges, np.float32)
    return S


def check(p, S, m, edges, budgets=ev.PAPER_BUDGETS):
    n, nb = p.shape
    summ, bins, br, cr = B.surrogate_evaluate(torch.from_numpy(p).to(DEV), torch.from_numpy(S).to(DEV),
                                              m, edges, budgets)
    ref = ev.evaluate(p.astype(np.float64), S.astype(np.float64), m, edges, budgets)
    summ = summ.cpu().numpy()
    assert np.array_equal(bins.cpu().numpy(), ref["bin"])
    tol_c = (nb + 2) * 2.0 ** -24
    assert np.abs(br.cpu().numpy() - ref["brier"]).max() <= tol_c
    assert np.abs(cr.cpu().numpy() - ref["crps"]).max() <= tol_c
    names = ["accuracy", "brier_mean", "crps_mean", "reward_brier", "reward_crps", "ece",
             "forecast_error"]
    for j, k in enumerate(names):
        tol = 1e-6 * (1 + abs(ref[k]))
        assert abs(summ[j] - ref[k]) <= tol, (k, summ[j], ref[k])
    # speedup recovered: the kernel ranks its own float32 expected speedups, within
    # (n_bins + 2) 2^-24 relative of the exact ones.  Candidates that close to the budget's
    # k-th score may fall on either side; the rest are decided.  With no such candidate the
    # result is exact; otherwise it lies between the two extreme resolutions.
    shat = of.expected_speedup(p.astype(np.float64), m)
    order = np.argsort(-shat, kind="stable")
    best = float(S.max())
    band = 2 * (nb + 2) * 2.0 ** -24 * np.abs(shat).max()
    exact = []
    for c, got, want in zip(budgets, summ[8:], ref["recovered_at"]):
        k = ev.budget_count(c, n)
        kth = shat[order[k - 1]]
        sure_in = shat > kth + band
        tied = np.abs(shat - kth) <= band
        if tied.sum() == 1 or k >= n:
            assert got == pytest.approx(want, abs=1e-9), (c, got, want)
            exact.append(c)
        else:
            # the summary is float64 on both sides: 1e-9 only absorbs its last-place rounding
            lo = 100 * float(S[sure_in].max()) / best if sure_in.any() else 0.0
            hi = 100 * float(S[sure_in | tied].max()) / best
            assert lo - 1e-9 <= got <= hi + 1e-9, (c, got, lo, hi)
    if len(exact) == len(budgets):
        assert summ[7] == pytest.approx(ref["recovered"], abs=1e-9)
    print(f"n={n} bins={nb}: accuracy {summ[0]:.4f} ECE {summ[5]:.4f} recovered {summ[7]:.2f} "
          f"(exact at {len(exact)}/{len(budgets)} budgets)", flush=True)


@pytest.mark.parametrize("n", [1, 7, 256, 1000, 65536])
def test_eight_bins_match_oracle(n):
    check(synth.bin_forecasts(n, 8, seed=n + 1), speedups(n, n + 2, E8), M8, E8)


@pytest.mark.parametrize("nb", [2, 5, 16])
def test_generic_bins_match_oracle(nb):
    rng = np.random.default_rng(nb)
    edges = np.sort(rng.uniform(0.2, 5.0, nb - 1))
    m = np.sort(rng.uniform(0.1, 6.0, nb))
    check(synth.bin_forecasts(3000, nb, seed=7 * nb), speedups(3000, nb, edges), m, edges,
          budgets=(0.02, 0.3, 1.0))


def test_perfect_forecasts():
    # one-hot on the measured bin with representatives equal to the speedups: accuracy 1,
    # Brier and CRPS 0, rewards 2, forecast error 0, ranking perfect (recovered 100%)
    n = 64
    S = np.array([M8[b % 8] for b in range(n)], np.float32)
    bins = ev.measured_bin(S.astype(np.float64), E8)
    p = np.zeros((n, 8), np.float32)
    p[np.arange(n), bins] = 1.0
    summ, _, _, _ = B.surrogate_evaluate(torch.from_numpy(p).to(DEV), torch.from_numpy(S).to(DEV),
                                         M8, E8)
    summ = summ.cpu().numpy()
    assert summ[0] == 1.0 and summ[1] == 0.0 and summ[2] == 0.0
    assert summ[3] == 2.0 and summ[4] == 2.0
    assert summ[6] == pytest.approx(0.0, abs=1e-6)
    assert summ[7] == 100.0
