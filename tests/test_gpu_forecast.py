"""GPU parity of the speedup-bin forecast head and of top-score selection (C ABI against
the float64 oracle).

Bound for S_hat and Pr[g >= x]: the kernel rounds each per-bin weight to float32 once and
accumulates n_bins fused multiply-adds in float32, so against the float64 value of the same
sum over the same float32 forecasts its error is at most (n_bins + 2) 2^-24 sum_b |p_b w_b|.
Top-score selection is bit-exact on a given score vector.
"""
import numpy as np
import pytest
import torch

from oracle import forecast as of
from oracle import transformer as ot
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

from conftest import arch_of

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
E8 = of.HALF_OCTAVE_EDGES
CUTOFFS = (1.25, 1.5, 2.0, 0.25, 4.0, 0.6, 1.0)


def bound(p, w):
    p = np.asarray(p, np.float64)
    return (p.shape[1] + 2) * 2.0 ** -24 * (np.abs(p) @ np.abs(np.asarray(w, np.float64))) + 1e-30


def check_head(p32, m, edges, cutoffs):
    dp = torch.from_numpy(p32).to(DEV)
    s, disc = B.surrogate_forecast_head(dp, m, edges, cutoffs)
    p = p32.astype(np.float64)
    want = of.expected_speedup(p, m)
    got = s.cpu().numpy().astype(np.float64)
    err = np.abs(got - want)
    print(f"n={len(p)} bins={p.shape[1]}: max |S_hat - oracle| = {err.max():.2e}", flush=True)
    assert np.all(err <= bound(p, m))
    for c, x in enumerate(cutoffs):
        frac = of.fraction_at_or_above(edges, x)
        want = of.discovery_score(p, edges, x)
        got = disc.cpu().numpy()[:, c].astype(np.float64)
        assert np.all(np.abs(got - want) <= bound(p, frac)), x


@pytest.mark.parametrize("n", [1, 63, 256, 1237, 70001])
def test_eight_bin_head_matches_oracle(n):
    p = synth.bin_forecasts(n, 8, seed=n)
    check_head(p, of.table3_bin_values(0.17, 5.6), E8, CUTOFFS)


@pytest.mark.parametrize("nb", [2, 3, 5, 16])
def test_generic_bins_match_oracle(nb):
    rng = np.random.default_rng(nb)
    edges = np.sort(rng.uniform(0.1, 10.0, nb - 1))
    m = np.sort(rng.uniform(0.05, 12.0, nb))
    cut = tuple(rng.uniform(edges[0], edges[-1], 3)) + (float(edges[0]), float(edges[-1]))
    check_head(synth.bin_forecasts(777, nb, seed=3 * nb), m, edges, cut)


def test_single_bin_and_optional_outputs():
    p = synth.bin_forecasts(100, 1, seed=4)
    s, disc = B.surrogate_forecast_head(torch.from_numpy(p).to(DEV), [2.5])
    assert disc is None
    # one float32 product: |error| <= 2.5 * 2^-24 * p < 1.5e-7
    assert np.allclose(s.cpu().numpy(), 2.5 * p[:, 0], rtol=0, atol=1e-6)
    p8 = synth.bin_forecasts(50, 8, seed=5)
    s, disc = B.surrogate_forecast_head(torch.from_numpy(p8).to(DEV), of.table3_bin_values(0.2, 5.0),
                                        E8, (2.0,), want_speedup=False)
    assert s is None and disc.shape == (50, 1)
    want = of.discovery_score(p8.astype(np.float64), E8, 2.0)
    # a float32 sum of at most 8 weighted probabilities, each <= 1: |error| <= 8 * 2^-23 < 1e-6
    assert np.abs(disc.cpu().numpy()[:, 0] - want).max() <= 1e-6
    empty = torch.empty(0, 8, dtype=torch.float32, device=DEV)
    s, disc = B.surrogate_forecast_head(empty, of.table3_bin_values(0.2, 5.0), E8, (2.0,))
    assert s.numel() == 0 and disc.numel() == 0


# ---------------------------------------------------------------- top-k by score
def score_cases():
    rng = np.random.default_rng(9)
    for n in (1, 2, 7, 256, 257, 5000, 65536):
        s = (rng.gamma(2.0, 0.7, n)).astype(np.float32)
        if n > 2:
            s[rng.integers(0, n, max(1, n // 10))] = np.nan
            s[rng.integers(0, n, max(1, n // 5))] = np.float32(1.19)
            s[rng.integers(0, n, max(1, n // 20))] = -0.0
            s[rng.integers(0, n, max(1, n // 20))] = 0.0
        yield n, s
    for n in (1024, 1025, 65535):
        yield n, rng.gamma(2.0, 0.7, n).astype(np.float32)
    yield 3000, np.full(3000, 1.19, np.float32)
    yield 100, np.full(100, np.nan, np.float32)
    yield 20000, (rng.integers(-3, 9, 20000) / 4).astype(np.float32)


@pytest.mark.parametrize("n,s", list(score_cases()), ids=lambda x: str(x) if np.isscalar(x) else "")
def test_top_score_select_matches_oracle_bit_exact(n, s):
    ds = torch.from_numpy(s).to(DEV)
    for k in sorted({0, 1, n // 4, n - 1, n, n + 5}):
        if k < 0:
            continue
        d, a, c = B.surrogate_select(ds, B.SURR_SELECT_TOP_SCORE, budget_k=k)
        rt, rr = of.select_top_score(s, k)
        c = c.cpu().numpy()
        assert list(c) == [len(rt), len(rr)]
        assert np.array_equal(d.cpu().numpy()[: c[0]], rt)
        assert np.array_equal(a.cpu().numpy()[: c[1]], rr)


# ---------------------------------------------------------------- end to end
def test_scored_eight_bin_forecasts_rank_like_the_oracle():
    """Score prompts with one verdict token per speedup bin, then rank by S_hat and measure
    the best quarter (Section 3.5), against the oracle's forward and head."""
    w = synth.CONFIGS["tiny"]
    shape = w.shape
    W = synth.make_weights(shape, seed=0, gain_std=0.1)
    names = [t[0] for t in synth.tensor_specs(shape)]
    scorer = B.Scorer(shape, W, names, DEV)
    tok, L = synth.make_prompts(w.replace(batch=32), seed=21)
    vid = np.arange(shape.vocab - 8, shape.vocab, dtype=np.int32)
    out = scorer.score(tok, L, vid)
    ref = ot.score(arch_of(shape), W, [tok[i, : L[i]] for i in range(len(L))], vid)
    m = of.table3_bin_values(0.17, 5.6)
    s, disc = B.surrogate_forecast_head(out["p"], m, E8, (1.5, 2.0))
    s_ref = of.expected_speedup(ref["p"], m)
    # p is within 1e-4 of the oracle in every bin (float32 model bar)
    tol = 1e-4 * np.abs(m).sum() + 1e-6
    assert np.abs(s.cpu().numpy() - s_ref).max() <= tol
    for c, x in enumerate((1.5, 2.0)):
        # a sum of 8 bin probabilities, each within 1e-4 of the oracle, with weights <= 1
        assert np.abs(disc.cpu().numpy()[:, c] - of.discovery_score(ref["p"], E8, x)).max() <= 8e-4
    k = len(L) // 4
    d, a, cnt = B.surrogate_select(s, B.SURR_SELECT_TOP_SCORE, budget_k=k)
    got = set(d.cpu().numpy()[: cnt.cpu().numpy()[0]].tolist())
    order = np.argsort(-s_ref, kind="stable")
    sure_in = set(i for i in order[:k] if s_ref[i] - s_ref[order[k]] > 2 * tol)
    sure_out = set(i for i in order[k:] if s_ref[order[k - 1]] - s_ref[i] > 2 * tol)
    assert len(got) == k and sure_in <= got and not (sure_out & got)
