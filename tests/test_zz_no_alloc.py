"""GPU check of surrogate_evaluate_noalloc, the evaluator on the library's fixed per-device
scratch, against surrogate_evaluate with a caller workspace: same kernels, same order of
every sum, so the outputs must agree bit for bit.  Two calls in a row, the second on a
smaller input, so the second reads scratch the first has left behind."""
import numpy as np
import pytest
import torch

from oracle import forecast as of
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def inputs(n, nb, seed):
    p = torch.from_numpy(synth.bin_forecasts(n, nb, seed=seed)).to(DEV)
    rng = np.random.default_rng(seed + 100)
    S = torch.from_numpy(np.exp(rng.normal(0.0, 1.0, n)).astype(np.float32)).to(DEV)
    return p, S


def test_evaluate_noalloc_matches_workspace_entry_point():
    m8 = of.table3_bin_values(0.17, 5.6)
    e8 = of.HALF_OCTAVE_EDGES
    cases = [(65536, 8, (0.01, 0.05, 0.10, 0.25, 0.50, 0.7, 0.9, 1.0), 3),
             (1000, 8, (0.01, 0.05, 0.10, 0.25, 0.50), 4)]
    for n, nb, budgets, seed in cases:
        print(f"noalloc evaluator: n={n} n_bins={nb} budgets={len(budgets)}", flush=True)
        p, S = inputs(n, nb, seed)
        ref = B.surrogate_evaluate(p, S, m8, e8, budgets)
        got = B.surrogate_evaluate_noalloc(p, S, m8, e8, budgets)
        torch.cuda.synchronize()
        for r, g, name in zip(ref, got, ("summary", "bins", "brier", "crps")):
            assert torch.equal(r, g), name
        assert torch.isfinite(got[0]).all()
