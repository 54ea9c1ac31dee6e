"""GPU parity at the benchmark's full sizes.

The whole batch of a config is scored on the GPU exactly as bench.py does (one
surrogate_score_pairs call over all prompts); the float64 oracle recomputes sampled
prompts one by one (the shortest prompt and prompt 0).  The deferral step is checked
for the properties that hold at any size on the confidence vector it was given, and on
the sampled prompts against the oracle's confidence away from the threshold (its
bit-exact parity on given vectors is in test_gpu_parity).  Shapes the oracle cannot finish at full
depth (14B) are checked at their full width with fewer layers.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as ot
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

from conftest import arch_of, assert_selection_near_oracle, assert_selection_valid
from test_gpu_parity import TOL, assert_parity, make_scorer, padded, rng_prompts

pytestmark = pytest.mark.gpu


def score_full_config(name, rows):
    w = synth.CONFIGS[name]
    scorer, W = make_scorer(w.shape)
    tok, L = synth.make_prompts(w)
    vid = synth.verdict_ids(w)
    out = scorer.score(tok, L, vid)
    assert B.surrogate_device_status(scorer.model) == B.SURR_OK
    rows = [int(np.argmin(L)) if r == "shortest" else r for r in rows]
    ref = ot.score(arch_of(w.shape), W, [tok[i, : L[i]] for i in rows], vid)
    assert_parity(out, ref, TOL["bf16"], rows)
    conf = out["confidence"]
    q = conf.cpu().numpy()
    if w.select[0] == "budget":
        d, a, c = B.surrogate_select(conf, B.SURR_SELECT_BUDGET, budget_k=w.budget_k)
        assert_selection_valid(q, d.cpu().numpy(), a.cpu().numpy(), c.cpu().numpy(), "budget",
                               k=w.budget_k)
    else:
        d, a, c = B.surrogate_select(conf, B.SURR_SELECT_THRESHOLD, threshold=w.select[1])
        assert_selection_valid(q, d.cpu().numpy(), a.cpu().numpy(), c.cpu().numpy(),
                               "threshold", tau=w.select[1])
        # the sampled prompts are deferred exactly when the oracle's confidence says so,
        # away from the threshold
        assert_selection_near_oracle(d.cpu().numpy()[: int(c[0])], len(L), ref["confidence"],
                                     TOL["bf16"], rows=rows, tau=w.select[1])
    return scorer, out, tok, L, vid


@pytest.mark.timeout(900)
def test_7b_config_full_batch_sampled_prompt():
    scorer, out, tok, L, vid = score_full_config("7b", ["shortest"])
    # the sampled prompt scored alone gives bitwise the same result as inside the batch
    i = int(np.argmin(L))
    t1, l1 = padded([tok[i, : L[i]]])
    alone = scorer.score(t1, l1, vid)
    assert torch.equal(alone["logprobs"][0], out["logprobs"][i])


@pytest.mark.timeout(600)
def test_1p5b_config_full_batch_sampled_prompts():
    score_full_config("1p5b", ["shortest", 0])


# At 14B width bf16 storage by itself reaches the 3e-2 bar: a float64 emulation that
# rounds to bf16 exactly where the kernels store bf16 (norm outputs, q/k/v, P, attention
# output, SwiGLU output, final hidden) gives on these inputs a max verdict log-prob error
# of 2.8e-2 at rms 1.4e-2 (unit norm gains: 2.0e-2 at rms 1.0e-2).  The full-vocabulary
# log-probs of this shape are held to that floor plus the kernels' own rounding order,
# 4e-2; the renormalised verdict distribution, the confidence and the argmax keep 3e-2.
LP_TOL_14B_WIDTH = 4e-2


@pytest.mark.timeout(600)
def test_14b_shape_full_width_reduced_depth():
    shape = synth.CONFIGS["14b"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape, gain_std=0.1)
    lengths = [1, 127, 300, 1100]
    tok, L = padded(rng_prompts(shape.vocab, lengths, 21))
    vid = list(range(shape.vocab - 5, shape.vocab))
    out = scorer.score(tok, L, vid)
    assert_parity(out, ot.score(arch_of(shape), W, [tok[i, : L[i]] for i in range(len(L))], vid),
                  TOL["bf16"], lp_tol=LP_TOL_14B_WIDTH)
