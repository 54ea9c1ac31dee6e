"""Pins of the bf16-storage emulation (tests/bf16_emulation.py) and of the oracle's
forecast margin (CPU only).

The emulation bounds the bf16 configurations' parity checks, so it is pinned to facts
other than itself: with rounding off it is the float64 oracle's forward; its rounding is
round-to-nearest-even to bfloat16 at the exact halfway cases; it rounds at every storage
point of the bf16 path and nowhere else; its ensemble members are deterministic and
differ from each other only through the roundings.
"""
import math

import numpy as np
import pytest
import torch

from oracle import transformer as ot
from paper_2605_31464_amd import synth

from bf16_emulation import Bf16Emulation, _Rounder
from conftest import arch_of

SHAPE = synth.ModelShape(2, 64, 4, 2, 16, 96, 300, 64)  # bf16 weights, GQA 4/2


def model(gain_std=0.1, seed=0, shape=SHAPE):
    return arch_of(shape), synth.make_weights(shape, seed=seed, gain_std=gain_std)


def prompts(vocab, lengths, seed=3):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, vocab, n).astype(np.int32) for n in lengths]


def test_exact_mode_is_the_oracle_forward():
    arch, W = model()
    ps = prompts(SHAPE.vocab, [1, 5, 33])
    vid = [0, 7, 299]
    em = Bf16Emulation(arch, W, rounding=False).score(ps, vid)
    ref = ot.score(arch, W, ps, vid)
    np.testing.assert_allclose(em["logprobs"][0], ref["logprobs"], atol=1e-11, rtol=0)
    np.testing.assert_allclose(em["p"][0], ref["p"], atol=1e-12, rtol=0)


def test_exact_mode_on_float32_weights_is_the_oracle_forward():
    shape = synth.CONFIGS["tiny"].shape
    arch, W = model(shape=shape)
    ps = prompts(shape.vocab, [2, 70])
    em = Bf16Emulation(arch, W, rounding=False).score(ps, [1, 2])
    ref = ot.score(arch, W, ps, [1, 2])
    np.testing.assert_allclose(em["logprobs"][0], ref["logprobs"], atol=1e-11, rtol=0)


def test_rounding_is_nearest_even_to_bfloat16():
    R = _Rounder(0, "cpu", True)
    ulp = 2.0 ** -7  # bfloat16 spacing in [1, 2)
    x = torch.tensor([1.0, 1 + ulp / 2, 1 + 3 * ulp / 2, 1 + ulp / 2 + 2 ** -20, -(1 + ulp),
                      1002.0, 1003.0, 2.0 ** -130], dtype=torch.float64)
    # ties go to the even neighbour, just above a tie rounds up, representable values stay
    # (in [512, 1024) the spacing is 4: 1000 has the even mantissa 122, 1004 the odd 123)
    want = [1.0, 1.0, 1 + 2 * ulp, 1 + ulp, -(1 + ulp), 1000.0, 1004.0, 2.0 ** -130]
    assert R.bf16(x).tolist() == want
    # on float32 values it is torch's float32 -> bfloat16 conversion, bit for bit
    v = torch.from_numpy(np.random.default_rng(1).normal(size=4096).astype(np.float32))
    np.testing.assert_array_equal(R.bf16(v.double()).numpy(), v.bfloat16().double().numpy())
    # the float32 storage of the residual stream
    assert R.f32(torch.tensor([1 + 2.0 ** -30], dtype=torch.float64)).item() == 1.0


def test_ensemble_members_round_to_nearest_and_probabilities_per_row():
    """Members k > 0 round to nearest even after a float32-sized perturbation (so a value
    far from a rounding boundary rounds as in member 0) and round each probability row on
    the bf16 grid scaled by one factor in [1, 2) (a relative error of at most 2^-8)."""
    x = torch.from_numpy(np.random.default_rng(4).normal(size=1 << 20)) * 3.0
    plain = _Rounder(0, "cpu", True).bf16(x)
    m1 = _Rounder(1, "cpu", True).bf16(x)
    same = (m1 == plain).double().mean().item()
    assert 0.99 < same < 1.0  # only values within 2^-16 of a boundary may round the other way
    assert torch.equal(m1, m1.float().bfloat16().double())  # still bfloat16 values
    p = torch.rand(64, 300, dtype=torch.float64)
    r = _Rounder(2, "cpu", True).bf16_rows(p)
    assert ((r - p).abs() / p).max().item() <= 2.0 ** -8 * (1 + 1e-12)
    assert not torch.equal(r, _Rounder(0, "cpu", True).bf16_rows(p))


def test_rounds_at_every_storage_point_and_nowhere_else():
    """Per layer: attention-norm output, q, k, v, the probabilities of each query head,
    attention output, MLP-norm output, SwiGLU output; then the final hidden state."""
    arch, W = model()
    calls = []
    orig = _Rounder.bf16

    def counting(self, x):
        calls.append(tuple(x.shape))
        return orig(self, x)

    _Rounder.bf16 = counting
    try:
        Bf16Emulation(arch, W).score(prompts(SHAPE.vocab, [9]), [1])
    finally:
        _Rounder.bf16 = orig
    L, d, hd = 9, SHAPE.d_model, SHAPE.head_dim
    nq, nkv, ff = SHAPE.n_q_heads, SHAPE.n_kv_heads, SHAPE.d_ff
    layer = [(L, d), (L, nq, hd), (L, nkv, hd), (L, nkv, hd)] + [(L, L)] * nq + \
            [(L, nq * hd), (L, d), (L, ff)]
    assert calls == layer * SHAPE.n_layers + [(1, d)]


def test_rounding_moves_the_result_by_a_bf16_sized_amount():
    arch, W = model()
    ps = prompts(SHAPE.vocab, [40, 64])
    vid = [0, 7, 299]
    exact = Bf16Emulation(arch, W, rounding=False).score(ps, vid)["logprobs"][0]
    em = Bf16Emulation(arch, W).score(ps, vid, members=(0, 1, 2))["logprobs"]
    err = np.abs(em - exact)
    # a few bf16 steps (2^-8 relative) of logits of size ~1, never zero, never O(1)
    assert 1e-5 < err.max() < 5e-2


def test_ensemble_members_are_deterministic_and_distinct():
    arch, W = model()
    ps = prompts(SHAPE.vocab, [50])
    em = Bf16Emulation(arch, W)
    a = em.score(ps, [3, 4], members=(0, 1, 2))["logprobs"]
    b = em.score(ps, [3, 4], members=(2, 0))["logprobs"]
    assert np.array_equal(a[2], b[0]) and np.array_equal(a[0], b[1])
    assert not np.array_equal(a[0], a[1]) and not np.array_equal(a[1], a[2])


# ---------------------------------------------------------------- forecast margin
def test_forecast_margin_is_top1_minus_top2():
    lp = np.log(np.array([[0.5, 0.2, 0.3],     # top-1 first: ln(.5) - ln(.3)
                          [0.1, 0.3, 0.6],     # top-1 last:  ln(.6) - ln(.3)
                          [0.4, 0.4, 0.2],     # exact tie: 0
                          [0.25, 0.05, 0.7]]))
    out = ot.forecast(lp)
    want = [math.log(0.5 / 0.3), math.log(0.6 / 0.3), 0.0, math.log(0.7 / 0.25)]
    np.testing.assert_allclose(out["margin"], want, atol=1e-15, rtol=0)
    assert np.all(out["margin"] >= 0)        # a swapped top-1/top-2 order gives < 0
    assert out["verdict"].tolist() == [0, 2, 0, 2]  # the tie takes the lowest index


def test_forecast_margin_single_verdict_is_infinite():
    out = ot.forecast(np.array([[-3.0], [-0.5]]))
    assert np.all(np.isposinf(out["margin"]))
    assert out["p"].tolist() == [[1.0], [1.0]] and out["verdict"].tolist() == [0, 0]


def test_forecast_margin_gates_argmax_checks():
    # only the first row is decisive at 0.1 nats
    out = ot.forecast(np.array([[-1.0, -1.2], [-1.0, -1.05], [-2.0, -2.0]]))
    np.testing.assert_allclose(out["margin"], [0.2, 0.05, 0.0], atol=1e-15)
    assert (out["margin"] > 0.1).tolist() == [True, False, False]
