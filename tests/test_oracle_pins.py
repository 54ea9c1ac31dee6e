"""Pins of the float64 oracle to facts other than itself (CPU only).

Each test checks the oracle against a closed form, an invariant, a hand-computed
case, an independent library routine or brute force, chosen so that a plausible
slip (a dropped term, a wrong sign or index, a transposed operand) fails one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

from oracle import select as osel
from oracle import transformer as ot
from paper_2605_31464_amd import synth

from conftest import arch_of

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_model(seed=0, gain_std=0.0, **shape_kw):
    shape = synth.CONFIGS["tiny"].shape.replace(**shape_kw)
    return arch_of(shape), synth.make_weights(shape, seed=seed, gain_std=gain_std)


def rand_prompt(vocab, L, seed):
    return np.random.default_rng(seed).integers(0, vocab, L).astype(np.int32)


# ---------------------------------------------------------------- P1 simplex
def test_attention_rows_are_causal_distributions():
    rng = np.random.default_rng(0)
    s = rng.normal(size=(37, 37)) * 3
    p = ot.causal_softmax_rows(s)
    assert np.all(p >= 0)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-12, rtol=0)
    assert np.all(p[np.triu_indices(37, 1)] == 0.0)


def test_forecast_is_on_the_simplex():
    arch, W = tiny_model()
    out = ot.score(arch, W, [rand_prompt(512, 50, 1), rand_prompt(512, 9, 2)], [3, 7, 511])
    p = out["p"]
    assert np.all(p >= 0)
    assert np.allclose(p.sum(axis=1), 1.0, atol=1e-12, rtol=0)
    assert np.array_equal(out["confidence"], p.max(axis=1))
    assert np.array_equal(out["verdict"], np.argmax(p, axis=1))


# ---------------------------------------------------------------- P2 causality
def test_future_tokens_do_not_change_earlier_rows():
    arch, W = tiny_model(gain_std=0.1)
    a = rand_prompt(512, 40, 3)
    b = a.copy()
    b[25:] = rand_prompt(512, 15, 4)
    xa, xb = ot.forward_hidden(arch, W, [a, b])
    assert np.array_equal(xa[:25], xb[:25])
    assert not np.allclose(xa[25:], xb[25:])


def test_prefix_scoring_equals_row_of_full_forward():
    arch, W = tiny_model()
    t = rand_prompt(512, 33, 5)
    (x_full,) = ot.forward_hidden(arch, W, [t])
    for j in (0, 7, 20):
        z_row = ot.last_position_logits(arch, W, [x_full[: j + 1]])
        z_pre = ot.last_position_logits(arch, W, ot.forward_hidden(arch, W, [t[: j + 1]]))
        np.testing.assert_allclose(z_pre, z_row, atol=1e-12, rtol=0)


# ---------------------------------------------------------------- P3 RoPE
def test_rope_identity_at_position_zero():
    x = np.random.default_rng(6).normal(size=(1, 3, 32))
    assert np.array_equal(ot.apply_rope(x, np.array([0]), 10000.0), x)


def test_rope_matches_complex_rotation_and_preserves_norm():
    # rotate-half RoPE is multiplication of (x_i + i*x_{i+hd/2}) by exp(i*theta_i),
    # theta_i = pos * base^(-2i/hd)  (RoFormer's complex form)
    rng = np.random.default_rng(7)
    hd, pos = 32, np.array([0, 1, 5, 1000, 16383])
    x = rng.normal(size=(len(pos), 2, hd))
    got = ot.apply_rope(x, pos, 10000.0)
    z = x[..., : hd // 2] + 1j * x[..., hd // 2:]
    freq = np.array([10000.0 ** (-2 * i / hd) for i in range(hd // 2)])
    zr = z * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    want = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(got, want, atol=1e-12, rtol=0)
    np.testing.assert_allclose(np.linalg.norm(got, axis=-1), np.linalg.norm(x, axis=-1),
                               rtol=1e-13)


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(8)
    q, k = rng.normal(size=(6, 1, 64)), rng.normal(size=(6, 1, 64))
    pos = np.arange(6)
    s0 = ot.apply_rope(q, pos, 1e4)[:, 0] @ ot.apply_rope(k, pos, 1e4)[:, 0].T
    s1 = ot.apply_rope(q, pos + 777, 1e4)[:, 0] @ ot.apply_rope(k, pos + 777, 1e4)[:, 0].T
    np.testing.assert_allclose(s0, s1, atol=1e-10, rtol=0)


# ---------------------------------------------------------------- P4 brute force
def test_single_token_attention_returns_v0():
    rng = np.random.default_rng(9)
    q, k, v = rng.normal(size=(1, 4, 8)), rng.normal(size=(1, 2, 8)), rng.normal(size=(1, 2, 8))
    o = ot.causal_attention(q, k, v)
    for a in range(4):
        assert np.array_equal(o[0, a], v[0, a // 2])


def hand_case():
    """d=4, one head (hd=4), V=4, d_ff=1, eps=0, prompt [0, 1]; see the derivation in
    test_hand_computed_one_layer_model."""
    z4 = lambda: np.zeros((4, 4))
    E = np.array([[1, 1, 1, 1], [2, 0, 0, 0], [0, 2, 0, 0], [0, 0, 2, 0]], float)
    wq = z4(); wq[0, 0] = 0.5; wq[0, 1] = 7.0          # q = [0.5 h0 + 7 h1, 0, 0, 0]
    wk = z4(); wk[0, 0] = 1.0; wk[1, 0] = 5.0          # k = [h0, 5 h0, 0, 0]
    wv = np.eye(4); wv[1, 1] = 2.0; wv[1, 0] = 1.0      # v = [h0, h0 + 2 h1, h2, h3]
    wo = z4(); wo[0, 1] = 1.0                           # attn out = [o1, 0, 0, 0]
    W = {"embed": E, "layers.0.attn_norm": np.ones(4), "layers.0.w_q": wq,
         "layers.0.w_k": wk, "layers.0.w_v": wv, "layers.0.w_o": wo,
         "layers.0.mlp_norm": np.ones(4), "layers.0.w_gate": np.array([[1.0, 0, 0, 0]]),
         "layers.0.w_up": np.array([[0.5, 0, 0, 0]]),
         "layers.0.w_down": np.array([[0.0], [0.0], [1.0], [0.0]]),
         "final_norm": np.ones(4),
         "lm_head": np.array([[1.0, 0, 0, 0], [0, 0, 1, 0], [0, 0, 0, 0], [0, 1, 0, 0]])}
    arch = dict(n_layers=1, d_model=4, n_q_heads=1, n_kv_heads=1, head_dim=4, d_ff=1,
                vocab=4, rope_base=10000.0, rms_eps=0.0)
    return arch, W


def test_hand_computed_one_layer_model():
    # Derivation for the last position (j = 1), by hand:
    #   h_0 = [1,1,1,1], h_1 = [2,0,0,0] (both have unit RMS).
    #   q_1 = [1,0,0,0]; k_0 = [1,5,0,0]; k_1 = [2,10,0,0]; v_0 = [1,3,1,1]; v_1 = [2,2,0,0].
    #   RoPE pairs dims (0,2) with angle pos*1 and (1,3) with angle pos*0.01.  q_1 has
    #   only dim 0, so only the (0,2) pair matters:
    #     score(1,0) = cos(1) / sqrt(4),  score(1,1) = 2 (cos^2 1 + sin^2 1) / 2 = 1.
    #   a = softmax([cos(1)/2, 1]);  o_1 = a0 v_0 + a1 v_1;  o_1[1] = 3 a0 + 2 a1 = w.
    #   x_1 = E[1] + [w,0,0,0] = [2+w,0,0,0];  RMSNorm -> h = [2,0,0,0];
    #   gate = 2, up = 1 -> x_1 = [2+w, 0, s, 0] with s = silu(2) = 2/(1+e^-2).
    #   y = x_1 / sqrt(((2+w)^2 + s^2)/4);  z = [y0, y2, 0, y1] = [(2+w)/r, s/r, 0, 0].
    #   verdicts [0, 1]: lp = z[:2] - log(e^z0 + e^z1 + 2).
    arch, W = hand_case()
    out = ot.score(arch, W, [np.array([0, 1])], [0, 1])
    e0, e1 = math.exp(math.cos(1.0) / 2), math.exp(1.0)
    a0, a1 = e0 / (e0 + e1), e1 / (e0 + e1)
    w = 3 * a0 + 2 * a1
    s = 2.0 / (1.0 + math.exp(-2.0))
    r = math.sqrt(((2 + w) ** 2 + s * s) / 4)
    z0, z1 = (2 + w) / r, s / r
    lse = math.log(math.exp(z0) + math.exp(z1) + 2.0)
    np.testing.assert_allclose(out["logprobs"][0], [z0 - lse, z1 - lse], atol=1e-12, rtol=0)
    assert out["verdict"][0] == 0


# ---------------------------------------------------------------- P5 zero head
def test_zero_head_gives_uniform_logprobs():
    arch, W = tiny_model()
    W = dict(W, lm_head=np.zeros_like(W["lm_head"]))
    out = ot.score(arch, W, [rand_prompt(512, 20, 10), rand_prompt(512, 3, 11)], [5, 6, 9])
    assert np.all(out["logprobs"] == -math.log(512))
    np.testing.assert_allclose(out["p"], 1 / 3, atol=1e-15)
    assert np.all(out["verdict"] == 0)


# ---------------------------------------------------------------- P6 zero mixing
def test_zero_output_projections_leave_the_embedding():
    arch, W = tiny_model(gain_std=0.1)
    W = dict(W)
    for l in range(arch["n_layers"]):
        W[f"layers.{l}.w_o"] = np.zeros_like(W[f"layers.{l}.w_o"])
        W[f"layers.{l}.w_down"] = np.zeros_like(W[f"layers.{l}.w_down"])
    t = rand_prompt(512, 30, 12)
    t2 = t.copy()
    t2[:-1] = rand_prompt(512, 29, 13)
    vid = [1, 2, 3]
    got, got2 = ot.score(arch, W, [t, t2], vid)["logprobs"]
    e = W["embed"][t[-1]].astype(np.float64)
    g = W["final_norm"].astype(np.float64)
    y = e / np.sqrt(np.mean(e ** 2) + arch["rms_eps"]) * g
    want = scipy.special.log_softmax(W["lm_head"].astype(np.float64) @ y)[vid]
    np.testing.assert_allclose(got, want, atol=1e-12, rtol=0)
    np.testing.assert_allclose(got2, want, atol=1e-12, rtol=0)


# ---------------------------------------------------------------- P7 GQA
def test_gqa_equals_mha_with_duplicated_kv_heads():
    arch, W = tiny_model(n_kv_heads=2)
    hd = arch["head_dim"]
    W_mha = dict(W)
    for l in range(arch["n_layers"]):
        for n in ("w_k", "w_v"):
            m = W[f"layers.{l}.{n}"].reshape(2, hd, -1)
            W_mha[f"layers.{l}.{n}"] = np.repeat(m, 2, axis=0).reshape(4 * hd, -1)
    arch_mha = dict(arch, n_kv_heads=4)
    t = [rand_prompt(512, 45, 14)]
    a = ot.score(arch, W, t, [0, 1])["logprobs"]
    b = ot.score(arch_mha, W_mha, t, [0, 1])["logprobs"]
    np.testing.assert_allclose(a, b, atol=1e-13, rtol=0)


# ---------------------------------------------------------------- P8 library routines
def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(15)
    L, nq, nkv, hd = 29, 6, 2, 16
    q, k, v = rng.normal(size=(L, nq, hd)), rng.normal(size=(L, nkv, hd)), rng.normal(size=(L, nkv, hd))
    o = ot.causal_attention(q, k, v)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(nq // nkv, dim=0)
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(nq // nkv, dim=0)
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, atol=1e-12, rtol=0)


def test_rms_norm_and_lse_match_library():
    rng = np.random.default_rng(16)
    x, g = rng.normal(size=(5, 64)), rng.normal(size=64)
    ref = F.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(ot.rms_norm(x, g, 1e-6), ref, atol=1e-13, rtol=0)
    z = rng.normal(size=1000) * 30
    np.testing.assert_allclose(ot.log_softmax_full(z), z - scipy.special.logsumexp(z),
                               atol=1e-11, rtol=0)


def torch_reference_scores(arch, W, prompts, vid):
    """Independent float64 forward from torch.nn.functional building blocks."""
    d, nq, nkv, hd = arch["d_model"], arch["n_q_heads"], arch["n_kv_heads"], arch["head_dim"]
    T = {k: torch.from_numpy(ot.to_f64(v)) for k, v in W.items()}
    freq = torch.tensor([arch["rope_base"] ** (-2 * i / hd) for i in range(hd // 2)],
                        dtype=torch.float64)

    def rope(x):  # x [heads, L, hd]
        L = x.shape[1]
        rot = torch.polar(torch.ones(L, hd // 2, dtype=torch.float64),
                          torch.arange(L, dtype=torch.float64)[:, None] * freq[None])
        z = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * rot
        return torch.cat([z.real, z.imag], dim=-1)

    out = []
    for t in prompts:
        x = T["embed"][torch.from_numpy(np.asarray(t, np.int64))]
        L = x.shape[0]
        for l in range(arch["n_layers"]):
            p = f"layers.{l}."
            h = F.rms_norm(x, (d,), T[p + "attn_norm"], eps=arch["rms_eps"])
            q = F.linear(h, T[p + "w_q"]).view(L, nq, hd).transpose(0, 1)
            k = F.linear(h, T[p + "w_k"]).view(L, nkv, hd).transpose(0, 1)
            v = F.linear(h, T[p + "w_v"]).view(L, nkv, hd).transpose(0, 1)
            k = k.repeat_interleave(nq // nkv, 0)
            v = v.repeat_interleave(nq // nkv, 0)
            o = F.scaled_dot_product_attention(rope(q), rope(k), v, is_causal=True)
            x = x + F.linear(o.transpose(0, 1).reshape(L, nq * hd), T[p + "w_o"])
            h = F.rms_norm(x, (d,), T[p + "mlp_norm"], eps=arch["rms_eps"])
            x = x + F.linear(F.silu(F.linear(h, T[p + "w_gate"])) * F.linear(h, T[p + "w_up"]),
                             T[p + "w_down"])
        y = F.rms_norm(x[-1], (d,), T["final_norm"], eps=arch["rms_eps"])
        out.append(F.log_softmax(F.linear(y, T["lm_head"]), dim=-1)[vid].numpy())
    return np.stack(out)


@pytest.mark.parametrize("kv", [4, 2, 1])
def test_whole_model_matches_torch_functional_forward(kv):
    arch, W = tiny_model(gain_std=0.1, n_kv_heads=kv)
    prompts = [rand_prompt(512, L, 20 + L) for L in (1, 17, 70)]
    vid = [0, 100, 511]
    got = ot.score(arch, W, prompts, vid)["logprobs"]
    want = torch_reference_scores(arch, W, prompts, vid)
    np.testing.assert_allclose(got, want, atol=1e-11, rtol=0)


def test_bf16_weights_decode_exactly():
    shape = synth.CONFIGS["small"].shape.replace(n_layers=1, vocab=64, d_model=64, d_ff=64,
                                                 n_q_heads=1, n_kv_heads=1)
    W = synth.make_weights(shape)
    bits = W["layers.0.w_q"]
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    assert np.array_equal(ot.to_f64(bits), ref)


# ---------------------------------------------------------------- P11 batch independence
def test_batch_scores_equal_single_scores():
    arch, W = tiny_model()
    prompts = [rand_prompt(512, L, 30 + L) for L in (5, 64, 13)]
    batch = ot.score(arch, W, prompts, [1, 2])["logprobs"]
    for i, t in enumerate(prompts):
        np.testing.assert_allclose(ot.score(arch, W, [t], [1, 2])["logprobs"][0], batch[i],
                                   atol=1e-13, rtol=0)


# ---------------------------------------------------------------- P9 select
def test_threshold_trivial_cases_and_partition():
    q = np.array([0.0, 0.3, 0.7, 1.0, -0.0, 0.5], np.float32)
    d, a = osel.select_threshold(q, 0.0)
    assert d.size == 0 and np.array_equal(a, np.arange(6))
    d, a = osel.select_threshold(q, 1.0000001)
    assert np.array_equal(d, np.arange(6)) and a.size == 0
    d, a = osel.select_threshold(q, 0.7)
    assert np.array_equal(d, [0, 1, 4, 5]) and np.array_equal(a, [2, 3])
    d, a = osel.select_threshold(np.array([np.nan, 0.9], np.float32), 0.0)
    assert np.array_equal(d, [0]) and np.array_equal(a, [1])


def test_threshold_defer_set_is_monotone_in_tau():
    q = np.random.default_rng(17).random(200).astype(np.float32)
    prev = set()
    for tau in np.linspace(0, 1.01, 60):
        d = set(osel.select_threshold(q, tau)[0].tolist())
        assert prev <= d
        prev = d


def test_budget_trivial_cases():
    q = np.random.default_rng(18).random(9).astype(np.float32)
    assert osel.select_budget(q, 0)[0].size == 0
    assert np.array_equal(osel.select_budget(q, 9)[0], np.arange(9))
    assert np.array_equal(osel.select_budget(q, 50)[0], np.arange(9))
    for k in range(10):
        d, a = osel.select_budget(q, k)
        assert d.size == k and np.array_equal(np.sort(np.concatenate([d, a])), np.arange(9))
    with pytest.raises(ValueError):
        osel.select_budget(q, -1)


def test_budget_brute_force_over_subsets():
    # Definition: D (|D| = k) is the defer set iff every i in D precedes every j not in D
    # in the order (NaN first, then ascending confidence, then ascending index).
    rng = np.random.default_rng(19)
    vals = np.array([np.nan, 0.1, 0.5, 0.5, -0.0, 0.0, 0.9], np.float32)
    for trial in range(40):
        n = int(rng.integers(1, 8))
        q = rng.choice(vals, n)

        def before(i, j):
            qi, qj = float(q[i]), float(q[j])
            if math.isnan(qi) != math.isnan(qj):
                return math.isnan(qi)
            if math.isnan(qi) or qi == qj:
                return i < j
            return qi < qj

        for k in range(n + 1):
            good = [set(D) for D in itertools.combinations(range(n), k)
                    if all(before(i, j) for i in D for j in range(n) if j not in D)]
            assert len(good) == 1
            d, a = osel.select_budget(q, k)
            assert set(d.tolist()) == good[0]
            assert list(d) == sorted(d) and list(a) == sorted(a)


# ---------------------------------------------------------------- P10 paper worked values
def test_paper_worked_values():
    with open(os.path.join(GOLDEN, "paper_selective_use.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        d, a = osel.select_threshold(np.array([c["confidence"]], np.float32), c["tau"])
        assert bool(a.size) == c["accepted"], c["source"]


# ---------------------------------------------------------------- next-token read-out
def test_next_token_rows_equal_prefix_scoring():
    """Row j of the teacher-forced read-out is the last-position read-out of the prefix
    ending at j (the pinned scoring path), and each row is a distribution."""
    arch, W = tiny_model(gain_std=0.1)
    t = rand_prompt(512, 40, 11)
    pos = [0, 7, 39]
    rows = ot.next_token_log_softmax(arch, W, t, pos)
    assert np.allclose(np.exp(rows).sum(axis=1), 1.0, atol=1e-12, rtol=0)
    for r, j in enumerate(pos):
        ids = [3, 100, 511]
        ref = ot.score(arch, W, [t[: j + 1]], ids)["logprobs"][0]
        assert np.allclose(rows[r, ids], ref, atol=1e-12, rtol=0)
