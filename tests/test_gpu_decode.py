"""GPU parity of decode continuation (cache entries extended by prefill and decode steps)
against the float64 oracle by teacher forcing: a fixed seeded prompt and continuation,
the prompt prefilled into a cache entry and the continuation appended one token per
step, each step scoring the next continuation token.  The oracle runs the whole
sequence once and reads the next-token log-softmax at every position.

Bars: target log-probs within 1e-4 (float32 model) and 3e-2 (bf16); the greedy next
token equal to the oracle's argmax wherever its top-1/top-2 log-prob margin exceeds the
model's bar twice over.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as ot
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

from conftest import arch_of
from test_gpu_parity import TOL, make_scorer, padded, rng_prompts

pytestmark = pytest.mark.gpu


def teacher_forced(scorer, W, shape, prompt_lengths, n_steps, seed, tol, decode_batch=True):
    seqs = rng_prompts(shape.vocab, [n + n_steps + 1 for n in prompt_lengths], seed)
    B_ = len(seqs)
    cache = scorer.create_cache([len(s) for s in seqs])
    ids = np.arange(B_, dtype=np.int32)
    # prefill the prompts, scoring each sequence's first continuation token
    tok, L = padded([s[:n] for s, n in zip(seqs, prompt_lengths)])
    nxt, lp = scorer.extend(cache, ids, tok, L, [s[n] for s, n in zip(seqs, prompt_lengths)])
    got_lp, got_tok = [lp.cpu().numpy()], [nxt.cpu().numpy()]
    for t in range(n_steps):
        step = np.array([[s[n + t]] for s, n in zip(seqs, prompt_lengths)], np.int32)
        tgt = [s[n + t + 1] for s, n in zip(seqs, prompt_lengths)]
        if decode_batch:
            nxt, lp = scorer.extend(cache, ids, step, np.ones(B_, np.int32), tgt)
            got_lp.append(lp.cpu().numpy())
            got_tok.append(nxt.cpu().numpy())
        else:  # one entry per call
            row_lp, row_tok = [], []
            for i in range(B_):
                nxt, lp = scorer.extend(cache, ids[i: i + 1], step[i: i + 1], [1], tgt[i: i + 1])
                row_lp.append(lp.cpu().numpy()[0])
                row_tok.append(nxt.cpu().numpy()[0])
            got_lp.append(np.array(row_lp))
            got_tok.append(np.array(row_tok))
    got_lp = np.stack(got_lp, axis=1)    # [B, n_steps + 1]
    got_tok = np.stack(got_tok, axis=1)
    lens = B.surrogate_cache_lengths(cache, B_)
    assert lens.tolist() == [n + n_steps for n in prompt_lengths]
    arch = arch_of(shape)
    worst = 0.0
    for i, (s, n) in enumerate(zip(seqs, prompt_lengths)):
        pos = list(range(n - 1, n + n_steps))
        rows = ot.next_token_log_softmax(arch, W, s[: n + n_steps], pos)
        ref_lp = rows[np.arange(len(pos)), [s[j + 1] for j in pos]]
        err = np.abs(got_lp[i] - ref_lp).max()
        worst = max(worst, err)
        top2 = np.sort(rows, axis=1)[:, -2:]
        sure = (top2[:, 1] - top2[:, 0]) > 2 * tol
        assert np.array_equal(got_tok[i][sure], np.argmax(rows, axis=1)[sure]), i
    print(f"prompts {prompt_lengths}, {n_steps} decode steps: max |lp - oracle| = {worst:.3e} "
          f"(tol {tol})", flush=True)
    assert worst <= tol
    return cache


def test_tiny_teacher_forced_decode_matches_oracle():
    shape = synth.CONFIGS["tiny"].shape
    scorer, W = make_scorer(shape, gain_std=0.1)
    teacher_forced(scorer, W, shape, [5, 64, 130, 1], 20, seed=71, tol=TOL["f32"])


@pytest.mark.parametrize("cfg", ["small", "1p5b"])
def test_bf16_teacher_forced_decode_matches_oracle(cfg):
    shape = synth.CONFIGS[cfg].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape, gain_std=0.1)
    teacher_forced(scorer, W, shape, [1, 63, 64, 65, 200], 70, seed=73, tol=TOL["bf16"])


def test_decode_does_not_depend_on_batching():
    """Entries stepped together or one per call give bitwise the same results."""
    shape = synth.CONFIGS["1p5b"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape)
    seqs = rng_prompts(shape.vocab, [40, 100, 7], 81)
    tgt = [1, 2, 3]

    def run(together):
        cache = scorer.create_cache([128, 128, 128])
        tok, L = padded(seqs)
        scorer.extend(cache, [0, 1, 2], tok, L)
        out = []
        for t in range(5):
            step = np.full((3, 1), 10 + t, np.int32)
            if together:
                out.append(scorer.extend(cache, [0, 1, 2], step, [1, 1, 1], tgt)[1].cpu().numpy())
            else:
                out.append(np.array([scorer.extend(cache, [i], step[i: i + 1], [1], tgt[i: i + 1])[1]
                                     .cpu().numpy()[0] for i in (2, 0, 1)])[[1, 2, 0]])
        return np.stack(out)

    assert np.array_equal(run(True), run(False))


def test_mixed_prefill_and_decode_in_one_call():
    """A call may prefill some entries while stepping others; the results equal the
    separate calls' (bitwise: per-row results do not depend on the batch)."""
    shape = synth.CONFIGS["small"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape)
    a, b = rng_prompts(shape.vocab, [90, 33], 91)
    c1 = scorer.create_cache([256, 256])
    scorer.extend(c1, [0], padded([a])[0], [90])
    _, lp_mixed = scorer.extend(c1, [0, 1], padded([[5], b])[0], [1, 33], [7, 9])
    c2 = scorer.create_cache([256, 256])
    scorer.extend(c2, [0], padded([a])[0], [90])
    _, lp0 = scorer.extend(c2, [0], np.array([[5]], np.int32), [1], [7])
    _, lp1 = scorer.extend(c2, [1], padded([b])[0], [33], [9])
    assert lp_mixed[0].item() == lp0[0].item() and lp_mixed[1].item() == lp1[0].item()


def test_cache_argument_errors_and_reset():
    shape = synth.CONFIGS["small"].shape.replace(n_layers=1)
    scorer, W = make_scorer(shape)
    cache = scorer.create_cache([64, 10])
    tok = np.zeros((2, 70), np.int32)
    with pytest.raises(B.SurrogateError) as e:  # 70 tokens exceed a 64-token entry
        scorer.extend(cache, [0], tok[:1], [70])
    assert e.value.status == B.SURR_E_SHAPE
    with pytest.raises(B.SurrogateError) as e:  # an entry twice in one call
        scorer.extend(cache, [1, 1], tok[:, :3], [3, 3])
    assert e.value.status == B.SURR_E_INVALID_ARG
    with pytest.raises(B.SurrogateError) as e:
        scorer.extend(cache, [2], tok[:1, :3], [3])
    assert e.value.status == B.SURR_E_INVALID_ARG
    with pytest.raises(B.SurrogateError) as e:
        scorer.extend(cache, [0], tok[:1, :3], [3], [shape.vocab])
    assert e.value.status == B.SURR_E_INVALID_ARG
    scorer.extend(cache, [1], tok[:1, :64], [64])  # capacity 10 rounds up to 64
    assert B.surrogate_cache_lengths(cache, 2).tolist() == [0, 64]
    B.surrogate_cache_reset(cache, [1])
    assert B.surrogate_cache_lengths(cache, 2).tolist() == [0, 0]
    with pytest.raises(B.SurrogateError):
        B.surrogate_cache_create(scorer.model, [shape.max_pos + 1])


def test_decode_entries_crossing_key_slices_match_oracle():
    """Decode steps of entries whose keys cross the 256-key slices of the decode
    attention (and end inside partly filled 16-key groups) against the oracle."""
    shape = synth.CONFIGS["1p5b"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape, gain_std=0.1)
    teacher_forced(scorer, W, shape, [250, 509, 1020], 9, seed=77, tol=TOL["bf16"])


@pytest.mark.parametrize("wide_ffn", [False, True], ids=["d_ff4864", "d_ff16384"])
def test_row_count_regimes_give_bitwise_equal_rows(wide_ffn):
    """The projections pick a kernel by row count (few-row kernel up to 64 rows, per 64
    rows up to 128 against narrow weights, 128 x 128 tiles up to 128 rows against weights
    of 32768 rows or more, 256 x 256 tiles above); every choice accumulates in the same
    order, so a decode step's results do not depend on how many entries share it.  With
    d_ff = 16384 the gate/up projection (N = 32768) takes the 128 x 128 tiles with the
    SwiGLU epilogue from 65 to 128 rows."""
    shape = synth.CONFIGS["small"].shape.replace(n_layers=2)
    if wide_ffn:
        shape = shape.replace(n_layers=1, d_ff=16384)
    scorer, W = make_scorer(shape, gain_std=0.1)
    n = 140
    seqs = rng_prompts(shape.vocab, [3 + i % 5 for i in range(n)], 95)
    tgt = [(7 * i) % shape.vocab for i in range(n)]
    step = np.array([[11 + i % 13] for i in range(n)], np.int32)

    def run(group):
        cache = scorer.create_cache([64] * n)
        for g0 in range(0, n, 70):  # prefill in two calls of 70 (per-64-row regime)
            ids = list(range(g0, min(n, g0 + 70)))
            tok, L = padded([seqs[i] for i in ids])
            scorer.extend(cache, ids, tok, L)
        lp = np.empty(n, np.float32)
        nt = np.empty(n, np.int32)
        for g0 in range(0, n, group):
            ids = list(range(g0, min(n, g0 + group)))
            nxt, l = scorer.extend(cache, ids, step[ids], np.ones(len(ids), np.int32),
                                   [tgt[i] for i in ids])
            lp[ids] = l.cpu().numpy()
            nt[ids] = nxt.cpu().numpy()
        return lp, nt

    ref_lp, ref_nt = run(n)  # 140 rows: tiled projections
    for group in (1, 13, 30, 64, 100):
        lp, nt = run(group)
        assert np.array_equal(lp, ref_lp), group
        assert np.array_equal(nt, ref_nt), group
    assert B.surrogate_device_status(scorer.model) == B.SURR_OK
