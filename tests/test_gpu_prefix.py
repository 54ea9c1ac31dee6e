"""GPU parity of shared-prefix scoring: prompts that continue a cached prefix against the
float64 oracle run on the concatenated prompt (prefix ++ suffix), at the bars of
test_gpu_parity (1e-4 float32, 3e-2 bf16), plus consistency with the plain scoring path.
"""
import numpy as np
import pytest
import torch

from oracle import transformer as ot
from paper_2605_31464_amd import binding as B
from paper_2605_31464_amd import synth

from conftest import arch_of
from bf16_emulation import Bf16Emulation
from floor_parity import FLOOR_FACTOR, assert_parity_floor, emulate, rows_of
from test_gpu_parity import TOL, assert_parity, make_scorer, padded, rng_prompts

pytestmark = pytest.mark.gpu


def run_case(scorer, W, shape, prefix_lengths, suffix_lengths, pid, seed, tol, vid=None):
    ptok, Lp = padded(rng_prompts(shape.vocab, prefix_lengths, seed))
    stok, Ls = padded(rng_prompts(shape.vocab, suffix_lengths, seed + 1))
    pid = np.asarray(pid, np.int32)
    vid = list(range(shape.vocab - 3, shape.vocab)) if vid is None else vid
    print(f"prefixes {list(Lp)}, suffixes {list(Ls)}, prefix ids {list(pid)}", flush=True)
    cache = scorer.build_prefixes(ptok, Lp)
    out = scorer.score_suffixes(cache, pid, stok, Ls, vid)
    full, fl = synth.concat_prompts(ptok, Lp, stok, Ls, pid)
    ref = ot.score(arch_of(shape), W, [full[i, : fl[i]] for i in range(len(fl))], vid)
    assert_parity(out, ref, tol)
    return cache, out, (full, fl, vid)


# ---------------------------------------------------------------- float32 model
def test_tiny_prefix_continuations_match_oracle():
    shape = synth.CONFIGS["tiny"].shape
    scorer, W = make_scorer(shape, gain_std=0.1)
    run_case(scorer, W, shape, [70, 129, 64], [1, 2, 63, 64, 65, 200, 33, 5],
             [0, 1, 2, 0, -1, 1, 0, 2], seed=31, tol=TOL["f32"])


# ---------------------------------------------------------------- bf16
@pytest.mark.parametrize("cfg,layers", [("small", 2), ("1p5b", 2)])
def test_bf16_prefix_continuations_match_oracle(cfg, layers):
    shape = synth.CONFIGS[cfg].shape.replace(n_layers=layers)
    scorer, W = make_scorer(shape, gain_std=0.1)
    prefix_lengths = [1, 63, 64, 65, 300]
    suffix_lengths = [1, 5, 64, 130, 257, 127, 128, 129, 40, 64]
    pid = [0, 1, 2, 3, 4, 4, 3, 2, 1, -1]
    cache, out, (full, fl, vid) = run_case(scorer, W, shape, prefix_lengths, suffix_lengths, pid,
                                           seed=41, tol=TOL["bf16"])
    assert cache.nbytes() >= 2 * layers * sum((n + 63) // 64 * 64 for n in prefix_lengths) \
        * shape.n_kv_heads * shape.head_dim * 2
    # the same prompts through the plain path: close (different key tiling, so not bitwise)
    plain = scorer.score(full, fl, vid)
    d = (out["logprobs"] - plain["logprobs"]).abs().max().item()
    print(f"max |prefix path - plain path| = {d:.3e}", flush=True)
    assert d <= TOL["bf16"]
    # a prompt with no prefix computes exactly what the plain path computes for it
    i = pid.index(-1)
    alone = scorer.score(full[i: i + 1, : fl[i]], fl[i: i + 1], vid)
    assert torch.equal(alone["logprobs"][0], out["logprobs"][i])


def test_prefix_results_do_not_depend_on_the_batch():
    shape = synth.CONFIGS["1p5b"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape)
    ptok, Lp = padded(rng_prompts(shape.vocab, [90, 200], 51))
    stok, Ls = padded(rng_prompts(shape.vocab, [17, 300, 64, 129], 52))
    pid = np.array([1, 0, 1, 0], np.int32)
    vid = [shape.vocab - 2, shape.vocab - 1]
    cache = scorer.build_prefixes(ptok, Lp)
    both = scorer.score_suffixes(cache, pid, stok, Ls, vid)
    for i in range(len(Ls)):
        one = scorer.score_suffixes(cache, pid[i: i + 1], stok[i: i + 1, : Ls[i]], Ls[i: i + 1], vid)
        assert torch.equal(one["logprobs"][0], both["logprobs"][i])
    again = scorer.score_suffixes(cache, pid, stok, Ls, vid)
    assert torch.equal(again["logprobs"], both["logprobs"])


def test_prefix_argument_errors():
    shape = synth.CONFIGS["small"].shape.replace(n_layers=1)
    scorer, W = make_scorer(shape)
    ptok, Lp = padded(rng_prompts(shape.vocab, [40], 61))
    cache = scorer.build_prefixes(ptok, Lp)
    stok, Ls = padded(rng_prompts(shape.vocab, [10, 10], 62))
    with pytest.raises(B.SurrogateError) as e:
        scorer.score_suffixes(cache, [0, 1], stok, Ls, [1])  # prefix 1 does not exist
    assert e.value.status == B.SURR_E_INVALID_ARG
    with pytest.raises(B.SurrogateError) as e:  # prefix + suffix beyond max_pos
        long = np.zeros((1, shape.max_pos - 39), np.int32)
        scorer.score_suffixes(cache, [0], long, [shape.max_pos - 39], [1])
    assert e.value.status == B.SURR_E_SHAPE
    with pytest.raises(B.SurrogateError) as e:  # a prefix must leave room for a suffix
        scorer.build_prefixes(np.zeros((1, shape.max_pos), np.int32), [shape.max_pos])
    assert e.value.status == B.SURR_E_SHAPE
    other, _ = make_scorer(shape, seed=3)
    with pytest.raises(B.SurrogateError) as e:
        other.score_suffixes(cache, [0, 0], stok, Ls, [1])
    assert e.value.status == B.SURR_E_INVALID_ARG


# ---------------------------------------------------------------- benchmark workload
@pytest.mark.timeout(900)
def test_7b_shared_prefix_workload_matches_oracle_and_plain_path():
    """The bench's shared-prefix workload at full 7B size.  The shortest candidate through
    the prefix path and the plain path against the float64 oracle on its concatenated
    prompt (full depth); every candidate's prefix-path result against the plain path on
    the concatenated prompts.  The two paths group a candidate's keys into different
    64-key tiles (the prefix's last tile is padded), so their bf16 roundings differ.

    Bounds come from the bf16 storage floor (floor_parity.py): against the oracle, the
    per-candidate bound; between the two paths, twice the largest bound over four
    candidates spanning the lengths (the shortest, the median and the two longest), each
    path being within its bound of the exact result.  There the floor is measured
    against the emulation's exact mode, which a CPU test pins to the oracle's forward."""
    w = synth.PREFIX_CONFIGS["7b-prefix"]
    scorer, W = make_scorer(w.shape)
    ptok, Lp, stok, Ls, pid = synth.make_prefix_prompts(w)
    vid = list(range(w.shape.vocab - w.n_verdict, w.shape.vocab))
    cache = scorer.build_prefixes(ptok, Lp)
    out = scorer.score_suffixes(cache, pid, stok, Ls, vid)
    assert B.surrogate_device_status(scorer.model) == B.SURR_OK
    full, fl = synth.concat_prompts(ptok, Lp, stok, Ls, pid)
    plain = scorer.score(full, fl, vid)
    out = {k: v.clone() for k, v in out.items()}
    plain = {k: v.clone() for k, v in plain.items()}
    del scorer, cache
    torch.cuda.empty_cache()

    order = np.argsort(fl, kind="stable")
    sub = [int(order[0]), int(order[len(order) // 2]), int(order[-2]), int(order[-1])]
    prompts = [full[i, : fl[i]] for i in sub]
    print(f"floor candidates {sub}, lengths {[int(fl[i]) for i in sub]}", flush=True)
    emu = emulate(w.shape, W, prompts, vid)
    exact = Bf16Emulation(arch_of(w.shape), W, "cuda:0", rounding=False).score(prompts, vid)
    f_lp = np.abs(emu["logprobs"] - exact["logprobs"]).max()
    f_p = np.abs(emu["p"] - exact["p"]).max()
    b_lp, b_p = max(TOL["bf16"], FLOOR_FACTOR * f_lp), max(TOL["bf16"], FLOOR_FACTOR * f_p)
    dlp = (out["logprobs"] - plain["logprobs"]).abs()
    dp = (out["p"] - plain["p"]).abs().max().item()
    print(f"7B shared-prefix workload: |prefix path - plain path| log-probs max "
          f"{dlp.max().item():.3e} rms {dlp.pow(2).mean().sqrt().item():.3e} (bound "
          f"{2 * b_lp:.3e}), p max {dp:.3e} (bound {2 * b_p:.3e}); floor log-probs {f_lp:.3e}, "
          f"p {f_p:.3e}", flush=True)
    assert dlp.max().item() <= 2 * b_lp
    assert dp <= 2 * b_p

    i = sub[0]
    print(f"oracle on candidate {i}: prefix {Lp[pid[i]]} + suffix {Ls[i]} tokens", flush=True)
    ref = rows_of(ot.score(arch_of(w.shape), W, [prompts[0]], vid))
    one = {k: v[:, :1] for k, v in emu.items()}
    assert_parity_floor(out, [i], ref, one, [f"prefix path, candidate {i}"])
    assert_parity_floor(plain, [i], ref, one, [f"plain path, candidate {i}"])


def test_token_budget_chunks_of_suffixes_and_cache_appends():
    """Chunked calls (a workspace for the longest prompt alone) give bitwise the one-pass
    outputs: suffix scoring against cached prefixes (prefix ids and outputs offset per
    chunk) and appends to cache entries with greedy and teacher-forced read-outs."""
    shape = synth.CONFIGS["1p5b"].shape.replace(n_layers=2)
    scorer, W = make_scorer(shape)
    ptok, Lp = padded(rng_prompts(shape.vocab, [90, 200, 64], 57))
    stok, Ls = padded(rng_prompts(shape.vocab, [17, 300, 64, 129, 250, 1], 58))
    pid = np.array([1, 0, -1, 2, 1, 0], np.int32)
    vid = [shape.vocab - 2, shape.vocab - 1]
    cache = scorer.build_prefixes(ptok, Lp)
    whole = scorer.score_suffixes(cache, pid, stok, Ls, vid)
    dtok = torch.from_numpy(stok).to("cuda:0")
    small = B.surrogate_workspace_size(scorer.model, 1, int(Ls.max()), int(Ls.max()))
    ws = torch.empty(small, dtype=torch.uint8, device="cuda:0")
    out = {k: torch.empty_like(v) for k, v in whole.items()}
    B.surrogate_score_suffixes(scorer.model, cache, pid, dtok, Ls, vid, ws, out["logprobs"],
                               out["confidence"], out["p"], out["verdict"])
    for k in whole:
        assert torch.equal(out[k], whole[k]), k
    # appends: two caches of the same entries, one filled in one pass, one in chunks
    caps = [512] * len(Ls)
    targets = [3, 5, 7, 11, 13, 17]
    c1, c2 = scorer.create_cache(caps), scorer.create_cache(caps)
    eids = list(range(len(Ls)))
    n1, t1 = scorer.extend(c1, eids, stok, Ls, targets)
    n2 = torch.empty_like(n1)
    t2 = torch.empty_like(t1)
    B.surrogate_cache_extend(scorer.model, c2, eids, dtok, Ls, ws, targets, n2, t2)
    assert torch.equal(n1, n2) and torch.equal(t1, t2)
    assert B.surrogate_cache_lengths(c2, len(Ls)).tolist() == Ls.tolist()
