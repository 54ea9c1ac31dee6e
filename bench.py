#!/usr/bin/env python3
"""Throughput of batched forecast scoring on one MI355X.

One step = one prefill-only scoring pass over a batch of ragged kernel-pair prompts
(surrogate_score_pairs: embedding, all decoder layers, last-position LM head with the
full-vocabulary log-softmax, verdict read-out) followed by the deferral step
(surrogate_select).  Inputs are seeded synthetic prompts and random weights of the
named shape, resident in HBM before the timed region starts.

Default workload: the 7B-shape bf16 decoder (28 layers, d_model 3584, 28/4 heads of
128, d_ff 18944, vocab 131072), 128 prompts with lognormal lengths (median 3072,
sigma 0.5, clipped to [1024, 8192]), 2 verdict tokens, budget deferral of
floor(0.2 * 128) = 25 candidates.

Prints one JSON line.  `value` is forecast pairs/s; prefill tokens/s and the fraction
of the bf16 MFMA peak are reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15  # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12   # MI355X HBM3E, B/s
METRIC = "forecast pairs/sec + prefill tokens/sec at 7B shape; % bf16 MFMA peak"


def flops_per_prompt(s, L: np.ndarray) -> np.ndarray:
    """Algorithmic FLOPs of scoring one prompt of length L: causal triangle only, final
    layer pruned to the K/V projection plus the last row, LM head at the last row."""
    d, dq, dkv, ff = s.d_model, s.d_q, s.d_kv, s.d_ff
    L = L.astype(np.float64)
    c_lin = 2 * d * (dq + 2 * dkv) + 2 * dq * d + 6 * d * ff
    c_att = 2 * s.n_q_heads * s.head_dim * L * (L + 1)
    return ((s.n_layers - 1) * (c_lin * L + c_att) + 4 * d * dkv * L + (c_lin - 4 * d * dkv)
            + 4 * s.n_q_heads * s.head_dim * L + 2 * d * s.vocab)


def phase_rates(s, L: np.ndarray, phases: dict, steps: int) -> dict:
    """Achieved rate of each phase against its roofline, from the phase times measured
    with HIP events on the launch stream: MFMA phases in TFLOP/s of algorithmic work,
    memory-bound phases in GB/s of algorithmic bytes (each tensor read or written once).
    Per step at the batch's lengths: QKV over all T tokens in the non-final layers, and
    in the final one K/V over all T tokens plus the queries of the B last rows; O, gate/up
    and down over T in the non-final
    layers; attention on the causal triangle in the non-final layers plus the last row of
    each prompt in the final one; RMSNorm = 2 n_layers - 1 full-batch norms (fp32 row in,
    bf16 row out) plus two on the last rows; the head reads W_head once (bf16 models write
    one 16-byte record per row and 128-column tile, the float32 model B rows of logits) and
    the read-out reads those back; embedding gathers bf16 rows into the fp32 residual."""
    d, dq, dkv, ff, V = s.d_model, s.d_q, s.d_kv, s.d_ff, s.vocab
    nl, T, B_ = s.n_layers, float(L.sum()), float(len(L))
    esz = 2 if s.dtype == "bf16" else 4
    Lf = L.astype(np.float64)
    head_out = B_ * (16 * ((V + 127) // 128) if s.dtype == "bf16" else 4 * V)
    work = {
        "gemm_qkv": ("mfma", 2.0 * d * (dq + 2 * dkv) * T * (nl - 1) + 4.0 * d * dkv * T
                     + 2.0 * d * dq * B_),
        "gemm_o": ("mfma", 2.0 * dq * d * T * (nl - 1)),
        "gemm_gate_up": ("mfma", 2.0 * d * 2 * ff * T * (nl - 1)),
        "gemm_down": ("mfma", 2.0 * ff * d * T * (nl - 1)),
        "attention": ("mfma", (nl - 1) * float((2 * s.n_q_heads * s.head_dim * Lf * (Lf + 1)).sum())
                      + float((4 * s.n_q_heads * s.head_dim * Lf).sum())),
        "embed": ("hbm", T * (esz * d + 4 * d + 12)),
        "rmsnorm": ("hbm", ((2 * nl - 1) * T + 2 * B_) * (4 * d + esz * d)),
        "lm_head": ("hbm", esz * V * d + esz * B_ * d + head_out),
        "lse_verdict": ("hbm", head_out),
    }
    out = {}
    for ph, (bound, amount) in work.items():
        ms, n = phases.get(ph, (0.0, 0))
        if not n or ms <= 0:
            continue
        t = ms / steps / 1e3
        if bound == "mfma":
            ach = amount / t
            out[ph] = {"bound": "mfma", "achieved": ach / 1e12, "unit": "TFLOP/s",
                       "frac": ach / PEAK_BF16, "ms_per_step": ms / steps}
        else:
            ach = amount / t
            out[ph] = {"bound": "hbm", "achieved": ach / 1e9, "unit": "GB/s",
                       "frac": ach / PEAK_HBM, "ms_per_step": ms / steps}
    return out


def prefix_flops(s, Lp: np.ndarray, Ls: np.ndarray, pid: np.ndarray):
    """Algorithmic FLOPs of the shared-prefix workload: building each prefix's K/V (all
    layers but the last in full, the last only its K/V projection) and scoring each suffix
    against its prefix (suffix rows attend every prefix key and their causal suffix keys;
    the final layer pruned as in flops_per_prompt)."""
    d, dq, dkv, ff, nl = s.d_model, s.d_q, s.d_kv, s.d_ff, s.n_layers
    c_lin = 2 * d * (dq + 2 * dkv) + 2 * dq * d + 6 * d * ff
    qh = 2 * s.n_q_heads * s.head_dim
    Lp = Lp.astype(np.float64)
    Ls = Ls.astype(np.float64)
    P = Lp[pid]
    build = float(((nl - 1) * (c_lin * Lp + qh * Lp * (Lp + 1)) + 4 * d * dkv * Lp).sum())
    score = float(((nl - 1) * (c_lin * Ls + qh * (2 * P * Ls + Ls * (Ls + 1))) + 4 * d * dkv * Ls
                   + (c_lin - 4 * d * dkv) + 2 * qh * (P + Ls) + 2 * d * s.vocab).sum())
    return build, score


def prefix_reuse_rates(B, torch, dev, model, steps: int, warmup: int) -> dict:
    """Shared-prefix workload (every candidate of a task shares that task's prompt prefix):
    per step, build the prefixes' K/V and score every candidate's suffix against it, then
    the budget selection; beside it the plain path on the concatenated prompts."""
    from paper_2605_31464_amd import synth
    w = synth.PREFIX_CONFIGS["7b-prefix"]
    s = w.shape
    ptok_np, Lp, stok_np, Ls, pid = synth.make_prefix_prompts(w)
    full_np, fl = synth.concat_prompts(ptok_np, Lp, stok_np, Ls, pid)
    vid = np.arange(s.vocab - w.n_verdict, s.vocab, dtype=np.int32)
    nb = len(Ls)
    ptok = torch.from_numpy(ptok_np).to(dev)
    stok = torch.from_numpy(stok_np).to(dev)
    ws_b = torch.empty(B.surrogate_workspace_size(model, len(Lp), int(Lp.sum()), int(Lp.max())),
                       dtype=torch.uint8, device=dev)
    ws_s = torch.empty(B.surrogate_workspace_size(model, nb, int(Ls.sum()), int(Ls.max())),
                       dtype=torch.uint8, device=dev)
    lp = torch.empty(nb, w.n_verdict, device=dev)
    conf = torch.empty(nb, device=dev)
    d_idx = torch.empty(nb, dtype=torch.int32, device=dev)
    a_idx = torch.empty(nb, dtype=torch.int32, device=dev)
    counts = torch.empty(2, dtype=torch.int32, device=dev)
    k = int(0.2 * nb)
    stream = torch.cuda.current_stream()

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(n):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n / 1e3

    # building the prefixes' K/V (the cache allocates its memory, so it is timed apart)
    caches = []
    t_build = timed(lambda: caches.append(B.surrogate_prefix_build(model, ptok, Lp, ws_b,
                                                                   stream=stream)), steps)
    cache = caches.pop()
    cache_bytes = cache.nbytes()
    for c in caches:
        c.close()

    def score():
        B.surrogate_score_suffixes(model, cache, pid, stok, Ls, vid, ws_s, lp, conf, stream=stream)
        B.surrogate_select(conf, B.SURR_SELECT_BUDGET, 0.0, k, d_idx, a_idx, counts, stream=stream)

    t_score = timed(score, steps)
    cache.close()
    del ws_b, ws_s
    full = torch.from_numpy(full_np).to(dev)
    ws_f = torch.empty(B.surrogate_workspace_size(model, nb, int(fl.sum()), int(fl.max())),
                       dtype=torch.uint8, device=dev)

    def plain():
        B.surrogate_score_pairs(model, full, fl, vid, ws_f, lp, conf, stream=stream)
        B.surrogate_select(conf, B.SURR_SELECT_BUDGET, 0.0, k, d_idx, a_idx, counts, stream=stream)

    t_plain = timed(plain, 1)
    del ws_f, full
    build, score = prefix_flops(s, Lp, Ls, pid)
    flop_plain = float(flops_per_prompt(s, fl).sum())
    t_pre = t_build + t_score
    return {"workload": w.name, "n_tasks": w.n_tasks, "batch": nb,
            "prefix_tokens": int(Lp.sum()), "suffix_tokens": int(Ls.sum()),
            "concatenated_tokens": int(fl.sum()),
            "lengths": {"prefix": list(w.prefix_lengths), "suffix": list(w.suffix_lengths)},
            "cache_bytes": cache_bytes,
            "pairs_per_s": nb / t_score, "ms_per_step": t_score * 1e3,
            "mfma_frac_of_peak": score / t_score / PEAK_BF16,
            "build_ms": t_build * 1e3,
            "build_mfma_frac_of_peak": build / t_build / PEAK_BF16,
            "pairs_per_s_with_build": nb / t_pre,
            "plain_pairs_per_s": nb / t_plain, "plain_ms_per_step": t_plain * 1e3,
            "plain_mfma_frac_of_peak": flop_plain / t_plain / PEAK_BF16,
            "speedup_vs_plain": t_plain / t_score,
            "speedup_vs_plain_with_build": t_plain / t_pre,
            "concatenated_tokens_per_s": float(fl.sum()) / t_score,
            "note": "pairs_per_s scores every candidate against the resident prefix cache "
                    "(a search reuses a task's prefix across steps); _with_build adds one "
                    "prefix build per batch; plain scores the concatenated prompts"}


def decode_rates(B, torch, dev, model, s, tok_np, L, steps: int = 32,
                 in_flight=(8, 32, 128), prompt_cap: int = 2048) -> dict:
    """Greedy decode throughput against the number of sequences in flight (the paper's
    surrogate reasons before its verdict).  For each P: the first P prompts of the
    workload, cut to prompt_cap tokens, are prefilled into cache entries (untimed); then
    `steps` decode steps, each appending every sequence's greedy token, are timed with
    HIP events.  Algorithmic HBM bytes per step: every weight matrix once, the entries'
    cached keys and values once, the new keys and values written once."""
    d, dq, dkv, ff, nl, V = s.d_model, s.d_q, s.d_kv, s.d_ff, s.n_layers, s.vocab
    esz = 2 if s.dtype == "bf16" else 4
    w_bytes = esz * (nl * (d * (dq + 2 * dkv) + dq * d + 3 * d * ff) + V * d)
    stream = torch.cuda.current_stream()
    out = {"steps": steps, "prompt_cap": prompt_cap, "points": []}
    for P in in_flight:
        Lp = np.minimum(L[:P], prompt_cap).astype(np.int32)
        cache = B.surrogate_cache_create(model, Lp + steps + 4)
        ids = np.arange(P, dtype=np.int32)
        tok = torch.from_numpy(np.ascontiguousarray(tok_np[:P, : int(Lp.max())])).to(dev)
        ws = torch.empty(B.surrogate_workspace_size(model, P, int(Lp.sum()), int(Lp.max())),
                         dtype=torch.uint8, device=dev)
        nxt = torch.empty(P, dtype=torch.int32, device=dev)
        B.surrogate_cache_extend(model, cache, ids, tok, Lp, ws, next_token=nxt, stream=stream)
        del ws
        ws = torch.empty(B.surrogate_workspace_size(model, P, P, 1), dtype=torch.uint8, device=dev)
        ones = np.ones(P, np.int32)
        step_tok = nxt.view(P, 1)

        def step():
            B.surrogate_cache_extend(model, cache, ids, step_tok, ones, ws, next_token=nxt,
                                     stream=stream)

        for _ in range(2):
            step()
        torch.cuda.synchronize()
        ctx0 = Lp.astype(np.float64) + 2
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 1e3 / steps
        kv_read = float(sum((ctx0.sum() + P * i) for i in range(steps))) / steps * nl * 2 * dkv * esz
        kv_write = P * nl * 2 * dkv * esz
        bytes_step = w_bytes + kv_read + kv_write
        out["points"].append({"in_flight": P, "ms_per_step": t * 1e3, "tokens_per_s": P / t,
                              "mean_context": float(ctx0.mean()) + steps / 2,
                              "hbm_bytes_per_step": bytes_step,
                              "achieved_GBps": bytes_step / t / 1e9,
                              "frac_of_hbm": bytes_step / t / PEAK_HBM})
        cache.close()
        del ws, tok
        torch.cuda.empty_cache()
    return out


def forecast_head_rates(B, torch, dev, n: int = 65536, reps: int = 200) -> dict:
    """Latency and achieved HBM rate of the eight-bin forecast head (expected speedup and
    three discovery cutoffs) and of top-quarter selection by expected speedup, on n
    seeded forecasts resident in HBM.  Algorithmic bytes per head call: the forecasts
    (4 n_bins B per row) read once, 4 (1 + n_cutoffs) B per row written."""
    from paper_2605_31464_amd import synth
    nb, cut = 8, (1.25, 1.5, 2.0)
    edges = [2.0 ** e for e in (-2.0, -1.0, -0.5, 0.0, 0.5, 1.0, 2.0)]
    m = [0.17, 0.35, 0.59, 0.84, 1.19, 1.68, 2.83, 5.6]  # open-bin means: synthetic values
    probs = torch.from_numpy(synth.bin_forecasts(n, nb, seed=3)).to(dev)
    sp = torch.empty(n, device=dev)
    disc = torch.empty(n, len(cut), device=dev)
    d_idx = torch.empty(n, dtype=torch.int32, device=dev)
    a_idx = torch.empty(n, dtype=torch.int32, device=dev)
    counts = torch.empty(2, dtype=torch.int32, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3  # microseconds

    us_head = timed(lambda: B.surrogate_forecast_head(probs, m, edges, cut, sp, disc))
    S = torch.from_numpy(np.exp(np.random.default_rng(4).normal(0.0, 1.0, n)).astype(np.float32)).to(dev)
    ws_ev = torch.empty(B.surrogate_evaluate_workspace_size(n, 5), dtype=torch.uint8, device=dev)
    us_eval = timed(lambda: B.surrogate_evaluate(probs, S, m, edges, workspace=ws_ev,
                                                 per_candidate=False))
    us_sel = timed(lambda: B.surrogate_select(sp, B.SURR_SELECT_TOP_SCORE, 0.0, n // 4, d_idx,
                                              a_idx, counts))
    nbytes = n * (4 * nb + 4 * (1 + len(cut)))
    return {"n": n, "n_bins": nb, "n_cutoffs": len(cut), "us_per_call": us_head,
            "bytes": nbytes, "achieved_GBps": nbytes / (us_head * 1e-6) / 1e9,
            "frac_of_hbm": nbytes / (us_head * 1e-6) / PEAK_HBM, "bound": "launch latency",
            "select_top_quarter_us": us_sel,
            "evaluate_us": us_eval,
            "evaluate_note": "rewards, ECE, forecast error and speedup recovered at the five "
                             "budgets of Section 3.1 over the same n forecasts"}


def cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), else the platform's processor."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(shape, W, tok, L, vid, budget_s: float = 25.0) -> dict:
    """Time the float64 oracle on a bounded sample of the same workload: the whole shortest
    prompt of the batch (one of the sampled prompts {0, 1, shortest, longest}), every layer
    and the full-vocabulary head, when one layer's measured time says that fits in
    budget_s; otherwise as many layers as fit, scaled to all of them.  The batch time is
    then extrapolated by the algorithmic FLOP model (flops_per_prompt: linear in tokens
    plus the causal attention triangle), so the quadratic attention cost of the longer
    prompts is counted; the result is labelled as extrapolated."""
    from oracle import transformer as ot
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"] or [os.cpu_count() or 1])
    except Exception:
        threads = os.cpu_count() or 1
    i0 = int(np.argmin(L))
    prompt = tok[i0, : int(L[i0])]
    arch = dict(n_layers=1, d_model=shape.d_model, n_q_heads=shape.n_q_heads,
                n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, d_ff=shape.d_ff,
                vocab=shape.vocab, rope_base=shape.rope_base, rms_eps=shape.rms_eps)
    t0 = time.perf_counter()
    ot.forward_hidden(arch, W, [prompt])
    one = time.perf_counter() - t0
    n_run = max(1, min(shape.n_layers, int(budget_s / max(one, 1e-3))))
    arch["n_layers"] = n_run
    t0 = time.perf_counter()
    xs = ot.forward_hidden(arch, W, [prompt])
    t1 = time.perf_counter()
    z = ot.last_position_logits(arch, W, xs)
    ot.log_softmax_full(z[0])
    t2 = time.perf_counter()
    t_prompt = (t1 - t0) * shape.n_layers / n_run + (t2 - t1)
    f_all = float(flops_per_prompt(shape, L).sum())
    f_one = float(flops_per_prompt(shape, L[i0: i0 + 1]).sum())
    t_batch = t_prompt * f_all / f_one
    what = (f"all {shape.n_layers} layers" if n_run == shape.n_layers else
            f"layers 0-{n_run - 1} of {shape.n_layers}, scaled to all of them")
    return {"value": len(L) / t_batch, "unit": "pairs/s", "cores": int(threads), "kind": "oracle",
            "sample": f"float64 oracle on the whole of prompt {i0} (the shortest, {len(prompt)} "
                      f"tokens; {what}) plus its full-vocabulary head: {t2 - t0:.1f} s measured, "
                      f"{t_prompt:.1f} s per prompt; batch time extrapolated by the algorithmic "
                      f"FLOP model over all {len(L)} prompts",
            "extrapolated": True, "measured_s": t2 - t0, "prompt_s": t_prompt,
            "tokens_per_s": float(L.sum()) / t_batch, "cpu": cpu_model()}


TRAFFIC_REPORT = os.path.join(ROOT, "profiles", "gemm_gate_up_{config}_traffic.md")
GEMM_SOURCE = os.path.join(ROOT, "paper_2605_31464_amd", "csrc", "k_gemm.hip")


def measured_traffic(config: str):
    """HBM bytes per launch of the gate/up GEMM from the committed rocprofv3 counter
    report, or None when there is none or the GEMM source changed since it was taken."""
    from paper_2605_31464_amd.rocprof_summary import source_sha256
    path = TRAFFIC_REPORT.format(config=config)
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("bench-traffic:"):
            _, val, sha = line.split()
            return float(val) if sha == source_sha256(GEMM_SOURCE) else None
    return None


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="7b", help="tiny | small | 1p5b | 7b | 14b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the per-phase HIP-event timing (the roofline block)")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode-throughput section (7B shape only)")
    ap.add_argument("--no-prefix", action="store_true",
                    help="skip the shared-prefix workload (7B shape only)")
    ap.add_argument("--no-forecast-head", action="store_true",
                    help="skip timing the eight-bin forecast head and top-score selection")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one device-to-device copy of this size first (reference "
                         "dispatch for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build scores on exactly one GPU; runs with --gpus above 1 are "
              "not supported (prompts shard by data parallelism, which is not built here).",
              file=sys.stderr)
        return 2

    import torch
    from paper_2605_31464_amd import binding as B
    from paper_2605_31464_amd import synth

    w = synth.CONFIGS[args.config]
    s = w.shape
    t_setup = time.perf_counter()
    W = synth.make_weights(s)
    names = [x[0] for x in synth.tensor_specs(s)]
    tok_np, L = synth.make_prompts(w)
    vid = synth.verdict_ids(w)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = B.make_config(s)
    model = B.surrogate_load_weights_tensors(cfg, [W[n] for n in names])
    B_ = len(L)
    T = int(L.sum())
    tok = torch.from_numpy(tok_np).to(dev)
    ws = torch.empty(B.surrogate_workspace_size(model, B_, T, int(L.max())), dtype=torch.uint8,
                     device=dev)
    nv = len(vid)
    lp = torch.empty(B_, nv, device=dev)
    p = torch.empty(B_, nv, device=dev)
    conf = torch.empty(B_, device=dev)
    verdict = torch.empty(B_, dtype=torch.int32, device=dev)
    d_idx = torch.empty(B_, dtype=torch.int32, device=dev)
    a_idx = torch.empty(B_, dtype=torch.int32, device=dev)
    counts = torch.empty(2, dtype=torch.int32, device=dev)
    if w.select[0] == "budget":
        mode, tau, k = B.SURR_SELECT_BUDGET, 0.0, w.budget_k
    else:
        mode, tau, k = B.SURR_SELECT_THRESHOLD, w.select[1], 0
    stream = torch.cuda.current_stream()
    print(f"[bench] {w.name}: B={B_} T={T} setup {time.perf_counter() - t_setup:.1f}s",
          file=sys.stderr, flush=True)

    if args.copy_calibration_mib:
        src = torch.ones(args.copy_calibration_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step():
        B.surrogate_score_pairs(model, tok, L, vid, ws, lp, conf, p, verdict, stream=stream)
        B.surrogate_select(conf, mode, tau, k, d_idx, a_idx, counts, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if B.surrogate_device_status(model) != B.SURR_OK:
        raise RuntimeError("device error during warm-up")
    if not args.no_profile:
        B.surrogate_profile_enable(model, True)
        B.surrogate_profile_collect(model)  # start from zero
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step()
        print(f"[bench] step {i + 1}/{args.steps} enqueued", file=sys.stderr, flush=True)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_s = ev0.elapsed_time(ev1) / 1e3
    phases = B.surrogate_profile_collect(model) if not args.no_profile else {}
    B.surrogate_profile_enable(model, False)

    t_step = gpu_s / args.steps
    flop = float(flops_per_prompt(s, L).sum())
    out = {
        "metric": METRIC,
        "value": B_ / t_step,
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if s.dtype == "bf16" else "f32",
        "data": "synthetic (seeded Zipf(1.1) prompts, N(0,0.02) weights)",
        "config": {"workload": w.name, "batch": B_, "total_tokens": T,
                   "lengths": list(w.lengths), "n_verdict": nv,
                   "select": f"{w.select[0]} {k if w.select[0] == 'budget' else tau}"},
        "prefill_tokens_per_s": T / t_step,
        "mfma_frac_of_peak": flop / t_step / PEAK_BF16,
        "algorithmic_tflop_per_step": flop / 1e12,
        "wall_s_timed": wall,
    }
    if phases:
        out["phases_ms_per_step"] = {ph: ms / args.steps for ph, (ms, n) in phases.items() if n}
        # Dominant kernel: the gate/up projection with its SwiGLU epilogue, one launch per
        # non-final layer over all T tokens: 2 * T * (2 d_ff) * d_model FLOP per launch.
        ms, n = phases["gemm_gate_up"]
        if n:
            per_launch = 2.0 * T * (2 * s.d_ff) * s.d_model
            avg_s = ms / n / 1e3
            ach = per_launch / avg_s
            out["roofline"] = {"kernel": "gemm_bf16 SwiGLU epilogue (gate/up projection)",
                               "bound": "mfma", "achieved": ach / 1e12,
                               "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                               "frac": ach / PEAK_BF16,
                               "traffic": measured_traffic(args.config),
                               "avg_launch_ms": avg_s * 1e3, "launches": n}
        out["phase_rates"] = phase_rates(s, L.astype(np.int64), phases, args.steps)
    if not args.no_forecast_head:
        out["forecast_head"] = forecast_head_rates(B, torch, dev)
    if not args.no_decode and args.config == "7b":
        print("[bench] decode throughput", file=sys.stderr, flush=True)
        if "ws" in locals():
            del ws
        torch.cuda.empty_cache()
        out["decode"] = decode_rates(B, torch, dev, model, s, tok_np, L)
    if not args.no_prefix and args.config == "7b":
        print("[bench] shared-prefix workload", file=sys.stderr, flush=True)
        if "ws" in locals():
            del ws
        torch.cuda.empty_cache()
        out["prefix_reuse"] = prefix_reuse_rates(B, torch, dev, model, max(1, min(args.steps, 3)),
                                                 1)
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on a bounded sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(s, W, tok_np, L, vid)
    print(json.dumps(out), flush=True)
    B.surrogate_free(model)
    return 0


if __name__ == "__main__":
    sys.exit(main())
