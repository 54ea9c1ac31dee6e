"""Seeded synthetic inputs for batched forecast scoring: model shapes, weights, prompts.

This module only *draws data*.  It holds none of the scoring arithmetic, so both the
HIP path and the float64 oracle can consume its outputs without sharing code.

Workloads stand in for the paper's kernel-pair prompts (the forecast query
x_i = (reference kernel, candidate kernel, hardware) of Section 2.1): the prompt text
itself is not available, so prompts are i.i.d. Zipf(1.1) token streams with the
length mixes below, and the decoder weights are random.

Definitions (fixed here so every consumer gets identical bytes):

* Weights.  Tensor number ``i`` in :func:`tensor_specs` order is drawn in flat
  row-major chunks of ``CHUNK`` elements; chunk ``c`` comes from
  ``PCG64(SeedSequence(seed, spawn_key=(i, c)))`` via ``standard_normal(float32)``,
  multiplied by ``0.02`` in float32.  bf16 models round that float32 value to
  bfloat16 (round to nearest even) and store the 16-bit patterns as ``uint16``.
  Norm gains are float32 ones, or ``1 + gain_std * N(0, 1)`` when ``gain_std > 0``.
* Prompts.  ``default_rng(seed)`` draws the lengths first, then the tokens of all
  prompts back to back.  Uniform lengths are inclusive integers; lognormal lengths are
  ``clip(rint(exp(N(ln median, sigma^2))), lo, hi)``.  Token ranks follow a finite
  Zipf law P(r) proportional to r^-1.1, r = 1..V, sampled by inverse CDF; token id =
  r - 1.  Verdict ids are the last ``n_verdict`` ids of the vocabulary.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

CHUNK = 1 << 22


@dataclasses.dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    max_pos: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-6
    dtype: str = "bf16"  # "f32" or "bf16": storage and GEMM-input type

    @property
    def d_q(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def d_kv(self) -> int:
        return self.n_kv_heads * self.head_dim

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: ModelShape
    batch: int
    lengths: tuple  # ("uniform", lo, hi) or ("lognormal", median, sigma, lo, hi)
    n_verdict: int
    select: tuple  # ("threshold", tau) or ("budget", fraction_of_batch)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def budget_k(self) -> int:
        """Deferral budget k = floor(fraction * batch) (never above the budget)."""
        if self.select[0] != "budget":
            raise ValueError("workload uses threshold selection")
        return int(math.floor(self.select[1] * self.batch))


CONFIGS = {
    "tiny": Workload(
        "tiny-fp32-2L-d128",
        ModelShape(2, 128, 4, 4, 32, 352, 512, 1024, dtype="f32"),
        4, ("uniform", 64, 256), 2, ("threshold", 0.7)),
    "small": Workload(
        "small-0.5B-bf16-24L-d896",
        ModelShape(24, 896, 14, 2, 64, 4864, 32768, 4096),
        32, ("uniform", 512, 2048), 2, ("budget", 0.25)),
    "1p5b": Workload(
        "1.5B-bf16-28L-d1536",
        ModelShape(28, 1536, 12, 2, 128, 8960, 65536, 8192),
        64, ("lognormal", 2048, 0.5, 512, 6144), 5, ("threshold", 0.6)),
    "7b": Workload(
        "7B-bf16-28L-d3584-b128",
        ModelShape(28, 3584, 28, 4, 128, 18944, 131072, 8192),
        128, ("lognormal", 3072, 0.5, 1024, 8192), 2, ("budget", 0.20)),
    "14b": Workload(
        "14B-bf16-48L-d5120-b32",
        ModelShape(48, 5120, 40, 8, 128, 13824, 131072, 16384),
        32, ("uniform", 8192, 16384), 5, ("threshold", 0.8)),
}


def layer_tensor_names(layer: int) -> list:
    p = f"layers.{layer}."
    return [p + n for n in ("attn_norm", "w_q", "w_k", "w_v", "w_o",
                            "mlp_norm", "w_gate", "w_up", "w_down")]


def tensor_specs(shape: ModelShape) -> list:
    """Canonical tensor order: (name, rows, cols, is_norm).  Matrices are [out, in]."""
    d, dq, dkv, ff, V = shape.d_model, shape.d_q, shape.d_kv, shape.d_ff, shape.vocab
    specs = [("embed", V, d, False)]
    for l in range(shape.n_layers):
        n = layer_tensor_names(l)
        specs += [(n[0], 1, d, True), (n[1], dq, d, False), (n[2], dkv, d, False),
                  (n[3], dkv, d, False), (n[4], d, dq, False), (n[5], 1, d, True),
                  (n[6], ff, d, False), (n[7], ff, d, False), (n[8], d, ff, False)]
    specs += [("final_norm", 1, d, True), ("lm_head", V, d, False)]
    return specs


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (torch's CPU cast)."""
    import torch
    return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _fill_chunk(out_flat, tensor_index, chunk, seed, bf16, scale, offset):
    lo = chunk * CHUNK
    hi = min(lo + CHUNK, out_flat.size)
    g = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence(seed, spawn_key=(tensor_index, chunk))))
    v = g.standard_normal(hi - lo, dtype=np.float32)
    v *= np.float32(scale)
    if offset:
        v += np.float32(offset)
    out_flat[lo:hi] = _to_bf16_bits(v) if bf16 else v


def make_weights(shape: ModelShape, seed: int = 0, gain_std: float = 0.0,
                 threads: int | None = None, std: float = 0.02) -> dict:
    """All model tensors as numpy arrays (uint16 bf16 bits or float32), by name."""
    specs = tensor_specs(shape)
    bf16 = shape.dtype == "bf16"
    out, jobs = {}, []
    for i, (name, rows, cols, is_norm) in enumerate(specs):
        if is_norm:
            a = np.ones(cols, np.float32)
            if gain_std > 0:
                jobs += [(a, i, c, seed, False, gain_std, 1.0)
                         for c in range(-(-a.size // CHUNK))]
        else:
            a = np.empty((rows, cols), np.uint16 if bf16 else np.float32)
            jobs += [(a.reshape(-1), i, c, seed, bf16, std, 0.0)
                     for c in range(-(-a.size // CHUNK))]
        out[name] = a
    n = threads or min(16, os.cpu_count() or 1)
    import torch
    prev = torch.get_num_threads()
    torch.set_num_threads(1)  # parallelism comes from the chunk workers
    try:
        with ThreadPoolExecutor(n) as ex:
            for f in [ex.submit(_fill_chunk, *j) for j in jobs]:
                f.result()
    finally:
        torch.set_num_threads(prev)
    return out


FILE_MAGIC = b"SURRWGT1"
FILE_ALIGN = 4096


def file_tensors(shape: ModelShape, weights: dict) -> list:
    """(name, dtype, shape, array) of every tensor in weight-file order: the per-layer
    q, k and v matrices are stored as one w_qkv matrix (q rows, then k, then v)."""
    dt = shape.dtype
    out = [("embed", dt, list(weights["embed"].shape), weights["embed"])]
    for l in range(shape.n_layers):
        p = f"layers.{l}."
        qkv = np.concatenate([weights[p + "w_q"], weights[p + "w_k"], weights[p + "w_v"]], axis=0)
        out += [(p + "attn_norm", "f32", [shape.d_model], weights[p + "attn_norm"]),
                (p + "w_qkv", dt, list(qkv.shape), qkv),
                (p + "w_o", dt, list(weights[p + "w_o"].shape), weights[p + "w_o"]),
                (p + "mlp_norm", "f32", [shape.d_model], weights[p + "mlp_norm"])]
        out += [(p + n, dt, list(weights[p + n].shape), weights[p + n])
                for n in ("w_gate", "w_up", "w_down")]
    out += [("final_norm", "f32", [shape.d_model], weights["final_norm"]),
            ("lm_head", dt, list(weights["lm_head"].shape), weights["lm_head"])]
    return out


def write_weight_file(path, shape: ModelShape, weights: dict) -> None:
    """Write a weight file: the magic, the header length (uint64 little-endian), the JSON
    header (config and tensor table), then each tensor's raw little-endian bytes at an
    offset that is a multiple of 4096 (bf16 as 16-bit patterns, f32 as IEEE floats)."""
    import json
    entries = file_tensors(shape, weights)
    config = {"n_layers": shape.n_layers, "d_model": shape.d_model,
              "n_q_heads": shape.n_q_heads, "n_kv_heads": shape.n_kv_heads,
              "head_dim": shape.head_dim, "d_ff": shape.d_ff, "vocab": shape.vocab,
              "max_pos": shape.max_pos, "rope_base": float(shape.rope_base),
              "rms_eps": float(shape.rms_eps), "dtype": shape.dtype}

    def header(start):
        table, off = [], start
        for name, dt, shp, a in entries:
            table.append({"name": name, "dtype": dt, "shape": shp, "offset": off})
            off += -(-np.asarray(a).nbytes // FILE_ALIGN) * FILE_ALIGN
        return json.dumps({"format": "surrogate-weights", "version": 1, "config": config,
                           "tensors": table}).encode("ascii")

    start = FILE_ALIGN
    while True:  # the first tensor starts at the first 4096 boundary past the header
        h = header(start)
        need = -(-(16 + len(h)) // FILE_ALIGN) * FILE_ALIGN
        if need == start:
            break
        start = need
    with open(path, "wb") as f:
        f.write(FILE_MAGIC + len(h).to_bytes(8, "little") + h)
        for (name, dt, shp, a), t in zip(entries, json.loads(h)["tensors"]):
            a = np.ascontiguousarray(a, np.float32 if dt == "f32" else np.uint16)
            if a.size != int(np.prod(shp)):
                raise ValueError(f"{name}: {a.size} elements, shape {shp}")
            f.seek(t["offset"])
            f.write(a.astype(a.dtype.newbyteorder("<"), copy=False).tobytes())


def zipf_cdf(vocab: int, s: float = 1.1) -> np.ndarray:
    r = np.arange(1, vocab + 1, dtype=np.float64)
    c = np.cumsum(r ** -s)
    return c / c[-1]


def draw_lengths(w: Workload, rng: np.random.Generator) -> np.ndarray:
    spec = w.lengths
    if spec[0] == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=w.batch).astype(np.int32)
    if spec[0] == "lognormal":
        _, median, sigma, lo, hi = spec
        raw = np.exp(rng.normal(math.log(median), sigma, size=w.batch))
        return np.clip(np.rint(raw), lo, hi).astype(np.int32)
    raise ValueError(spec)


def make_prompts(w: Workload, seed: int = 1, pad: int = 0, lengths=None):
    """Padded token matrix [B, Lmax] int32 and lengths [B] int32."""
    rng = np.random.default_rng(seed)
    L = draw_lengths(w, rng) if lengths is None else np.asarray(lengths, np.int32)
    cdf = zipf_cdf(w.shape.vocab)
    ids = np.searchsorted(cdf, rng.random(int(L.sum())), side="right")
    ids = np.minimum(ids, w.shape.vocab - 1).astype(np.int32)
    tok = np.full((len(L), int(L.max())), pad, np.int32)
    off = 0
    for b, n in enumerate(L):
        tok[b, :n] = ids[off:off + n]
        off += n
    return tok, L


def verdict_ids(w: Workload) -> np.ndarray:
    V = w.shape.vocab
    return np.arange(V - w.n_verdict, V, dtype=np.int32)


def bin_forecasts(n: int, n_bins: int = 8, seed: int = 2) -> np.ndarray:
    """Forecast distributions over speedup bins, float32 [n, n_bins].

    Row i is a Dirichlet draw with all concentrations equal to alpha_i, where
    log10(alpha_i) is uniform on [-1, 1]: small alpha gives peaked forecasts, large
    alpha nearly flat ones.  ``default_rng(seed)`` draws the alphas, then the rows.
    """
    rng = np.random.default_rng(seed)
    alpha = 10.0 ** rng.uniform(-1.0, 1.0, size=n)
    g = rng.gamma(alpha[:, None], 1.0, size=(n, n_bins))
    g = np.maximum(g, 1e-30)
    return (g / g.sum(axis=1, keepdims=True)).astype(np.float32)


@dataclasses.dataclass(frozen=True)
class PrefixWorkload:
    """Candidates that share per-task prompt prefixes (the system prompt plus the task's
    reference kernel), each followed by its own candidate suffix."""
    name: str
    shape: ModelShape
    n_tasks: int
    batch: int
    prefix_lengths: tuple  # ("lognormal", median, sigma, lo, hi) or ("uniform", lo, hi)
    suffix_lengths: tuple
    n_verdict: int


PREFIX_CONFIGS = {
    "7b-prefix": PrefixWorkload("7B-bf16-shared-prefix", CONFIGS["7b"].shape, 6, 128,
                                ("lognormal", 2048, 0.5, 1024, 4096),
                                ("lognormal", 1024, 0.5, 256, 4096), 2),
}


def _draw(spec, n, rng):
    if spec[0] == "uniform":
        return rng.integers(spec[1], spec[2] + 1, size=n).astype(np.int32)
    _, median, sigma, lo, hi = spec
    return np.clip(np.rint(np.exp(rng.normal(math.log(median), sigma, size=n))), lo, hi).astype(np.int32)


def make_prefix_prompts(w: PrefixWorkload, seed: int = 1):
    """(prefix tokens [G, Pmax], prefix lengths [G], suffix tokens [B, Smax], suffix lengths
    [B], prefix id of each candidate [B]).  ``default_rng(seed)`` draws the prefix lengths,
    the suffix lengths, then all prefix tokens and all suffix tokens back to back (Zipf(1.1)
    ranks as in make_prompts); candidate i belongs to task i mod G."""
    rng = np.random.default_rng(seed)
    V = w.shape.vocab
    Lp = _draw(w.prefix_lengths, w.n_tasks, rng)
    Ls = _draw(w.suffix_lengths, w.batch, rng)
    cdf = zipf_cdf(V)

    def tokens(L):
        ids = np.minimum(np.searchsorted(cdf, rng.random(int(L.sum())), side="right"), V - 1)
        tok = np.zeros((len(L), int(L.max())), np.int32)
        off = 0
        for b, n in enumerate(L):
            tok[b, :n] = ids[off:off + n]
            off += n
        return tok

    ptok = tokens(Lp)
    stok = tokens(Ls)
    pid = (np.arange(w.batch) % w.n_tasks).astype(np.int32)
    return ptok, Lp, stok, Ls, pid


def concat_prompts(ptok, Lp, stok, Ls, pid):
    """Padded [B, max(Lp[pid] + Ls)] matrix of the full prompts prefix ++ suffix (-1: none)."""
    full_len = np.array([(Lp[g] if g >= 0 else 0) + n for g, n in zip(pid, Ls)], np.int32)
    tok = np.zeros((len(Ls), int(full_len.max())), np.int32)
    for i, (g, n) in enumerate(zip(pid, Ls)):
        p = int(Lp[g]) if g >= 0 else 0
        if p:
            tok[i, :p] = ptok[g, :p]
        tok[i, p:p + n] = stok[i, :n]
    return tok, full_len
