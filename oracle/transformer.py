"""Float64 decoder forward and forecast read-out (test infrastructure, see package doc).

The forecast follows Section 2.1 of the paper: the surrogate produces a distribution
p_i over verdicts (p_{i,b} >= 0, sum_b p_{i,b} = 1), the predicted bin is its argmax
and the confidence is q_i = max_b p_{i,b}.  Here p_i is read from the model's next-
token log-probabilities of a fixed set of verdict tokens at the last prompt position
(prefill-only scoring), renormalised over those tokens.

The decoder is the standard pre-norm dense transformer: RMSNorm, rotate-half RoPE,
causal grouped-query attention, SwiGLU MLP, final RMSNorm and an untied LM head,
without biases.  ``arch`` is a mapping with keys n_layers, d_model, n_q_heads,
n_kv_heads, head_dim, d_ff, vocab, rope_base, rms_eps.  ``weights`` maps the tensor
names (embed, layers.<l>.{attn_norm,w_q,w_k,w_v,w_o,mlp_norm,w_gate,w_up,w_down},
final_norm, lm_head) to arrays; uint16 arrays hold bfloat16 bit patterns and are
decoded exactly, everything else is converted with astype(float64).  Matrices are
[out, in], so a projection is h @ W.T.
"""
from __future__ import annotations

import numpy as np


def to_f64(a) -> np.ndarray:
    """Exact float64 value of a weight array (bfloat16 bit patterns or any float)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g along the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope_angles(positions: np.ndarray, head_dim: int, base: float) -> np.ndarray:
    """theta[j, i] = pos_j * base^(-2i/head_dim), i < head_dim/2."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / head_dim)
    return np.asarray(positions, np.float64)[:, None] * inv_freq[None, :]


def apply_rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half RoPE on x[L, heads, hd]: dims (i, i + hd/2) rotate by theta_i."""
    hd = x.shape[-1]
    half = hd // 2
    th = rope_angles(positions, hd, base)[:, None, :]
    c, s = np.cos(th), np.sin(th)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def causal_softmax_rows(scores: np.ndarray) -> np.ndarray:
    """Row j of the result is the exact softmax of scores[j, :j+1]; columns m > j are
    excluded (their probability is exactly 0)."""
    L = scores.shape[0]
    future = np.triu(np.ones((L, L), dtype=bool), 1)
    s = np.where(future, -np.inf, scores)
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Causal GQA attention.  q[L, n_q, hd], k/v[L, n_kv, hd] -> o[L, n_q, hd].
    Query head a reads kv head floor(a * n_kv / n_q) (consecutive groups)."""
    L, n_q, hd = q.shape
    n_kv = k.shape[1]
    o = np.empty_like(q)
    for a in range(n_q):
        c = (a * n_kv) // n_q
        p = causal_softmax_rows(q[:, a, :] @ k[:, c, :].T / np.sqrt(hd))
        o[:, a, :] = p @ v[:, c, :]
    return o


def silu(z: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def layer_weights(weights, layer: int) -> dict:
    p = f"layers.{layer}."
    return {n: to_f64(weights[p + n]) for n in
            ("attn_norm", "w_q", "w_k", "w_v", "w_o", "mlp_norm", "w_gate", "w_up", "w_down")}


def decoder_layer(arch, lw: dict, x: np.ndarray) -> np.ndarray:
    """One pre-norm layer on the residual x[L, d] of a single prompt (positions 0..L-1)."""
    L = x.shape[0]
    hd, nq, nkv = arch["head_dim"], arch["n_q_heads"], arch["n_kv_heads"]
    pos = np.arange(L)
    h = rms_norm(x, lw["attn_norm"], arch["rms_eps"])
    q = (h @ lw["w_q"].T).reshape(L, nq, hd)
    k = (h @ lw["w_k"].T).reshape(L, nkv, hd)
    v = (h @ lw["w_v"].T).reshape(L, nkv, hd)
    q = apply_rope(q, pos, arch["rope_base"])
    k = apply_rope(k, pos, arch["rope_base"])
    o = causal_attention(q, k, v).reshape(L, nq * hd)
    x = x + o @ lw["w_o"].T
    h = rms_norm(x, lw["mlp_norm"], arch["rms_eps"])
    u = silu(h @ lw["w_gate"].T) * (h @ lw["w_up"].T)
    return x + u @ lw["w_down"].T


def forward_hidden(arch, weights, prompts) -> list:
    """Final residual stream x[L_i, d] of every prompt (before the final norm).

    Prompts are independent; the loop runs layer by layer so each weight matrix is
    converted to float64 once per call."""
    E = to_f64(weights["embed"])
    prompts = [np.asarray(t, np.int64) for t in prompts]
    for t in prompts:
        if t.ndim != 1 or t.size == 0 or t.min() < 0 or t.max() >= E.shape[0]:
            raise ValueError("each prompt needs >= 1 token id in [0, vocab)")
    xs = [E[t] for t in prompts]
    del E
    for l in range(arch["n_layers"]):
        lw = layer_weights(weights, l)
        xs = [decoder_layer(arch, lw, x) for x in xs]
    return xs


def log_softmax_full(z: np.ndarray) -> np.ndarray:
    m = z.max()
    return z - (m + np.log(np.sum(np.exp(z - m))))


def last_position_logits(arch, weights, xs) -> np.ndarray:
    """z_i = W_head . RMSNorm(x_i[L_i - 1]) for every prompt -> [B, V]."""
    g = to_f64(weights["final_norm"])
    y = np.stack([rms_norm(x[-1], g, arch["rms_eps"]) for x in xs])
    return y @ to_f64(weights["lm_head"]).T


def next_token_log_softmax(arch, weights, tokens, positions) -> np.ndarray:
    """Full-vocabulary log-softmax of the next-token logits after each of `positions`
    of one token sequence: row r is log p(. | tokens[0 .. positions[r]]).  The causal
    forward makes every row the last-position read-out of the corresponding prefix."""
    x = forward_hidden(arch, weights, [tokens])[0]
    g = to_f64(weights["final_norm"])
    y = np.stack([rms_norm(x[j], g, arch["rms_eps"]) for j in positions])
    z = y @ to_f64(weights["lm_head"]).T
    return np.stack([log_softmax_full(zi) for zi in z])


def forecast(lp: np.ndarray) -> dict:
    """Verdict log-probs lp[B, n] -> p (renormalised), confidence q = max p,
    predicted verdict = first argmax, and the top-1 minus top-2 log-prob margin."""
    lp = np.atleast_2d(lp)
    m = lp.max(axis=1, keepdims=True)
    e = np.exp(lp - m)
    p = e / e.sum(axis=1, keepdims=True)
    q = p.max(axis=1)
    yhat = np.argmax(p, axis=1).astype(np.int32)
    if lp.shape[1] >= 2:
        srt = np.sort(lp, axis=1)
        margin = srt[:, -1] - srt[:, -2]
    else:
        margin = np.full(lp.shape[0], np.inf)
    return {"p": p, "confidence": q, "verdict": yhat, "margin": margin}


def score(arch, weights, prompts, verdict_ids) -> dict:
    """Full-vocab log-probs of the verdict tokens at each prompt's last position,
    plus the forecast read-out.  prompts: list of 1-D token arrays."""
    xs = forward_hidden(arch, weights, prompts)
    z = last_position_logits(arch, weights, xs)
    lp_full = np.stack([log_softmax_full(zi) for zi in z])
    lp = lp_full[:, np.asarray(verdict_ids)]
    out = forecast(lp)
    out["logprobs"] = lp
    return out
