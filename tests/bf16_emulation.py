"""Float64 model of the bf16 path's storage roundings: the error floor of the bf16 configs.

TEST INFRASTRUCTURE ONLY (imported by ``tests/``).  It shares no code with the HIP path
and does not import the oracle.

The bf16 configurations compute in float32 but store intermediate tensors in bfloat16
wherever a tensor feeds a bf16 matrix product: the attention-norm output, q and k after
RoPE and v, the attention probabilities of the P V product, the attention output, the
MLP-norm output, the SwiGLU output and the final hidden state.  The residual stream is
stored in float32; the row sum of the attention probabilities, norms, softmax and
log-sum-exp are float32 arithmetic.  This module runs the decoder forward in float64 and
rounds exactly at those storage points (to float32 first, as the kernels round their
float32 accumulators, then to bfloat16 with round-to-nearest-even; float32 for the
residual stream).  Nothing else is rounded.  Its error against the exact float64 forward
is therefore the error that the bf16 storage by itself causes: a kernel with these
storage types cannot do better, whatever its summation order.

A single run gives one sample of that error.  Another correct bf16 path rounds the same
values at the same points, so the structured part of the error (which way a given value
rounds) is shared; it differs in float32 noise (summation order, a hardware exp), which
flips the roundings of values that lie near a rounding boundary, and in the scale at which
it rounds the attention probabilities: the kernel keeps them relative to a running maximum
that it updates lazily, i.e. multiplied by a per-row factor that is not a power of two.
``members`` selects an ensemble of such runs: member 0 rounds the exact values to nearest
even; member k > 0, from a generator seeded with k, first multiplies every value it rounds
by (1 + 2^-16 u) with u uniform in [-1, 1) (float32-sized noise; the roundings stay
nearest-even), and rounds each row of attention probabilities at a scale 2^v, v uniform in
[0, 1) per row (the rounded row is divided by the scale again).

With ``rounding=False`` the module computes the exact forward; a CPU test pins that mode
to the float64 oracle.
"""
from __future__ import annotations

import math

import numpy as np
import torch

PERTURB = 2.0 ** -16



def weight_tensor(a, device) -> torch.Tensor:
    """float64 tensor of a weight array (uint16 = bfloat16 bit patterns, else float)."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
        return t.to(device).to(torch.float64)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).to(device)


class _Rounder:
    """Storage roundings of one ensemble member."""

    def __init__(self, member: int, device, rounding: bool):
        self.rounding = rounding
        self.gen = None
        if rounding and member > 0:
            self.gen = torch.Generator(device=device)
            self.gen.manual_seed(member)

    @staticmethod
    def _rne(x):
        return x.to(torch.float32).to(torch.bfloat16).to(torch.float64)

    def _uniform(self, shape, device):
        return torch.rand(shape, generator=self.gen, device=device, dtype=torch.float64)

    def bf16(self, x):
        if not self.rounding:
            return x
        if self.gen is None:
            return self._rne(x)
        return self._rne(x * (1.0 + PERTURB * (2.0 * self._uniform(x.shape, x.device) - 1.0)))

    def bf16_rows(self, p):
        """Attention probabilities p[rows, keys], each row rounded at its own scale."""
        if not self.rounding or self.gen is None:
            return self.bf16(p)
        scale = torch.exp2(self._uniform((p.shape[0], 1), p.device))
        return self.bf16(p * scale) / scale

    def f32(self, x):
        if not self.rounding:
            return x
        return x.to(torch.float32).to(torch.float64)


def _rms_norm(x, g, eps):
    return x / torch.sqrt((x * x).mean(dim=-1, keepdim=True) + eps) * g


def _rope(x, base):
    """Rotate-half RoPE on x[L, heads, hd] at positions 0..L-1."""
    L, _, hd = x.shape
    half = hd // 2
    i = torch.arange(half, dtype=torch.float64, device=x.device)
    th = torch.arange(L, dtype=torch.float64, device=x.device)[:, None] * base ** (-2.0 * i / hd)
    c, s = torch.cos(th)[:, None, :], torch.sin(th)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], dim=-1)


def _attention(q, k, v, R):
    """Causal GQA attention with the probabilities stored in bf16 for the P V product
    and their row sum kept unrounded.  q[L, nq, hd], k/v[L, nkv, hd]."""
    L, nq, hd = q.shape
    nkv = k.shape[1]
    future = torch.ones(L, L, dtype=torch.bool, device=q.device).triu(1)
    o = torch.empty_like(q)
    for a in range(nq):
        c = (a * nkv) // nq
        s = (q[:, a, :].contiguous() @ k[:, c, :].T.contiguous()) / math.sqrt(hd)
        s.masked_fill_(future, -math.inf)
        pf = torch.exp(s - s.amax(dim=1, keepdim=True))
        l = pf.sum(dim=1, keepdim=True)
        o[:, a, :] = (R.bf16_rows(pf) @ v[:, c, :].contiguous()) / l
        del s, pf
    return o


class Bf16Emulation:
    """arch: mapping with n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab,
    rope_base, rms_eps.  weights: tensor name -> numpy array (the synthetic generator's
    layout: embed, layers.<l>.{attn_norm, w_q, w_k, w_v, w_o, mlp_norm, w_gate, w_up,
    w_down}, final_norm, lm_head; matrices [out, in])."""

    def __init__(self, arch, weights, device="cpu", rounding=True):
        self.arch, self.W, self.device, self.rounding = arch, weights, device, rounding

    def _w(self, name):
        return weight_tensor(self.W[name], self.device)

    def _layer(self, lw, x, R):
        a = self.arch
        L = x.shape[0]
        hd, nq, nkv = a["head_dim"], a["n_q_heads"], a["n_kv_heads"]
        h = R.bf16(_rms_norm(x, lw["attn_norm"], a["rms_eps"]))
        q = R.bf16(_rope((h @ lw["w_q"].T).reshape(L, nq, hd), a["rope_base"]))
        k = R.bf16(_rope((h @ lw["w_k"].T).reshape(L, nkv, hd), a["rope_base"]))
        v = R.bf16((h @ lw["w_v"].T).reshape(L, nkv, hd))
        o = R.bf16(_attention(q, k, v, R).reshape(L, nq * hd))
        del q, k, v
        x = R.f32(x + o @ lw["w_o"].T)
        h = R.bf16(_rms_norm(x, lw["mlp_norm"], a["rms_eps"]))
        g = h @ lw["w_gate"].T
        u = R.bf16(g / (1.0 + torch.exp(-g)) * (h @ lw["w_up"].T))
        del g, h
        return R.f32(x + u @ lw["w_down"].T)

    @torch.no_grad()
    def score(self, prompts, verdict_ids, members=(0,), progress=False):
        """Verdict log-probs (full-vocabulary log-softmax at the last position) and their
        renormalised distribution for every prompt and ensemble member.
        Returns {"logprobs": [M, B, n], "p": [M, B, n]} as float64 numpy arrays.
        progress: print a line after every layer."""
        a = self.arch
        E = self._w("embed")
        toks = [torch.as_tensor(np.asarray(t, np.int64), device=self.device) for t in prompts]
        Rs = [_Rounder(m, self.device, self.rounding) for m in members]
        xs = [[E[t].clone() for t in toks] for _ in members]
        del E
        for l in range(a["n_layers"]):
            p = f"layers.{l}."
            lw = {n: self._w(p + n) for n in ("attn_norm", "w_q", "w_k", "w_v", "w_o",
                                              "mlp_norm", "w_gate", "w_up", "w_down")}
            for mi, R in enumerate(Rs):
                xs[mi] = [self._layer(lw, x, R) for x in xs[mi]]
            del lw
            if progress:
                print(f"emulation: layer {l + 1}/{a['n_layers']} done ({len(Rs)} members, "
                      f"{len(toks)} prompts)", flush=True)
        g = self._w("final_norm")
        head = self._w("lm_head")
        vid = torch.as_tensor(np.asarray(verdict_ids, np.int64), device=self.device)
        lps, ps = [], []
        for mi, R in enumerate(Rs):
            y = R.bf16(torch.stack([_rms_norm(x[-1], g, a["rms_eps"]) for x in xs[mi]]))
            z = y @ head.T
            lp = (z - torch.logsumexp(z, dim=1, keepdim=True))[:, vid]
            lps.append(lp)
            ps.append(torch.softmax(lp, dim=1))
        return {"logprobs": torch.stack(lps).cpu().numpy(), "p": torch.stack(ps).cpu().numpy()}
