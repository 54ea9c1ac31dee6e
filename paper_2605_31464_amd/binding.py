"""ctypes binding of libsurrogate.so: the C ABI of include/surrogate.h under the same names.

Argument marshalling only: torch tensors supply device memory and the current HIP
stream; every step of scoring and selection runs in the library's HIP kernels.  There
is no CPU fallback - loading fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libsurrogate.so")

SURR_OK = 0
SURR_E_INVALID_ARG = -1
SURR_E_SHAPE = -2
SURR_E_TOKEN_RANGE = -3
SURR_E_OOM = -4
SURR_E_HIP = -5
SURR_E_WEIGHTS = -6
SURR_E_WORKSPACE = -7
SURR_E_IO = -8
SURR_F32, SURR_BF16 = 0, 1
SURR_SELECT_THRESHOLD, SURR_SELECT_BUDGET, SURR_SELECT_TOP_SCORE = 0, 1, 2

EXPORTS = ("surrogate_tensor_count", "surrogate_tensor_shape", "surrogate_load_weights",
           "surrogate_load_weights_tensors", "surrogate_weight_file_config",
           "surrogate_get_config", "surrogate_workspace_size", "surrogate_score_pairs",
           "surrogate_select", "surrogate_device_status", "surrogate_free",
           "surrogate_status_string", "surrogate_last_error", "surrogate_profile_enable",
           "surrogate_profile_collect", "surrogate_forecast_head", "surrogate_prefix_build",
           "surrogate_score_suffixes", "surrogate_prefix_cache_bytes", "surrogate_prefix_free",
           "surrogate_evaluate_workspace_size", "surrogate_evaluate", "surrogate_evaluate_noalloc",
           "surrogate_cache_create",
           "surrogate_cache_extend", "surrogate_cache_lengths", "surrogate_cache_reset")
PHASES = ("embed", "rmsnorm", "gemm_qkv", "rope", "attention", "gemm_o", "gemm_gate_up",
          "gemm_down", "last_rows", "lm_head", "lse_verdict", "prefix_capture")


class SurrogateError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class surrogate_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layers", "d_model", "n_q_heads", "n_kv_heads", "head_dim", "d_ff", "vocab",
                 "max_pos")] + [("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                                ("dtype", ctypes.c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libsurrogate.so (built by build_lib); raise if it is not there."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2605_31464_amd.build_lib` (no CPU fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    cfgp = ctypes.POINTER(surrogate_config)
    sig = {
        "surrogate_tensor_count": (I32, [cfgp, ctypes.POINTER(I32)]),
        "surrogate_tensor_shape": (I32, [cfgp, I32, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                         ctypes.POINTER(I32)]),
        "surrogate_load_weights_tensors": (I32, [cfgp, ctypes.POINTER(P), I32, I32, P, ctypes.POINTER(P)]),
        "surrogate_load_weights": (I32, [ctypes.c_char_p, P, ctypes.POINTER(P)]),
        "surrogate_weight_file_config": (I32, [ctypes.c_char_p, cfgp]),
        "surrogate_get_config": (I32, [P, cfgp]),
        "surrogate_workspace_size": (I32, [P, I32, I64, I32, ctypes.POINTER(SZ)]),
        "surrogate_score_pairs": (I32, [P, P, I64, P, I32, P, I32, P, SZ, P, P, P, P, P]),
        "surrogate_select": (I32, [P, I32, I32, F, I32, P, P, P, P]),
        "surrogate_device_status": (I32, [P, P]),
        "surrogate_free": (None, [P]),
        "surrogate_status_string": (ctypes.c_char_p, [I32]),
        "surrogate_last_error": (ctypes.c_char_p, []),
        "surrogate_profile_enable": (I32, [P, I32]),
        "surrogate_profile_collect": (I32, [P, P, P]),
        "surrogate_forecast_head": (I32, [P, I64, I32, P, P, P, I32, P, P, P]),
        "surrogate_prefix_build": (I32, [P, P, I64, P, I32, P, SZ, P, ctypes.POINTER(P)]),
        "surrogate_score_suffixes": (I32, [P, P, P, P, I64, P, I32, P, I32, P, SZ, P, P, P, P, P]),
        "surrogate_prefix_cache_bytes": (I32, [P, ctypes.POINTER(SZ)]),
        "surrogate_prefix_free": (None, [P]),
        "surrogate_evaluate_workspace_size": (I32, [I32, I32, ctypes.POINTER(SZ)]),
        "surrogate_cache_create": (I32, [P, I32, P, ctypes.POINTER(P)]),
        "surrogate_cache_extend": (I32, [P, P, P, P, I64, P, I32, P, P, SZ, P, P, P]),
        "surrogate_cache_lengths": (I32, [P, P]),
        "surrogate_cache_reset": (I32, [P, P, I32]),
        "surrogate_evaluate": (I32, [P, P, I32, I32, P, P, P, I32, P, SZ, P, P, P, P, P]),
        "surrogate_evaluate_noalloc": (I32, [P, P, I32, I32, P, P, P, I32, P, P, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype, fn.argtypes = res, args
    _lib = L
    return L


def _check(status: int, where: str):
    if status != SURR_OK:
        L = lib()
        raise SurrogateError(status, where, L.surrogate_last_error().decode())


def make_config(shape) -> surrogate_config:
    """surrogate_config from an object with the ModelShape fields."""
    return surrogate_config(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                            shape.head_dim, shape.d_ff, shape.vocab, shape.max_pos,
                            float(shape.rope_base), float(shape.rms_eps),
                            SURR_BF16 if shape.dtype == "bf16" else SURR_F32)


def _stream(stream=None) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


def surrogate_tensor_count(cfg: surrogate_config) -> int:
    n = ctypes.c_int32()
    _check(lib().surrogate_tensor_count(ctypes.byref(cfg), ctypes.byref(n)), "surrogate_tensor_count")
    return n.value


def surrogate_tensor_shape(cfg: surrogate_config, index: int):
    r, c, dt = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int32()
    _check(lib().surrogate_tensor_shape(ctypes.byref(cfg), index, ctypes.byref(r), ctypes.byref(c),
                                        ctypes.byref(dt)), "surrogate_tensor_shape")
    return r.value, c.value, dt.value


class Model:
    """Owns a surrogate_model handle (device weights)."""

    def __init__(self, handle: int, cfg: surrogate_config):
        self.handle = ctypes.c_void_p(handle)
        self.cfg = cfg

    def close(self):
        if self.handle:
            lib().surrogate_free(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def surrogate_load_weights(path, stream=None) -> Model:
    """A model from a weight file (synth.write_weight_file writes them)."""
    h = ctypes.c_void_p()
    _check(lib().surrogate_load_weights(os.fsencode(path), ctypes.c_void_p(_stream(stream)),
                                        ctypes.byref(h)), "surrogate_load_weights")
    cfg = surrogate_config()
    _check(lib().surrogate_get_config(h, ctypes.byref(cfg)), "surrogate_get_config")
    return Model(h.value, cfg)


def surrogate_weight_file_config(path) -> surrogate_config:
    """The configuration a weight file declares (header checks only, no device work)."""
    cfg = surrogate_config()
    _check(lib().surrogate_weight_file_config(os.fsencode(path), ctypes.byref(cfg)),
           "surrogate_weight_file_config")
    return cfg


def surrogate_load_weights_tensors(cfg: surrogate_config, tensors, stream=None) -> Model:
    """tensors: canonical-order list of numpy host arrays or torch device tensors."""
    n = len(tensors)
    on_device = 0
    ptrs = (ctypes.c_void_p * n)()
    keep = []
    for i, t in enumerate(tensors):
        rows, cols, dt = surrogate_tensor_shape(cfg, i)
        if isinstance(t, np.ndarray):
            a = np.ascontiguousarray(t)
            want = np.float32 if dt == SURR_F32 else np.uint16
            if a.dtype != want or a.size != rows * cols:
                raise ValueError(f"tensor {i}: want {want.__name__} x {rows * cols}, got {a.dtype} x {a.size}")
            keep.append(a)
            ptrs[i] = a.ctypes.data
        else:
            on_device = 1
            if not t.is_contiguous() or t.numel() != rows * cols:
                raise ValueError(f"tensor {i}: need a contiguous device tensor of {rows * cols} elements")
            keep.append(t)
            ptrs[i] = t.data_ptr()
    if on_device and any(isinstance(t, np.ndarray) for t in tensors):
        raise ValueError("tensors must be all host arrays or all device tensors")
    h = ctypes.c_void_p()
    _check(lib().surrogate_load_weights_tensors(ctypes.byref(cfg), ptrs, n, on_device,
                                                ctypes.c_void_p(_stream(stream)), ctypes.byref(h)),
           "surrogate_load_weights_tensors")
    return Model(h.value, cfg)


def surrogate_workspace_size(model: Model, batch: int, total_tokens: int, max_len: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().surrogate_workspace_size(model.handle, batch, total_tokens, max_len,
                                          ctypes.byref(out)), "surrogate_workspace_size")
    return out.value


def surrogate_score_pairs(model: Model, tokens, lengths, verdict_ids, workspace, logprobs,
                          confidence, probs=None, verdict=None, stream=None):
    """tokens: int32 device [B, S]; lengths, verdict_ids: host int sequences;
    workspace: device byte tensor; outputs: preallocated device tensors."""
    import torch
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 [B, S] device tensor")
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    vid = np.ascontiguousarray(np.asarray(verdict_ids, dtype=np.int32))
    B = int(tokens.shape[0])
    if L.shape != (B,):
        raise ValueError("lengths must have one entry per row of tokens")
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().surrogate_score_pairs(
        model.handle, ptr(tokens), int(tokens.shape[1]), L.ctypes.data_as(ctypes.c_void_p), B,
        vid.ctypes.data_as(ctypes.c_void_p), int(vid.size), ptr(workspace),
        workspace.numel() * workspace.element_size(), ptr(logprobs), ptr(probs), ptr(confidence),
        ptr(verdict), ctypes.c_void_p(_stream(stream))), "surrogate_score_pairs")


class PrefixCache:
    """Owns a surrogate_prefix_cache handle (device keys and values of shared prefixes)."""

    def __init__(self, handle: int, lengths):
        self.handle = ctypes.c_void_p(handle)
        self.lengths = list(int(x) for x in lengths)

    def nbytes(self) -> int:
        out = ctypes.c_size_t()
        _check(lib().surrogate_prefix_cache_bytes(self.handle, ctypes.byref(out)),
               "surrogate_prefix_cache_bytes")
        return out.value

    def close(self):
        if self.handle:
            lib().surrogate_prefix_free(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def surrogate_cache_create(model: Model, capacities) -> PrefixCache:
    """Empty cache entries of the given token capacities (decode continuation)."""
    cap = np.ascontiguousarray(np.asarray(capacities, dtype=np.int32))
    h = ctypes.c_void_p()
    _check(lib().surrogate_cache_create(model.handle, int(cap.size),
                                        cap.ctypes.data_as(ctypes.c_void_p), ctypes.byref(h)),
           "surrogate_cache_create")
    return PrefixCache(h.value, np.zeros(cap.size, np.int32))


def surrogate_cache_extend(model: Model, cache: PrefixCache, entry_ids, tokens, lengths, workspace,
                           target_ids=None, next_token=None, target_logprob=None, stream=None):
    """Append row i of tokens (int32 device [B, S], lengths[i] valid) to entry
    entry_ids[i]; writes the greedy next token and, with target_ids, its log-prob."""
    import torch
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 [B, S] device tensor")
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    eid = np.ascontiguousarray(np.asarray(entry_ids, dtype=np.int32))
    B = int(tokens.shape[0])
    if L.shape != (B,) or eid.shape != (B,):
        raise ValueError("lengths and entry_ids must have one entry per row of tokens")
    tgt = None if target_ids is None else np.ascontiguousarray(np.asarray(target_ids, dtype=np.int32))
    if tgt is not None and tgt.shape != (B,):
        raise ValueError("target_ids must have one entry per row of tokens")
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().surrogate_cache_extend(
        model.handle, cache.handle, eid.ctypes.data_as(ctypes.c_void_p), ptr(tokens),
        int(tokens.shape[1]), L.ctypes.data_as(ctypes.c_void_p), B,
        tgt.ctypes.data_as(ctypes.c_void_p) if tgt is not None else None, ptr(workspace),
        workspace.numel() * workspace.element_size(), ptr(next_token), ptr(target_logprob),
        ctypes.c_void_p(_stream(stream))), "surrogate_cache_extend")


def surrogate_cache_lengths(cache: PrefixCache, n_entries: int) -> np.ndarray:
    out = np.zeros(n_entries, np.int32)
    _check(lib().surrogate_cache_lengths(cache.handle, out.ctypes.data_as(ctypes.c_void_p)),
           "surrogate_cache_lengths")
    return out


def surrogate_cache_reset(cache: PrefixCache, entry_ids):
    eid = np.ascontiguousarray(np.asarray(entry_ids, dtype=np.int32))
    _check(lib().surrogate_cache_reset(cache.handle, eid.ctypes.data_as(ctypes.c_void_p),
                                       int(eid.size)), "surrogate_cache_reset")


def surrogate_prefix_build(model: Model, tokens, lengths, workspace, stream=None) -> PrefixCache:
    """tokens: int32 device [G, S]; lengths: host ints; workspace: device byte tensor."""
    import torch
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 [G, S] device tensor")
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    G = int(tokens.shape[0])
    if L.shape != (G,):
        raise ValueError("lengths must have one entry per row of tokens")
    h = ctypes.c_void_p()
    _check(lib().surrogate_prefix_build(
        model.handle, ctypes.c_void_p(tokens.data_ptr()), int(tokens.shape[1]),
        L.ctypes.data_as(ctypes.c_void_p), G, ctypes.c_void_p(workspace.data_ptr()),
        workspace.numel() * workspace.element_size(), ctypes.c_void_p(_stream(stream)),
        ctypes.byref(h)), "surrogate_prefix_build")
    return PrefixCache(h.value, L)


def surrogate_score_suffixes(model: Model, cache: PrefixCache, prefix_ids, tokens, lengths,
                             verdict_ids, workspace, logprobs, confidence, probs=None,
                             verdict=None, stream=None):
    """As surrogate_score_pairs for prompts = cached prefix prefix_ids[i] (-1: none) +
    row i of tokens."""
    import torch
    if tokens.dtype != torch.int32 or tokens.dim() != 2 or not tokens.is_contiguous():
        raise ValueError("tokens must be a contiguous int32 [B, S] device tensor")
    L = np.ascontiguousarray(np.asarray(lengths, dtype=np.int32))
    pid = np.ascontiguousarray(np.asarray(prefix_ids, dtype=np.int32))
    vid = np.ascontiguousarray(np.asarray(verdict_ids, dtype=np.int32))
    B = int(tokens.shape[0])
    if L.shape != (B,) or pid.shape != (B,):
        raise ValueError("lengths and prefix_ids must have one entry per row of tokens")
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().surrogate_score_suffixes(
        model.handle, cache.handle, pid.ctypes.data_as(ctypes.c_void_p), ptr(tokens),
        int(tokens.shape[1]), L.ctypes.data_as(ctypes.c_void_p), B,
        vid.ctypes.data_as(ctypes.c_void_p), int(vid.size), ptr(workspace),
        workspace.numel() * workspace.element_size(), ptr(logprobs), ptr(probs), ptr(confidence),
        ptr(verdict), ctypes.c_void_p(_stream(stream))), "surrogate_score_suffixes")


def surrogate_select(confidence, mode: int, threshold: float = 0.0, budget_k: int = 0,
                     defer_idx=None, accept_idx=None, counts=None, stream=None):
    """Returns (defer_idx, accept_idx, counts) device int32 tensors."""
    import torch
    n = int(confidence.numel())
    dev = confidence.device
    defer_idx = torch.empty(n, dtype=torch.int32, device=dev) if defer_idx is None else defer_idx
    accept_idx = torch.empty(n, dtype=torch.int32, device=dev) if accept_idx is None else accept_idx
    counts = torch.empty(2, dtype=torch.int32, device=dev) if counts is None else counts
    _check(lib().surrogate_select(ctypes.c_void_p(confidence.data_ptr()), n, mode, float(threshold),
                                  int(budget_k), ctypes.c_void_p(defer_idx.data_ptr()),
                                  ctypes.c_void_p(accept_idx.data_ptr()),
                                  ctypes.c_void_p(counts.data_ptr()),
                                  ctypes.c_void_p(_stream(stream))), "surrogate_select")
    return defer_idx, accept_idx, counts


def surrogate_forecast_head(probs, bin_values, bin_edges=None, cutoffs=(), expected_speedup=None,
                            discovery=None, want_speedup=True, stream=None):
    """probs: float32 device [n, n_bins]; bin_values, bin_edges, cutoffs: host sequences.
    Returns (expected_speedup [n] or None, discovery [n, n_cutoffs] or None)."""
    import torch
    if probs.dtype != torch.float32 or probs.dim() != 2 or not probs.is_contiguous():
        raise ValueError("probs must be a contiguous float32 [n, n_bins] device tensor")
    n, nb = int(probs.shape[0]), int(probs.shape[1])
    m = np.ascontiguousarray(np.asarray(bin_values, np.float64))
    if m.shape != (nb,):
        raise ValueError("bin_values must have n_bins entries")
    cut = np.ascontiguousarray(np.asarray(cutoffs, np.float64).reshape(-1))
    nc = int(cut.size)
    e = None if bin_edges is None else np.ascontiguousarray(np.asarray(bin_edges, np.float64))
    if want_speedup and expected_speedup is None:
        expected_speedup = torch.empty(n, dtype=torch.float32, device=probs.device)
    if nc and discovery is None:
        discovery = torch.empty(n, nc, dtype=torch.float32, device=probs.device)
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    host = lambda a: ctypes.c_void_p(a.ctypes.data if a is not None and a.size else 0)
    _check(lib().surrogate_forecast_head(
        ptr(probs), n, nb, host(m), host(e), host(cut), nc, ptr(expected_speedup),
        ptr(discovery if nc else None), ctypes.c_void_p(_stream(stream))), "surrogate_forecast_head")
    return expected_speedup, (discovery if nc else None)


SUMMARY_FIELDS = ("accuracy", "brier", "crps", "reward_brier", "reward_crps", "ece",
                  "forecast_error", "recovered")


def surrogate_evaluate_workspace_size(n: int, n_budgets: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().surrogate_evaluate_workspace_size(n, n_budgets, ctypes.byref(out)),
           "surrogate_evaluate_workspace_size")
    return out.value


def surrogate_evaluate(probs, speedup, bin_values, bin_edges, budgets=(0.01, 0.05, 0.10, 0.25, 0.50),
                       per_candidate=True, workspace=None, stream=None):
    """probs: float32 device [n, n_bins]; speedup: float32 device [n].  Returns (summary
    float64 device tensor [8 + n_budgets], bins, brier, crps) with the per-candidate
    tensors None unless per_candidate."""
    import torch
    if probs.dtype != torch.float32 or probs.dim() != 2 or not probs.is_contiguous():
        raise ValueError("probs must be a contiguous float32 [n, n_bins] device tensor")
    if speedup.dtype != torch.float32 or speedup.numel() != probs.shape[0]:
        raise ValueError("speedup must be float32 with one entry per forecast")
    n, nb = int(probs.shape[0]), int(probs.shape[1])
    m = np.ascontiguousarray(np.asarray(bin_values, np.float64))
    e = np.ascontiguousarray(np.asarray(bin_edges, np.float64))
    c = np.ascontiguousarray(np.asarray(budgets, np.float64))
    dev = probs.device
    if workspace is None:
        workspace = torch.empty(surrogate_evaluate_workspace_size(n, int(c.size)),
                                dtype=torch.uint8, device=dev)
    summary = torch.empty(8 + c.size, dtype=torch.float64, device=dev)
    bins = torch.empty(n, dtype=torch.int32, device=dev) if per_candidate else None
    br = torch.empty(n, dtype=torch.float32, device=dev) if per_candidate else None
    cr = torch.empty(n, dtype=torch.float32, device=dev) if per_candidate else None
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().surrogate_evaluate(
        ptr(probs), ptr(speedup), n, nb, m.ctypes.data_as(ctypes.c_void_p),
        e.ctypes.data_as(ctypes.c_void_p), c.ctypes.data_as(ctypes.c_void_p), int(c.size),
        ptr(workspace), workspace.numel() * workspace.element_size(), ptr(bins), ptr(br), ptr(cr),
        ptr(summary), ctypes.c_void_p(_stream(stream))), "surrogate_evaluate")
    return summary, bins, br, cr


def surrogate_evaluate_noalloc(probs, speedup, bin_values, bin_edges,
                               budgets=(0.01, 0.05, 0.10, 0.25, 0.50), out=None, stream=None):
    """As surrogate_evaluate, on the library's fixed per-device scratch instead of a workspace.
    out: optional (summary float64 [8 + n_budgets], bins int32 [n], brier float32 [n], crps
    float32 [n]) device tensors to write into; the per-candidate ones may be None.  Returns
    the four tensors."""
    import torch
    if probs.dtype != torch.float32 or probs.dim() != 2 or not probs.is_contiguous():
        raise ValueError("probs must be a contiguous float32 [n, n_bins] device tensor")
    if speedup.dtype != torch.float32 or speedup.numel() != probs.shape[0]:
        raise ValueError("speedup must be float32 with one entry per forecast")
    n, nb = int(probs.shape[0]), int(probs.shape[1])
    m = np.ascontiguousarray(np.asarray(bin_values, np.float64))
    e = np.ascontiguousarray(np.asarray(bin_edges, np.float64))
    c = np.ascontiguousarray(np.asarray(budgets, np.float64))
    if out is None:
        dev = probs.device
        out = (torch.empty(8 + c.size, dtype=torch.float64, device=dev),
               torch.empty(n, dtype=torch.int32, device=dev),
               torch.empty(n, dtype=torch.float32, device=dev),
               torch.empty(n, dtype=torch.float32, device=dev))
    summary, bins, br, cr = out
    ptr = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    _check(lib().surrogate_evaluate_noalloc(
        ptr(probs), ptr(speedup), n, nb, m.ctypes.data_as(ctypes.c_void_p),
        e.ctypes.data_as(ctypes.c_void_p), c.ctypes.data_as(ctypes.c_void_p), int(c.size),
        ptr(bins), ptr(br), ptr(cr), ptr(summary), ctypes.c_void_p(_stream(stream))),
        "surrogate_evaluate_noalloc")
    return summary, bins, br, cr


def surrogate_device_status(model: Model, stream=None) -> int:
    """Synchronizes; returns SURR_OK or SURR_E_TOKEN_RANGE (sticky flag, then cleared)."""
    return lib().surrogate_device_status(model.handle, ctypes.c_void_p(_stream(stream)))


def surrogate_profile_enable(model: Model, enable: bool = True):
    _check(lib().surrogate_profile_enable(model.handle, int(bool(enable))), "surrogate_profile_enable")


def surrogate_profile_collect(model: Model) -> dict:
    """{phase: (milliseconds, launches)} since the previous collect."""
    ms = (ctypes.c_double * len(PHASES))()
    n = (ctypes.c_int64 * len(PHASES))()
    _check(lib().surrogate_profile_collect(model.handle, ms, n), "surrogate_profile_collect")
    return {p: (ms[i], n[i]) for i, p in enumerate(PHASES)}


def surrogate_free(model: Model):
    model.close()


# ---------------------------------------------------------------- convenience layer
class Scorer:
    """A loaded model plus a workspace sized for one batch shape."""

    def __init__(self, shape, weights: dict, names, device="cuda:0", weight_file=None):
        """weights/names: tensors in memory; or weight_file: a weight file (shape and
        weights None)."""
        import torch
        self.torch = torch
        self.device = torch.device(device)
        with torch.cuda.device(self.device):
            if weight_file is not None:
                self.model = surrogate_load_weights(weight_file)
                self.cfg = self.model.cfg
            else:
                self.cfg = make_config(shape)
                self.model = surrogate_load_weights_tensors(self.cfg, [weights[n] for n in names])
        self.workspace = None

    def ensure_workspace(self, batch, total_tokens, max_len):
        need = surrogate_workspace_size(self.model, batch, total_tokens, max_len)
        if self.workspace is None or self.workspace.numel() < need:
            self.workspace = None
            self.workspace = self.torch.empty(need, dtype=self.torch.uint8, device=self.device)
        return self.workspace

    def score(self, tokens, lengths, verdict_ids):
        torch = self.torch
        tok = torch.as_tensor(np.asarray(tokens, np.int32)).to(self.device) \
            if not isinstance(tokens, torch.Tensor) else tokens
        L = np.asarray(lengths, np.int32)
        B, nv = len(L), len(verdict_ids)
        ws = self.ensure_workspace(B, int(L.sum()), int(L.max()))
        out = {"logprobs": torch.empty(B, nv, dtype=torch.float32, device=self.device),
               "p": torch.empty(B, nv, dtype=torch.float32, device=self.device),
               "confidence": torch.empty(B, dtype=torch.float32, device=self.device),
               "verdict": torch.empty(B, dtype=torch.int32, device=self.device)}
        surrogate_score_pairs(self.model, tok, L, verdict_ids, ws, out["logprobs"], out["confidence"],
                              out["p"], out["verdict"])
        return out

    def build_prefixes(self, tokens, lengths) -> PrefixCache:
        torch = self.torch
        tok = torch.as_tensor(np.asarray(tokens, np.int32)).to(self.device) \
            if not isinstance(tokens, torch.Tensor) else tokens
        L = np.asarray(lengths, np.int32)
        ws = self.ensure_workspace(len(L), int(L.sum()), int(L.max()))
        return surrogate_prefix_build(self.model, tok, L, ws)

    def create_cache(self, capacities) -> PrefixCache:
        return surrogate_cache_create(self.model, capacities)

    def extend(self, cache: PrefixCache, entry_ids, tokens, lengths, target_ids=None):
        """Append tokens to cache entries; returns (next_token, target_logprob or None)."""
        torch = self.torch
        tok = torch.as_tensor(np.asarray(tokens, np.int32)).to(self.device) \
            if not isinstance(tokens, torch.Tensor) else tokens
        L = np.asarray(lengths, np.int32)
        B = len(L)
        ws = self.ensure_workspace(B, int(L.sum()), int(L.max()))
        nxt = torch.empty(B, dtype=torch.int32, device=self.device)
        lp = torch.empty(B, dtype=torch.float32, device=self.device) if target_ids is not None else None
        surrogate_cache_extend(self.model, cache, entry_ids, tok, L, ws, target_ids, nxt, lp)
        return nxt, lp

    def score_suffixes(self, cache: PrefixCache, prefix_ids, tokens, lengths, verdict_ids):
        torch = self.torch
        tok = torch.as_tensor(np.asarray(tokens, np.int32)).to(self.device) \
            if not isinstance(tokens, torch.Tensor) else tokens
        L = np.asarray(lengths, np.int32)
        B, nv = len(L), len(verdict_ids)
        ws = self.ensure_workspace(B, int(L.sum()), int(L.max()))
        out = {"logprobs": torch.empty(B, nv, dtype=torch.float32, device=self.device),
               "p": torch.empty(B, nv, dtype=torch.float32, device=self.device),
               "confidence": torch.empty(B, dtype=torch.float32, device=self.device),
               "verdict": torch.empty(B, dtype=torch.int32, device=self.device)}
        surrogate_score_suffixes(self.model, cache, prefix_ids, tok, L, verdict_ids, ws,
                                 out["logprobs"], out["confidence"], out["p"], out["verdict"])
        return out
