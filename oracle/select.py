"""Selective deferral (test infrastructure, see package doc).

Section 2.1 (Selective Use): forecasts whose confidence q_i clears a threshold are
accepted and the rest are measured on the device.  The comparison is q_i >= tau,
the convention Section 3.6 uses for turning a score into a positive prediction; it
is made in float32 (tau is cast first), and a NaN confidence never clears it.

Budget mode defers the k candidates of lowest confidence (Section 3.1 measures a
top-c% subset of the candidates; here the subset is the least confident one).
Order: confidence ascending with NaN first, ties broken by ascending index; -0.0
equals +0.0.  k is clamped to [0, N]; a negative k is an error.  Both index lists
are returned in ascending order and together partition range(N).
"""
from __future__ import annotations

import math

import numpy as np


def select_threshold(confidence, tau: float):
    q = np.asarray(confidence, np.float32)
    t = np.float32(tau)
    accept = [i for i in range(len(q)) if q[i] >= t]
    acc = set(accept)
    defer = [i for i in range(len(q)) if i not in acc]
    return np.array(defer, np.int32), np.array(accept, np.int32)


def select_budget(confidence, k: int):
    if k < 0:
        raise ValueError("budget k must be >= 0")
    q = np.asarray(confidence, np.float32)
    n = len(q)
    k = min(k, n)

    def key(i):
        v = float(q[i])
        return (-math.inf if math.isnan(v) else v, i)

    order = sorted(range(n), key=key)
    d = set(order[:k])
    defer = [i for i in range(n) if i in d]
    accept = [i for i in range(n) if i not in d]
    return np.array(defer, np.int32), np.array(accept, np.int32)
