import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (runs the HIP path)")


def arch_of(shape):
    """Architecture mapping the oracle reads, from a synthetic ModelShape."""
    return dict(n_layers=shape.n_layers, d_model=shape.d_model, n_q_heads=shape.n_q_heads,
                n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, d_ff=shape.d_ff,
                vocab=shape.vocab, rope_base=shape.rope_base, rms_eps=shape.rms_eps)


@pytest.fixture
def arch_of_shape():
    return arch_of


def assert_selection_valid(q, d, a, c, mode, tau=None, k=None):
    """Selection properties that hold at any size, on the confidence vector the kernel was
    given: the lists partition range(n) in ascending order; threshold: exactly the entries
    >= tau (float32) are accepted; budget: |defer| = min(k, n) and no accepted entry ranks
    below a deferred one in the order (NaN first, value ascending, index ascending)."""
    import numpy as np
    q = np.asarray(q, np.float32)
    n = len(q)
    c = [int(x) for x in c]
    d, a = np.asarray(d)[: c[0]], np.asarray(a)[: c[1]]
    assert c[0] + c[1] == n
    assert np.all(np.diff(d) > 0) and np.all(np.diff(a) > 0)
    assert sorted(d.tolist() + a.tolist()) == list(range(n))
    if mode == "threshold":
        t = np.float32(tau)
        assert np.all(q[a] >= t) and not np.any(q[d] >= t)
    else:
        assert c[0] == min(k, n)
        key = np.where(np.isnan(q), -np.inf, q)
        if c[0] and c[1]:
            worst_d = max(d, key=lambda i: (key[i], i))
            best_a = min(a, key=lambda i: (key[i], i))
            assert (key[worst_d], worst_d) < (key[best_a], best_a)


def assert_selection_near_oracle(defer, n, ref_conf, tol, rows=None, tau=None, k=None):
    """Deferral decisions agree with the oracle's wherever its confidence is farther than
    tol from the decision boundary.  rows: the prompts ref_conf covers (all if None; a
    budget needs all of them)."""
    import numpy as np
    defer = set(int(i) for i in defer)
    rows = list(range(n)) if rows is None else list(rows)
    ref = np.asarray(ref_conf, np.float64)
    if tau is not None:
        for r, v in zip(rows, ref):
            if v >= tau + tol:
                assert r not in defer, (r, v)
            elif v < tau - tol:
                assert r in defer, (r, v)
        return
    assert len(rows) == n
    order = np.argsort(ref, kind="stable")
    kk = min(k, n)
    if kk in (0, n):
        assert len(defer) == kk
        return
    lo_out, hi_in = ref[order[kk]], ref[order[kk - 1]]
    for r in order[:kk]:
        if ref[r] < lo_out - 2 * tol:
            assert rows[r] in defer
    for r in order[kk:]:
        if ref[r] > hi_in + 2 * tol:
            assert rows[r] not in defer
