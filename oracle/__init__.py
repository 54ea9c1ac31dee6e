"""Float64 CPU oracle for batched forecast scoring.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The HIP
path never calls it, and it shares no code with the HIP path: it reads the same
seeded input arrays and nothing else.

Every function restates a definition from the paper or from the standard decoder
forward in plain NumPy float64, with no blocking, fusion or reordering beyond the
definition:

* ``transformer`` - the decoder forward, the full-vocabulary log-softmax at the last
  prompt position, and the forecast distribution p_i, predicted bin and confidence
  q_i = max_b p_{i,b} of Section 2.1 (Forecasting Relative Performance).
* ``select``      - selective use (Section 2.1, Selective Use) with the threshold
  convention s >= tau of Section 3.6, and the budgeted measurement of the lowest-
  confidence k candidates (Section 3.1 measures a top-c% subset).
* ``forecast``    - the paper's eight-bin speedup head: expected speedup
  S_hat = sum_b p_b m_b (Section 3.1, Table 3), discovery score Pr[g >= x]
  (Section 3.6) and the top-k candidates by S_hat (Sections 3.1 and 3.5).
* ``evaluate``    - forecast quality against measured speedups: measured bins, the
  correctness, Brier and CRPS rewards (Section 2.2), ECE, forecast error and speedup
  recovered (Section 3.1).

Parity status: every function is pinned by ``tests/test_oracle_pins.py`` and
``tests/test_oracle_forecast_pins.py`` and ``tests/test_oracle_evaluate_pins.py`` (closed
forms, invariants, a hand-computed one-layer case, independent library routines,
brute force).  The absolute bf16 error at full depth has no closed form; it is
bounded only by comparison with this oracle at the stated tolerances.
"""
from . import evaluate, forecast, select, transformer  # noqa: F401
