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
