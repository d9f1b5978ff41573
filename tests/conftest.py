import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from synth.workloads import ModelShape  # noqa: E402


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def tiny_shape(dtype="fp32", **kw):
    """A very small model used by the oracle pins (GQA: 4 query heads over 2 kv heads)."""
    base = dict(n_layers=2, d_model=8, n_heads=4, n_kv_heads=2, head_dim=4, d_ff=12,
                vocab=10, dtype=dtype, init_std=0.5)
    base.update(kw)
    return ModelShape(**base)


def random_weights(m, seed=0):
    """Small random weights straight from numpy (bf16 models get bf16-exact values)."""
    from synth.gen import model_weights
    W = model_weights(m, seed=seed)
    rng = np.random.default_rng(seed + 99)
    # non-trivial norm gains so that a dropped gain fails a pin
    W["final_norm"] = (1.0 + 0.3 * rng.standard_normal(m.d_model)).astype(np.float32)
    for L in W["layers"]:
        L["attn_norm"] = (1.0 + 0.3 * rng.standard_normal(m.d_model)).astype(np.float32)
        L["mlp_norm"] = (1.0 + 0.3 * rng.standard_normal(m.d_model)).astype(np.float32)
    return W


@pytest.fixture
def rng():
    return np.random.default_rng(1234)
