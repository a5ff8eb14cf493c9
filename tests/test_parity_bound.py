"""The quantization-limited gate is not vacuous: a simulated bf16 pipeline
(features and outputs rounded to bf16) stays inside the rounding bound, and
the same pipeline with a planted mistake does not."""

import numpy as np
import torch

from _parity import bf16_half_ulp, rounding_bound


def _bf16(a):
    return torch.as_tensor(a, dtype=torch.float32).to(torch.bfloat16).double().numpy()


def test_half_ulp():
    assert bf16_half_ulp(1.0) == 2.0 ** -8
    assert bf16_half_ulp(9.0) == 2.0 ** -5
    assert bf16_half_ulp(-150.0) == 0.5


def test_bound_holds_for_bf16_pipeline_and_catches_a_dropped_term():
    rng = np.random.default_rng(0)
    T, d_in, H_r, d_h = 64, 256, 2, 64
    scale = rng.lognormal(0.0, 1.0, d_in)
    x = rng.standard_normal((T, d_in)) * scale
    A = rng.standard_normal((H_r * d_h, d_in)) / np.sqrt(d_in)
    ref = (x @ A.T).reshape(T, H_r, d_h).transpose(1, 0, 2)
    y = _bf16(_bf16(x) @ A.T).reshape(T, H_r, d_h).transpose(1, 0, 2)
    bound = rounding_bound(ref, x, A)
    assert np.all(np.abs(y - ref) <= bound)
    x_bad = x.copy()
    x_bad[:, 7] = 0.0                        # a dropped feature
    y_bad = _bf16(_bf16(x_bad) @ A.T).reshape(T, H_r, d_h).transpose(1, 0, 2)
    assert np.any((np.abs(y_bad - ref) > bound) & (np.abs(y_bad - ref) > 2e-2))
