"""The quantization-limited gate is not vacuous: a simulated bf16 pipeline
(features and outputs rounded to bf16) stays inside the rounding bound, and
the same pipeline with a planted mistake does not."""

import numpy as np
import torch

from _parity import bf16_half_ulp, rounding_bound, rounding_bound_normed
from oracle import rope as _rope
from oracle import transfer as _tr


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


def _normed_pipeline(x, A, b, g, eps, pos, theta, round_x, plant=None):
    """Simulated key path: (bf16) x -> y = A x + b -> RMSNorm per head with g
    -> RoPE at pos -> bf16.  plant: a mistake to put in."""
    T = x.shape[0]
    H_r, d_h = A.shape[0] // g.size, g.size
    xx = _bf16(x) if round_x else x
    if plant == "dropped feature":
        xx = xx.copy()
        xx[:, 11] = 0.0
    y = (xx @ A.T + b).reshape(T, H_r, d_h).transpose(1, 0, 2)
    gg = np.roll(g, 1) if plant == "shifted weight" else g
    if plant == "rotate first":
        y = _tr.rms_norm(_rope.rotate(y, pos, theta), gg, eps)
    else:
        y = _rope.rotate(_tr.rms_norm(y, gg, eps), pos, theta)
    return _bf16(y) if round_x else y


def test_normed_bound_holds_and_catches_planted_mistakes():
    rng = np.random.default_rng(1)
    T, d_in, H_r, d_h = 96, 256, 2, 64
    x = rng.standard_normal((T, d_in))
    A = rng.standard_normal((H_r * d_h, d_in)) / np.sqrt(d_in)
    b = 0.2 * rng.standard_normal(H_r * d_h)
    g = np.concatenate([rng.uniform(0.5, 1.0, d_h // 2), rng.uniform(1.0, 1.5, d_h // 2)])
    pos = 1000 + np.arange(T)
    ref = _normed_pipeline(x, A, b, g, 1e-6, pos, 5e5, round_x=False)
    bound = rounding_bound_normed(ref, x, A, b, g, 1e-6, rotated=True)
    got = _normed_pipeline(x, A, b, g, 1e-6, pos, 5e5, round_x=True)
    assert np.all(np.abs(got - ref) <= bound)
    for plant in ("dropped feature", "shifted weight", "rotate first"):
        bad = _normed_pipeline(x, A, b, g, 1e-6, pos, 5e5, round_x=True, plant=plant)
        assert np.any((np.abs(bad - ref) > bound) & (np.abs(bad - ref) > 2e-2)), plant
