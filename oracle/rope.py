"""Rotary position embedding oracle, fp64 (test infrastructure).

Rotate-half convention, applied to each head vector v of even size d: for
k < d/2 the pair (v_k, v_{k+d/2}) is rotated by the angle pos * w_k with
w_k = theta ** (-2k/d):

    v'_k       = v_k cos(a) - v_{k+d/2} sin(a)
    v'_{k+d/2} = v_{k+d/2} cos(a) + v_k sin(a)

Un-rotation at position p is rotation at -p.  The method maps keys before the
receiver's RoPE (Sec. 3 opening paragraph; App. B.1), so keys that a sender
stores after its RoPE are first un-rotated at the sender's positions with the
sender's theta, and mapped keys are rotated at the receiver's positions with
the receiver's theta.  Angles are formed in fp64.
"""

from __future__ import annotations

import numpy as np


def inv_freq(theta: float, d: int) -> np.ndarray:
    if d % 2:
        raise ValueError("head size must be even")
    k = np.arange(d // 2, dtype=np.float64)
    return np.float64(theta) ** (-2.0 * k / d)


def angles(pos, theta: float, d: int) -> np.ndarray:
    """[T, d/2] fp64 angles pos_t * w_k."""
    pos = np.asarray(pos, dtype=np.float64)
    return pos[:, None] * inv_freq(theta, d)[None, :]


def rotate(v, pos, theta: float) -> np.ndarray:
    """Rotate v[..., T, d] at positions pos[T]."""
    v = np.asarray(v, dtype=np.float64)
    d = v.shape[-1]
    a = angles(pos, theta, d)
    c, s = np.cos(a), np.sin(a)
    v1, v2 = v[..., : d // 2], v[..., d // 2:]
    return np.concatenate([v1 * c - v2 * s, v2 * c + v1 * s], axis=-1)


def unrotate(v, pos, theta: float) -> np.ndarray:
    """Inverse of ``rotate`` at the same positions: rotation at -pos."""
    return rotate(v, -np.asarray(pos, dtype=np.float64), theta)
