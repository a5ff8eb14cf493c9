"""Layer-map oracle (test infrastructure; see package docstring).

Receiver layers and sender layers are 0-based here.

* ``interp2``: receiver layer j sits at the fractional sender depth
  p = j (L_S - 1) / (L_R - 1) and linearly interpolates the two nearest sender
  layers floor(p) and floor(p) + 1 with weights (1 - frac(p), frac(p)).  The
  table keeps p exact as integers: lo = floor(p), rem / den = frac(p),
  hi = min(lo + 1, L_S - 1).  When rem == 0 the layer has a single tap.  With
  a single receiver layer the depth is taken as 0.

* ``neighbor3``: the paper's proportional depth alignment with three sender
  layers at offsets (-4, 0, +4) around the matched layer, clipped to the
  model (Eq. 1; App. B.1 "clipped at model boundaries").  Written 0-based:
  pi = round(j (L_S - 1) / (L_R - 1)), N(j) = clip(pi - 4, pi, pi + 4).
  Reading: ``round`` is round-half-to-even on the exact rational.
"""

from __future__ import annotations

from fractions import Fraction

import numpy as np


def interp2(L_s: int, L_r: int):
    """Integer table (lo, hi, rem, den), each int64 [L_r]."""
    if L_s < 1 or L_r < 1:
        raise ValueError("layer counts must be >= 1")
    lo = np.zeros(L_r, dtype=np.int64)
    hi = np.zeros(L_r, dtype=np.int64)
    rem = np.zeros(L_r, dtype=np.int64)
    den = np.ones(L_r, dtype=np.int64)
    if L_r == 1:
        return lo, hi, rem, den
    for j in range(L_r):
        num, d = j * (L_s - 1), L_r - 1
        lo[j], rem[j], den[j] = num // d, num % d, d
        hi[j] = min(lo[j] + 1, L_s - 1)
    return lo, hi, rem, den


def interp2_weights(lo, hi, rem, den):
    """fp64 weights (alpha_lo, alpha_hi) of the two taps of each layer."""
    rem = np.asarray(rem, dtype=np.float64)
    den = np.asarray(den, dtype=np.float64)
    return (den - rem) / den, rem / den


def proportional_depth(L_s: int, L_r: int):
    """0-based matched sender layer pi(j) of Eq. 1 (round half to even)."""
    if L_r == 1:
        return np.zeros(1, dtype=np.int64)
    return np.asarray([round(Fraction(j * (L_s - 1), L_r - 1)) for j in range(L_r)],
                      dtype=np.int64)


def neighbor3(L_s: int, L_r: int):
    """0-based sender layers (t1, t2, t3) feeding each receiver layer, [L_r, 3]."""
    pi = proportional_depth(L_s, L_r)
    taps = np.stack([pi - 4, pi, pi + 4], axis=1)
    return np.clip(taps, 0, L_s - 1)


def neighbor3_parameter_count(L_r: int, d_s_kv: int, d_r_kv: int) -> int:
    """Stored parameters of the folded 3-layer maps: per receiver layer and
    role one A of shape (3 d_S) x d_R plus one bias of d_R (Eq. 9 with the
    concatenated features of Eq. 2)."""
    return 2 * L_r * (3 * d_s_kv * d_r_kv + d_r_kv)
