"""Pins for the layer-map oracle: hand-worked tables, closed-form depth,
Eq. 1's neighbourhood, and the mapper parameter counts printed in the paper."""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import layer_map as lm


@pytest.fixture(scope="module")
def golden(golden_dir):
    with open(os.path.join(golden_dir, "layer_maps.json")) as f:
        return json.load(f)


def _table(L_s, L_r):
    return np.stack(lm.interp2(L_s, L_r), axis=1).tolist()


def test_interp2_hand_tables(golden):
    g = golden["interp2"]
    assert _table(4, 6) == g["4->6"]
    assert _table(32, 40)[:3] == g["32->40_head"]
    assert _table(32, 40)[-1] == g["32->40_last"]
    assert _table(28, 32)[:3] == g["28->32_head"]


@pytest.mark.parametrize("L_s,L_r", [(4, 6), (32, 28), (32, 40), (28, 32), (7, 7), (1, 5), (5, 1), (2, 9)])
def test_interp2_depth_closed_form(L_s, L_r):
    lo, hi, rem, den = lm.interp2(L_s, L_r)
    a_lo, a_hi = lm.interp2_weights(lo, hi, rem, den)
    for j in range(L_r):
        p = Fraction(j * (L_s - 1), L_r - 1) if L_r > 1 else Fraction(0)
        # the weighted tap depth is the exact fractional depth
        assert Fraction(int(lo[j])) + Fraction(int(rem[j]), int(den[j])) == p
        assert 0 <= lo[j] <= hi[j] <= L_s - 1 and hi[j] - lo[j] <= 1
        assert a_lo[j] + a_hi[j] == 1.0
        if rem[j] == 0:
            assert a_hi[j] == 0.0
    # endpoints map to the first and last sender layer
    assert lo[0] == 0 and rem[0] == 0
    if L_r > 1:
        assert lo[-1] == L_s - 1 and rem[-1] == 0


def test_interp2_equal_depth_is_identity():
    lo, hi, rem, den = lm.interp2(9, 9)
    assert lo.tolist() == list(range(9)) and not rem.any()


def test_neighbor3_eq1(golden):
    g = golden["neighbor3"]
    t = lm.neighbor3(32, 40).tolist()
    assert t[:3] == g["32->40_head"] and t[-1] == g["32->40_last"]
    # offsets (-4, 0, +4) away from the clip
    for row, p in zip(lm.neighbor3(32, 40), lm.proportional_depth(32, 40)):
        if 4 <= p <= 27:
            assert row.tolist() == [p - 4, p, p + 4]


@pytest.mark.parametrize("L_s,L_r", [(28, 32), (32, 36), (32, 40), (36, 40), (40, 28), (36, 32)])
def test_proportional_depth_has_no_ties(L_s, L_r):
    # Half-way cases would make the rounding rule matter; the paper's layer
    # counts never produce one.
    for j in range(L_r):
        f = Fraction(j * (L_s - 1), L_r - 1)
        assert f - int(f) != Fraction(1, 2)


def test_mapper_parameter_counts(golden):
    g = golden["mapper_parameters"]
    d = g["d_kv"]
    for name, r in g["receivers"].items():
        n = lm.neighbor3_parameter_count(r["layers"], d, d)
        assert round(n / 1e6) == r["millions"], name
    # 0.40-0.50 GB in BF16
    assert 0.40 <= lm.neighbor3_parameter_count(32, d, d) * 2 / 1e9 < 0.41
    assert 0.50 <= lm.neighbor3_parameter_count(40, d, d) * 2 / 1e9 < 0.51
