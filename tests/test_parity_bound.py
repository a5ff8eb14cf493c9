"""The kernel-arithmetic gate (tests/_parity.py, gate 3) is not vacuous.

A CPU emulation of the bf16 path's arithmetic -- features rounded once to
bf16, fp32 products and accumulation, fp32 bias, key norm and rotation with
fp32 cos/sin tables, one bf16 rounding of the output -- passes it.  The same
emulation with one planted mistake in the oracle steps it runs (a CSR weight
off by one, swapped interpolation weights, features rounded twice, a RoPE
position off by one on either side, the other role's bias, a dropped feature)
fails it.  CPU only; the mistakes are planted in the oracle's arithmetic, never
in the GPU path.
"""

import numpy as np
import pytest

from _parity import (MAX_ABS, bf16_half_ulp, bf16_round, check_layer, kernel_gate,
                     near_midpoint)
from oracle import alignment as al
from oracle import layer_map as lm
from oracle import rope as _rope
from oracle import transfer as tr
from paper_2609_32259_amd import synth


def test_half_ulp_and_rounding():
    assert bf16_half_ulp(1.0) == 2.0 ** -8
    assert bf16_half_ulp(9.0) == 2.0 ** -5
    assert bf16_half_ulp(-150.0) == 0.5
    # round to nearest even at the bf16 midpoints of [1, 2): ulp 2^-7
    assert bf16_round(1.0 + 2.0 ** -8) == 1.0                   # tie, even below
    assert bf16_round(1.0 + 3 * 2.0 ** -8) == 1.0 + 2 * 2.0 ** -7  # tie, even above
    assert bf16_round(1.0 + 2.0 ** -8 + 2.0 ** -20) == 1.0 + 2.0 ** -7
    assert bf16_round(-3.0) == -3.0
    assert bool(near_midpoint(np.array([1.0 + 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20]))[1])
    assert not bool(near_midpoint(np.array([1.0 + 2.0 ** -9]))[0])


CFG = synth.LLAMA8B_14B_8K.with_(name="gate emulation", T_s=320, L_s=5, L_r=7, H_r=4,
                                 k_scale_sigma=1.0)


@pytest.fixture(scope="module")
def wl():
    return synth.make_workload(CFG, seed=21, device="cpu")


def _inputs(wl, opts=None):
    S = wl.S[0].float().numpy().astype(np.float64)
    csr = al.build_alignment(*wl.seg.seq(0), "overlap")
    lt = lm.interp2(CFG.L_s, CFG.L_r)
    rope = dict(wl.rope, pos0_s=0, pos0_r=0)
    A = wl.A.float().numpy().astype(np.float64)
    b = wl.bias.float().numpy().astype(np.float64)
    return S, csr, lt, rope, A, b


def _f32_rotate(y, pos, theta):
    d = y.shape[-1]
    a = _rope.angles(pos, theta, d)
    c, s = np.cos(a).astype(np.float32), np.sin(a).astype(np.float32)
    y1, y2 = y[..., : d // 2], y[..., d // 2:]
    return np.concatenate([y1 * c - y2 * s, y2 * c + y1 * s], axis=-1)


def _emulate(xs, A_lc, b_lc, role, layer, rope, opts, rows, rope_shift=0, product_scale=None):
    """The path's arithmetic on scaled features xs (fp64 [n, K]); with
    product_scale, the fp32 product is multiplied by it before the bias (the
    staged path's 1/r with concatenated taps)."""
    xb = bf16_round(xs).astype(np.float32)
    y = xb @ A_lc.astype(np.float32).T
    if product_scale is not None:
        y = y * np.float32(product_scale)
    if b_lc is not None:
        y = y + b_lc.astype(np.float32)[None, :]
    n = xs.shape[0]
    d_h = CFG.d_h
    y = y.reshape(n, -1, d_h).transpose(1, 0, 2)
    _, k_norm, eps = tr._opts(opts)
    if role == 0 and k_norm is not None:
        g = np.asarray(k_norm, np.float32)[layer]
        y = y / np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + np.float32(eps)) * g
    if role == 0 and rope.get("rotate_receiver_k", False):
        y = _f32_rotate(y, np.asarray(rows) + rope_shift, rope["theta_r"])
    return bf16_round(y)


def _features_rounded_twice(S, lt, csr, rope, layer, role):
    # planted: the interpolated, un-rotated sender rows are rounded to bf16
    # before the weighted sum (the features are rounded again afterwards)
    lo, hi, rem, den = lt
    a_lo, a_hi = lm.interp2_weights(lo, hi, rem, den)
    m = a_lo[layer] * S[lo[layer], role]
    if rem[layer]:
        m = m + a_hi[layer] * S[hi[layer], role]
    T_s = S.shape[3]
    if role == 0:
        m = _rope.unrotate(m, np.arange(T_s), rope["theta_s"])
    u = bf16_round(m.transpose(1, 0, 2).reshape(T_s, -1))
    return tr._weights_matrix(csr, T_s) @ u


PLANTS = ["none", "csr weight num+1", "swapped interpolation weights", "features rounded twice",
          "receiver rope position +1", "sender rope position +1", "other role's bias",
          "dropped feature"]


def _run(wl, plant, layer, role, opts=None):
    S, csr, lt, rope, A, b = _inputs(wl)
    T_r = csr[0].size - 1
    rows = np.arange(T_r)
    x = tr.scaled_features(tr.features(S, lt, csr, rope, layer, role), layer, role, opts)
    ref = tr.map_features(x, A[layer, role], b[layer, role], role, CFG.d_h, layer, rope, opts)
    gate = kernel_gate(x, A[layer, role], b[layer, role], role, CFG.d_h, layer, rope, opts)
    xp, b_lc, shift = x, b[layer, role], 0
    if plant == "csr weight num+1":
        rp, col, num, den = (t.copy() for t in csr)
        j = int(np.nonzero(np.diff(rp) >= 2)[0][0])
        num[rp[j]] += 1
        xp = tr.scaled_features(tr.features(S, lt, (rp, col, num, den), rope, layer, role),
                                layer, role, opts)
    elif plant == "swapped interpolation weights":
        lo, hi, rem, den = lt
        xp = tr.scaled_features(tr.features(S, (lo, hi, den - rem, den), csr, rope, layer, role),
                                layer, role, opts)
    elif plant == "features rounded twice":
        xp = tr.scaled_features(_features_rounded_twice(S, lt, csr, rope, layer, role), layer,
                                role, opts)
    elif plant == "receiver rope position +1":
        shift = 1
    elif plant == "sender rope position +1":
        xp = tr.scaled_features(tr.features(S, lt, csr, dict(rope, pos0_s=1), layer, role),
                                layer, role, opts)
    elif plant == "other role's bias":
        b_lc = b[layer, 1 - role]
    elif plant == "dropped feature":
        xp = x.copy()
        xp[:, 200] = 0.0
    got = _emulate(xp, A[layer, role], b_lc, role, layer, rope, opts, rows, shift)
    return got, ref, gate


# layer 2 of 5 -> 7 interpolates at depth 4/3 (weights 2/3, 1/3), keys carry
# log-normal(0, 1) outlier channels and RoPE 5e5 -> 1e9
@pytest.mark.parametrize("role", [0, 1])
def test_emulated_path_passes_the_gate(wl, role):
    got, ref, gate = _run(wl, "none", 2, role)
    s = check_layer(got, ref, f"emulation role {role}", max_abs="report" if role == 0 else "ulp",
                    gate=gate)
    assert s["gate"] <= 1.0
    if role == 1:
        assert s["max"] <= MAX_ABS


@pytest.mark.parametrize("plant", PLANTS[1:])
def test_planted_mistake_fails_the_gate(wl, plant):
    role = 1 if plant == "other role's bias" else 0
    if plant == "swapped interpolation weights":
        role = 1
    got, ref, gate = _run(wl, plant, 2, role)
    ref_q, bound = gate
    assert np.any(np.abs(got - ref_q) > bound), plant
    with pytest.raises(AssertionError):
        check_layer(got, ref, plant, max_abs="report", gate=gate)


def _paper_opts():
    opts = synth.make_opts(CFG.with_(paper_opts=True), seed=21, device="cpu")
    return dict(inv_r=opts["inv_r"].numpy().astype(np.float64),
                k_norm=opts["k_norm"].numpy().astype(np.float64), k_norm_eps=opts["k_norm_eps"])


def test_scaled_product_passes_its_gate_and_planted_scales_fail(wl):
    # The staged path with concatenated taps rounds x_j without 1/r and scales
    # the product A x_j by 1/r: the gate then rounds x_j unscaled and maps it
    # with A / r (equal to the oracle's A (x_j / r) in exact arithmetic).
    opts = _paper_opts()
    layer, role = 3, 0
    S, csr, lt, rope, A, b = _inputs(wl)
    rows = np.arange(csr[0].size - 1)
    x = tr.features(S, lt, csr, rope, layer, role)
    inv = float(opts["inv_r"][layer, role])
    ref = tr.map_features(tr.scaled_features(x, layer, role, opts), A[layer, role], b[layer, role],
                          role, CFG.d_h, layer, rope, opts)
    o = dict(opts, inv_r=None)
    gate = kernel_gate(x, A[layer, role] * inv, b[layer, role], role, CFG.d_h, layer, rope, o)
    got = _emulate(x, A[layer, role], b[layer, role], role, layer, rope, o, rows, product_scale=inv)
    s = check_layer(got, ref, "scaled product", max_abs="report", gate=gate)
    assert s["gate"] <= 1.0
    ref_q, bound = gate
    for bad in (1.0, inv * inv):  # 1/r left out, 1/r applied twice
        got = _emulate(x, A[layer, role], b[layer, role], role, layer, rope, o, rows,
                       product_scale=bad)
        assert np.any(np.abs(got - ref_q) > bound), bad


def test_planted_mistakes_fail_with_key_norm(wl):
    # The paper's construction: 1/r on the features, key RMSNorm, then RoPE.
    opts = synth.make_opts(CFG.with_(paper_opts=True), seed=21, device="cpu")
    opts = dict(inv_r=opts["inv_r"].numpy().astype(np.float64),
                k_norm=opts["k_norm"].numpy().astype(np.float64), k_norm_eps=opts["k_norm_eps"])
    got, ref, gate = _run(wl, "none", 3, 0, opts)
    check_layer(got, ref, "normed keys", max_abs="report", gate=gate)
    for plant in ("csr weight num+1", "features rounded twice", "receiver rope position +1",
                  "dropped feature"):
        got, ref, gate = _run(wl, plant, 3, 0, opts)
        ref_q, bound = gate
        assert np.any(np.abs(got - ref_q) > bound), plant
