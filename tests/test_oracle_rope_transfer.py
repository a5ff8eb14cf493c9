"""Pins for the RoPE and transfer oracles: closed forms, group identities,
special cases that reduce to a plain matrix product, linearity, and a
brute-force loop implementation written independently from the definitions."""

import math

import numpy as np
import pytest

from oracle import alignment as al
from oracle import layer_map as lm
from oracle import rope
from oracle import transfer as tr
from paper_2609_32259_amd import synth


# --- RoPE ---------------------------------------------------------------------

def test_rope_closed_form_single_pair():
    # d = 2: one pair with frequency 1, so the angle is the position itself.
    pos = np.array([0.0, 1.0, 2.5, -3.0, 1000.0])
    v = np.tile(np.array([1.0, 0.0]), (pos.size, 1))
    out = rope.rotate(v, pos, theta=12345.0)
    assert np.allclose(out[:, 0], np.cos(pos), atol=1e-15)
    assert np.allclose(out[:, 1], np.sin(pos), atol=1e-15)
    w = np.tile(np.array([0.0, 1.0]), (pos.size, 1))
    out = rope.rotate(w, pos, theta=12345.0)
    assert np.allclose(out[:, 0], -np.sin(pos), atol=1e-15)
    assert np.allclose(out[:, 1], np.cos(pos), atol=1e-15)


def test_rope_second_frequency_pairs_rotate_half():
    # d = 4, theta = 100: frequencies 1 and 100**-0.5 = 0.1; element k pairs with k + 2.
    v = np.zeros((1, 4))
    v[0, 1] = 1.0
    out = rope.rotate(v, [7.0], theta=100.0)[0]
    assert np.allclose(out, [0.0, math.cos(0.7), 0.0, math.sin(0.7)], atol=1e-15)


def test_rope_group_identities():
    rng = np.random.default_rng(0)
    v = rng.standard_normal((3, 50, 128))
    pos = rng.integers(0, 40000, 50).astype(np.float64)
    assert np.array_equal(rope.rotate(v, np.zeros(50), 5e5), v)  # R(0) = I
    back = rope.unrotate(rope.rotate(v, pos, 5e5), pos, 5e5)
    assert np.max(np.abs(back - v)) < 1e-12
    # rotation preserves the norm of every pair
    r = rope.rotate(v, pos, 1e9)
    n0 = v[..., :64] ** 2 + v[..., 64:] ** 2
    n1 = r[..., :64] ** 2 + r[..., 64:] ** 2
    assert np.max(np.abs(n0 - n1)) < 1e-12


def test_rope_relative_position():
    rng = np.random.default_rng(1)
    q, k = rng.standard_normal((2, 1, 1, 64))
    dots = []
    for p in (0.0, 17.0, 3000.0):
        qq = rope.rotate(q, [p + 5.0], 1e4)
        kk = rope.rotate(k, [p], 1e4)
        dots.append(float(np.sum(qq * kk)))
    assert np.allclose(dots, dots[0], rtol=0, atol=1e-10)


# --- transfer -----------------------------------------------------------------

def _tiny(seed=0, L_s=3, L_r=5, H_s=2, H_r=3, d_h=8, n_chars=60, rope_on=True):
    rng = np.random.default_rng(seed)
    sb, se = synth.segment_chars(rng, n_chars, 1, 5)
    rb, re_ = synth.segment_chars(rng, n_chars, 1, 7)
    S = rng.standard_normal((L_s, 2, H_s, sb.size, d_h))
    A = rng.standard_normal((L_r, 2, H_r * d_h, H_s * d_h)) / math.sqrt(H_s * d_h)
    b = 0.3 * rng.standard_normal((L_r, 2, H_r * d_h))
    rp = dict(theta_s=500.0, theta_r=2.0e4, unrotate_sender_k=True, rotate_receiver_k=True,
              pos0_s=3, pos0_r=11) if rope_on else None
    return (sb, se, rb, re_), S, A, b, rp


def test_identity_transfer_reproduces_sender_exactly():
    rng = np.random.default_rng(2)
    b_, e_ = synth.segment_chars(rng, 300, 1, 6)
    L, H, d = 4, 3, 16
    S = rng.standard_normal((L, 2, H, b_.size, d)).astype(np.float32).astype(np.float64)
    A = np.broadcast_to(np.eye(H * d), (L, 2, H * d, H * d))
    for mode in ("overlap", "ta"):
        csr = al.build_alignment(b_, e_, b_, e_, mode)
        out = tr.transfer(S, lm.interp2(L, L), csr, A, None, None)
        assert np.array_equal(out, S)


def test_equal_rope_round_trip_is_identity():
    rng = np.random.default_rng(4)
    b_, e_ = synth.segment_chars(rng, 200, 1, 6)
    L, H, d = 2, 2, 32
    S = rng.standard_normal((L, 2, H, b_.size, d))
    A = np.broadcast_to(np.eye(H * d), (L, 2, H * d, H * d))
    rp = dict(theta_s=5e5, theta_r=5e5, unrotate_sender_k=True, rotate_receiver_k=True,
              pos0_s=7, pos0_r=7)
    out = tr.transfer(S, lm.interp2(L, L), al.overlap_csr(b_, e_, b_, e_), A, None, rp)
    assert np.max(np.abs(out - S)) < 1e-12


def test_single_tap_identity_alignment_is_a_matrix_product():
    """With identical tokenizations and one sender layer per receiver layer,
    the transfer is y = A x + b on each flattened token: a plain matmul."""
    rng = np.random.default_rng(5)
    b_, e_ = synth.segment_chars(rng, 150, 1, 6)
    L, H_s, H_r, d = 3, 2, 3, 8
    S = rng.standard_normal((L, 2, H_s, b_.size, d))
    A = rng.standard_normal((L, 2, H_r * d, H_s * d))
    bias = rng.standard_normal((L, 2, H_r * d))
    out = tr.transfer(S, lm.interp2(L, L), al.overlap_csr(b_, e_, b_, e_), A, bias, None)
    for l in range(L):
        for c in range(2):
            X = S[l, c].transpose(1, 0, 2).reshape(b_.size, H_s * d)   # [T, H_s*d], head-major
            Y = np.matmul(X, A[l, c].T) + bias[l, c]
            assert np.allclose(out[l, c], Y.reshape(b_.size, H_r, d).transpose(1, 0, 2),
                               rtol=1e-12, atol=1e-12)


def test_layer_interpolation_recovers_fractional_depth():
    # Sender layer l holds the constant l; with identity alignment and A = I the
    # receiver layer j holds its fractional sender depth j (L_s-1)/(L_r-1).
    rng = np.random.default_rng(6)
    b_, e_ = synth.segment_chars(rng, 40, 1, 4)
    L_s, L_r, H, d = 5, 8, 1, 4
    S = np.broadcast_to(np.arange(L_s, dtype=np.float64)[:, None, None, None, None],
                        (L_s, 2, H, b_.size, d))
    A = np.broadcast_to(np.eye(H * d), (L_r, 2, H * d, H * d))
    out = tr.transfer(S, lm.interp2(L_s, L_r), al.overlap_csr(b_, e_, b_, e_), A, None, None)
    for j in range(L_r):
        assert np.allclose(out[j], j * (L_s - 1) / (L_r - 1), rtol=0, atol=1e-14)


def test_segment_mean_of_constant_rows():
    # Sender token i holds the constant i: receiver row j holds the
    # overlap-weighted mean of the indices it reads.
    rng = np.random.default_rng(7)
    sb, se = synth.segment_chars(rng, 80, 1, 6)
    rb, re_ = synth.segment_chars(rng, 80, 1, 8)
    S = np.broadcast_to(np.arange(sb.size, dtype=np.float64)[None, None, None, :, None],
                        (1, 2, 1, sb.size, 2))
    A = np.broadcast_to(np.eye(2), (1, 2, 2, 2))
    csr = al.overlap_csr(sb, se, rb, re_)
    out = tr.transfer(S, lm.interp2(1, 1), csr, A, None, None)
    for j in range(rb.size):
        tot = sum(max(0, min(se[i], re_[j]) - max(sb[i], rb[j])) * i for i in range(sb.size))
        assert abs(out[0, 0, 0, j, 0] - tot / (re_[j] - rb[j])) < 1e-12


def test_linearity_in_cache_and_maps():
    seg, S1, A1, b1, rp = _tiny(8)
    rng = np.random.default_rng(9)
    S2 = rng.standard_normal(S1.shape)
    A2 = rng.standard_normal(A1.shape)
    b2 = rng.standard_normal(b1.shape)
    L_s, L_r = S1.shape[0], A1.shape[0]
    csr = al.overlap_csr(*seg)
    lt = lm.interp2(L_s, L_r)
    f = lambda S, A, b: tr.transfer(S, lt, csr, A, b, rp)  # noqa: E731
    lhs = f(S1 + 2.5 * S2, A1, None)
    rhs = f(S1, A1, None) + 2.5 * f(S2, A1, None)
    assert np.max(np.abs(lhs - rhs)) < 1e-12
    lhs = f(S1, A1 + A2, b1 + b2)
    rhs = f(S1, A1, b1) + f(S1, A2, b2)
    assert np.max(np.abs(lhs - rhs)) < 1e-12


def brute_transfer(S, sb, se, rb, re_, L_r, A, bias, rp):
    """Per-token, per-head, per-element loops straight from the definitions,
    with character-level overlap counting and explicit 2x2 rotations."""
    L_s, _, H_s, T_s, d = S.shape
    d_r = A.shape[2]
    H_r = d_r // d
    half = d // 2
    T_r = len(rb)
    a_ta = al.ta_alignment(sb, se, rb, re_)
    out = np.zeros((L_r, 2, H_r, T_r, d))
    for j in range(T_r):
        counts = {}
        for ch in range(int(rb[j]), int(re_[j])):
            for i in range(T_s):
                if sb[i] <= ch < se[i]:
                    counts[i] = counts.get(i, 0) + 1
        if not counts:
            counts = {int(a_ta[j]): 1}
        tot = sum(counts.values())
        for l in range(L_r):
            p = Fraction(l * (L_s - 1), L_r - 1) if L_r > 1 else Fraction(0)
            lo = int(p)
            f = float(p - lo)
            hi = min(lo + 1, L_s - 1)
            for c in range(2):
                x = [0.0] * (H_s * d)
                for i, n in counts.items():
                    for h in range(H_s):
                        m = [(1 - f) * S[lo, c, h, i, e] + (f * S[hi, c, h, i, e] if f else 0.0)
                             for e in range(d)]
                        if c == 0 and rp is not None:
                            pos = rp["pos0_s"] + i
                            u = [0.0] * d
                            for k in range(half):
                                ang = -pos * rp["theta_s"] ** (-2.0 * k / d)
                                u[k] = m[k] * math.cos(ang) - m[k + half] * math.sin(ang)
                                u[k + half] = m[k + half] * math.cos(ang) + m[k] * math.sin(ang)
                            m = u
                        for e in range(d):
                            x[h * d + e] += n / tot * m[e]
                y = [sum(A[l, c, o, k] * x[k] for k in range(H_s * d)) + bias[l, c, o]
                     for o in range(d_r)]
                for h in range(H_r):
                    v = y[h * d:(h + 1) * d]
                    if c == 0 and rp is not None:
                        pos = rp["pos0_r"] + j
                        w = [0.0] * d
                        for k in range(half):
                            ang = pos * rp["theta_r"] ** (-2.0 * k / d)
                            w[k] = v[k] * math.cos(ang) - v[k + half] * math.sin(ang)
                            w[k + half] = v[k + half] * math.cos(ang) + v[k] * math.sin(ang)
                        v = w
                    out[l, c, h, j, :] = v
    return out


from fractions import Fraction  # noqa: E402


@pytest.mark.parametrize("seed,rope_on", [(10, True), (11, False), (12, True)])
def test_transfer_matches_brute_force(seed, rope_on):
    seg, S, A, b, rp = _tiny(seed, rope_on=rope_on)
    L_s, L_r = S.shape[0], A.shape[0]
    csr = al.overlap_csr(*seg)
    out = tr.transfer(S, lm.interp2(L_s, L_r), csr, A, b, rp)
    ref = brute_transfer(S, *seg, L_r, A, b, rp)
    assert np.max(np.abs(out - ref)) < 1e-11


def test_transfer_rows_matches_transfer():
    seg, S, A, b, rp = _tiny(13, L_s=4, L_r=6, n_chars=120)
    lt = lm.interp2(4, 6)
    csr = al.overlap_csr(*seg)
    full = tr.transfer(S, lt, csr, A, b, rp)
    get = lambda l, c, idx: S[l, c][:, idx, :]  # noqa: E731
    rows = [0, 3, 7, len(seg[2]) - 1]
    for l in (0, 2, 5):
        for c in (0, 1):
            part = tr.transfer_rows(get, lt, csr, A[l, c], b[l, c], rp, S.shape[-1], l, c, rows)
            assert np.max(np.abs(part - full[l, c][:, rows, :])) < 1e-12
