"""Pins for the transfer oracle's paper-faithful options (Eq. 3 / Eq. 9: the
map sees x / r; App. B.1: the receiver's key normalization, then its RoPE):
closed forms of the per-head RMSNorm, the scalar 1/r against a scaled map,
the normalize-then-rotate order, and a brute force with both options."""

import math

import numpy as np
import pytest

from oracle import alignment as al
from oracle import layer_map as lm
from oracle import rope
from oracle import transfer as tr
from paper_2609_32259_amd import synth


def test_rms_norm_closed_forms():
    # [3, 4]: mean square 12.5, so the unit-weight result is [3, 4] / sqrt(12.5)
    out = tr.rms_norm(np.array([3.0, 4.0]), np.ones(2), 0.0)
    assert np.allclose(out, [3.0 / math.sqrt(12.5), 4.0 / math.sqrt(12.5)], rtol=0, atol=1e-15)
    rng = np.random.default_rng(0)
    y = rng.standard_normal((5, 7, 128))
    n = tr.rms_norm(y, np.ones(128), 0.0)
    assert np.allclose(np.mean(n * n, axis=-1), 1.0, rtol=0, atol=1e-12)      # unit RMS
    assert np.allclose(tr.rms_norm(3.5 * y, np.ones(128), 0.0), n, atol=1e-12)  # scale-free
    g = rng.standard_normal(128)
    assert np.allclose(tr.rms_norm(y, g, 0.0), n * g, atol=1e-12)             # weight per feature
    # eps enters under the root: a zero head stays zero, a tiny head is damped
    assert np.array_equal(tr.rms_norm(np.zeros(8), np.ones(8), 1e-6), np.zeros(8))
    t = tr.rms_norm(np.full(4, 1e-4), np.ones(4), 1e-6)
    assert np.allclose(t, 1e-4 / math.sqrt(1e-8 + 1e-6), rtol=1e-14)


def _tiny(seed, L_s=3, L_r=4, H_s=2, H_r=3, d_h=8, n_chars=50):
    rng = np.random.default_rng(seed)
    sb, se = synth.segment_chars(rng, n_chars, 1, 5)
    rb, re_ = synth.segment_chars(rng, n_chars, 1, 7)
    S = rng.standard_normal((L_s, 2, H_s, sb.size, d_h))
    A = rng.standard_normal((L_r, 2, H_r * d_h, H_s * d_h)) / math.sqrt(H_s * d_h)
    b = 0.3 * rng.standard_normal((L_r, 2, H_r * d_h))
    rp = dict(theta_s=700.0, theta_r=3.0e4, unrotate_sender_k=True, rotate_receiver_k=True,
              pos0_s=2, pos0_r=9)
    opts = dict(inv_r=rng.uniform(0.2, 3.0, (L_r, 2)), k_norm=rng.uniform(0.5, 1.5, (L_r, d_h)),
                k_norm_eps=1e-5)
    return (sb, se, rb, re_), S, A, b, rp, opts


def test_inv_r_equals_a_scaled_map():
    seg, S, A, b, rp, opts = _tiny(1)
    csr = al.overlap_csr(*seg)
    lt = lm.interp2(S.shape[0], A.shape[0])
    out = tr.transfer(S, lt, csr, A, b, rp, opts=dict(inv_r=opts["inv_r"]))
    ref = tr.transfer(S, lt, csr, A * opts["inv_r"][:, :, None, None], b, rp)
    assert np.max(np.abs(out - ref)) < 1e-12


def test_key_norm_is_applied_before_the_receiver_rope():
    """With identity alignment, an identity map and no bias, the keys are
    rope(rmsnorm(S)); the weights differ between the two halves of each RoPE
    pair, so the other order gives a different result."""
    rng = np.random.default_rng(2)
    b_, e_ = synth.segment_chars(rng, 80, 1, 5)
    L, H, d = 2, 2, 8
    S = rng.standard_normal((L, 2, H, b_.size, d))
    A = np.broadcast_to(np.eye(H * d), (L, 2, H * d, H * d))
    g = np.concatenate([np.full(d // 2, 0.5), np.full(d // 2, 2.0)])
    opts = dict(k_norm=np.tile(g, (L, 1)), k_norm_eps=0.0)
    rp = dict(theta_s=1.0, theta_r=100.0, unrotate_sender_k=False, rotate_receiver_k=True,
              pos0_s=0, pos0_r=5)
    out = tr.transfer(S, lm.interp2(L, L), al.overlap_csr(b_, e_, b_, e_), A, None, rp, opts=opts)
    pos = 5 + np.arange(b_.size)
    for l in range(L):
        y = S[l, 0]
        rms = np.sqrt(np.mean(y * y, axis=-1, keepdims=True))
        first = rope.rotate(y / rms * g, pos, 100.0)                      # normalize, then rotate
        other = rope.rotate(y, pos, 100.0)
        other = other / np.sqrt(np.mean(other * other, axis=-1, keepdims=True)) * g
        assert np.max(np.abs(out[l, 0] - first)) < 1e-12
        assert np.max(np.abs(first - other)) > 1e-2
        assert np.max(np.abs(out[l, 1] - S[l, 1])) < 1e-12               # values untouched


def brute_opts(S, sb, se, rb, re_, L_r, A, bias, rp, opts):
    """Per-element loops from the definitions with 1/r and the key norm."""
    L_s, _, H_s, T_s, d = S.shape
    d_r = A.shape[2]
    H_r = d_r // d
    half = d // 2
    out = np.zeros((L_r, 2, H_r, len(rb), d))
    a_ta = al.ta_alignment(sb, se, rb, re_)
    for j in range(len(rb)):
        counts = {}
        for ch in range(int(rb[j]), int(re_[j])):
            for i in range(T_s):
                if sb[i] <= ch < se[i]:
                    counts[i] = counts.get(i, 0) + 1
        if not counts:
            counts = {int(a_ta[j]): 1}
        tot = sum(counts.values())
        for l in range(L_r):
            num = l * (L_s - 1)
            lo, rem = divmod(num, L_r - 1) if L_r > 1 else (0, 0)
            f = rem / (L_r - 1) if L_r > 1 else 0.0
            hi = min(lo + 1, L_s - 1)
            for c in range(2):
                x = [0.0] * (H_s * d)
                for i, n in counts.items():
                    for h in range(H_s):
                        m = [(1 - f) * S[lo, c, h, i, e] + f * S[hi, c, h, i, e] for e in range(d)]
                        if c == 0:
                            u = [0.0] * d
                            for k in range(half):
                                ang = -(rp["pos0_s"] + i) * rp["theta_s"] ** (-2.0 * k / d)
                                u[k] = m[k] * math.cos(ang) - m[k + half] * math.sin(ang)
                                u[k + half] = m[k + half] * math.cos(ang) + m[k] * math.sin(ang)
                            m = u
                        for e in range(d):
                            x[h * d + e] += n / tot * m[e] * opts["inv_r"][l, c]
                y = [sum(A[l, c, o, k] * x[k] for k in range(H_s * d)) + bias[l, c, o]
                     for o in range(d_r)]
                for h in range(H_r):
                    v = y[h * d:(h + 1) * d]
                    if c == 0:
                        ms = sum(t * t for t in v) / d
                        v = [v[e] / math.sqrt(ms + opts["k_norm_eps"]) * opts["k_norm"][l, e]
                             for e in range(d)]
                        w = [0.0] * d
                        for k in range(half):
                            ang = (rp["pos0_r"] + j) * rp["theta_r"] ** (-2.0 * k / d)
                            w[k] = v[k] * math.cos(ang) - v[k + half] * math.sin(ang)
                            w[k + half] = v[k + half] * math.cos(ang) + v[k] * math.sin(ang)
                        v = w
                    out[l, c, h, j, :] = v
    return out


@pytest.mark.parametrize("seed", [3, 4])
def test_options_match_brute_force(seed):
    seg, S, A, b, rp, opts = _tiny(seed)
    L_r = A.shape[0]
    out = tr.transfer(S, lm.interp2(S.shape[0], L_r), al.overlap_csr(*seg), A, b, rp, opts=opts)
    ref = brute_opts(S, *seg, L_r, A, b, rp, opts)
    assert np.max(np.abs(out - ref)) < 1e-11


def test_options_on_taps_and_rows_agree():
    seg, S, A, b, rp, opts = _tiny(5, L_s=9)
    L_r = A.shape[0]
    taps = lm.neighbor3(S.shape[0], L_r)
    rng = np.random.default_rng(6)
    A3 = rng.standard_normal((L_r, 2, A.shape[2], 3 * A.shape[3])) / 8.0
    csr = al.overlap_csr(*seg)
    full = tr.transfer_taps(S, taps, csr, A3, b, rp, opts=opts)
    # the single-block case reduces to transfer() with the same options
    A1 = np.zeros_like(A3)
    A1[..., :A.shape[3]] = A
    t1 = taps[:, 0]
    table = (t1, t1, np.zeros(L_r, np.int64), np.ones(L_r, np.int64))
    assert np.max(np.abs(tr.transfer_taps(S, taps, csr, A1, b, rp, opts=opts)
                         - tr.transfer(S, table, csr, A, b, rp, opts=opts))) < 1e-12
    get = lambda l, c, idx: S[l, c][:, idx, :]  # noqa: E731
    rows = [0, 4, len(seg[2]) - 1]
    for l in (0, 3):
        for c in (0, 1):
            part = tr.transfer_rows_taps(get, taps, csr, A3[l, c], b[l, c], rp, S.shape[-1], l, c,
                                         rows, opts=opts)
            assert np.max(np.abs(part - full[l, c][:, rows, :])) < 1e-12
    lt = lm.interp2(S.shape[0], L_r)
    full2 = tr.transfer(S, lt, csr, A, b, rp, opts=opts)
    for l in (1, 2):
        for c in (0, 1):
            part = tr.transfer_rows(get, lt, csr, A[l, c], b[l, c], rp, S.shape[-1], l, c, rows,
                                    opts=opts)
            assert np.max(np.abs(part - full2[l, c][:, rows, :])) < 1e-12
