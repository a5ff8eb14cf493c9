"""Pins for the concatenated-feature transfer oracle (the paper's layer
alignment, Sec. 3.1 Eq. 1-2): an independent per-element brute force, the
reduction to the already pinned single-layer transfer, the plain-matmul
special case, linearity, and row/full agreement."""

import math

import numpy as np
import pytest

from oracle import alignment as al
from oracle import layer_map as lm
from oracle import transfer as tr
from paper_2609_32259_amd import synth


def _tiny(seed=0, L_s=9, L_r=5, H_s=2, H_r=3, d_h=8, n_taps=3, n_chars=60, rope_on=True):
    rng = np.random.default_rng(seed)
    sb, se = synth.segment_chars(rng, n_chars, 1, 5)
    rb, re_ = synth.segment_chars(rng, n_chars, 1, 7)
    S = rng.standard_normal((L_s, 2, H_s, sb.size, d_h))
    A = rng.standard_normal((L_r, 2, H_r * d_h, n_taps * H_s * d_h)) / math.sqrt(n_taps * H_s * d_h)
    b = 0.3 * rng.standard_normal((L_r, 2, H_r * d_h))
    taps = rng.integers(0, L_s, (L_r, n_taps))
    rp = dict(theta_s=500.0, theta_r=2.0e4, unrotate_sender_k=True, rotate_receiver_k=True,
              pos0_s=3, pos0_r=11) if rope_on else None
    return (sb, se, rb, re_), S, A, b, taps, rp


def brute_taps(S, sb, se, rb, re_, taps, A, bias, rp):
    """Per-token, per-tap, per-head, per-element loops from the definitions,
    with character-level overlap counting and explicit 2x2 rotations."""
    L_s, _, H_s, T_s, d = S.shape
    L_r, _, d_r, _ = A.shape
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
            for c in range(2):
                x = []
                for t in taps[l]:
                    xt = [0.0] * (H_s * d)
                    for i, n in counts.items():
                        for h in range(H_s):
                            m = [S[t, c, h, i, e] for e in range(d)]
                            if c == 0 and rp is not None:
                                pos = rp["pos0_s"] + i
                                u = [0.0] * d
                                for k in range(half):
                                    ang = -pos * rp["theta_s"] ** (-2.0 * k / d)
                                    u[k] = m[k] * math.cos(ang) - m[k + half] * math.sin(ang)
                                    u[k + half] = m[k + half] * math.cos(ang) + m[k] * math.sin(ang)
                                m = u
                            for e in range(d):
                                xt[h * d + e] += n / tot * m[e]
                    x += xt
                y = [sum(A[l, c, o, k] * x[k] for k in range(len(x))) + bias[l, c, o]
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


@pytest.mark.parametrize("seed,rope_on,n_taps", [(20, True, 3), (21, False, 3), (22, True, 2)])
def test_taps_transfer_matches_brute_force(seed, rope_on, n_taps):
    seg, S, A, b, taps, rp = _tiny(seed, rope_on=rope_on, n_taps=n_taps)
    csr = al.overlap_csr(*seg)
    out = tr.transfer_taps(S, taps, csr, A, b, rp)
    ref = brute_taps(S, *seg, taps, A, b, rp)
    assert np.max(np.abs(out - ref)) < 1e-11


def test_one_nonzero_block_is_the_single_layer_transfer():
    """A = [A0 | 0 | 0] reads tap t1 alone: the result equals the (separately
    pinned) single-layer transfer whose layer table names t1 with weight 1."""
    seg, S, A, b, taps, rp = _tiny(23)
    csr = al.overlap_csr(*seg)
    L_r, _, d_r, d3 = A.shape
    d_in = d3 // 3
    A3 = np.zeros_like(A)
    A3[..., :d_in] = A[..., :d_in]
    out = tr.transfer_taps(S, taps, csr, A3, b, rp)
    t1 = taps[:, 0]
    table = (t1, t1, np.zeros(L_r, dtype=np.int64), np.ones(L_r, dtype=np.int64))
    ref = tr.transfer(S, table, csr, A[..., :d_in], b, rp)
    assert np.max(np.abs(out - ref)) < 1e-12


def test_equal_taps_with_split_map_equal_the_single_layer_transfer():
    seg, S, A, b, taps, rp = _tiny(24)
    csr = al.overlap_csr(*seg)
    L_r, _, d_r, d3 = A.shape
    d_in = d3 // 3
    A0 = A[..., :d_in]
    same = np.repeat(taps[:, :1], 3, axis=1)
    out = tr.transfer_taps(S, same, csr, np.concatenate([A0 / 4, A0 / 2, A0 / 4], axis=-1), b, rp)
    table = (same[:, 0], same[:, 0], np.zeros(L_r, dtype=np.int64), np.ones(L_r, dtype=np.int64))
    ref = tr.transfer(S, table, csr, A0, b, rp)
    assert np.max(np.abs(out - ref)) < 1e-12


def test_identity_alignment_is_a_sum_of_matrix_products():
    """Identical tokenizations, no RoPE: y = sum_t A_t S[t] + b on each token."""
    rng = np.random.default_rng(25)
    b_, e_ = synth.segment_chars(rng, 120, 1, 6)
    L_s, L_r, H_s, H_r, d = 10, 4, 2, 3, 8
    S = rng.standard_normal((L_s, 2, H_s, b_.size, d))
    taps = lm.neighbor3(L_s, L_r)
    A = rng.standard_normal((L_r, 2, H_r * d, 3 * H_s * d))
    bias = rng.standard_normal((L_r, 2, H_r * d))
    out = tr.transfer_taps(S, taps, al.overlap_csr(b_, e_, b_, e_), A, bias, None)
    for l in range(L_r):
        for c in range(2):
            Y = bias[l, c][None, :].copy()
            for q, t in enumerate(taps[l]):
                X = S[t, c].transpose(1, 0, 2).reshape(b_.size, H_s * d)
                Y = Y + np.matmul(X, A[l, c][:, q * H_s * d:(q + 1) * H_s * d].T)
            assert np.allclose(out[l, c], Y.reshape(b_.size, H_r, d).transpose(1, 0, 2),
                               rtol=1e-12, atol=1e-12)


def test_identity_map_on_first_block_reproduces_the_sender_layer():
    rng = np.random.default_rng(26)
    b_, e_ = synth.segment_chars(rng, 200, 1, 6)
    L, H, d = 6, 2, 16
    S = rng.standard_normal((L, 2, H, b_.size, d)).astype(np.float32).astype(np.float64)
    taps = lm.neighbor3(L, L)
    A = np.zeros((L, 2, H * d, 3 * H * d))
    A[..., :H * d] = np.eye(H * d)
    for mode in ("overlap", "ta"):
        out = tr.transfer_taps(S, taps, al.build_alignment(b_, e_, b_, e_, mode), A, None, None)
        assert np.array_equal(out, S[taps[:, 0]])


def test_linearity_in_cache_and_maps():
    seg, S1, A1, b1, taps, rp = _tiny(27)
    rng = np.random.default_rng(28)
    S2 = rng.standard_normal(S1.shape)
    A2 = rng.standard_normal(A1.shape)
    b2 = rng.standard_normal(b1.shape)
    csr = al.overlap_csr(*seg)
    f = lambda S, A, b: tr.transfer_taps(S, taps, csr, A, b, rp)  # noqa: E731
    assert np.max(np.abs(f(S1 - 1.5 * S2, A1, None) - (f(S1, A1, None) - 1.5 * f(S2, A1, None)))) < 1e-12
    assert np.max(np.abs(f(S1, A1 + A2, b1 + b2) - (f(S1, A1, b1) + f(S1, A2, b2)))) < 1e-12


def test_rows_form_matches_full_form():
    seg, S, A, b, taps, rp = _tiny(29, n_chars=120)
    csr = al.overlap_csr(*seg)
    full = tr.transfer_taps(S, taps, csr, A, b, rp)
    get = lambda l, c, idx: S[l, c][:, idx, :]  # noqa: E731
    rows = [0, 2, 9, len(seg[2]) - 1]
    for l in (0, 3, 4):
        for c in (0, 1):
            part, xs = tr.transfer_rows_taps(get, taps, csr, A[l, c], b[l, c], rp, S.shape[-1],
                                             l, c, rows, return_features=True)
            assert np.max(np.abs(part - full[l, c][:, rows, :])) < 1e-12
            assert np.max(np.abs(xs - tr.features_taps(S, taps, csr, rp, l, c)[rows])) < 1e-12
