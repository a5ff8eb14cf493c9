"""Transfer oracle: sender KV cache -> receiver KV cache, fp64 (test
infrastructure; see package docstring).

For one sequence, receiver layer l, role c in {K=0, V=1} and receiver token j:

1. Layer interpolation (two nearest sender layers, weights from the integer
   layer table):  m_i = a_lo * S[lo, c, :, i, :] + a_hi * S[hi, c, :, i, :]
   (the hi tap is absent when rem == 0).
2. Keys stored after the sender's RoPE are un-rotated at sender position
   p_i = pos0_s + i with the sender's theta: u_i = U_s(p_i) m_i.  Values and
   pre-RoPE keys pass unchanged.
3. Token alignment: x_j = sum over the CSR row of (num / den_j) * u_i,
   flattened head-major (feature index h * d_h + e) -- the flattened role-c
   KV feature of Sec. 3.1 (Eq. 2 with one interpolated tap).
4. Folded affine map of Eq. 9, written in column form: y_j = A[l, c] (x_j / r)
   + b[l, c] with A stored [d_R, d_S] (the transpose of the paper's row-vector
   A_final).  The scalar r of Eq. 3 is given per (layer, role) as inv_r =
   1/r (absent: 1, i.e. folded into A by the caller).
5. Reshape into receiver KV heads.  For keys, apply the receiver's key
   normalization when given -- RMSNorm over each head's d_h features with
   weight g[l] and epsilon eps: y <- y / sqrt(mean(y^2) + eps) * g -- and
   then the receiver's RoPE at q_j = pos0_r + j with the receiver's theta
   (Sec. 3.3 "Folding for inference"; App. B.1: keys are mapped before key
   normalization and RoPE, which the receiver applies once).
6. R[l, c, h', j, e'] = y_j[h' * d_h + e'].

The optional inv_r / key normalization come in an ``opts`` dict:
``{"inv_r": [L_R, 2] or None, "k_norm": [L_R, d_h] or None, "k_norm_eps": e}``.

Inputs are the exact stored values widened to fp64; the result stays fp64.
"""

from __future__ import annotations

import numpy as np
import scipy.sparse as sp

from . import rope as _rope
from .layer_map import interp2_weights

K, V = 0, 1


def rms_norm(y, g, eps):
    """RMSNorm over the last axis (one receiver head's d_h features)."""
    y = np.asarray(y, dtype=np.float64)
    return y / np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + float(eps)) * np.asarray(g, np.float64)


def _opts(opts):
    opts = opts or {}
    return opts.get("inv_r"), opts.get("k_norm"), float(opts.get("k_norm_eps", 1e-6))


def _mix(S_lo, S_hi, a_lo, a_hi, rem):
    m = a_lo * S_lo
    if rem != 0:
        m = m + a_hi * S_hi
    return m


def _weights_matrix(csr, T_s):
    row_ptr, col, num, den = (np.asarray(t, dtype=np.int64) for t in csr)
    T_r = row_ptr.size - 1
    rows = np.repeat(np.arange(T_r), np.diff(row_ptr))
    w = num.astype(np.float64) / den[rows].astype(np.float64)
    return sp.csr_matrix((w, col, row_ptr), shape=(T_r, T_s))


def features(S, layer_table, csr, rope, layer, role):
    """Steps 1-3 for one receiver layer and role: the aligned, interpolated,
    un-rotated flattened sender features x_j, fp64 [T_R, H_S * d_h]."""
    S = np.asarray(S, dtype=np.float64)
    _, _, H_s, T_s, d_h = S.shape
    lo, hi, rem, den_l = (np.asarray(t) for t in layer_table)
    a_lo, a_hi = interp2_weights(lo, hi, rem, den_l)
    m = _mix(S[lo[layer], role], S[hi[layer], role], a_lo[layer], a_hi[layer], rem[layer])
    if role == K and rope is not None and rope.get("unrotate_sender_k", False):
        m = _rope.unrotate(m, rope.get("pos0_s", 0) + np.arange(T_s), rope["theta_s"])
    u = m.transpose(1, 0, 2).reshape(T_s, H_s * d_h)                    # head-major
    return _weights_matrix(csr, T_s) @ u


def map_features(x, A_lc, b_lc, role, d_h, layer=0, rope=None, opts=None, rows=None):
    """Steps 4-6 for one receiver layer and role, from the features the map
    sees (x_j / r, i.e. 1/r already applied): y_j = A_lc x_j + b_lc (Eq. 9 in
    column form), reshaped into receiver heads; keys then take the receiver's
    key normalization (weights k_norm[layer]) and its rotation at
    q_j = pos0_r + j.
    x     fp64 [n, d_in]; rows: the receiver indices j of x's rows (default
          0..n-1), used only for the rotation
    returns fp64 [H_R, n, d_h]"""
    _, k_norm, eps = _opts(opts)
    x = np.asarray(x, dtype=np.float64)
    A_lc = np.asarray(A_lc, dtype=np.float64)
    n = x.shape[0]
    H_r = A_lc.shape[0] // d_h
    y = x @ A_lc.T
    if b_lc is not None:
        y = y + np.asarray(b_lc, dtype=np.float64)[None, :]
    y = y.reshape(n, H_r, d_h).transpose(1, 0, 2)                           # [H_r, n, d_h]
    if role == K and k_norm is not None:
        y = rms_norm(y, np.asarray(k_norm)[layer], eps)
    if role == K and rope is not None and rope.get("rotate_receiver_k", False):
        j = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
        y = _rope.rotate(y, rope.get("pos0_r", 0) + j, rope["theta_r"])
    return y


def scaled_features(x, layer, role, opts=None):
    """x_j / r: the features scaled by the 1/r of Eq. 3 when opts gives it."""
    inv_r, _, _ = _opts(opts)
    if inv_r is None:
        return np.asarray(x, dtype=np.float64)
    return np.asarray(x, dtype=np.float64) * float(np.asarray(inv_r, np.float64)[layer, role])


def transfer(S, layer_table, csr, A, b=None, rope=None, H_r=None, opts=None):
    """Whole receiver cache of one sequence.

    S           fp64-convertible [L_S, 2, H_S, T_S, d_h]
    layer_table (lo, hi, rem, den) int arrays [L_R]
    csr         (row_ptr[T_R+1], col, num, den[T_R]) for this sequence
    A           [L_R, 2, d_R, d_S];  b  [L_R, 2, d_R] or None
    rope        None or dict(theta_s, theta_r, unrotate_sender_k,
                rotate_receiver_k, pos0_s, pos0_r)
    opts        None or dict(inv_r, k_norm, k_norm_eps) (module docstring)
    returns     [L_R, 2, H_R, T_R, d_h] fp64
    """
    S = np.asarray(S, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    L_s, _, H_s, T_s, d_h = S.shape
    L_r, _, d_r, d_in = A.shape
    if d_in != H_s * d_h:
        raise ValueError("A's input size must be H_S * d_h")
    H_r = d_r // d_h if H_r is None else H_r
    T_r = np.asarray(csr[0]).size - 1
    out = np.empty((L_r, 2, H_r, T_r, d_h), dtype=np.float64)
    for l in range(L_r):
        for c in (K, V):
            x = features(S, layer_table, csr, rope, l, c)                  # [T_r, d_S]
            x = scaled_features(x, l, c, opts)
            out[l, c] = map_features(x, A[l, c], None if b is None else np.asarray(b)[l, c],
                                     c, d_h, l, rope, opts)
    return out


def transfer_rows(get_sender, layer_table, csr, A_lc, b_lc, rope, d_h,
                  layer, role, rows, return_features=False, opts=None):
    """Selected receiver rows of one (layer, role), entry by entry.

    get_sender(l, c, idx) -> fp64 [H_S, len(idx), d_h] gives sender rows idx
    of sender layer l, role c (only the rows the CSR entries name are asked
    for).  A_lc is A[layer, role] ([d_R, d_S]); b_lc its bias or None.
    Returns fp64 [H_R, len(rows), d_h] (and the features x, fp64
    [len(rows), d_S], when return_features).  opts as in ``transfer``.
    """
    inv_r, k_norm, eps = _opts(opts)
    lo, hi, rem, den_l = (np.asarray(t) for t in layer_table)
    a_lo, a_hi = interp2_weights(lo, hi, rem, den_l)
    row_ptr, col, num, den = (np.asarray(t, dtype=np.int64) for t in csr)
    A_lc = np.asarray(A_lc, dtype=np.float64)
    d_r, d_in = A_lc.shape
    H_r = d_r // d_h
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((H_r, rows.size, d_h), dtype=np.float64)
    xs = np.empty((rows.size, d_in), dtype=np.float64)
    unrot = role == K and rope is not None and rope.get("unrotate_sender_k", False)
    rot = role == K and rope is not None and rope.get("rotate_receiver_k", False)
    for n, j in enumerate(rows):
        ents = range(row_ptr[j], row_ptr[j + 1])
        idx = np.asarray([col[e] for e in ents], dtype=np.int64)
        S_lo = get_sender(int(lo[layer]), role, idx)
        S_hi = get_sender(int(hi[layer]), role, idx) if rem[layer] != 0 else None
        x = np.zeros(d_in, dtype=np.float64)
        for q, e in enumerate(ents):
            m = a_lo[layer] * S_lo[:, q, :]
            if rem[layer] != 0:
                m = m + a_hi[layer] * S_hi[:, q, :]
            if unrot:
                p = rope.get("pos0_s", 0) + int(col[e])
                m = _rope.unrotate(m[:, None, :], [p], rope["theta_s"])[:, 0, :]
            x += (float(num[e]) / float(den[j])) * m.reshape(-1)
        if inv_r is not None:
            x = x * float(np.asarray(inv_r, np.float64)[layer, role])
        xs[n] = x
        y = A_lc @ x
        if b_lc is not None:
            y = y + np.asarray(b_lc, dtype=np.float64)
        y = y.reshape(H_r, d_h)
        if role == K and k_norm is not None:
            y = rms_norm(y, np.asarray(k_norm)[layer], eps)
        if rot:
            qpos = rope.get("pos0_r", 0) + int(j)
            y = _rope.rotate(y[:, None, :], [qpos], rope["theta_r"])[:, 0, :]
        out[:, n, :] = y
    return (out, xs) if return_features else out


# ---------------------------------------------------------------------------
# Concatenated-feature maps (the paper's own layer alignment, Sec. 3.1 Eq. 2).
#
# Receiver layer l reads n sender layers taps[l] = (t_1, .., t_n) -- for the
# paper's map the three layers of Eq. 1 -- without interpolation.  For each
# tap t the aligned feature is
#     x_j^t = sum over the CSR row of (num / den_j) * U_s(p_i) S[t, c, :, i, :]
# (un-rotation for post-RoPE keys only), flattened head-major, and the map
# sees their concatenation x_j = [x_j^{t_1} | .. | x_j^{t_n}] (Eq. 2), so
# A[l, c] is [d_R, n * d_S].  The rest (bias, receiver RoPE, reshape) is as
# in ``transfer``.
# ---------------------------------------------------------------------------

def aligned_layer(S, sender_layer, csr, rope, role):
    """x^t of one sender layer t, fp64 [T_R, H_S * d_h]."""
    S = np.asarray(S, dtype=np.float64)
    _, _, H_s, T_s, d_h = S.shape
    m = S[sender_layer, role]
    if role == K and rope is not None and rope.get("unrotate_sender_k", False):
        m = _rope.unrotate(m, rope.get("pos0_s", 0) + np.arange(T_s), rope["theta_s"])
    u = m.transpose(1, 0, 2).reshape(T_s, H_s * d_h)                    # head-major
    return _weights_matrix(csr, T_s) @ u


def features_taps(S, taps, csr, rope, layer, role):
    """Concatenated features of Eq. 2, fp64 [T_R, n * H_S * d_h]."""
    return np.concatenate([aligned_layer(S, int(t), csr, rope, role)
                           for t in np.asarray(taps)[layer]], axis=1)


def transfer_taps(S, taps, csr, A, b=None, rope=None, H_r=None, opts=None):
    """Whole receiver cache with concatenated-feature maps.

    taps  int [L_R, n] sender layers of each receiver layer
    A     [L_R, 2, d_R, n * d_S];  b  [L_R, 2, d_R] or None
    other arguments and the result as in ``transfer``
    """
    S = np.asarray(S, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    taps = np.asarray(taps)
    _, _, H_s, _, d_h = S.shape
    L_r, _, d_r, d_in = A.shape
    if d_in != taps.shape[1] * H_s * d_h:
        raise ValueError("A's input size must be n_taps * H_S * d_h")
    H_r = d_r // d_h if H_r is None else H_r
    T_r = np.asarray(csr[0]).size - 1
    out = np.empty((L_r, 2, H_r, T_r, d_h), dtype=np.float64)
    for l in range(L_r):
        for c in (K, V):
            x = scaled_features(features_taps(S, taps, csr, rope, l, c), l, c, opts)
            out[l, c] = map_features(x, A[l, c], None if b is None else np.asarray(b)[l, c],
                                     c, d_h, l, rope, opts)
    return out


def transfer_rows_taps(get_sender, taps, csr, A_lc, b_lc, rope, d_h, layer, role, rows,
                       return_features=False, opts=None):
    """Selected receiver rows of one (layer, role) with concatenated-feature
    maps, entry by entry (get_sender as in ``transfer_rows``)."""
    inv_r, k_norm, eps = _opts(opts)
    taps = np.asarray(taps)[layer]
    row_ptr, col, num, den = (np.asarray(t, dtype=np.int64) for t in csr)
    A_lc = np.asarray(A_lc, dtype=np.float64)
    d_r, d_in = A_lc.shape
    H_r = d_r // d_h
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((H_r, rows.size, d_h), dtype=np.float64)
    xs = np.empty((rows.size, d_in), dtype=np.float64)
    unrot = role == K and rope is not None and rope.get("unrotate_sender_k", False)
    rot = role == K and rope is not None and rope.get("rotate_receiver_k", False)
    for n, j in enumerate(rows):
        ents = range(row_ptr[j], row_ptr[j + 1])
        idx = np.asarray([col[e] for e in ents], dtype=np.int64)
        blocks = []
        for t in taps:
            St = get_sender(int(t), role, idx)                           # [H_S, len, d_h]
            x = np.zeros(St.shape[0] * d_h, dtype=np.float64)
            for q, e in enumerate(ents):
                m = St[:, q, :]
                if unrot:
                    p = rope.get("pos0_s", 0) + int(col[e])
                    m = _rope.unrotate(m[:, None, :], [p], rope["theta_s"])[:, 0, :]
                x += (float(num[e]) / float(den[j])) * m.reshape(-1)
            blocks.append(x)
        x = np.concatenate(blocks)
        if inv_r is not None:
            x = x * float(np.asarray(inv_r, np.float64)[layer, role])
        xs[n] = x
        y = A_lc @ x
        if b_lc is not None:
            y = y + np.asarray(b_lc, dtype=np.float64)
        y = y.reshape(H_r, d_h)
        if role == K and k_norm is not None:
            y = rms_norm(y, np.asarray(k_norm)[layer], eps)
        if rot:
            qpos = rope.get("pos0_r", 0) + int(j)
            y = _rope.rotate(y[:, None, :], [qpos], rope["theta_r"])[:, 0, :]
        out[:, n, :] = y
    return (out, xs) if return_features else out
