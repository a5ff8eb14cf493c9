"""Offline construction of the folded affine maps, fp64 (test infrastructure;
see package docstring).

For one receiver layer and role, N paired samples: x_n (aligned sender
feature, dimension p = d~_S) and y_n (receiver feature, dimension q = d_R), with
sample weights w_n.

1. Sender RMS (Eq. 3): r = sqrt(sum_n w_n |x_n|^2 / (p sum_n w_n)), Z = X / r.
2. Weighted moments of Z and Y: means mu_Z, mu_Y; covariances Sigma_Z, Sigma_Y
   and the cross-covariance Sigma_ZY (Sec. 3.2, between Eq. 3 and Eq. 4).
   Reading: the weighted covariance is normalized by sum_n w_n.  A and b below
   do not depend on that normalizer (it cancels between the whitening and the
   recoloring).
3. Whitening and Procrustes alignment (Eq. 4): the thin SVD
   Sigma_Z^{-1/2} Sigma_ZY Sigma_Y^{-1/2} = U Lambda Q^T gives R* = U Q^T.
   Sigma^{+-1/2} are the symmetric (principal) roots.
4. Recolor (Eq. 5): A = Sigma_Z^{-1/2} R* Sigma_Y^{1/2} (p x q),
   b = mu_Y - mu_Z A, and y = (x/r) A + b (row-vector form).
   Reading of the unnamed numerical stabilization: a relative ridge
   Sigma + ridge * (tr Sigma / dim) * I on Sigma_Z and on Sigma_Y before their
   roots; ridge = 0 is the unregularized map.
5. Low-rank correction (Sec. 3.3, the residual equation): y^ = y0 + (y0 B) G
   with B (q x rho) and G (rho x q).
6. Fold (Eq. 9): A_final = A (I + B G), b_final = b (I + B G).

The transfer path stores the map transposed ([d_R][d_S], column form
y = A x + b); ``abi_orientation`` converts.
"""

from __future__ import annotations

import numpy as np


def _weights(w, n):
    if w is None:
        return np.ones(n, np.float64)
    w = np.asarray(w, np.float64)
    if w.shape != (n,):
        raise ValueError("weights must have one entry per sample")
    return w


def sender_rms(X, w=None):
    """Eq. 3: one scalar RMS over all weighted samples and feature dimensions."""
    X = np.asarray(X, np.float64)
    n, p = X.shape
    w = _weights(w, n)
    return float(np.sqrt(np.sum(w * np.sum(X * X, axis=1)) / (p * np.sum(w))))


def weighted_moments(X, Y, w=None):
    """Weighted means and (co)variances, normalized by the weight sum.

    Returns (mu_X, mu_Y, S_XX, S_XY, S_YY).
    """
    X = np.asarray(X, np.float64)
    Y = np.asarray(Y, np.float64)
    n = X.shape[0]
    if Y.shape[0] != n:
        raise ValueError("X and Y must pair the same samples")
    w = _weights(w, n)
    W = np.sum(w)
    mu_x = (w @ X) / W
    mu_y = (w @ Y) / W
    Xc = X - mu_x
    Yc = Y - mu_y
    S_xx = (Xc * w[:, None]).T @ Xc / W
    S_xy = (Xc * w[:, None]).T @ Yc / W
    S_yy = (Yc * w[:, None]).T @ Yc / W
    return mu_x, mu_y, S_xx, S_xy, S_yy


def ridge(S, lam):
    """The stabilization reading: S + lam * (tr S / dim) * I."""
    S = np.asarray(S, np.float64)
    if lam == 0:
        return S.copy()
    d = S.shape[0]
    return S + float(lam) * (np.trace(S) / d) * np.eye(d)


def psd_power(S, power):
    """Symmetric power S^power of a symmetric positive definite matrix from its
    eigendecomposition (power = 1/2 or -1/2 for the principal roots)."""
    S = np.asarray(S, np.float64)
    S = 0.5 * (S + S.T)
    lam, V = np.linalg.eigh(S)
    # numerically singular: the usual rank tolerance dim * eps * largest eigenvalue
    if lam.min() <= S.shape[0] * np.finfo(np.float64).eps * max(lam.max(), 0.0):
        raise np.linalg.LinAlgError("covariance is not positive definite")
    return (V * lam ** power) @ V.T


def procrustes(M):
    """Eq. 4: R* = U Q^T from the thin SVD M = U Lambda Q^T."""
    U, _, Qt = np.linalg.svd(np.asarray(M, np.float64), full_matrices=False)
    return U @ Qt


def recolor(mu_z, mu_y, S_zz, S_zy, S_yy, lam=0.0):
    """Eq. 4-5 from the moments of Z = X / r and Y.  Returns (A, b) with A of
    shape (p, q) in the paper's row-vector orientation."""
    Wz = psd_power(ridge(S_zz, lam), -0.5)
    Syr = ridge(S_yy, lam)
    Wy = psd_power(Syr, -0.5)
    Ry = psd_power(Syr, 0.5)
    R = procrustes(Wz @ np.asarray(S_zy, np.float64) @ Wy)
    A = Wz @ R @ Ry
    b = np.asarray(mu_y, np.float64) - np.asarray(mu_z, np.float64) @ A
    return A, b


def recolor_from_samples(X, Y, w=None, lam=0.0):
    """Eq. 3 then Eq. 4-5 on paired samples.  Returns (r, A, b)."""
    r = sender_rms(X, w)
    mu_z, mu_y, S_zz, S_zy, S_yy = weighted_moments(np.asarray(X, np.float64) / r, Y, w)
    A, b = recolor(mu_z, mu_y, S_zz, S_zy, S_yy, lam)
    return r, A, b


def apply_map(X, r, A, b):
    """y = (x / r) A + b for each row x of X (Eq. 5 and Eq. 9)."""
    return np.asarray(X, np.float64) / r @ np.asarray(A, np.float64) + np.asarray(b, np.float64)


def correct(Y0, B, G):
    """The rank-rho output-aware correction added to the Recolor output:
    y^ = y0 + (y0 B) G (Sec. 3.3)."""
    Y0 = np.asarray(Y0, np.float64)
    return Y0 + (Y0 @ np.asarray(B, np.float64)) @ np.asarray(G, np.float64)


def fold(A, b, B, G):
    """Eq. 9: A_final = A (I + B G), b_final = b (I + B G)."""
    B = np.asarray(B, np.float64)
    G = np.asarray(G, np.float64)
    F = np.eye(B.shape[0]) + B @ G
    return np.asarray(A, np.float64) @ F, np.asarray(b, np.float64) @ F


def abi_orientation(A):
    """The transfer path's [d_R][d_in] storage of a row-vector map A (d_in x d_R)."""
    return np.ascontiguousarray(np.asarray(A, np.float64).T)
