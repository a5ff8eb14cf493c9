"""Pins of the offline map construction oracle (Eq. 3-5, Eq. 9) against closed
forms, library routines and the identities the paper states.

The paper prints no worked example for Recolor; every pin here is a closed
form, a library routine on a special case, an invariant the paper states
(mu_Z A + b = mu_Y and A^T Sigma_Z A = Sigma_Y for p >= q and nonsingular
covariances), or exact recovery of a planted affine relation.
"""

import numpy as np
import pytest
import scipy.linalg

from oracle import recolor as rc


def _samples(rng, n, p, q, noise=0.3, mean_scale=1.0):
    """Correlated paired samples: X with a spread of variances, Y a noisy linear
    function of X.  Generates inputs only."""
    L = rng.standard_normal((p, p)) * np.logspace(0, -1.5, p)[None, :]
    X = rng.standard_normal((n, p)) @ L.T + mean_scale * rng.standard_normal(p)
    C = rng.standard_normal((p, q)) / np.sqrt(p)
    Y = X @ C + noise * rng.standard_normal((n, q)) + mean_scale * rng.standard_normal(q)
    return X, Y


# ---- Eq. 3 -------------------------------------------------------------------

def test_sender_rms_hand_example():
    # rows (3, 4) and (0, 0): sum |x|^2 = 25 over p = 2 features and 2 samples.
    assert rc.sender_rms([[3.0, 4.0], [0.0, 0.0]]) == pytest.approx(2.5, rel=1e-15)
    # a constant matrix has RMS |c|
    assert rc.sender_rms(np.full((7, 5), -1.75)) == pytest.approx(1.75, rel=1e-15)


def test_sender_rms_weights_are_row_multiplicities():
    rng = np.random.default_rng(0)
    X = rng.standard_normal((6, 4))
    w = np.array([1, 3, 0, 2, 1, 5], float)
    Xd = np.repeat(X, w.astype(int), axis=0)
    assert rc.sender_rms(X, w) == pytest.approx(rc.sender_rms(Xd), rel=1e-14)
    # scale of the weights does not matter; Z = X / r has unit weighted mean square
    assert rc.sender_rms(X, 7.5 * w) == pytest.approx(rc.sender_rms(X, w), rel=1e-14)
    r = rc.sender_rms(X, w)
    Z = X / r
    assert np.sum(w * np.sum(Z * Z, axis=1)) / (4 * w.sum()) == pytest.approx(1.0, rel=1e-14)


# ---- weighted moments ----------------------------------------------------------

def test_weighted_moments_match_numpy_cov():
    rng = np.random.default_rng(1)
    X, Y = _samples(rng, 200, 5, 3)
    w = rng.uniform(0.1, 2.0, 200)
    mx, my, Sxx, Sxy, Syy = rc.weighted_moments(X, Y, w)
    J = np.cov(np.hstack([X, Y]).T, aweights=w, bias=True)
    np.testing.assert_allclose(mx, np.average(X, axis=0, weights=w), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(my, np.average(Y, axis=0, weights=w), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(Sxx, J[:5, :5], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(Sxy, J[:5, 5:], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(Syy, J[5:, 5:], rtol=1e-12, atol=1e-13)


def test_weighted_moments_integer_weights_duplicate_rows():
    rng = np.random.default_rng(2)
    X, Y = _samples(rng, 9, 3, 2)
    w = np.array([2, 1, 1, 4, 1, 3, 1, 1, 2], float)
    a = rc.weighted_moments(X, Y, w)
    k = w.astype(int)
    b = rc.weighted_moments(np.repeat(X, k, axis=0), np.repeat(Y, k, axis=0))
    for u, v in zip(a, b):
        np.testing.assert_allclose(u, v, rtol=1e-12, atol=1e-13)


# ---- symmetric roots and Procrustes ----------------------------------------------

def test_psd_power_roots():
    rng = np.random.default_rng(3)
    G = rng.standard_normal((6, 6))
    S = G @ G.T + 0.5 * np.eye(6)
    Wm = rc.psd_power(S, -0.5)
    Wp = rc.psd_power(S, 0.5)
    np.testing.assert_allclose(Wm, Wm.T, atol=1e-13)
    np.testing.assert_allclose(Wm @ S @ Wm, np.eye(6), atol=1e-11)
    np.testing.assert_allclose(Wp @ Wp, S, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Wp, scipy.linalg.sqrtm(S).real, rtol=1e-10, atol=1e-11)
    # diagonal closed form
    D = np.diag([4.0, 9.0, 0.25])
    np.testing.assert_allclose(rc.psd_power(D, -0.5), np.diag([0.5, 1 / 3, 2.0]), rtol=1e-15)
    with pytest.raises(np.linalg.LinAlgError):
        rc.psd_power(np.diag([1.0, 0.0]), -0.5)


def test_procrustes_square_matches_scipy():
    rng = np.random.default_rng(4)
    M = rng.standard_normal((7, 7))
    R_lib, _ = scipy.linalg.orthogonal_procrustes(np.eye(7), M)
    np.testing.assert_allclose(rc.procrustes(M), R_lib, atol=1e-12)


def test_procrustes_rectangular_is_the_best_isometry():
    rng = np.random.default_rng(5)
    M = rng.standard_normal((9, 4))
    R = rc.procrustes(M)
    np.testing.assert_allclose(R.T @ R, np.eye(4), atol=1e-13)
    best = np.trace(R.T @ M)
    for _ in range(200):
        Qc, _ = np.linalg.qr(rng.standard_normal((9, 4)))
        assert np.trace(Qc.T @ M) <= best + 1e-12
    # a column vector's polar factor is its normalization
    v = rng.standard_normal((5, 1))
    np.testing.assert_allclose(rc.procrustes(v), v / np.linalg.norm(v), atol=1e-15)


# ---- Recolor (Eq. 4-5) -----------------------------------------------------------

def test_recolor_scalar_closed_form():
    # p = q = 1: A = sign(cov_zy) sd_y / sd_z and b = mu_y - mu_z A.
    x = np.array([[1.0], [2.0], [3.0], [6.0]])
    for y in (np.array([[2.0], [0.0], [1.0], [5.0]]), np.array([[2.0], [3.0], [1.0], [-4.0]])):
        r, A, b = rc.recolor_from_samples(x, y)
        assert r == pytest.approx(np.sqrt(50 / 4), rel=1e-15)
        z = x[:, 0] / r
        cz = z - z.mean()
        cy = y[:, 0] - y[:, 0].mean()
        expect = np.sign(np.mean(cz * cy)) * np.sqrt(np.mean(cy * cy) / np.mean(cz * cz))
        assert A[0, 0] == pytest.approx(expect, rel=1e-13)
        assert b[0] == pytest.approx(y.mean() - z.mean() * expect, rel=1e-13, abs=1e-14)


def test_recolor_two_to_one_closed_form():
    # p = 2 uncorrelated sender features, q = 1: M is a column vector, R* = M / |M|,
    # so A = Sigma_Z^{-1/2} M sd_y / |M| with M_i = cov(z_i, y) / (sd_i sd_y).
    rng = np.random.default_rng(6)
    z = rng.standard_normal((4000, 2))
    z -= z.mean(0)
    z = z @ np.linalg.inv(np.linalg.cholesky(np.cov(z.T, bias=True))).T  # exactly white
    z = z * np.array([2.0, 0.5]) + np.array([1.0, -3.0])
    y = 0.7 * z[:, :1] - 1.3 * z[:, 1:] + 0.4 * rng.standard_normal((4000, 1)) + 2.0
    mz, my, Szz, Szy, Syy = rc.weighted_moments(z, y)
    np.testing.assert_allclose(Szz, np.diag([4.0, 0.25]), atol=1e-12)
    A, b = rc.recolor(mz, my, Szz, Szy, Syy)
    sd = np.array([2.0, 0.5])
    sy = np.sqrt(Syy[0, 0])
    M = Szy[:, 0] / (sd * sy)
    expect = (M / np.linalg.norm(M)) / sd * sy
    np.testing.assert_allclose(A[:, 0], expect, rtol=1e-10)
    np.testing.assert_allclose(b, my - mz @ A, rtol=1e-13)


@pytest.mark.parametrize("p,q", [(6, 6), (12, 4), (30, 10)])
def test_recolor_identities_of_the_paper(p, q):
    rng = np.random.default_rng(7 + p)
    X, Y = _samples(rng, 3000, p, q)
    w = rng.uniform(0.2, 3.0, 3000)
    r, A, b = rc.recolor_from_samples(X, Y, w)
    mz, my, Szz, Szy, Syy = rc.weighted_moments(X / r, Y, w)
    np.testing.assert_allclose(mz @ A + b, my, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(A.T @ Szz @ A, Syy, rtol=1e-9, atol=1e-10 * np.abs(Syy).max())


@pytest.mark.parametrize("p,q", [(5, 5), (8, 3)])
def test_recolor_recovers_an_exact_affine_relation(p, q):
    # If y = z C + d exactly, Sigma_Z^{1/2} C Sigma_Y^{-1/2} has orthonormal columns,
    # so R* is that matrix and Recolor returns C and d.
    rng = np.random.default_rng(11 + p)
    X, _ = _samples(rng, 500, p, 1)
    C = rng.standard_normal((p, q))
    d = rng.standard_normal(q)
    r = rc.sender_rms(X)
    Y = (X / r) @ C + d
    r2, A, b = rc.recolor_from_samples(X, Y)
    assert r2 == pytest.approx(r, rel=1e-15)
    np.testing.assert_allclose(A, C, rtol=1e-8, atol=1e-9)
    np.testing.assert_allclose(b, d, rtol=1e-8, atol=1e-9)
    np.testing.assert_allclose(rc.apply_map(X, r2, A, b), Y, rtol=1e-8, atol=1e-8)


def test_recolor_is_invariant_to_the_covariance_normalizer():
    rng = np.random.default_rng(13)
    X, Y = _samples(rng, 60, 4, 3)
    mz, my, Szz, Szy, Syy = rc.weighted_moments(X, Y)
    A1, b1 = rc.recolor(mz, my, Szz, Szy, Syy)
    k = 60 / 59  # unbiased instead of weight-sum normalization
    A2, b2 = rc.recolor(mz, my, k * Szz, k * Szy, k * Syy)
    np.testing.assert_allclose(A1, A2, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(b1, b2, rtol=1e-9, atol=1e-12)


def test_ridge_reading():
    S = np.array([[2.0, 1.0], [1.0, 4.0]])
    np.testing.assert_allclose(rc.ridge(S, 0.1), S + 0.1 * 3.0 * np.eye(2), rtol=1e-15)
    # with a ridge, the covariance identity holds for the stabilized covariances
    rng = np.random.default_rng(14)
    X, Y = _samples(rng, 800, 10, 4)
    # duplicate sender features make Sigma_Z singular, as clipped layer taps do
    X = np.hstack([X, X[:, :3]])
    r = rc.sender_rms(X)
    mz, my, Szz, Szy, Syy = rc.weighted_moments(X / r, Y)
    with pytest.raises(np.linalg.LinAlgError):
        rc.recolor(mz, my, Szz, Szy, Syy)
    A, b = rc.recolor(mz, my, Szz, Szy, Syy, lam=1e-3)
    np.testing.assert_allclose(A.T @ rc.ridge(Szz, 1e-3) @ A, rc.ridge(Syy, 1e-3), rtol=1e-8,
                               atol=1e-9)
    np.testing.assert_allclose(mz @ A + b, my, atol=1e-11)


def test_planted_mistakes_fail_the_recovery_pin():
    rng = np.random.default_rng(15)
    X, _ = _samples(rng, 400, 5, 1)
    C = rng.standard_normal((5, 5))
    d = rng.standard_normal(5)
    r = rc.sender_rms(X)
    Y = (X / r) @ C + d
    mz, my, Szz, Szy, Syy = rc.weighted_moments(X / r, Y)
    Wz = rc.psd_power(Szz, -0.5)
    Wy = rc.psd_power(Syy, -0.5)
    Ry = rc.psd_power(Syy, 0.5)
    U, _, Qt = np.linalg.svd(Wz @ Szy @ Wy)
    wrong = {
        "transposed rotation": Wz @ (Qt.T @ U.T) @ Ry,
        "roots swapped": Wz @ (U @ Qt) @ Wy,
        "cross-covariance transposed": Wz @ rc.procrustes(Wz @ Szy.T @ Wy) @ Ry,
        "no whitening": rc.procrustes(Szy) @ Ry,
    }
    for name, A in wrong.items():
        assert np.abs(A - C).max() > 1e-3, name


# ---- correction and fold (Eq. 9) -------------------------------------------------

def test_fold_equals_correction_after_the_map():
    rng = np.random.default_rng(16)
    p, q, rho = 12, 8, 3
    X = rng.standard_normal((50, p))
    A = rng.standard_normal((p, q))
    b = rng.standard_normal(q)
    B = 0.02 * rng.standard_normal((q, rho))
    G = rng.standard_normal((rho, q))
    r = 1.7
    Y0 = rc.apply_map(X, r, A, b)
    Af, bf = rc.fold(A, b, B, G)
    np.testing.assert_allclose(rc.apply_map(X, r, Af, bf), rc.correct(Y0, B, G), rtol=1e-12,
                               atol=1e-12)
    # G = 0 (the calibration's initialization) leaves the map unchanged
    A0, b0 = rc.fold(A, b, B, np.zeros_like(G))
    np.testing.assert_array_equal(A0, A)
    np.testing.assert_array_equal(b0, b)


def test_fold_rank_one_hand_example():
    A = np.array([[1.0, 2.0], [0.0, 1.0], [3.0, -1.0]])  # p = 3, q = 2
    b = np.array([1.0, -2.0])
    B = np.array([[1.0], [2.0]])
    G = np.array([[0.5, -1.0]])
    # I + B G = [[1.5, -1], [1, -1]]
    Af, bf = rc.fold(A, b, B, G)
    np.testing.assert_array_equal(Af, [[3.5, -3.0], [1.0, -1.0], [3.5, -2.0]])
    np.testing.assert_array_equal(bf, [-0.5, 1.0])
    np.testing.assert_array_equal(rc.abi_orientation(Af), np.array(Af).T)
