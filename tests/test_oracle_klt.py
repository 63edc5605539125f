"""Pins of the KLT-rotated store's oracle (Sec. 3.5) to what the mathematics fixes.

The calibration pin uses keys whose mean and covariance are known exactly:
K = Z diag(sigma) Q^T + mu with Z = [H; -H] for a 128 x 128 Hadamard matrix H,
so every column of Z has mean 0 and Z^T Z = n I (n = 256).  The population
covariance of K is then Q diag(sigma^2) Q^T: eigenvalues sigma^2, eigenvectors
the columns of Q.  A dropped mean, an n - 1 normalisation, a transposed
product or an ascending order each fails it.
"""
import numpy as np
import pytest
import scipy.linalg

from oracle import klt

D = 128


def _design(seed, sig=None):
    rng = np.random.default_rng(seed)
    H = scipy.linalg.hadamard(D).astype(np.float64)
    Z = np.vstack([H, -H])
    Q, _ = np.linalg.qr(rng.standard_normal((D, D)))
    if sig is None:
        sig = np.linspace(3.0, 0.2, D)
    mu = rng.standard_normal(D)
    return Z @ np.diag(sig) @ Q.T + mu, mu, Q, np.asarray(sig)


def test_calibrate_recovers_a_known_covariance():
    K, mu, Q, sig = _design(3)
    m, V, lam = klt.klt_calibrate(K)
    assert np.allclose(m, mu, atol=1e-12)
    assert np.allclose(lam, sig ** 2, atol=1e-12)          # population covariance, descending
    assert np.allclose(np.abs(V.T @ Q), np.eye(D), atol=1e-10)  # the same axes, column by column


def test_calibrate_eigen_equation_and_orthonormality():
    rng = np.random.default_rng(5)
    A = rng.standard_normal((D, D)) * np.linspace(2.0, 0.05, D)
    K = rng.standard_normal((3000, D)) @ A.T + 0.5
    m, V, lam = klt.klt_calibrate(K)
    X = K - K.mean(0)
    C = X.T @ X / K.shape[0]
    assert np.abs(C @ V - V * lam).max() <= 1e-10 * lam[0]
    assert np.abs(V.T @ V - np.eye(D)).max() <= 1e-12
    assert (np.diff(lam) <= 0).all()
    # sign convention: the largest-magnitude entry of every column is positive
    j = np.argmax(np.abs(V), axis=0)
    assert (V[j, np.arange(D)] > 0).all()


def test_calibrate_degenerate_units():
    m, V, lam = klt.klt_calibrate(np.zeros((0, D)))
    assert (m == 0).all() and (V == np.eye(D)).all() and (lam == 0).all()
    one = np.random.default_rng(1).standard_normal((1, D))
    m, V, lam = klt.klt_calibrate(one)
    assert np.allclose(m, one[0]) and np.allclose(lam, 0.0)


def test_rotate_identity_and_permutation_are_exact():
    rng = np.random.default_rng(7)
    K = rng.standard_normal((300, D)).astype(np.float32)
    mu = rng.standard_normal(D).astype(np.float32)
    assert np.array_equal(klt.klt_rotate_keys(K, np.zeros(D, np.float32), np.eye(D, dtype=np.float32)), K)
    perm = rng.permutation(D)
    P = np.zeros((D, D), np.float32)
    P[perm, np.arange(D)] = 1.0  # column c of the output is channel perm[c]
    assert np.array_equal(klt.klt_rotate_keys(K, mu, P), (K - mu)[:, perm])
    q = rng.standard_normal((4, D)).astype(np.float32)
    assert np.array_equal(klt.klt_rotate_q(q, np.eye(D, dtype=np.float32)), q)


def test_rotate_keys_within_fp32_bound_and_norm_preserving():
    rng = np.random.default_rng(9)
    K = (3 * rng.standard_normal((500, D))).astype(np.float16)
    mu = rng.standard_normal(D).astype(np.float32)
    Q, _ = np.linalg.qr(rng.standard_normal((D, D)))
    V = Q.astype(np.float32)
    y = klt.klt_rotate_keys(K, mu, V).astype(np.float64)
    d = K.astype(np.float32) - mu  # the fp32 centring the oracle states
    exact = d.astype(np.float64) @ V.astype(np.float64)
    # each of the D products and D sums rounds once: |err| <= 2 D u sum_j |d_j V_jc|
    bound = 2 * D * 2.0 ** -24 * (np.abs(d).astype(np.float64) @ np.abs(V).astype(np.float64))
    assert (np.abs(y - exact) <= bound).all()
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(d.astype(np.float64), axis=1), rtol=1e-5)


def test_rotated_scores_equal_centred_raw_scores():
    """q' . k' = (q V) . ((k - mu) V) = q . (k - mu) for orthonormal V."""
    rng = np.random.default_rng(11)
    K, mu, Q, _ = _design(13)
    K = K.astype(np.float32)
    m, V, lam = klt.klt_calibrate(K)
    V32, mu32 = V.astype(np.float32), m.astype(np.float32)
    q = rng.standard_normal((4, D)).astype(np.float32)
    s_rot = klt.klt_rotate_q(q, V32).astype(np.float64) @ klt.klt_rotate_keys(K, mu32, V32).T.astype(np.float64)
    s_raw = q.astype(np.float64) @ (K.astype(np.float64) - mu32.astype(np.float64)).T
    scale = np.abs(q).astype(np.float64) @ np.abs(K.astype(np.float64) - mu32).T
    assert (np.abs(s_rot - s_raw) <= 1e-5 * scale + 1e-6).all()


def test_rotated_importance_sums_to_the_score_variance():
    """Sec. 3.5: with g_j = sum_h (q_h V)_j^2 lambda_j, sum_j g_j = sum_h q_h^T C q_h."""
    rng = np.random.default_rng(17)
    A = rng.standard_normal((D, D)) * np.linspace(1.5, 0.1, D)
    K = rng.standard_normal((4000, D)) @ A.T
    m, V, lam = klt.klt_calibrate(K)
    X = K - m
    C = X.T @ X / K.shape[0]
    q = rng.standard_normal((4, D))
    qr = q @ V
    g = (qr ** 2).sum(0) * lam
    assert g.sum() == pytest.approx(sum(q[h] @ C @ q[h] for h in range(4)), rel=1e-10)
