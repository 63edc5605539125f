"""KLT-rotated store (Sec. 3.5, basis rule) -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module; the product library never does, and this
module never imports the product.

The rotated variant of the method stores the planes of (k - mu) V instead of
k, where mu is the mean of the unit's calibration keys and V the orthonormal
eigenbasis of their covariance (one basis per KV head and layer), and it
allocates depths with g_j = sum_h ((q_h V)_j)^2 lambda_j, lambda_j the
eigenvalue of column j.  Everything downstream (pack, water-filling, scan,
top-k) is unchanged.  Calibration keys here are the unit's own keys.

Readings (the paper is silent on these):
  * covariance normalised by n (the population covariance of the keys);
  * columns ordered by eigenvalue, largest first (the paper orders by the
    calibration score variance, which needs calibration queries; with
    isotropic queries the two orders agree), ties by the solver's order;
  * each eigenvector's sign fixed so that its largest-magnitude entry (the
    first one among equal magnitudes) is positive;
  * the rotations are computed in fp32 in a fixed order: d_j = fl(k_j - mu_j),
    then for j = 0, 1, ..., D-1: acc_c = fl(acc_c + fl(d_j * V[j][c])), acc_c
    starting at +0 (no fused multiply-add).  The query is rotated the same way
    without the mean.

Parity status:
  klt_calibrate    pinned: keys with an exactly known mean and covariance
                   (a Hadamard design) give the known eigenvalues and
                   eigenvectors; eigen-equation and orthonormality residuals.
  klt_rotate_keys  pinned: identity and permutation bases reproduce the
                   (centred) keys exactly; a general basis is within the fp32
                   error bound of the fp64 product and preserves norms.
  klt_rotate_q     pinned: identity basis; q' . k' equals q . (k - mu) within
                   the fp32 bound (the two rotations use V consistently).
"""
from __future__ import annotations

import numpy as np

__all__ = ["klt_calibrate", "klt_rotate_keys", "klt_rotate_q", "klt_fix_signs"]


def klt_fix_signs(V: np.ndarray) -> np.ndarray:
    """Sign convention: the largest-magnitude entry of each column (the first
    among equal magnitudes) is made positive."""
    V = np.array(V, copy=True)
    for c in range(V.shape[1]):
        j = int(np.argmax(np.abs(V[:, c])))  # argmax returns the first maximum
        if V[j, c] < 0:
            V[:, c] = -V[:, c]
    return V


def klt_calibrate(K: np.ndarray):
    """Sec. 3.5: mean, eigenbasis and eigenvalues of one unit's keys.

    K [n][D] (any float dtype; taken exactly in fp64).  Returns (mu [D] fp64,
    V [D][D] fp64 with eigenvector c in column c, lam [D] fp64), columns by
    eigenvalue descending.  n = 0 gives mu = 0, V = I, lam = 0.
    """
    K = np.asarray(K, dtype=np.float64)
    n, D = K.shape
    if n == 0:
        return np.zeros(D), np.eye(D), np.zeros(D)
    mu = K.sum(axis=0) / n
    X = K - mu
    C = (X.T @ X) / n
    lam, V = np.linalg.eigh(C)  # ascending eigenvalues, orthonormal columns
    order = np.argsort(-lam, kind="stable")
    return mu, np.ascontiguousarray(klt_fix_signs(V[:, order])), lam[order]


def _rotate_f32(X: np.ndarray, V: np.ndarray) -> np.ndarray:
    """acc_c = sum over j ascending of fl(X_j * V[j][c]), each sum rounded to fp32."""
    X = np.asarray(X, dtype=np.float32)
    V = np.asarray(V, dtype=np.float32)
    D = V.shape[0]
    acc = np.zeros((X.shape[0], V.shape[1]), dtype=np.float32)
    for j in range(D):
        acc = acc + X[:, j:j + 1] * V[j:j + 1, :]  # both operations round to fp32
    return acc


def klt_rotate_keys(K: np.ndarray, mu: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Sec. 3.5: the stored coordinates (k - mu) V of each key, fp32 [n][D].

    K [n][D] fp32 or fp16 values (converted exactly to fp32); mu [D] and
    V [D][D] are taken as fp32.
    """
    d = np.asarray(K, dtype=np.float32) - np.asarray(mu, dtype=np.float32)
    return _rotate_f32(d, V)


def klt_rotate_q(q: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Sec. 3.5: q_h V per head, fp32 [G][D] (q fp32 or fp16 values)."""
    return _rotate_f32(np.asarray(q, dtype=np.float32), V)
