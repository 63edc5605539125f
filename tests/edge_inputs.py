"""Seeded key generators for the edge cases of Sec. 3.2's fp16 block scales,
shared by the oracle pins and the GPU parity tests (inputs only: no arithmetic
of the method)."""
import numpy as np


def scale_edge_keys(rng, n, D=16):
    """Blocks whose absmax is a binary16 subnormal (several magnitudes, ties
    between subnormals, absmax below half the smallest subnormal), in
    [65504, 65520) (finite: rounds to 65504), exactly 65520 (rounds to
    infinity), and fp32 subnormal keys beside a subnormal-scale channel."""
    K = (rng.standard_normal((n, D)) * 0.3).astype(np.float32)
    edges = [3e-6, 2.0 ** -24, 2.0 ** -25, 1.5 * 2.0 ** -24, 6.0e-5, 2.0 ** -14 - 2.0 ** -25,
             65504.0, 65519.99, 65510.0, 1e-38]
    for c, a in enumerate(edges):
        col = rng.uniform(-1.0, 1.0, n).astype(np.float64) * a
        col[rng.integers(0, n, 3)] = a * np.sign(rng.standard_normal(3))
        K[:, c] = col.astype(np.float32)
        if a == 65519.99:
            K[0, c] = np.nextafter(np.float32(65520.0), np.float32(0))
    K[:, 10] = np.float32(1e-40) * np.sign(rng.standard_normal(n)).astype(np.float32)  # fp32 subnormals
    K[::7, 11] = -np.float32(1e-41)
    K[1::7, 11] = np.float32(2.0 ** -20)
    return K
