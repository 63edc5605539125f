"""Pins the CPU oracle to what the paper and the mathematics fix, on random inputs.

Each check computes its expectation independently of the oracle's code path:
numpy's own float16 conversion, closed forms, brute-force enumeration, a
Monte-Carlo estimate of a stated law, or a full sort.
"""
import itertools

import numpy as np
import pytest

from edge_inputs import scale_edge_keys


def _keys(rng, n, D, scale=None):
    sig = np.exp(rng.standard_normal(D)) if scale is None else np.full(D, scale)
    return (rng.standard_normal((n, D)) * sig).astype(np.float32)


def _codes(planes, n):
    """Decode 4-bit codes [n][D] from planes by reading bits (independent of the oracle)."""
    D, _, nb = planes.shape
    words = planes.astype(np.uint64)
    i = np.arange(n)
    out = np.zeros((n, D), np.int64)
    for p in range(4):
        bits = (words[:, p, i // 64] >> (i % 64).astype(np.uint64)) & np.uint64(1)
        out += bits.T.astype(np.int64) << (3 - p)
    return out


@pytest.mark.parametrize("n", [1, 63, 64, 65, 1000, 4096])
def test_pack_prefix_is_t_bit_quantiser(orc, n):
    """Sec. 3.2: the first t planes are exactly the t-bit mid-rise quantiser of
    [-a, a): c >> (4-t) = clip(floor(2^(t-1) k / a), -2^(t-1), 2^(t-1)-1) + 2^(t-1);
    the MSB is the sign; the scale is fp16(block absmax); pad bits are zero."""
    rng = np.random.default_rng(n)
    K = _keys(rng, n, 16)
    K[0, 3] = -0.0
    K[:, 5] = 0.0  # an all-zero channel
    nb = (n + 63) // 64
    planes, scales, st = orc.pack(K, nb_cap=nb + 2)
    assert st == 0
    c = _codes(planes, n)
    for b in range(nb):
        blk = K[64 * b:min(n, 64 * b + 64)]
        a16 = np.abs(blk).max(0).astype(np.float16)  # numpy's own round-to-nearest-even
        assert (scales[:, b] == a16.view(np.uint16)).all()
        a = a16.astype(np.float64)
        kk = blk.astype(np.float64)
        cb = c[64 * b:64 * b + blk.shape[0]]
        for t in range(1, 5):
            h = 2.0 ** (t - 1)
            with np.errstate(divide="ignore", invalid="ignore"):
                want = np.clip(np.floor(h * kk / a), -h, h - 1) + h
            want = np.where(a > 0, want, h)  # a zero block holds the zero code
            assert ((cb >> (4 - t)) == want).all(), (b, t)
        msb = (cb >> 3) == 1
        assert (msb == ((kk >= 0) | (a == 0))).all()
    # pad bits past n and whole pad blocks are zero
    if n % 64:
        assert ((planes[:, :, nb - 1] >> np.uint64(n % 64)) == 0).all()
    assert (planes[:, :, nb:] == 0).all() and (scales[:, nb:] == 0).all()


def test_store_is_68_bytes_per_token(orc):
    """Sec. 3.2: 64 B of codes + 4 B of fp16 scales per token per KV head (D = 128)."""
    n = 4096
    planes, scales, _ = orc.pack(_keys(np.random.default_rng(0), n, 128))
    assert planes.nbytes + scales.nbytes == 68 * n


def test_dequant_values(orc):
    """Sec. 3.2: at t = 4 the value is (c - 8 + 1/2) s; every prefix value is a
    half-integer multiple of a/2^(t-1) and lies in (-a, a); exact in fp32."""
    rng = np.random.default_rng(1)
    K = _keys(rng, 256, 8)
    planes, scales, _ = orc.pack(K)
    c = _codes(planes, 256)
    for i in range(0, 256, 7):
        for j in range(8):
            a = float(np.uint16(scales[j, i // 64]).view(np.float16))
            v4 = orc.dequant(planes, scales, j, 4, i)
            assert v4 == (c[i, j] - 8 + 0.5) * a / 8
            for t in range(1, 5):
                v = orc.dequant(planes, scales, j, t, i)
                assert abs(v) < a and float(np.float32(v)) == v
                u = v / (a / 2 ** (t - 1)) - 0.5
                assert u == round(u)


def test_error_variance_law(orc):
    """Sec. 3.3: a depth-t read of values spread uniformly over [-a, a) errs with
    variance a^2 / (3 * 4^t).  Monte Carlo with a = 1 per block."""
    rng = np.random.default_rng(2)
    n = 64 * 4000
    K = rng.uniform(-1.0, 1.0, (n, 1)).astype(np.float32)
    K[::64, 0] = 1.0  # pin every block absmax to exactly 1
    planes, scales, _ = orc.pack(K)
    for t in range(1, 5):
        vals = np.array([orc.dequant(planes, scales, 0, t, i) for i in range(0, n, 5)])
        err = vals - K[::5, 0].astype(np.float64)
        m = ~np.isin(np.arange(0, n, 5) % 64, [0])
        want = 1.0 / (3 * 4 ** t)
        assert abs(np.mean(err[m] ** 2) / want - 1) < 0.06, t


def _brute_waterfill(g, B):
    best, arg = None, None
    for t in itertools.product(range(5), repeat=len(g)):
        if sum(t) <= B:
            e = sum(gj * 4.0 ** -tj for gj, tj in zip(g, t))
            if best is None or e < best - 1e-15:
                best, arg = e, t
    return list(arg)


@pytest.mark.parametrize("seed", range(12))
def test_waterfill_equals_brute_force_optimum(orc, seed):
    """Sec. 3.3: Eq. (wf) minimises sum_j g_j 4^-t_j under sum t_j <= B (distinct
    marginal gains); checked by enumerating all 5^D depth vectors, D <= 5."""
    rng = np.random.default_rng(seed)
    D = 3 + seed % 3
    q = rng.standard_normal((2, D)).astype(np.float32)
    var = np.exp(rng.standard_normal(D)).astype(np.float32)
    g = orc.importance(q, var).astype(np.float64)
    np.testing.assert_allclose(g, ((q.astype(np.float64) ** 2).sum(0)) * var, rtol=1e-6)
    for B in range(0, 4 * D + 1):
        d, th, _ = orc.alloc_waterfill(q, var, B)
        assert d.tolist() == _brute_waterfill(g, B), (B, g)


@pytest.mark.parametrize("seed", range(6))
def test_waterfill_properties(orc, seed):
    """Sec. 3.3: sum t <= B; one more candidate would overflow; depths grow with B;
    zero-importance channels are never read; Eq. (wf) evaluated directly (fp64
    log4, round half up) at a theta just above theta* gives the same depths;
    the paper's 30-step geometric bisection lands on them too."""
    rng = np.random.default_rng(100 + seed)
    D, G = 128, 4
    sig = np.exp(rng.standard_normal(D))
    sig[rng.choice(D, 4, replace=False)] *= 8
    var = (sig ** 2).astype(np.float32)
    q = rng.standard_normal((G, D)).astype(np.float16).astype(np.float32)
    q[:, 7] = 0.0
    g = orc.importance(q, var).astype(np.float64)
    cands = np.sort((g[:, None] * 2.0 ** -(2 * np.arange(1, 5) - 1)).ravel())[::-1]
    prev = None
    for B in [0, 1, 17, 40, 48, 80, 200, 4 * D - 4, 4 * D - 1, 4 * D, 4 * D + 10]:
        d, th, st = orc.alloc_waterfill(q, var, B)
        assert st == 0 and d.sum() <= B and d[7] == 0
        if B < 4 * D - 4:  # channel 7 alone has zero candidates
            th_star = cands[B]
            assert float(th) == np.float32(th_star)
            assert d.sum() + (cands == th_star).sum() > B
            nxt = cands[cands > th_star].min() if (cands > th_star).any() else 2 * th_star
            d2, s2 = orc.depths_at(g, np.sqrt(th_star * nxt))
            assert d2.tolist() == d.tolist() and s2 == d.sum()
            if B > 0:
                hi, d3, _, _ = orc.bisect(g, B, cands[-5] / 2 + 1e-30, 2 * cands[0], steps=200)
                assert d3.tolist() == d.tolist()
        if prev is not None:
            assert (d >= prev).all()
        prev = d
    # active channels at B = 48, G = 4 land near the paper's 30-34 of 128
    d48, _, _ = orc.alloc_waterfill(q, var, 48)
    assert 20 <= int((d48 > 0).sum()) <= 40


def test_topr_rule(orc):
    """Sec. 2 (SparQ): top-r channels by sum_h |q_hj|, ties to the lower index."""
    rng = np.random.default_rng(3)
    for r in [0, 1, 16, 32, 127, 128]:
        q = rng.integers(-3, 4, (4, 128)).astype(np.float32)  # many ties
        d, th, _ = orc.alloc_topr(q, r)
        w = np.abs(q).sum(0)
        order = sorted(range(128), key=lambda j: (-w[j], j))
        want = np.zeros(128, np.uint8)
        want[order[:r]] = 4
        assert d.tolist() == want.tolist()
        assert float(th) == (w[order[r - 1]] if r else 0.0)


@pytest.mark.parametrize("seed", range(4))
def test_scores_reference_and_replica(orc, seed):
    """fp64 scores equal a direct dequantise-and-dot written with numpy; linear in
    q; all-depth-4 is the full 4-bit scan; the fp32 replica lies within its own
    error bound (A fma roundings) of the fp64 value."""
    rng = np.random.default_rng(seed)
    n, D, G = 300, 128, 4
    K = _keys(rng, n, D)
    planes, scales, _ = orc.pack(K)
    q = rng.standard_normal((G, D)).astype(np.float16).astype(np.float32)
    var = np.exp(rng.standard_normal(D)).astype(np.float32)
    d, _, _ = orc.alloc_waterfill(q, var, 48)
    s64, sab = orc.scores_f64(planes, scales, n, q, d, with_abs=True)
    c = _codes(planes, n)
    a = scales.view(np.float16).astype(np.float64)[:, np.arange(n) // 64].T  # [n][D]
    t = d.astype(np.int64)
    with np.errstate(invalid="ignore"):
        khat = np.where(t > 0, ((c >> (4 - t)) + 0.5 - 2.0 ** (t - 1)) * a * 2.0 ** (1 - t), 0.0)
    np.testing.assert_allclose(s64, q.astype(np.float64) @ khat.T, rtol=1e-12, atol=1e-12)
    q2 = rng.standard_normal((G, D)).astype(np.float32)
    lin = orc.scores_f64(planes, scales, n, q + q2, d) - orc.scores_f64(planes, scales, n, q2, d)
    np.testing.assert_allclose(lin, orc.scores_f64(planes, scales, n, q, d), atol=1e-4)
    full = orc.scores_f64(planes, scales, n, q, np.full(D, 4, np.uint8))
    np.testing.assert_allclose(full, q.astype(np.float64) @ ((c - 8 + 0.5) * a / 8).T, rtol=1e-12, atol=1e-12)
    s32 = orc.scores_f32(planes, scales, n, q, d).astype(np.float64)
    A = int((d > 0).sum())
    bound = 2 * A * 2.0 ** -24 * sab + 1e-30
    assert (np.abs(s32 - s64) <= bound).all()
    assert (np.abs(s32 - s64) <= 1e-5 * sab + 1e-30).all()


@pytest.mark.parametrize("seed", range(8))
def test_topk_brute_force(orc, seed):
    """Sec. 2: per-head top-k over [lo, n - tail), (score desc, index asc),
    -0 equal to +0, NaN last; short rows padded with -1 and flagged."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    s = rng.integers(-5, 6, n).astype(np.float32)  # heavy ties
    s[rng.random(n) < 0.1] = -0.0
    if seed % 2:
        s[rng.random(n) < 0.05] = np.nan
    lo = int(rng.integers(0, 5))
    tail = int(rng.integers(0, 5))
    k = int(rng.integers(1, n + 3))
    idx, val, st = orc.topk(s, k, lo, tail)
    elig = list(range(lo, max(lo, n - tail)))
    key = sorted(elig, key=lambda i: (1 if np.isnan(s[i]) else 0, 0 if np.isnan(s[i]) else -float(s[i]), i))
    want = key[:k] + [-1] * max(0, k - len(key))
    assert idx.tolist() == want
    assert bool(st & orc.TOPK_SHORT) == (k > len(elig))
    assert bool(st & orc.NONFINITE) == bool(np.isnan(s[elig]).any())


def test_sparse_attention_closed_forms(orc):
    """Sec. 2: with every key selected the result is dense softmax attention; a
    one-row set returns that V row; sink and local rows are always included."""
    rng = np.random.default_rng(4)
    n, D, G = 200, 128, 4
    K16 = rng.standard_normal((n, D)).astype(np.float16)
    V16 = rng.standard_normal((n, D)).astype(np.float16)
    q = rng.standard_normal((G, D)).astype(np.float32)
    sm = np.float32(1 / np.sqrt(D))
    idx = np.tile(np.arange(4, n - 32, dtype=np.int32), (G, 1))
    out = orc.sparse_attn(q, K16, V16, idx, 4, 32, sm)
    z = (q.astype(np.float64) @ K16.astype(np.float64).T) * np.float64(sm)
    p = np.exp(z - z.max(1, keepdims=True))
    dense = (p / p.sum(1, keepdims=True)) @ V16.astype(np.float64)
    np.testing.assert_allclose(out, dense, rtol=1e-12, atol=1e-12)
    one = orc.sparse_attn(q, K16, V16, np.array([[17]] * G, np.int32), 0, 0, sm)
    np.testing.assert_allclose(one, np.tile(V16[17].astype(np.float64), (G, 1)))
    only = orc.sparse_attn(q, K16, V16, np.full((G, 3), -1, np.int32), 4, 32, sm)
    rows = list(range(4)) + list(range(n - 32, n))
    zz = z[:, rows]
    pp = np.exp(zz - zz.max(1, keepdims=True))
    np.testing.assert_allclose(only, (pp / pp.sum(1, keepdims=True)) @ V16[rows].astype(np.float64), rtol=1e-12, atol=1e-12)


def test_nonfinite_and_overflow_flags(orc):
    """Device-status conventions: a block absmax beyond fp16 raises SCALE_OVERFLOW
    and stores zero codes; NaN keys raise NONFINITE and take the zero code."""
    K = np.ones((64, 2), np.float32)
    K[5, 0] = 70000.0
    K[9, 1] = np.nan
    planes, scales, st = orc.pack(K)
    assert st & orc.SCALE_OVERFLOW and st & orc.NONFINITE
    c = _codes(planes, 64)
    assert (c[:, 0] == 8).all() and c[9, 1] == 8 and c[0, 1] == 15


def _f16_edge_inputs():
    """Every finite binary16 value, every midpoint between neighbours (exact in
    fp32: 12 significant bits), the fp32 neighbours of each midpoint, values
    past the largest finite half, and the signed zeros."""
    h = np.arange(0, 0x7C00, dtype=np.uint32).astype(np.uint16)  # +0 .. 65504
    v = h.view(np.float16).astype(np.float32)
    mids = ((v[:-1].astype(np.float64) + v[1:].astype(np.float64)) / 2).astype(np.float32)
    assert (mids.astype(np.float64) == (v[:-1].astype(np.float64) + v[1:]) / 2).all()
    top = np.float32(65520.0)  # halfway between 65504 and the first power past the range
    extra = np.array([top, 70000.0, 3.0e38, np.inf, 2.0 ** -25, 2.0 ** -26, 1e-40, 1e-45], np.float32)
    pos = np.concatenate([v, mids, np.nextafter(mids, np.float32(np.inf)),
                          np.nextafter(mids, np.float32(0)), extra,
                          np.nextafter(np.float32(top), np.float32(0))[None]])
    return np.concatenate([pos, -pos]).astype(np.float32)


def test_f32_to_f16_exhaustive_against_numpy(orc):
    """Sec. 3.2 stores fp16 block scales: the oracle's binary16 conversion,
    written from the format's definition, equals numpy's round-to-nearest-even
    conversion on every finite half, every midpoint (ties to even), the fp32
    neighbours of every midpoint, the subnormal range down to 2^-26 and fp32
    subnormals, and the overflow edge (65504 + 16 = 65520 rounds to infinity,
    the fp32 value just below it to 65504)."""
    x = _f16_edge_inputs()
    got = orc.f32_to_f16_bits_array(x)
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, want)
    # spot values that a wrong rounding or range test would move
    below = np.nextafter(np.float32(65520.0), np.float32(0))
    assert orc.f32_to_f16_bits(below) == 0x7BFF and orc.f32_to_f16_bits(65520.0) == 0x7C00
    assert orc.f32_to_f16_bits(2.0 ** -25) == 0 and orc.f32_to_f16_bits(3 * 2.0 ** -26) == 1
    assert orc.f32_to_f16_bits(-(2.0 ** -24)) == 0x8001
    assert orc.f32_to_f16_bits(float("nan")) & 0x7C00 == 0x7C00 and orc.f32_to_f16_bits(float("nan")) & 0x3FF
    for h in range(0, 0x7C00, 97):  # the inverse is exact on finite halves
        assert orc.f16_bits_to_f64(h) == float(np.uint16(h).view(np.float16))


@pytest.mark.parametrize("n", [64, 200])
def test_pack_fp16_scale_edges(orc, n):
    """Sec. 3.2, Eq. (2) at the edges of the fp16 scale: the stored scale is
    numpy's fp16 of the block absmax, the codes are the exact real floor against
    that scale (checked per prefix as the t-bit quantiser, from the keys), and an
    absmax that rounds to infinity gives zero codes (8) and SCALE_OVERFLOW."""
    rng = np.random.default_rng(1000 + n)
    K = scale_edge_keys(rng, n)
    nb = (n + 63) // 64
    planes, scales, st = orc.pack(K, nb_cap=nb)
    assert st == 0
    c = _codes(planes, n)
    for b in range(nb):
        blk = K[64 * b:min(n, 64 * b + 64)]
        a16 = np.abs(blk).max(0).astype(np.float16)
        assert (scales[:, b] == a16.view(np.uint16)).all(), b
        a = a16.astype(np.float64)
        kk = blk.astype(np.float64)
        cb = c[64 * b:64 * b + blk.shape[0]]
        for t in range(1, 5):
            h = 2.0 ** (t - 1)
            with np.errstate(divide="ignore", invalid="ignore"):
                want = np.clip(np.floor(h * kk / a), -h, h - 1) + h
            want = np.where(a > 0, want, h)
            assert ((cb >> (4 - t)) == want).all(), (b, t)
    # absmax exactly 65520: fp16 infinity, codes 8, flagged
    K2 = K.copy()
    K2[5, 3] = np.float32(65520.0)
    p2, s2, st2 = orc.pack(K2, nb_cap=nb)
    assert st2 & 1 and s2[3, 0] == 0x7C00
    assert (_codes(p2, n)[:min(n, 64), 3] == 8).all()
