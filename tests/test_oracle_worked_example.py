"""Pins the CPU oracle to the worked example of App. A (printed values).

Fixture: tests/golden/worked_example.json, every value copied from App. A.
Values are compared at the precision the paper prints them.
"""
import numpy as np
import pytest


def _K(golden):
    return np.array(golden["K"], np.float32)


def _q(golden):
    return np.array([golden["q"]["A"], golden["q"]["B"]], np.float32)


def _var(golden):
    # App. A: Var is the unbiased sample variance of the six keys (it matches the
    # printed 3-decimal values and, unlike the rounded values, the printed g).
    return np.array(golden["K"], np.float64).var(axis=0, ddof=1).astype(np.float32)


def _codes(planes, j, n):
    return [sum(((int(planes[j, p, 0]) >> i) & 1) << (3 - p) for p in range(4)) for i in range(n)]


def test_variance_matches_print(golden):
    np.testing.assert_allclose(_var(golden), golden["var_printed"], atol=0.5e-3 + 1e-9)


def test_channel2_codes_scale_and_one_plane(orc, golden):
    """App. A, 'One plane of channel 2': a = 0.5, s = 0.0625, codes, +-0.25."""
    ref = golden["channel2"]
    planes, scales, st = orc.pack(_K(golden))
    assert st == 0
    assert orc.f16_bits_to_f64(scales[2, 0]) == ref["a"]
    assert orc.f16_bits_to_f64(scales[2, 0]) / 8 == ref["s"]
    assert _codes(planes, 2, 6) == ref["codes"]
    one = [orc.dequant(planes, scales, 2, 1, i) for i in range(6)]
    assert one == ref["one_plane_values"]


def test_importance_matches_print(orc, golden):
    """App. A, 'Importance weights' (Eq. g)."""
    g = orc.importance(_q(golden), _var(golden))
    np.testing.assert_allclose(g[:3], golden["g_printed"], atol=0.5e-2 + 1e-9)
    assert golden["g3_is_about_zero"] and abs(g[3]) < 0.005


@pytest.mark.parametrize("B,key", [(8, "bisection"), (6, "budget6")])
def test_waterfill_closed_form(orc, golden, B, key):
    """App. A: theta ~ 0.079 -> t = (4,3,1,0) at B = 8; theta ~ 0.118 -> (3,2,1,0) at B = 6."""
    d, th, st = orc.alloc_waterfill(_q(golden), _var(golden), B)
    ref = golden[key]
    want_t = ref["final_t"] if key == "bisection" else ref["t"]
    want_th = ref["final_theta"] if key == "bisection" else ref["theta"]
    assert st == 0
    assert d.tolist() == want_t
    assert abs(float(th) - want_th) < 0.5e-3
    assert int(d.sum()) == B  # App. A: the depths use all of the budget in both cases


def test_bisection_trace(orc, golden):
    """App. A bisection table, row by row, from the bracket [0.001, 10]."""
    b = golden["bisection"]
    g = np.array(b["g_used"], np.float64)
    hi, d, trials, sums = orc.bisect(g, b["B"], b["bracket"][0], b["bracket"][1], steps=30)
    lo_hi = list(b["bracket"])
    for r, row in enumerate(b["rows"]):
        th = trials[r]
        # trial = geometric mean of the current bracket, printed to 3 significant digits
        assert th == pytest.approx(np.sqrt(lo_hi[0] * lo_hi[1]))
        assert th == pytest.approx(row["trial"], rel=2e-3)
        l4 = np.log(g[:3] / th) / np.log(4.0)
        assert np.round(l4, 2).tolist() == pytest.approx(row["log4"], abs=1e-9)
        dt, s = orc.depths_at(g, th)
        assert dt.tolist() == row["t"] and s == row["sum"] == sums[r]
        assert (s <= b["B"]) == row["fits"]
        lo_hi = [lo_hi[0], th] if row["fits"] else [th, lo_hi[1]]
    assert abs(hi - b["final_theta"]) < 0.5e-3
    assert d.tolist() == b["final_t"]
    lo_i, hi_i = b["one_plane_interval_for_channel2"]
    assert abs(g[2] / 4 ** 1.5 - lo_i) < 1e-4 and abs(g[2] / 4 ** 0.5 - hi_i) < 1e-3
    # B = 6 by the same procedure
    hi6, d6, _, _ = orc.bisect(g, 6, b["bracket"][0], b["bracket"][1], steps=30)
    ref6 = golden["budget6"]
    assert abs(hi6 - ref6["theta"]) < 0.5e-3 and d6.tolist() == ref6["t"]
    assert np.round(np.log(g[:3] / hi6) / np.log(4.0), 2).tolist() == pytest.approx(ref6["log4"])
    assert abs(g[1] / 4 ** 2.5 - ref6["channel1_third_plane_below"]) < 1e-4


@pytest.mark.parametrize("which", ["f64", "f32"])
def test_scores_at_t4310(orc, golden, which):
    """App. A: approximate scores of heads A and B at depths (4,3,1,0), and exact ones."""
    K, q = _K(golden), _q(golden)
    planes, scales, _ = orc.pack(K)
    d = np.array([4, 3, 1, 0], np.uint8)
    f = orc.scores_f64 if which == "f64" else orc.scores_f32
    s = np.asarray(f(planes, scales, 6, q, d), np.float64)
    ref = golden["scores_at_t4310"]
    tol = 0.5 * 10 ** -ref["decimals"] + 1e-6
    np.testing.assert_allclose(s[0], ref["A_approx"], atol=tol)
    np.testing.assert_allclose(s[1], ref["B_approx"], atol=tol)
    exact = np.array(golden["K"], np.float64) @ np.array([golden["q"]["A"], golden["q"]["B"]]).T
    np.testing.assert_allclose(exact[:, 0], ref["A_exact"], atol=tol)
    np.testing.assert_allclose(exact[:, 1], ref["B_exact"], atol=tol)


def _top2(orc, row):
    idx, _, _ = orc.topk(np.asarray(row, np.float32), 2)
    return idx.tolist()


def test_selection_and_failures(orc, golden):
    """App. A: exact top-2 sets; Fathom at 8 bits selects them; B = 6 mis-ranks head B;
    SparQ r = 2 (sum |q| = (4,3,3,0.3), tie to the lower index) and the 2-bit thumbnail fail."""
    K, q = _K(golden), _q(golden)
    exact = np.array(golden["K"], np.float64) @ np.array([golden["q"]["A"], golden["q"]["B"]]).T
    assert _top2(orc, exact[:, 0]) == golden["exact_top2"]["A"]
    assert _top2(orc, exact[:, 1]) == golden["exact_top2"]["B"]
    planes, scales, _ = orc.pack(K)
    s8 = orc.scores_f32(planes, scales, 6, q, np.array([4, 3, 1, 0], np.uint8))
    assert _top2(orc, s8[0]) == golden["selection_at_t4310"]["A"]
    assert _top2(orc, s8[1]) == golden["selection_at_t4310"]["B"]
    d6, _, _ = orc.alloc_waterfill(q, _var(golden), 6)
    s6 = orc.scores_f32(planes, scales, 6, q, d6)
    assert golden["budget6_misranks_B"] and set(_top2(orc, s6[1])) != set(golden["exact_top2"]["B"])
    dr, wth, _ = orc.alloc_topr(q, 2)
    sp = golden["sparq_r2"]
    np.testing.assert_allclose(np.abs(q).sum(0), sp["sum_abs_q"], rtol=1e-6)
    assert np.flatnonzero(dr).tolist() == sp["channels"] and float(wth) == 3.0
    sq = orc.scores_f32(planes, scales, 6, q, dr)
    assert _top2(orc, sq[1]) == sp["B_top2"]
    st = orc.scores_f32(planes, scales, 6, q, np.full(4, 2, np.uint8))
    for h, name in enumerate("AB"):
        assert name in golden["thumbnail_2bit_misranks"]
        assert set(_top2(orc, st[h])) != set(golden["exact_top2"][name])
