"""The method's qualitative claims on its own synthetic layer (Sec. 3.3, Sec. 4):
at equal bytes per key, water-filled read depths select keys whose sparse
attention is closer to dense attention than the uniform top-r rule does, and
more bits bring water-filling closer to the exact-top-k selection.  On a layer
whose keys are not normalised per channel (its channels mixed by a random
rotation), KLT-rotated planes beat raw planes at equal bits (Sec. 3.5).

Relative L2 of the attention output against dense fp32 attention over all n
keys, per (unit, head), mean over the layer (bench.py --fidelity prints the
same table).  The inputs are seeded, so the comparison is deterministic.
"""
import importlib.util
import os

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
REF_UNITS = [0, 5]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def table():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spec = importlib.util.spec_from_file_location("bench_fidelity", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    full = bench.fidelity(refs_for=REF_UNITS)
    torch.cuda.empty_cache()
    return {k: v["mean"] for k, v in full["results"].items()}, full["refs"]


@pytest.mark.parametrize("B", [32, 48, 80])
def test_waterfill_beats_uniform_at_equal_bytes(table, B):
    t = table[0]
    assert t[f"waterfill_B{B}"] < t[f"uniform_B{B}"], t


def test_waterfill_approaches_exact_topk_with_more_bits(table):
    t = table[0]
    assert t["exact_topk"] <= t["waterfill_B80"] <= t["waterfill_B48"] <= t["waterfill_B32"], t


@pytest.mark.parametrize("u", REF_UNITS)
def test_dense_reference_equals_oracle_attention_over_every_key(table, u):
    """The harness's dense reference (torch fp32 matmul + softmax over all n
    keys) equals the oracle's exact attention (fp64) with every key selected,
    within fp32 accumulation error, for every head of sampled units."""
    r = table[1][u]
    n, G = r["K16"].shape[0], r["q"].shape[0]
    q32 = r["q"].astype(np.float32)
    every = np.tile(np.arange(n, dtype=np.int32), (G, 1))
    oo = oracle.sparse_attn(q32, r["K16"], r["V16"], every, 0, 0, 1 / np.sqrt(128))
    scale = np.abs(r["V16"].astype(np.float64)).max()
    assert np.abs(r["dense"] - oo).max() <= 1e-4 * scale, np.abs(r["dense"] - oo).max()


@pytest.mark.parametrize("u", REF_UNITS)
def test_exact_topk_reference_is_the_fp64_top_k(table, u):
    """The harness's exact-top-k bound (torch.topk over fp32 q.k) selects the k
    largest fp64 dot products up to fp32 near-ties: every key clearly above the
    fp64 k-th score is selected, and no selected key is clearly below it."""
    r = table[1][u]
    K64, q64 = r["K"].astype(np.float64), r["q"].astype(np.float64)
    k = r["exact_idx"].shape[1]
    for h in range(q64.shape[0]):
        s = K64 @ q64[h]
        tol = 1e-5 * (np.abs(K64) @ np.abs(q64[h]))  # above the fp32 dot-product error bound (128 terms)
        kth = np.sort(s)[::-1][k - 1]
        sel = np.zeros(s.shape, bool)
        sel[r["exact_idx"][h]] = True
        assert len(np.unique(r["exact_idx"][h])) == k
        assert sel[s - tol > kth].all(), h
        assert not (sel & (s + tol < kth)).any(), h


@pytest.fixture(scope="module")
def basis_table():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spec = importlib.util.spec_from_file_location("bench_fidelity_basis", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    res = bench.fidelity_basis()["results"]
    torch.cuda.empty_cache()
    return {k: v["mean"] for k, v in res.items()}


@pytest.mark.parametrize("B", [32, 48, 80])
def test_klt_planes_beat_raw_planes_on_mixed_channels(basis_table, B):
    assert basis_table[f"klt_B{B}"] < basis_table[f"raw_B{B}"], basis_table
