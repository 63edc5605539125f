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

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def table():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    spec = importlib.util.spec_from_file_location("bench_fidelity", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    res = bench.fidelity()["results"]
    torch.cuda.empty_cache()
    return {k: v["mean"] for k, v in res.items()}


@pytest.mark.parametrize("B", [32, 48, 80])
def test_waterfill_beats_uniform_at_equal_bytes(table, B):
    assert table[f"waterfill_B{B}"] < table[f"uniform_B{B}"], table


def test_waterfill_approaches_exact_topk_with_more_bits(table):
    assert table["exact_topk"] <= table["waterfill_B80"] <= table["waterfill_B48"] <= table["waterfill_B32"], table


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
