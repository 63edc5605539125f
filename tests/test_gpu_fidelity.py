"""The method's qualitative claim on its own synthetic layer (Sec. 3.3, Sec. 4):
at equal bytes per key, water-filled read depths select keys whose sparse
attention is closer to dense attention than the uniform top-r rule does, and
more bits bring water-filling closer to the exact-top-k selection.

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
