"""fathom_scan_topk_noalloc (the entry point for callers that cannot allocate)
against fathom_scan_topk_ex with a caller workspace: bit-identical indices,
values and status on two calls in a row through the C ABI, the second with a
smaller input (fewer units, shorter rows, smaller k, sink/local protocol), so
what the first call left in the library's array must not leak into it."""
import numpy as np
import pytest
import torch

import paper_2609_17652_amd as F

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.lib()


def _case(ns, seed, G, B):
    rng = np.random.default_rng(seed)
    U, nmax = len(ns), max(ns)
    sig = np.exp(rng.standard_normal((U, 1, 128)))
    K = (rng.standard_normal((U, nmax, 128)) * sig).astype(np.float32)
    nt = torch.tensor(ns, dtype=torch.int64, device=DEV)
    planes, scales = F.fathom_pack(torch.from_numpy(K).to(DEV), nt)
    q = torch.from_numpy(rng.standard_normal((U, G, 128)).astype(np.float16)).to(DEV)
    var = torch.from_numpy(np.exp(rng.standard_normal((U, 128))).astype(np.float32)).to(DEV)
    d, _ = F.fathom_alloc_depths(q, var, F.FATHOM_WATERFILL, B)
    return planes, scales, nt, q, d


def test_noalloc_equals_workspace_call_twice_shrinking():
    cases = [
        # 8 units, long rows, k = 2048 (filtered rows, a direct row, a forced exact row)
        (dict(ns=[131072, 131072, 100000, 77777, 131072, 3000, 131072, 65536], seed=7, G=4, B=48), 2048, 0, 0,
         48),
        # then a smaller call: 3 units, shorter rows, k = 300, the sink/local protocol
        (dict(ns=[20000, 5000, 41], seed=8, G=4, B=40), 300, 4, 32, 0),
    ]
    for kw, k, lo, tail, bound in cases:
        planes, scales, nt, q, d = _case(**kw)
        if kw["seed"] == 7:
            d[4] = 4  # 512 bits: beyond the bound of 48, recomputed by the exact path
        U, G = q.shape[0], q.shape[1]
        nb = planes.shape[-1]
        assert F.fathom_scan_topk_workspace_size(U, G, 64 * nb, k) <= F.fathom_scan_topk_noalloc_capacity()
        st0, st1 = F.new_status(), F.new_status()
        i0, v0 = F.fathom_scan_topk(planes, scales, nt, q, d, k, lo, tail, dev_status=st0, max_unit_bits=bound)
        i1 = torch.full((U, G, k), -7, dtype=torch.int32, device=DEV)
        v1 = torch.full((U, G, k), 7.0, dtype=torch.float32, device=DEV)
        F.fathom_scan_topk_noalloc(planes, scales, nt, q, d, k, lo, tail, i1, v1, dev_status=st1,
                                   max_unit_bits=bound)
        torch.cuda.synchronize()
        assert torch.equal(i0, i1), kw
        assert torch.equal(v0.view(torch.int32), v1.view(torch.int32)), kw
        assert int(st0.item()) == int(st1.item()), kw
        if kw["seed"] == 7:
            assert int(st1.item()) & F.FATHOM_DEV_TOPK_FALLBACK


def test_noalloc_rejects_shapes_beyond_its_array():
    """64 units x 4 heads at k = 8192 need more workspace than the library's
    array holds: FATHOM_ERR_WORKSPACE before anything is launched, and the
    outputs are left as they were."""
    U, k = 64, 8192
    planes, scales, nt, q, d = _case(ns=[1000] * U, seed=9, G=4, B=48)
    assert F.fathom_scan_topk_workspace_size(U, 4, 64 * planes.shape[-1], k) > F.fathom_scan_topk_noalloc_capacity()
    idx = torch.full((U, 4, k), -3, dtype=torch.int32, device=DEV)
    val = torch.zeros((U, 4, k), dtype=torch.float32, device=DEV)
    with pytest.raises(F.FathomError) as e:
        F.fathom_scan_topk_noalloc(planes, scales, nt, q, d, k, 0, 0, idx, val)
    assert e.value.code == F.FATHOM_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (idx == -3).all()
