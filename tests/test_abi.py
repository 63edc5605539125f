"""CPU checks of the C ABI: the library loads, exports every symbol declared in
include/fathom.h, and rejects bad arguments on the host before any launch.
No call here reaches a kernel (all of them fail validation or are no-ops)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def fl():
    import paper_2609_17652_amd as F
    if not os.path.exists(F.LIB_PATH):
        from paper_2609_17652_amd import build
        build.build()
    return F


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "fathom.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fathom_[a-z_]+)\s*\(", src)))


def test_header_declares_the_five_steps():
    syms = declared_symbols()
    for s in ("fathom_pack", "fathom_alloc_depths", "fathom_scan", "fathom_topk", "fathom_sparse_attn"):
        assert s in syms


def test_library_exports_every_declared_symbol(fl):
    L = fl.lib()
    for s in declared_symbols():
        assert hasattr(L, s), s
    assert sorted(fl.EXPORTED) == declared_symbols()


def test_status_strings_and_version(fl):
    assert fl.fathom_status_string(0) == "FATHOM_OK"
    assert fl.fathom_status_string(-5) == "FATHOM_ERR_WORKSPACE"
    assert "gfx950" in fl.fathom_version()


def test_constants_match_header(fl):
    src = open(os.path.join(ROOT, "include", "fathom.h")).read()
    for name in ("FATHOM_DEV_SCALE_OVERFLOW", "FATHOM_DEV_NONFINITE", "FATHOM_DEV_TOPK_FALLBACK",
                 "FATHOM_DEV_TOPK_SHORT", "FATHOM_DEV_BAD_N", "FATHOM_MAX_K"):
        m = re.search(rf"#define {name} (\d+)u?", src)
        assert m and int(m.group(1)) == getattr(fl, name), name
    for name, val in (("FATHOM_ERR_INVALID", -1), ("FATHOM_ERR_UNSUPPORTED", -2), ("FATHOM_ERR_RANGE", -3),
                      ("FATHOM_ERR_HIP", -4), ("FATHOM_ERR_WORKSPACE", -5)):
        assert re.search(rf"{name} = {val}", src) and getattr(fl, name) == val


def test_workspace_sizes(fl):
    a = fl.fathom_topk_workspace_size(8, 4, 1 << 20, 2048)
    b = fl.fathom_topk_workspace_size(8, 4, 1 << 20, 4096)
    assert 0 < a < b
    s = fl.fathom_scan_topk_workspace_size(8, 4, 1 << 20, 2048)
    # the fused scan + top-k keeps no score array: well below 8 x 4 x 2^20 fp32 scores
    # (the exact pass's per-chunk partial lists are its largest part)
    assert 0 < s < 8 * 4 * (1 << 20) * 4 // 3
    assert fl.fathom_topk_workspace_size(0, 4, 10, 10) == 0


NULL = None
S = C.c_void_p(0)
FAKE = C.c_void_p(0x1000)  # never dereferenced: every call below fails host validation


def test_host_validation(fl):
    L = fl.lib()
    # pack: D != 128, bad dtype, negative U, null pointers, misaligned K, bad ld_tok
    assert L.fathom_pack(FAKE, 0, 128, 0, FAKE, 1, 64, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_pack(FAKE, 7, 128, 0, FAKE, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_pack(FAKE, 0, 128, 0, FAKE, -1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack(NULL, 0, 128, 0, FAKE, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack(C.c_void_p(0x1004), 0, 128, 0, FAKE, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack(FAKE, 0, 100, 0, FAKE, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack(FAKE, 0, 130, 0, FAKE, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack(NULL, 0, 128, 0, NULL, 0, 128, 1, NULL, NULL, NULL, S) == fl.FATHOM_OK  # U = 0: no-op
    # gather_store: D, null pointers, misaligned bases (rejected before any HIP call)
    assert L.fathom_gather_store(FAKE, FAKE, FAKE, 1, 64, 1, FAKE, FAKE, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_gather_store(NULL, FAKE, FAKE, 1, 128, 1, FAKE, FAKE, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_gather_store(C.c_void_p(0x1008), FAKE, FAKE, 1, 128, 1, FAKE, FAKE, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_gather_store(NULL, NULL, NULL, 0, 128, 1, NULL, NULL, S) == fl.FATHOM_OK  # U = 0: no-op
    # pack_append: as pack, plus n_old and a non-negative bound on new tokens
    assert L.fathom_pack_append(FAKE, 0, 128, 0, NULL, FAKE, 1, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack_append(FAKE, 0, 128, 0, FAKE, FAKE, -1, 1, 128, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack_append(FAKE, 0, 128, 0, FAKE, FAKE, 1, 1, 64, 1, FAKE, FAKE, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_pack_append(FAKE, 0, 128, 0, C.c_void_p(0x1004), FAKE, 1, 1, 128, 1, FAKE, FAKE, NULL,
                                S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_pack_append(NULL, 0, 128, 0, NULL, NULL, 1, 0, 128, 1, NULL, NULL, NULL, S) == fl.FATHOM_OK
    # alloc: budget / r range, G range, mode
    assert L.fathom_alloc_depths(FAKE, 0, 1, 4, 128, FAKE, 0, 513, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_RANGE
    assert L.fathom_alloc_depths(FAKE, 0, 1, 4, 128, FAKE, 0, -1, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_RANGE
    assert L.fathom_alloc_depths(FAKE, 0, 1, 4, 128, FAKE, 1, 129, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_RANGE
    assert L.fathom_alloc_depths(FAKE, 0, 1, 9, 128, FAKE, 0, 48, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_alloc_depths(FAKE, 0, 1, 4, 128, FAKE, 5, 48, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_alloc_depths(FAKE, 0, 1, 4, 128, NULL, 0, 48, FAKE, NULL, NULL, S) == fl.FATHOM_ERR_INVALID
    # scan: G = 0, D = 64, null depths, ld_s < 1
    assert L.fathom_scan(FAKE, FAKE, FAKE, 1, 128, 4, FAKE, 0, 0, FAKE, FAKE, 256, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_scan(FAKE, FAKE, FAKE, 1, 64, 4, FAKE, 0, 4, FAKE, FAKE, 256, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_scan(FAKE, FAKE, FAKE, 1, 128, 4, FAKE, 0, 4, NULL, FAKE, 256, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_scan(FAKE, FAKE, FAKE, 1, 128, 4, FAKE, 0, 4, FAKE, FAKE, 0, NULL, S) == fl.FATHOM_ERR_INVALID
    # top-k: k too large, k < 1, small workspace, misaligned workspace
    ws = fl.fathom_topk_workspace_size(1, 4, 4096, 64)
    assert L.fathom_topk(FAKE, 4096, FAKE, 1, 4, 9000, 0, 0, FAKE, NULL, FAKE, ws, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_topk(FAKE, 4096, FAKE, 1, 4, 0, 0, 0, FAKE, NULL, FAKE, ws, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_topk(FAKE, 4096, FAKE, 1, 4, 64, 0, 0, FAKE, NULL, FAKE, ws - 1, NULL, S) == fl.FATHOM_ERR_WORKSPACE
    assert L.fathom_topk(FAKE, 4096, FAKE, 1, 4, 64, -1, 0, FAKE, NULL, FAKE, ws, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_topk(FAKE, 4096, FAKE, 1, 4, 64, 0, 0, FAKE, NULL, C.c_void_p(0x1010), ws, NULL, S) == \
        fl.FATHOM_ERR_INVALID
    ws2 = fl.fathom_scan_topk_workspace_size(1, 4, 4096, 64)
    assert L.fathom_scan_topk(FAKE, FAKE, FAKE, 1, 128, 64, FAKE, 1, 4, FAKE, 64, 0, 0, FAKE, NULL, FAKE, ws2 - 1,
                              NULL, S) == fl.FATHOM_ERR_WORKSPACE
    # the no-workspace variant: a shape beyond the library's array, k too large, null idx (no HIP call made)
    cap = fl.fathom_scan_topk_noalloc_capacity()
    assert cap == 64 << 20
    assert fl.fathom_scan_topk_workspace_size(64, 4, 1 << 20, 8192) > cap
    assert fl.fathom_scan_topk_workspace_size(8, 4, 1 << 20, 2048) <= cap
    assert L.fathom_scan_topk_noalloc(FAKE, FAKE, FAKE, 64, 128, 1 << 14, FAKE, 1, 4, FAKE, 8192, 0, 0, 0, FAKE,
                                      NULL, NULL, S) == fl.FATHOM_ERR_WORKSPACE
    assert L.fathom_scan_topk_noalloc(FAKE, FAKE, FAKE, 1, 128, 64, FAKE, 1, 4, FAKE, 9000, 0, 0, 0, FAKE, NULL,
                                      NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_scan_topk_noalloc(FAKE, FAKE, FAKE, 1, 128, 64, FAKE, 1, 4, FAKE, 64, 0, 0, 0, NULL, NULL,
                                      NULL, S) == fl.FATHOM_ERR_INVALID
    # sparse attention: sink + local too large, odd ld_tok, null out
    wsa = fl.fathom_sparse_attn_workspace_size(1, 4, 8, 4, 32)
    assert wsa > 0
    assert L.fathom_sparse_attn(FAKE, 0, FAKE, FAKE, 128, 0, FAKE, 1, 4, 128, FAKE, 8, 1000, 100, C.c_float(1.0),
                                FAKE, FAKE, wsa, NULL, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_sparse_attn(FAKE, 0, FAKE, FAKE, 129, 0, FAKE, 1, 4, 128, FAKE, 8, 4, 32, C.c_float(1.0),
                                FAKE, FAKE, wsa, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_sparse_attn(FAKE, 0, FAKE, FAKE, 128, 0, FAKE, 1, 4, 128, FAKE, 8, 4, 32, C.c_float(1.0),
                                NULL, FAKE, wsa, NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_sparse_attn(FAKE, 0, FAKE, FAKE, 128, 0, FAKE, 1, 4, 128, FAKE, 8, 4, 32, C.c_float(1.0),
                                FAKE, FAKE, wsa - 1, NULL, S) == fl.FATHOM_ERR_WORKSPACE


def test_klt_host_validation(fl):
    L = fl.lib()
    wsk = fl.fathom_klt_calibrate_workspace_size(2)
    assert wsk >= 2 * 32 * 128 * 128 * 8 and fl.fathom_klt_calibrate_workspace_size(0) == 0
    A256 = C.c_void_p(0x10000)
    # calibrate: D, dtype, U < 0, null outputs, short or misaligned workspace, ld_tok < D
    assert L.fathom_klt_calibrate(FAKE, 0, 128, 0, FAKE, 64, 2, 64, FAKE, FAKE, FAKE, A256, wsk, NULL,
                                  S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_klt_calibrate(FAKE, 5, 128, 0, FAKE, 64, 2, 128, FAKE, FAKE, FAKE, A256, wsk, NULL,
                                  S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_klt_calibrate(FAKE, 0, 128, 0, FAKE, 64, -1, 128, FAKE, FAKE, FAKE, A256, wsk, NULL,
                                  S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_calibrate(FAKE, 0, 128, 0, FAKE, 64, 2, 128, FAKE, NULL, FAKE, A256, wsk, NULL,
                                  S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_calibrate(FAKE, 0, 128, 0, FAKE, 64, 2, 128, FAKE, FAKE, FAKE, A256, wsk - 1, NULL,
                                  S) == fl.FATHOM_ERR_WORKSPACE
    assert L.fathom_klt_calibrate(FAKE, 0, 128, 0, FAKE, 64, 2, 128, FAKE, FAKE, FAKE, C.c_void_p(0x10080), wsk,
                                  NULL, S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_calibrate(FAKE, 0, 100, 0, FAKE, 64, 2, 128, FAKE, FAKE, FAKE, A256, wsk, NULL,
                                  S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_calibrate(NULL, 0, 128, 0, NULL, 0, 0, 128, NULL, NULL, NULL, NULL, 0, NULL,
                                  S) == fl.FATHOM_OK  # U = 0: no-op
    # rotate keys: output block shorter than n_cap rows, null mu, misaligned fp16 keys
    assert L.fathom_klt_rotate_keys(FAKE, 0, 128, 0, FAKE, 64, 1, 128, FAKE, FAKE, FAKE, 63 * 128, NULL,
                                    S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_rotate_keys(FAKE, 0, 128, 0, FAKE, 64, 1, 128, NULL, FAKE, FAKE, 64 * 128, NULL,
                                    S) == fl.FATHOM_ERR_INVALID
    assert L.fathom_klt_rotate_keys(C.c_void_p(0x1001), 1, 128, 0, FAKE, 64, 1, 128, FAKE, FAKE, FAKE, 64 * 128,
                                    NULL, S) == fl.FATHOM_ERR_INVALID
    # rotate q: G outside 1..8, D != 128, null V
    assert L.fathom_klt_rotate_q(FAKE, 0, 1, 9, 128, FAKE, FAKE, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_klt_rotate_q(FAKE, 0, 1, 4, 64, FAKE, FAKE, S) == fl.FATHOM_ERR_UNSUPPORTED
    assert L.fathom_klt_rotate_q(FAKE, 0, 1, 4, 128, NULL, FAKE, S) == fl.FATHOM_ERR_INVALID


def test_synth_is_deterministic_and_shaped():
    from paper_2609_17652_amd import synth
    cfg = synth.WORKLOADS["head4k"]
    a = synth.host_units(cfg)
    b = synth.host_units(cfg)
    assert np.array_equal(a.K, b.K) and np.array_equal(a.q, b.q) and np.array_equal(a.var, b.var)
    assert a.K.shape == (1, 4096, 128) and a.q.shape == (1, 1, 128) and a.q.dtype == np.float32
    c1 = synth.WORKLOADS["layer128k"]
    h = synth.host_units(c1, units=[0, 1], n_override=256)
    assert h.q.dtype == np.float16 and h.q.shape == (2, 4, 128)
    assert not np.array_equal(h.K[0], h.K[1])
    n3 = synth.unit_lengths(synth.WORKLOADS["ragged16"])
    assert n3.shape == (128,) and n3.min() >= 65536 and n3.max() <= 524288
    assert (n3.reshape(16, 8) == n3.reshape(16, 8)[:, :1]).all()  # one length per session
    # 4 outlier channels at 8x
    rng = synth.unit_rng(0, 0, 0, 0)
    z = np.exp(rng.standard_normal(128))
    rng = synth.unit_rng(0, 0, 0, 0)
    s = synth.channel_sigma(rng)
    assert np.isclose(s / z, 8.0).sum() == 4 and np.isclose(s / z, 1.0).sum() == 124
