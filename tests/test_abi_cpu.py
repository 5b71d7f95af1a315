"""The C-ABI library without a GPU: it loads, exports every function
include/kara.h and include/kara_harness.h declare, and its host-side argument checks reject bad calls
before anything is launched."""
import ctypes
import os

import pytest

from paper_2607_01237_amd import kara

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(kara.LIB_PATH):
        from paper_2607_01237_amd import build
        build.build()
    return kara.load()


def good_params(**kw):
    p = dict(window=1024, buffer=0, budget=205, chunk_budget=16, max_chunk_len=8, head_dim=128,
             n_q_heads=32, n_kv_heads=8, block_size=16, num_pages=4096, max_blocks_per_seq=200,
             dtype="bf16", scale=0.0)
    p.update(kw)
    return kara.make_params(p, n_seqs=8)


def test_exports_every_declared_function(lib):
    names = kara.header_functions()
    # 15 in kara.h, 3 in kara_harness.h, 9 in kara_sched.h, 3 in kara_recompute.h
    assert len(names) == 30, names
    for n in names:
        assert hasattr(lib, n), n


def test_library_is_built_from_these_sources(lib):
    from paper_2607_01237_amd import build
    assert lib.kara_source_hash().decode() == build.source_hash()


def test_version_and_status_strings(lib):
    assert kara.abi_version() == 3
    for code in (0, -1, -2, -3, -4, -5, -6, -7):
        assert kara.status_string(code).startswith("KARA_")
    assert "unknown" in kara.status_string(12345)
    # nothing has failed on this thread: no HIP call is made to say so
    assert lib.kara_last_hip_error() == b"no HIP error"


def test_workspace_size_scales(lib):
    a = kara.workspace_size(good_params(), 8, 1)
    b = kara.workspace_size(good_params(), 8, 2)
    assert a > 0 and b > a
    # at least the scores, index sets and one partial slab per unit
    units = 8 * 8
    assert a >= units * (1024 * 4 * 2 + 189 * 4 + 205 * 4)


@pytest.mark.parametrize("field,value,code", [
    ("window", 0, kara.ERR_INVALID_ARG),
    ("buffer", 1024, kara.ERR_INVALID_ARG),
    ("buffer", -1, kara.ERR_INVALID_ARG),
    ("budget", 0, kara.ERR_INVALID_ARG),
    ("budget", 1025, kara.ERR_INVALID_ARG),
    ("chunk_budget", 205, kara.ERR_INVALID_ARG),
    ("chunk_budget", -1, kara.ERR_INVALID_ARG),
    ("max_chunk_len", 2, kara.ERR_INVALID_ARG),
    ("n_q_heads", 30, kara.ERR_INVALID_ARG),
    ("head_dim", 96, kara.ERR_UNSUPPORTED),
    ("dtype", 7, kara.ERR_INVALID_ARG),
    ("block_size", 0, kara.ERR_INVALID_ARG),
    ("scale", float("inf"), kara.ERR_INVALID_ARG),
    ("score_queries", -1, kara.ERR_INVALID_ARG),
    ("score_queries", 1025, kara.ERR_INVALID_ARG),
])
def test_bad_params_rejected(lib, field, value, code):
    p = good_params()
    setattr(p, field, value)
    out = ctypes.c_size_t(0)
    assert lib.kara_workspace_size(ctypes.byref(p), 8, 1, ctypes.byref(out)) == code


def test_compressible_limit(lib):
    p = good_params(window=kara.MAX_COMPRESSIBLE + 1, budget=10, chunk_budget=4)
    out = ctypes.c_size_t(0)
    assert lib.kara_workspace_size(ctypes.byref(p), 1, 1, ctypes.byref(out)) == kara.ERR_UNSUPPORTED
    p = good_params(window=kara.MAX_COMPRESSIBLE + 1, buffer=1, budget=10, chunk_budget=4)
    assert lib.kara_workspace_size(ctypes.byref(p), 1, 1, ctypes.byref(out)) == kara.OK


def test_null_pointers_rejected_before_launch(lib):
    p = good_params()
    r = ctypes.byref(p)
    assert lib.kara_validate(r, 4, None, None, None, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_select(r, 4, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_token2chunk(r, 4, None, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_select_kept(r, 4, None, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_commit_tables(r, 4, None, None, None, None, None, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_compact_pages(r, 4, None, 1, None, None, None, None, None, None, None, None) == kara.ERR_INVALID_ARG
    assert lib.kara_score_window(r, 4, None, 1, None, None, None, None, None, None, None, None, 0, None) == kara.ERR_INVALID_ARG
    assert lib.kara_compress_window(r, 4, None, 1, None, None, None, None, None, None, 1, None, None, None, None,
                                    None, None, None, 0, None) == kara.ERR_INVALID_ARG
    # nothing to do is not an error, and touches no pointer
    assert lib.kara_select(r, 0, None, None, None) == kara.OK
    assert lib.kara_validate(r, 0, None, None, None, None, None, None) == kara.OK
    assert lib.kara_token2chunk(r, 0, None, None, None, None) == kara.OK
    assert lib.kara_select_kept(r, 0, None, None, None, None) == kara.OK
    assert lib.kara_commit_tables(r, 0, None, None, None, None, None, None, None, None) == kara.OK
    assert lib.kara_compact_pages(r, 0, None, 1, None, None, None, None, None, None, None, None) == kara.OK
    assert lib.kara_score_window(r, 0, None, 1, None, None, None, None, None, None, None, None, 0, None) == kara.OK
    assert lib.kara_compress_window(r, 0, None, 1, None, None, None, None, None, None, 1, None, None, None, None,
                                    None, None, None, 0, None) == kara.OK
    assert lib.kara_compress_prefill(r, 0, None, 2, 1, None, None, None, None, None, None, 1, None, None, None,
                                     None, None, None, None, 0, None) == kara.OK


def test_workspace_checked_before_launch(lib):
    p = good_params()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: the size check fails first
    pools = (ctypes.c_void_p * 1)(0x1000)
    rc = lib.kara_compress_window(ctypes.byref(p), 2, fake, 1, fake, pools, pools, fake, fake, fake, 1, None,
                                  None, None, fake, fake, fake, fake, 16, None)
    assert rc == kara.ERR_WORKSPACE


def test_noalloc_rejects_calls_past_its_scratch(lib):
    """The allocation-free entry point refuses, before touching any pointer,
    a call whose workspace would not fit its static scratch; empty calls
    succeed."""
    p = good_params()
    fake = ctypes.c_void_p(0x1000)   # never dereferenced
    pools = (ctypes.c_void_p * 40)(*([0x1000] * 40))
    need = kara.workspace_size(p, 64, 40)
    assert need > kara.NOALLOC_SCRATCH_BYTES
    rc = lib.kara_compress_window_noalloc(ctypes.byref(p), 64, fake, 40, fake, pools, pools, fake, fake, fake, 1,
                                          None, None, None, fake, fake, fake, None)
    assert rc == kara.ERR_SCRATCH_LIMIT
    assert "KARA_NOALLOC_SCRATCH_BYTES" in kara.status_string(rc)
    assert lib.kara_compress_window_noalloc(ctypes.byref(p), 0, None, 1, None, None, None, None, None, None, 1,
                                            None, None, None, None, None, None, None) == kara.OK
    # one layer of 200 such sequences fits, as the header says
    assert kara.workspace_size(p, 200, 1) <= kara.NOALLOC_SCRATCH_BYTES
    assert kara.workspace_size(good_params(), 30, 7) <= kara.NOALLOC_SCRATCH_BYTES


def test_harness_checks_before_launch(lib):
    p = good_params()
    r = ctypes.byref(p)
    out = ctypes.c_size_t(0)
    assert lib.kara_harness_decode_workspace_size(r, 4, 2, 1000, ctypes.byref(out)) == kara.OK
    # 4 sequences x 2 layers x 32 query heads x 4 splits of 256 keys x (m, l, o[128])
    assert out.value == 4 * 2 * 32 * 4 * 130 * 4
    # longer than the block table can hold
    assert lib.kara_harness_decode_workspace_size(r, 4, 2, 200 * 16 + 1, ctypes.byref(out)) == kara.ERR_INVALID_ARG
    assert lib.kara_harness_kv_append(r, 4, None, 8, 1, None, None, None, None, None, None, None, None) \
        == kara.ERR_INVALID_ARG
    assert lib.kara_harness_kv_append(r, 0, None, 8, 1, None, None, None, None, None, None, None, None) == kara.OK
    fake = ctypes.c_void_p(0x1000)
    pools = (ctypes.c_void_p * 1)(0x1000)
    assert lib.kara_harness_decode_attention(r, 4, fake, 1, fake, pools, pools, fake, fake, 1000, fake, fake, 16,
                                             None) == kara.ERR_WORKSPACE
    wide = good_params(n_q_heads=256, n_kv_heads=8)
    assert lib.kara_harness_decode_attention(ctypes.byref(wide), 4, fake, 1, fake, pools, pools, fake, fake, 1000,
                                             fake, fake, 1 << 30, None) == kara.ERR_UNSUPPORTED


def test_scoring_queries_shrink_the_workspace(lib):
    # the partial column sums scale with the scoring rows (G * Wq)
    full = kara.workspace_size(good_params(), 8, 1)
    part = kara.workspace_size(good_params(buffer=64, budget=192, score_queries=64), 8, 1)
    assert part < full
    assert kara.workspace_size(good_params(score_queries=1024), 8, 1) == full


def test_recompute_host_checks(lib):
    """The recompute entry points reject bad arguments on the host (nothing
    is launched) and accept empty calls."""
    p = good_params()
    m = kara.make_model(4096, 12288)
    assert kara.recompute_workspace_size(p, m, 4) > 0
    assert kara.recompute_workspace_size(p, m, 8) > kara.recompute_workspace_size(p, m, 4)
    for bad in (kara.make_model(4094, 12288), kara.make_model(4096, 12284), kara.make_model(4096, 12288, 0.5),
                kara.make_model(4096, 12288, 1e4, -1.0)):
        with pytest.raises(kara.KaraError) as e:
            kara.recompute_workspace_size(p, bad, 4)
        assert e.value.code == kara.ERR_INVALID_ARG
    f32 = good_params(dtype="f32", window=256, budget=52)
    with pytest.raises(kara.KaraError) as e:
        kara.recompute_workspace_size(f32, m, 4)
    assert e.value.code == kara.ERR_UNSUPPORTED
    import ctypes
    out = ctypes.c_size_t(0)
    assert lib.kara_recompute_workspace_size(ctypes.byref(p), ctypes.byref(m), 4, None) == kara.ERR_INVALID_ARG
    # empty calls succeed without touching the device; missing pointers are argument errors
    assert lib.kara_recompute_attention(ctypes.byref(p), 0, None, None, None, None, None, None, None, None, None,
                                        None) == kara.OK
    assert lib.kara_recompute_attention(ctypes.byref(p), 2, None, None, None, None, None, None, None, None, None,
                                        None) == kara.ERR_INVALID_ARG
    w = (kara.LayerWeights * 1)()
    assert lib.kara_recompute_queries(ctypes.byref(p), ctypes.byref(m), 0, None, 1, w, None, None, None, None, None,
                                      None, None, None, None, None, None, 0, None) == kara.OK
    assert lib.kara_recompute_queries(ctypes.byref(p), ctypes.byref(m), 2, None, 1, w, None, None, None, None, None,
                                      None, None, None, None, None, None, 0, None) == kara.ERR_INVALID_ARG
    assert lib.kara_recompute_queries(ctypes.byref(p), ctypes.byref(m), 2, None, 0, w, None, None, None, None, None,
                                      None, None, None, None, None, None, 0, None) == kara.ERR_INVALID_ARG


def test_binding_shape_checks():
    """The binding's host checks (the library cannot see tensor sizes):
    wrong dtype or too few elements raise before any call."""
    torch = pytest.importorskip("torch")
    p = good_params()
    kara._need("x", None, 10, torch.int32)                     # optional argument left out
    kara._need("x", torch.zeros(8, dtype=torch.int32), 8, torch.int32)
    with pytest.raises(kara.KaraError, match="dtype"):
        kara._need("trig", torch.zeros(8, dtype=torch.int64), 8, torch.int32)
    with pytest.raises(kara.KaraError, match="at least 9"):
        kara._need("status", torch.zeros(8, dtype=torch.int32), 9, torch.int32)
    # the per-step outputs scale with units and the window's compressible length
    units = kara._units(p, 2, 3)
    assert units == 2 * 3 * p.n_kv_heads
    kara._step_outputs(p, units, torch.zeros(units * (p.window - p.buffer)), None, None)
    with pytest.raises(kara.KaraError, match="kept"):
        kara._step_outputs(p, units, None, None, torch.zeros(units * p.budget - 1, dtype=torch.int32))
    with pytest.raises(kara.KaraError, match="block_table"):
        kara._tables(p, torch.zeros(p.n_seqs * p.max_blocks_per_seq - 1, dtype=torch.int32), None)
    with pytest.raises(kara.KaraError, match="k_pools"):
        kara._pools(p, [torch.zeros(4, dtype=torch.bfloat16)], "k_pools")
