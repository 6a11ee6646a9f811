"""The C-ABI library loads and exports every symbol include/oasis.h declares (CPU only).

No compute call is made here; argument checks that fail before any HIP call
are exercised through ctypes.
"""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oasis.h")
LIB = os.path.join(ROOT, "paper_2608_08097_amd", "liboasis.so")


def declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^OASIS_API\s+[\w\s\*]+?\b(oasis_\w+)\s*\(", txt, re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2608_08097_amd.build_lib import build
        build()
    import paper_2608_08097_amd as P
    return P


def test_header_declares_the_path():
    names = declared()
    for fn in ("oasis_score_blocks", "oasis_select_topk", "oasis_stage_blocks", "oasis_sparse_decode_attn",
               "oasis_build_summaries", "oasis_update_summaries", "oasis_copy_blocks", "oasis_attn_workspace_bytes",
               "oasis_pipeline_create", "oasis_pipeline_step", "oasis_last_error", "oasis_abi_version"):
        assert fn in names


def test_exports_match_header(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True, check=True).stdout
    exported = sorted({l.split()[-1] for l in out.splitlines() if l.split() and l.split()[-1].startswith("oasis_")})
    assert exported == declared()
    cdll = ctypes.CDLL(LIB)
    for fn in declared():
        assert hasattr(cdll, fn)
    assert sorted(lib._lib.EXPORTS) == declared()


def test_abi_version(lib):
    assert lib.oasis_abi_version() == 7


def test_argument_checks_without_gpu(lib):
    L = lib.lib()
    bad_hd = lib.dims(1, 32, 8, 64, 16, 512)
    assert L.oasis_score_blocks(ctypes.byref(bad_hd), None, 5, 1, 4, None, None, None, None, None) == 2
    assert "head_dim" in lib.oasis_last_error()
    bad_b = lib.dims(1, 32, 8, 128, 8, 512)
    assert L.oasis_select_topk(ctypes.byref(bad_b), None, None, 4, None, None, None) == 2
    bad_g = lib.dims(1, 30, 8, 128, 16, 512)
    assert L.oasis_sparse_decode_attn(ctypes.byref(bad_g), None, 5, None, None, None, 4, None, 1.0, None, None,
                                      None, 0, None) == 1
    d = lib.dims(1, 32, 8, 128, 16, 512)
    assert L.oasis_score_blocks(ctypes.byref(d), None, 5, 1, 4, None, None, None, None, None) == 1
    assert "q is NULL" in lib.oasis_last_error()
    assert L.oasis_score_blocks(ctypes.byref(d), None, 5, 2, 4, None, None, None, None, None) == 1  # rows past T
    assert L.oasis_select_topk(ctypes.byref(d), None, None, 0, None, None, None) == 1
    rows65 = lib.dims(1, 72, 8, 128, 16, 512)  # G = 9, D = 8 -> 72 scoring rows
    assert L.oasis_score_blocks(ctypes.byref(rows65), None, 9, 1, 8, None, None, None, None, None) == 2
    big = lib.dims(1, 96, 8, 128, 16, 512)     # G = 12, T = 9 -> 108 attention rows
    assert L.oasis_sparse_decode_attn(ctypes.byref(big), None, 9, None, None, None, 4, None, 1.0, None, None,
                                      None, 0, None) == 2
    # a fetch cap below 1 admits nothing and is rejected
    assert L.oasis_stage_blocks(ctypes.byref(d), None, None, 10, None, None, None, None, None, 128, None, None, 0,
                                0, 1, None, None, None, None) == 1
    assert "fetch_cap" in lib.oasis_last_error()
    # local-only form needs copy_local
    assert L.oasis_stage_blocks(ctypes.byref(d), None, None, 10, None, None, None, None, None, 128, None, None, 0,
                                128, 0, None, None, None, None) == 1
    # zero requests: a no-op that succeeds without touching the device
    z = lib.dims(0, 32, 8, 128, 16, 512)
    assert L.oasis_score_blocks(ctypes.byref(z), None, 5, 1, 4, None, None, None, None, None) == 0
    assert lib.oasis_last_error() == ""


def test_growth_argument_checks_without_gpu(lib):
    L = lib.lib()
    d = lib.dims(2, 32, 8, 128, 16, 64)
    assert L.oasis_update_summaries(ctypes.byref(d), None, 10, None, None, None, 0, None, None, None) == 1
    assert "max_new_blocks" in lib.oasis_last_error()
    assert L.oasis_update_summaries(ctypes.byref(d), None, 10, None, None, None, 1, None, None, None) == 1
    assert "k_pages is NULL" in lib.oasis_last_error()
    assert L.oasis_copy_blocks(ctypes.byref(d), None, None, 4, None, None, None, 4, None, None, None, 0, None) == 1
    assert "max_blocks" in lib.oasis_last_error()
    assert L.oasis_copy_blocks(ctypes.byref(d), None, None, 0, None, None, None, 4, None, None, None, 8, None) == 1
    z = lib.dims(0, 32, 8, 128, 16, 64)                      # no requests: a no-op
    assert L.oasis_copy_blocks(ctypes.byref(z), None, None, 4, None, None, None, 4, None, None, None, 8, None) == 0


def test_pipeline_argument_checks_without_gpu(lib):
    L = lib.lib()
    h = ctypes.c_void_p(123)
    d = lib.dims(1, 32, 8, 128, 16, 512)
    assert L.oasis_pipeline_create(ctypes.byref(d), 5, 1, 4, 128, 6, 1.0, None, None, 10, None, 8, None, None,
                                   None) == 1
    bad = lib.dims(1, 32, 8, 64, 16, 512)
    assert L.oasis_pipeline_create(ctypes.byref(bad), 5, 1, 4, 128, 6, 1.0, None, None, 10, None, 8, None, None,
                                   ctypes.byref(h)) == 2
    assert h.value is None                      # cleared on failure
    assert L.oasis_pipeline_create(ctypes.byref(d), 5, 1, 4, 128, 6, 1.0, None, None, 10, None, 0, None, None,
                                   ctypes.byref(h)) == 1
    assert "max_layers" in lib.oasis_last_error()
    assert L.oasis_pipeline_create(ctypes.byref(d), 5, 1, 4, 128, 6, 1.0, None, None, 10, None, 8, 1, None,
                                   ctypes.byref(h)) == 1
    assert L.oasis_pipeline_set_layer(None, 0, None) == 1
    assert L.oasis_pipeline_step(None, 0, None, None, None, 0, 0, 0, None, None) == 1
    assert L.oasis_pipeline_join(None, None) == 1
    assert L.oasis_pipeline_profile_begin(None, 4) == 1
    assert L.oasis_pipeline_profile_end(None, None, None, None) == 1
    assert L.oasis_pipeline_set_local_source(None, None, None, 0, None) == 1
    assert L.oasis_pipeline_set_plan_stream(None, 0) == 1
    L.oasis_pipeline_destroy(None)


def test_score_select_checks_without_gpu(lib):
    """The fused score + select entry point rejects the sizes it does not cover before any HIP call."""
    L = lib.lib()
    P = [ctypes.c_void_p(64 * (i + 1)) for i in range(6)]  # non-NULL stand-ins, never dereferenced
    ok = lib.dims(2, 32, 8, 128, 16, 512)
    # 4 scoring rows (G = 4, one draft): the vector-ALU scorer's range
    assert L.oasis_score_select(ctypes.byref(ok), P[0], 2, 1, 1, P[1], P[2], P[3], 64, P[4], P[5], P[0], None) == 2
    assert "scoring rows" in lib.oasis_last_error()
    # 40 scoring rows (G = 8, five drafts)
    g8 = lib.dims(2, 64, 8, 128, 16, 512)
    assert L.oasis_score_select(ctypes.byref(g8), P[0], 6, 1, 5, P[1], P[2], P[3], 64, P[4], P[5], P[0], None) == 2
    long_rows = lib.dims(2, 32, 8, 128, 16, 20000)
    assert L.oasis_score_select(ctypes.byref(long_rows), P[0], 5, 1, 4, P[1], P[2], P[3], 64, P[4], P[5], P[0],
                                None) == 2
    assert "max_blocks" in lib.oasis_last_error()
    assert L.oasis_score_select(ctypes.byref(ok), None, 5, 1, 4, P[1], P[2], P[3], 64, P[4], P[5], P[0], None) == 1
    assert L.oasis_pipeline_set_fused_prediction(None, 0) == 1
    assert L.oasis_pipeline_set_wait_limit(None, 5) == 1
    assert L.oasis_pipeline_set_prediction_order(None, 0) == 1
    assert L.oasis_pipeline_check(None) == 1


def test_workspace_sizes(lib):
    d = lib.dims(8, 32, 8, 128, 16, 8192)
    ws = lib.oasis_attn_workspace_bytes(d, 5, 128)
    # 64 (request, KV head) pairs x 4 splits x 20 rows x (128 outputs + max + sum) floats
    assert ws == 64 * 4 * 20 * 130 * 4
    assert lib.oasis_attn_workspace_bytes(lib.dims(1, 32, 8, 64, 16, 1), 5, 4) == 0
    # 512 pairs fill the chip with one split each: no partials, no workspace
    assert lib.oasis_attn_workspace_bytes(lib.dims(64, 32, 8, 128, 16, 1024), 5, 128) == 0


def test_noalloc_attention_checks_without_gpu(lib):
    """The allocation-free attention entry point checks like the workspace form and rejects sizes whose
    partials exceed its scratch, all before any HIP call."""
    L = lib.lib()
    bad_hd = lib.dims(1, 32, 8, 64, 16, 512)
    assert L.oasis_sparse_decode_attn_noalloc(ctypes.byref(bad_hd), None, 5, None, None, None, 128, None, 0.1,
                                              None, None, None) == 2
    ok = lib.dims(8, 32, 8, 128, 16, 8192)
    assert L.oasis_sparse_decode_attn_noalloc(ctypes.byref(ok), None, 0, None, None, None, 128, None, 0.1, None,
                                              None, None) == 1
    assert L.oasis_sparse_decode_attn_noalloc(ctypes.byref(ok), None, 5, None, None, None, 128, None, 0.1, None,
                                              None, None) == 1
    assert "is NULL" in lib.oasis_last_error()
    # 255 pairs (G = 16: 80 rows) x 2 splits x 80 rows x 130 floats = 21.2 MB of partials > the 16 MiB scratch
    big = lib.dims(255, 16, 1, 128, 16, 8192)
    need = lib.oasis_attn_workspace_bytes(big, 5, 128)
    assert need == 255 * 2 * 80 * 130 * 4 and need > lib._lib.NOALLOC_SCRATCH_BYTES
    assert L.oasis_sparse_decode_attn_noalloc(ctypes.byref(big), None, 5, None, None, None, 128, None, 0.1, None,
                                              None, None) == 2
    assert "scratch" in lib.oasis_last_error()


def test_local_block_pages_cover_every_local_block():
    """The device copy of the active blocks holds, for every request and step, the block that is
    local at that step, at the index its table gives."""
    from workloads import make_workload
    w = make_workload("c3", num_reqs=4, ctx_args=(16, 1, 40), steps=37, budget=16 * 4)
    pages, table = w.local_block_pages(37)
    B = w.cfg.block_size
    seen = set()
    for s in range(37):
        for r, L in enumerate(w.ctx_len(s)):
            b = (int(L) - 1) // B
            i = table[r, b]
            assert i >= 0 and pages[i] == w.block_table[r, b]
            seen.add((r, b))
    assert len(seen) == len(pages) == int((table >= 0).sum())

