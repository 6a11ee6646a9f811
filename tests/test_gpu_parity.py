"""GPU parity: every kernel of the decode path through the C ABI vs the CPU oracle.

Sizes are chosen so the oracle finishes in seconds while the kernels still see
several tiles, splits and a ragged tail (contexts that are not multiples of
the block size or of the 16-block scoring tile, budgets larger than the
candidate count, empty and one-token contexts).
"""
import math
import time

import numpy as np
import pytest
import torch

import paper_2608_08097_amd as P
from oracle import oasis_oracle as O
from paper_2608_08097_amd.path import DecodePath, LayerState
from tests.gpu_util import (as_np_bits, assert_attn_close, assert_lse_close, assert_scores_close, dev_bf16,
                            dev_i32, host_bits, note, oracle_layer, pinned_pages, pool_v_from_htd, pool_v_to_htd,
                            selection_diff)
from workloads import (config, f32_to_bf16_bits, make_workload, random_bf16, random_scores,
                       random_selection, random_selection_h)

pytestmark = pytest.mark.gpu


def _dims(w):
    c = w.cfg
    return P.dims(c.num_reqs, c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size, w.NBmax)


def _summ_bits(x):
    """Oracle summaries (exact bf16 values, NaN where undefined) -> bf16 bits."""
    return f32_to_bf16_bits(np.nan_to_num(x, nan=0.0).astype(np.float32))


CASES = {
    # ragged contexts from 1 token to a few hundred blocks, B = 16
    "ragged16": lambda: make_workload("c2", num_reqs=5, ctx_args=(1, 3000), budget=512),
    "c1": lambda: make_workload("c1"),
    # B = 32, 64 scoring rows (G = 8, D = 8), 72 attention rows
    "gqa8_b32": lambda: make_workload("c5", num_reqs=2, ctx_args=(3000,), budget=1024),
    # G = 4, D = 1: 4 scoring rows (vector-ALU scorer), 8 attention rows
    "d1": lambda: make_workload("c1", num_draft=1, ctx_args=(2500,), budget=256),
    # one KV head group with 2 query heads, D = 2
    "g2": lambda: make_workload("c2", num_reqs=3, num_q_heads=16, num_draft=2, ctx_args=(700, 2200), budget=320),
    # G = 4, D = 6: 24 scoring rows (two row tiles), 28 attention rows
    "g4_d6": lambda: make_workload("c2", num_reqs=2, num_draft=6, ctx_args=(900, 2600), budget=384),
    # G = 8, D = 6, B = 32: 48 scoring rows (three row tiles), 56 attention rows (four tiles)
    "g8_d6_b32": lambda: make_workload("c5", num_reqs=2, num_draft=6, ctx_args=(2000,), budget=512),
    # 2 requests x 2 KV heads: a staging grid of 4 workgroups with batches of 8 entries
    "h2": lambda: make_workload("c2", num_reqs=2, num_q_heads=8, num_kv_heads=2, ctx_args=(600, 2500),
                                budget=16 * 20),
}


@pytest.fixture(scope="module", params=sorted(CASES))
def case(request):
    note(f"building inputs for {request.param}")
    w = CASES[request.param]()
    hk_t, hv_t = pinned_pages(w)
    return request.param, w, hk_t, hv_t


# ---------------------------------------------------------------------------
# a0 summaries: bit-exact
# ---------------------------------------------------------------------------

def test_summaries_bit_exact(case):
    name, w, hk_t, hv_t = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    ref_max, ref_min = O.block_summaries(as_np_bits(hk_t), w.block_table, ctx, c.block_size, w.NBmax)
    for source in ("pinned", "device"):
        note(f"summaries {name} from {source} pages")
        pages = hk_t if source == "pinned" else hk_t.cuda()
        kmax = torch.zeros((c.num_reqs, c.num_kv_heads, w.NBmax, c.head_dim), dtype=torch.bfloat16, device="cuda")
        kmin = torch.zeros_like(kmax)
        P.oasis_build_summaries(d, pages, dev_i32(w.block_table), dev_i32(ctx), kmax, kmin)
        torch.cuda.synchronize()
        gmax, gmin = O.bf16_to_f64(host_bits(kmax)), O.bf16_to_f64(host_bits(kmin))
        for r in range(c.num_reqs):
            _, nc, _ = O.block_counts(ctx[r], c.block_size)
            assert np.array_equal(gmax[r, :, :nc], ref_max[r, :, :nc]), (r, "kmax")
            assert np.array_equal(gmin[r, :, :nc], ref_min[r, :, :nc]), (r, "kmin")
            assert np.all(gmax[r, :, nc:] == 0), "rows past the candidates must stay untouched"


# ---------------------------------------------------------------------------
# a1 scores on the oracle's summaries
# ---------------------------------------------------------------------------

def test_scores(case):
    name, w, hk_t, _ = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    q = w.queries(0)
    kmax, kmin = O.block_summaries(as_np_bits(hk_t), w.block_table, ctx, c.block_size, w.NBmax)
    ref = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    note(f"scores {name}")
    scores = torch.full((c.num_reqs, c.num_kv_heads, w.NBmax), 7.0, device="cuda")
    P.oasis_score_blocks(d, dev_bf16(q), c.T, 1, c.num_draft, dev_bf16(_summ_bits(kmax)), dev_bf16(_summ_bits(kmin)),
                         dev_i32(ctx), scores)
    torch.cuda.synchronize()
    assert_scores_close(scores.cpu().numpy(), ref)


# ---------------------------------------------------------------------------
# a2 selection on given scores: bit-exact
# ---------------------------------------------------------------------------

SCORE_ROW_CASES = [
    # (seed, R, Hq, Hkv, T, first_draft, num_draft, NBmax, B, ctx lengths): rows = G * num_draft
    (1, 2, 8, 8, 2, 1, 1, 300, 16, [4800, 1000]),          # 1 row (vector-ALU scorer)
    (2, 2, 16, 8, 2, 1, 1, 130, 16, [2080, 17]),           # 2 rows
    (3, 3, 8, 8, 4, 1, 3, 200, 32, [6400, 33, 0]),         # 3 rows, B = 32, an empty context
    (10, 2, 32, 8, 2, 1, 1, 333, 16, [5328, 700]),         # 4 rows: the largest vector-ALU case
    (4, 2, 40, 8, 2, 1, 1, 257, 16, [4112, 4000]),         # 5 rows (G = 5): the smallest MFMA case
    (5, 2, 32, 8, 3, 0, 2, 129, 16, [2064, 1500]),         # 8 rows, the verify row scoring too
    (6, 2, 24, 8, 4, 1, 3, 300, 16, [4800, 2222]),         # 9 rows
    (7, 1, 17, 1, 2, 1, 1, 1000, 16, [16000]),             # 17 rows: two row tiles
    (8, 2, 64, 8, 6, 1, 5, 150, 32, [4800, 1234]),         # 40 rows: three row tiles
    (9, 1, 64, 8, 9, 1, 8, 64, 32, [2048]),                # 64 rows: four row tiles
]


@pytest.mark.parametrize("seed,R,Hq,Hkv,T,first_draft,num_draft,NB,B,lens", SCORE_ROW_CASES)
def test_scores_rows(seed, R, Hq, Hkv, T, first_draft, num_draft, NB, B, lens):
    """Every scorer variant (vector ALUs up to 4 rows, MFMA with 1 to 4 row tiles) against the oracle."""
    d_head = 128
    q = random_bf16(500 + seed, (R, T, Hq, d_head))
    a = random_bf16(510 + seed, (R, Hkv, NB, d_head))
    b = random_bf16(520 + seed, (R, Hkv, NB, d_head), scale=2.0)
    av, bv = O.bf16_to_f64(a), O.bf16_to_f64(b)
    kmax_bits = np.where(av >= bv, a, b)
    kmin_bits = np.where(av >= bv, b, a)
    ctx = np.array(lens, np.int32)
    ref = O.block_scores(q, O.bf16_to_f64(kmax_bits), O.bf16_to_f64(kmin_bits), ctx, Hkv, B, first_draft, num_draft)
    note(f"scores rows={Hq // Hkv * num_draft} seed={seed}")
    d = P.dims(R, Hq, Hkv, d_head, B, NB)
    scores = torch.full((R, Hkv, NB), 7.0, device="cuda")
    P.oasis_score_blocks(d, dev_bf16(q), T, first_draft, num_draft, dev_bf16(kmax_bits), dev_bf16(kmin_bits),
                         dev_i32(ctx), scores)
    torch.cuda.synchronize()
    assert_scores_close(scores.cpu().numpy(), ref)


SCORE_SELECT_CASES = [
    # (seed, R, Hq, Hkv, T, first_draft, num_draft, NBmax, B, ctx lengths, k, tied): rows = G * num_draft, 5 to 32
    (1, 2, 40, 8, 2, 1, 1, 257, 16, [4112, 4000], 64, False),              # 5 rows
    (2, 3, 32, 8, 5, 1, 4, 700, 16, [11200, 16 * 300 + 5, 0], 128, False),  # 16 rows, ragged, an empty context
    (3, 2, 24, 8, 4, 1, 3, 300, 16, [4800, 2222], 128, True),              # 9 rows, duplicated blocks (ties)
    (4, 1, 17, 1, 2, 1, 1, 1000, 16, [16000], 200, False),                 # 17 rows: two row tiles
    (5, 2, 64, 8, 5, 1, 4, 150, 32, [4800, 1234], 32, True),               # 32 rows, B = 32
    (6, 2, 32, 8, 5, 1, 4, 9000, 16, [144000, 100000], 128, False),        # > 8 keys per thread
    (7, 2, 32, 8, 5, 1, 4, 64, 16, [1024, 700], 128, False),               # fewer candidates than k
]


@pytest.mark.parametrize("seed,R,Hq,Hkv,T,first_draft,num_draft,NB,B,lens,k,tied", SCORE_SELECT_CASES)
def test_score_select_fused(seed, R, Hq, Hkv, T, first_draft, num_draft, NB, B, lens, k, tied):
    """The fused score + select kernel gives bit for bit the scores and selections of the two kernels,
    and the selection matches the oracle's under the near-tie rule."""
    d_head = 128
    q = random_bf16(600 + seed, (R, T, Hq, d_head))
    a = random_bf16(610 + seed, (R, Hkv, NB, d_head))
    b = random_bf16(620 + seed, (R, Hkv, NB, d_head), scale=2.0)
    if tied:  # many blocks share one summary: equal scores, broken by block id
        a = a[:, :, np.arange(NB) % 7]
        b = b[:, :, np.arange(NB) % 7]
    av, bv = O.bf16_to_f64(a), O.bf16_to_f64(b)
    kmax_bits = np.ascontiguousarray(np.where(av >= bv, a, b))
    kmin_bits = np.ascontiguousarray(np.where(av >= bv, b, a))
    ctx = np.array(lens, np.int32)
    note(f"score+select rows={Hq // Hkv * num_draft} seed={seed} NB={NB} k={k}")
    d = P.dims(R, Hq, Hkv, d_head, B, NB)
    args = (dev_bf16(q), T, first_draft, num_draft, dev_bf16(kmax_bits), dev_bf16(kmin_bits), dev_i32(ctx))
    s2 = torch.full((R, Hkv, NB), 7.0, device="cuda")
    sel2 = torch.full((R, Hkv, k), -7, dtype=torch.int32, device="cuda")
    cnt2 = torch.full((R, Hkv), -7, dtype=torch.int32, device="cuda")
    P.oasis_score_blocks(d, *args, s2)
    P.oasis_select_topk(d, s2, args[-1], k, sel2, cnt2)
    s1 = torch.full((R, Hkv, NB), 5.0, device="cuda")
    sel1 = torch.full((R, Hkv, k), -5, dtype=torch.int32, device="cuda")
    cnt1 = torch.full((R, Hkv), -5, dtype=torch.int32, device="cuda")
    P.oasis_score_select(d, *args, k, s1, sel1, cnt1)
    torch.cuda.synchronize()
    assert np.array_equal(s1.cpu().numpy(), s2.cpu().numpy()), "scores differ from the scoring kernel"
    assert np.array_equal(sel1.cpu().numpy(), sel2.cpu().numpy()), "selection differs from the top-K kernel"
    assert np.array_equal(cnt1.cpu().numpy(), cnt2.cpu().numpy())
    ref = O.block_scores(q, O.bf16_to_f64(kmax_bits), O.bf16_to_f64(kmin_bits), ctx, Hkv, B, first_draft, num_draft)
    assert_scores_close(s1.cpu().numpy(), ref)
    ref_sel, ref_cnt = O.select_topk(ref, ctx, k, B)
    selection_diff(sel1.cpu().numpy(), cnt1.cpu().numpy(), ref_sel, ref_cnt, ref)


SELECT_CASES = [
    # (seed, R, H, NBmax, B, ctx lengths, k, n_distinct)
    (1, 3, 8, 700, 16, [16 * 700, 16 * 300 + 5, 16 * 129], 128, None),
    (2, 2, 8, 9000, 16, [16 * 9000, 16 * 8192], 128, None),
    (3, 4, 2, 600, 16, [9600, 16, 1, 0], 64, None),           # one candidate, none, empty
    (4, 3, 4, 520, 16, [8320, 8000, 4000], 128, 5),           # heavy ties: 5 distinct values
    (5, 2, 8, 300, 32, [9600, 9000], 1, 3),                   # k = 1 with ties
    (6, 2, 3, 2100, 32, [67200, 50000], 256, None),
    (7, 1, 1, 64, 16, [1024], 4096, None),                    # k far above the candidates
    (8, 2, 2, 5000, 16, [80000, 80000], 4000, 50),            # large k, ties
    (9, 1, 2, 40000, 16, [640000], 128, None),                # keys re-read from memory (> 32768 candidates)
    (10, 2, 2, 20000, 16, [320000, 200000], 300, 7),          # 16-32 keys per thread
]


@pytest.mark.parametrize("seed,R,H,NB,B,lens,k,nd", SELECT_CASES)
def test_select_exact(seed, R, H, NB, B, lens, k, nd):
    scores = random_scores(300 + seed, (R, H, NB), n_distinct=nd)
    if seed % 2:  # signed zeros must compare equal
        scores[..., ::7] = np.float32(-0.0)
        scores[..., 3::7] = np.float32(0.0)
    ctx = np.array(lens, np.int32)
    ref_sel, ref_cnt = O.select_topk(scores, ctx, k, B)
    note(f"select seed={seed} R={R} H={H} NB={NB} k={k}")
    d = P.dims(R, 8 * H, H, 128, B, NB)
    sel = torch.full((R, H, k), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((R, H), -7, dtype=torch.int32, device="cuda")
    P.oasis_select_topk(d, torch.from_numpy(scores).cuda(), dev_i32(ctx), k, sel, cnt)
    torch.cuda.synchronize()
    assert np.array_equal(cnt.cpu().numpy(), ref_cnt)
    assert np.array_equal(sel.cpu().numpy(), ref_sel)


# ---------------------------------------------------------------------------
# a3 staging: plan (slot map, stamps, counts) and bytes, bit-exact
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("copy_local", [True, False])
def test_stage_exact(case, copy_local):
    name, w, hk_t, hv_t = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    k = c.K
    n_cand = np.array([O.block_counts(L, c.block_size)[1] for L in ctx])
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table))
    st = LayerState(d, c.T, k)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    sel, cnt = random_selection_h(500, n_cand, c.num_kv_heads, k)
    ctx_d = dev_i32(ctx)
    for step in range(1, 5):
        if step == 3:
            pass  # same selection again: nothing may move
        elif step > 1:
            sel, cnt = random_selection(500 + step, n_cand, k, prev=(sel, cnt), keep_frac=0.6)
        moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, step, pk, pv, ctx, c.block_size,
                               copy_local=copy_local)
        note(f"stage {name} step={step} copy_local={copy_local}")
        st.sel.copy_(torch.from_numpy(sel))
        st.sel_count.copy_(torch.from_numpy(cnt))
        path.stage(st, ctx_d, step, copy_local=copy_local)
        torch.cuda.synchronize()
        assert np.array_equal(st.slot_map.cpu().numpy(), smap), step
        assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp), step
        assert np.array_equal(st.moved.cpu().numpy(), moved), step
        if step == 3:
            assert moved.sum() == 0
        assert np.array_equal(host_bits(st.pool_k), pk), step
        assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv), step


@pytest.mark.parametrize("cap", [1, 3, 17])
def test_stage_capped_exact(case, cap):
    """Fetch cap (paper §4.2.3, §5.5.1): admitted misses ranked on the same fp32 scores on both sides."""
    name, w, hk_t, hv_t = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    k = c.K
    n_cand = np.array([O.block_counts(L, c.block_size)[1] for L in ctx])
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap)
    st = LayerState(d, c.T, k)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    sel, cnt = random_selection_h(600 + cap, n_cand, c.num_kv_heads, k)
    ctx_d = dev_i32(ctx)
    for step in range(1, 7):
        if step > 1 and step != 4:
            sel, cnt = random_selection(600 + cap + step, n_cand, k, prev=(sel, cnt), keep_frac=0.7)
        # ties on every other step: 9 distinct values
        scores = random_scores(650 + 10 * cap + step, (c.num_reqs, c.num_kv_heads, w.NBmax),
                               n_distinct=9 if step % 2 else None)
        moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, step, pk, pv, ctx, c.block_size,
                               copy_local=True, scores=scores, fetch_cap=cap)
        note(f"stage capped {name} cap={cap} step={step}")
        st.sel.copy_(torch.from_numpy(sel))
        st.sel_count.copy_(torch.from_numpy(cnt))
        st.scores.copy_(torch.from_numpy(scores))
        path.stage(st, ctx_d, step)
        torch.cuda.synchronize()
        assert np.array_equal(st.slot_map.cpu().numpy(), smap), step
        assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp), step
        assert np.array_equal(st.moved.cpu().numpy(), moved), step
        assert moved.max(initial=0) <= cap
        assert np.array_equal(host_bits(st.pool_k), pk), step
        assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv), step


STAGE_PASS_CASES = [
    # (seed, requests, k, fetch cap or None, context range): (request, KV head) pairs per staging
    # workgroup and per plan pass (a pass holds up to 1024 / k pairs, 64 at most)
    (1, 40, 100, None, (200, 2400)),   # 320 pairs: 5 per workgroup, planned in one pass of 500 items
    (2, 40, 300, 7, (1, 5200)),        # 3 pairs per pass: passes of 3 and 2, capped
    (3, 40, 13, 2, (1, 400)),          # k not a multiple of 4, capped
    (4, 64, 128, 6, (1000, 2600)),     # 8 pairs per workgroup: one full pass of 1024 items
    (5, 600, 3, None, (1, 90)),        # 75 pairs per workgroup: passes of 64 and 11
    (6, 5, 1024, 40, (100, 20000)),    # k = 1024: one pair per pass, two passes on some workgroups
]


@pytest.mark.parametrize("seed,R,k,cap,ctx_args", STAGE_PASS_CASES)
def test_stage_many_pairs_exact(seed, R, k, cap, ctx_args):
    """Several (request, KV head) plans per workgroup pass: slot maps, stamps, counts and bytes bit-exact."""
    w = make_workload("c2", num_reqs=R, ctx_args=ctx_args, budget=16 * k)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    d = _dims(w)
    ctx = w.ctx_len(0)
    n_cand = np.array([O.block_counts(L, c.block_size)[1] for L in ctx])
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap if cap else k)
    st = LayerState(d, c.T, k)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    sel, cnt = random_selection_h(700 + seed, n_cand, c.num_kv_heads, k)
    ctx_d = dev_i32(ctx)
    for step in range(1, 4):
        if step > 1:
            sel, cnt = random_selection(700 + seed + step, n_cand, k, prev=(sel, cnt), keep_frac=0.7)
        scores = random_scores(750 + seed + step, (c.num_reqs, c.num_kv_heads, w.NBmax),
                               n_distinct=9 if step == 2 else None)
        moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, step, pk, pv, ctx, c.block_size,
                               copy_local=True, scores=scores, fetch_cap=cap if cap else k)
        note(f"stage many pairs seed={seed} R={R} k={k} cap={cap} step={step}")
        st.sel.copy_(torch.from_numpy(sel))
        st.sel_count.copy_(torch.from_numpy(cnt))
        st.scores.copy_(torch.from_numpy(scores))
        path.stage(st, ctx_d, step)
        torch.cuda.synchronize()
        assert np.array_equal(st.slot_map.cpu().numpy(), smap), step
        assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp), step
        assert np.array_equal(st.moved.cpu().numpy(), moved), step
        if cap:
            assert moved.max(initial=0) <= cap
        assert np.array_equal(host_bits(st.pool_k), pk), step
        assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv), step
    # the local blocks alone (no plan; up to 256 workgroups, several pairs each beyond 256 pairs)
    st.pool_k[:, k].zero_()
    st.pool_v[:, k].zero_()
    pk[:, k] = 0
    pv[:, k] = 0
    note(f"stage many pairs local-only seed={seed} R={R} k={k}")
    path.refresh_local(st, ctx_d)
    torch.cuda.synchronize()
    smap_before = smap.copy()
    O.stage_blocks(hk, hv, w.block_table, np.full_like(smap, -1), np.zeros_like(cnt), smap.copy(), stamp.copy(),
                   0, pk, pv, ctx, c.block_size, copy_local=True)
    assert np.array_equal(host_bits(st.pool_k), pk)
    assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv)
    assert np.array_equal(st.slot_map.cpu().numpy(), smap_before)


def test_stage_local_only(case):
    name, w, hk_t, hv_t = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    k = c.K
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table))
    st = LayerState(d, c.T, k)
    note(f"stage local-only {name}")
    path.refresh_local(st, dev_i32(ctx))
    torch.cuda.synchronize()
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    O.stage_blocks(as_np_bits(hk_t), as_np_bits(hv_t), w.block_table, np.full_like(smap, -1),
                   np.zeros((c.num_reqs, c.num_kv_heads), np.int32), smap, np.zeros_like(smap), 0, pk, pv, ctx,
                   c.block_size, copy_local=True)
    assert np.array_equal(host_bits(st.pool_k), pk)
    assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv)
    assert np.all(st.slot_map.cpu().numpy() == -1)


# ---------------------------------------------------------------------------
# a4 attention on random pools and slot maps
# ---------------------------------------------------------------------------

ATTN_CASES = [
    # (seed, R, Hq, Hkv, T, B, k_slots, ctx lengths, free fraction)
    (1, 2, 32, 8, 5, 16, 128, [131072, 2000], 0.0),
    (2, 3, 32, 8, 5, 16, 7, [100, 17, 16], 0.3),         # odd unit tail, local_len 1 and 16
    (3, 2, 64, 8, 9, 32, 128, [65536, 33], 0.2),         # 72 rows, B = 32
    (4, 2, 8, 8, 1, 16, 40, [5000, 5001], 0.5),          # 1 row per head (T = 1, G = 1)
    (5, 2, 32, 8, 5, 16, 0, [10, 1], 0.0),               # local block only
    (6, 2, 32, 8, 5, 16, 16, [0, 300], 1.0),             # empty context; all slots free
    (7, 1, 40, 8, 4, 16, 300, [8192], 0.1),              # G = 5: 20 rows, many splits
    (8, 2, 16, 2, 5, 32, 33, [1000, 64], 0.25),
    (9, 2, 64, 8, 7, 16, 50, [4000, 777], 0.2),          # 56 rows: four row tiles
    (10, 2, 48, 8, 6, 32, 20, [3000, 100], 0.3),         # G = 6: 36 rows, three row tiles, B = 32
    (11, 2, 40, 8, 8, 16, 60, [4000, 950], 0.2),         # G = 5: 40 rows, three row tiles, B = 16
    (12, 2, 64, 8, 7, 32, 40, [2600, 1000], 0.2),        # 56 rows, four row tiles, B = 32
    (13, 2, 64, 8, 9, 16, 70, [3000, 1111], 0.3),        # 72 rows, five row tiles, B = 16
    # 256 (request, KV head) pairs: one split each, the many-row kernel writes the outputs itself
    (14, 32, 64, 8, 9, 32, 6, [6 * 32 + 5 + 3 * r for r in range(32)], 0.2),
    (15, 2, 64, 8, 9, 16, 0, [10, 1], 0.0),               # many-row kernel, local block only
    (16, 2, 64, 8, 9, 32, 16, [0, 300], 1.0),             # many-row kernel, empty context; all slots free
    (17, 3, 40, 8, 8, 16, 7, [100, 17, 16], 0.3),         # many-row kernel, odd unit tail, local_len 1 and 16
]


@pytest.mark.parametrize("seed,R,Hq,Hkv,T,B,ks,lens,free", ATTN_CASES)
def test_attn(seed, R, Hq, Hkv, T, B, ks, lens, free):
    d_head = 128
    q = random_bf16(700 + seed, (R, T, Hq, d_head))
    pk = random_bf16(710 + seed, (R, ks + 1, Hkv, B, d_head))
    pv = random_bf16(720 + seed, (R, ks + 1, Hkv, B, d_head))
    rng = np.random.default_rng(730 + seed)
    smap = np.where(rng.random((R, Hkv, ks)) < free, -1, rng.integers(0, 10 ** 6, (R, Hkv, ks))).astype(np.int32)
    ctx = np.array(lens, np.int32)
    # garbage (NaN bf16) in free slots and past the local block's end must not leak
    nan = np.uint16(0x7FC0)
    for r in range(R):
        for h in range(Hkv):
            for s in range(ks):
                if smap[r, h, s] < 0:
                    pk[r, s, h] = nan
                    pv[r, s, h] = nan
        _, _, ll = O.block_counts(ctx[r], B)
        pk[r, ks, :, ll:] = nan
        pv[r, ks, :, ll:] = nan
    ref_o, ref_l = O.sparse_attend(q, pk, pv, smap, ctx, B)
    note(f"attn seed={seed} R={R} Hq={Hq} Hkv={Hkv} T={T} B={B} ks={ks}")
    d = P.dims(R, Hq, Hkv, d_head, B, max(1, (int(ctx.max()) + B - 1) // B))
    out = torch.zeros((R, T, Hq, d_head), dtype=torch.bfloat16, device="cuda")
    lse = torch.zeros((R, T, Hq), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.oasis_attn_workspace_bytes(d, T, ks), dtype=torch.uint8, device="cuda")
    P.oasis_sparse_decode_attn(d, dev_bf16(q), T, dev_bf16(pk), dev_bf16(pool_v_from_htd(pv)),
                               dev_i32(smap) if ks else None, ks, dev_i32(ctx), None, out, lse, ws)
    torch.cuda.synchronize()
    assert_attn_close(host_bits(out), ref_o)
    assert_lse_close(lse.cpu().numpy(), ref_l)


# ---------------------------------------------------------------------------
# the whole step (summaries -> scores -> selection -> staging -> attention)
# ---------------------------------------------------------------------------

def test_full_step(case):
    name, w, hk_t, hv_t = case
    c = w.cfg
    d = _dims(w)
    ctx = w.ctx_len(0)
    q = w.queries(0)
    k = c.K
    ref = oracle_layer(w, as_np_bits(hk_t), as_np_bits(hv_t), ctx, q, k)
    note(f"full step {name}")
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table))
    st = LayerState(d, c.T, k)
    ctx_d, q_d = dev_i32(ctx), dev_bf16(q)
    path.build_summaries(st, ctx_d)
    path.step_serial(st, q_d, ctx_d, 0)
    torch.cuda.synchronize()
    assert_scores_close(st.scores.cpu().numpy(), ref["scores"])
    swapped = selection_diff(st.sel.cpu().numpy(), st.sel_count.cpu().numpy(), ref["sel"], ref["cnt"],
                             ref["scores"])
    assert not swapped, f"near-tie swaps in {swapped}"
    if c.key_dist == "planted":
        sel = st.sel.cpu().numpy()
        for r in range(c.num_reqs):
            for h in range(c.num_kv_heads):
                assert set(w.planted_ids(r, h)) <= set(sel[r, h]), (r, h)
    assert np.array_equal(st.slot_map.cpu().numpy(), ref["slot_map"])
    assert np.array_equal(st.moved.cpu().numpy(), ref["moved"])
    assert_attn_close(host_bits(st.out), ref["out"])
    assert_lse_close(st.lse.cpu().numpy(), ref["lse"])


def test_dense_equivalence():
    """Budget above every context: the sparse path reproduces dense attention (paper §5.2 threshold)."""
    w = make_workload("c2", num_reqs=3, ctx_args=(100, 1500), budget=16 * 100)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    d = _dims(w)
    ctx = w.ctx_len(0)
    k = w.NBmax
    note("dense equivalence")
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table))
    st = LayerState(d, c.T, k)
    ctx_d, q_d = dev_i32(ctx), dev_bf16(w.queries(0))
    path.build_summaries(st, ctx_d)
    path.step_serial(st, q_d, ctx_d, 0)
    torch.cuda.synchronize()
    ref_o, ref_l = O.dense_attend(w.queries(0), as_np_bits(hk_t), as_np_bits(hv_t), w.block_table, ctx, c.block_size)
    assert_attn_close(host_bits(st.out), ref_o)
    assert_lse_close(st.lse.cpu().numpy(), ref_l)


@pytest.mark.parametrize("issue", ["native", "native_plan_pred", "native_plan_alternating", "python"])
@pytest.mark.parametrize("cap", [None, 2])
def test_pipelined_multistep(cap, issue):
    """Reasoning-style loop: AR(1) queries, one token per step, attention on the previous step's staging.

    With a fetch cap, later steps attend stale residents in place of the misses
    that were not admitted (paper §5.5.1), on both sides alike. ``native_plan_pred``
    plans each transfer in the top-K kernel on the prediction stream;
    ``native_plan_alternating`` switches between the two streams every step (the
    first switch comes after the layer is registered).
    """
    steps = 6
    w = make_workload("c3", num_reqs=3, ctx_args=(200, 300, 1400), steps=steps, budget=16 * 24)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    d = _dims(w)
    k = c.K
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap, native=issue != "python",
                      plan_on_prediction=issue == "native_plan_pred")
    st = LayerState(d, c.T, k)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    none_sel = np.full_like(smap, -1)
    zero_cnt = np.zeros((c.num_reqs, c.num_kv_heads), np.int32)
    for s in range(steps):
        ctx = w.ctx_len(s)
        q = w.queries(s)
        # oracle, same schedule: local block, attention, then prediction and staging for the next step
        O.stage_blocks(hk, hv, w.block_table, none_sel, zero_cnt, smap, stamp, s, pk, pv, ctx, c.block_size)
        ref_o, ref_l = O.sparse_attend(q, pk, pv, smap, ctx, c.block_size)
        kmax, kmin = O.block_summaries(hk, w.block_table, ctx, c.block_size, w.NBmax)
        sc = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
        sel, cnt = O.select_topk(sc, ctx, k, c.block_size)
        moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, s, pk, pv, ctx, c.block_size,
                               copy_local=False, scores=sc, fetch_cap=cap)
        note(f"pipelined step {s} cap={cap} issue={issue}")
        ctx_d, q_d = dev_i32(ctx), dev_bf16(q)
        path.build_summaries(st, ctx_d)   # summaries of blocks completed so far
        if issue == "native_plan_alternating":
            path.set_plan_on_prediction(s % 2 == 1)
        path.step_pipelined(st, q_d, ctx_d, s, growing=True)
        path.join()
        torch.cuda.synchronize()
        assert_attn_close(host_bits(st.out), ref_o, f"step {s} out")
        assert_lse_close(st.lse.cpu().numpy(), ref_l)
        assert not selection_diff(st.sel.cpu().numpy(), st.sel_count.cpu().numpy(), sel, cnt, sc)
        assert np.array_equal(st.slot_map.cpu().numpy(), smap), s
        assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp), s
        assert np.array_equal(st.moved.cpu().numpy(), moved), s
        if s > 0:
            assert moved.sum() < cnt.sum(), "AR(1) drift: later steps are deltas"
        if cap is not None:
            assert moved.max() <= cap


@pytest.mark.parametrize("order", ["beside", "after"])
@pytest.mark.parametrize("plan_pred", [False, True])
@pytest.mark.parametrize("fused", [False, True])
def test_pipelined_layers_native(plan_pred, fused, order):
    """Several layers interleaved on the native issuer with no host synchronization
    between steps (paper §4.2.2: per-layer chains, layer-local waits); every
    layer's final state equals its own oracle chain, with the transfer planned on
    either stream, the prediction by the separate kernels or by the fused
    score + select (+ plan) kernel, and started beside or after the attention."""
    n_layers, rounds, cap = 3, 4, 3
    w = make_workload("c2", num_reqs=3, ctx_args=(900, 2500), budget=16 * 20, ar_queries=True)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    d = _dims(w)
    k = c.K
    ctx = w.ctx_len(0)
    ctx_d = dev_i32(ctx)
    qs = [w.layer_queries(l, rounds + 1) for l in range(n_layers)]
    kmax, kmin = O.block_summaries(hk, w.block_table, ctx, c.block_size, w.NBmax)
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap, plan_on_prediction=plan_pred,
                      fused_prediction=P.FUSED_PREDICTION_ON if fused else P.FUSED_PREDICTION_OFF,
                      prediction_order=P.PREDICT_BESIDE_ATTENTION if order == "beside" else P.PREDICT_AFTER_ATTENTION)
    layers = [LayerState(d, c.T, k) for _ in range(n_layers)]
    ref = []
    for l, st in enumerate(layers):
        # initial working set: one uncapped fill from the layer's first prediction
        path.build_summaries(st, ctx_d)
        path.predict(st, dev_bf16(qs[l][0]), ctx_d)
        path.stage(st, ctx_d, 0, fetch_cap=k)
        smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
        stamp = np.zeros_like(smap)
        pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
        pv = np.zeros_like(pk)
        sc = O.block_scores(qs[l][0], kmax, kmin, ctx, c.num_kv_heads, c.block_size)
        sel, cnt = O.select_topk(sc, ctx, k, c.block_size)
        O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
        ref.append(dict(smap=smap, stamp=stamp, pk=pk, pv=pv))
    q_dev = [[dev_bf16(x) for x in qs[l]] for l in range(n_layers)]
    note(f"native pipelined layers: issuing (plan on prediction: {plan_pred}, fused prediction: {fused}, "
         f"prediction {order} the attention)")
    for s in range(1, rounds + 1):
        for l in range(n_layers):
            path.step_pipelined(layers[l], q_dev[l][s], ctx_d, s)
    path.join()
    torch.cuda.synchronize()
    for l in range(n_layers):
        r = ref[l]
        for s in range(1, rounds + 1):
            q = qs[l][s]
            ref_o, ref_l = O.sparse_attend(q, r["pk"], r["pv"], r["smap"], ctx, c.block_size)
            sc = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
            sel, cnt = O.select_topk(sc, ctx, k, c.block_size)
            O.stage_blocks(hk, hv, w.block_table, sel, cnt, r["smap"], r["stamp"], s, r["pk"], r["pv"], ctx,
                           c.block_size, scores=sc, fetch_cap=cap)
        st = layers[l]
        assert_attn_close(host_bits(st.out), ref_o, f"layer {l} out")
        assert_lse_close(st.lse.cpu().numpy(), ref_l)
        assert np.array_equal(st.slot_map.cpu().numpy(), r["smap"]), l
        assert np.array_equal(st.slot_stamp.cpu().numpy(), r["stamp"]), l
        assert np.array_equal(host_bits(st.pool_k), r["pk"]), l
        assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), r["pv"]), l
    path.close()


def _independent_stream_pair(tries: int = 8):
    """Two streams on different hardware queues: a bounded sleep kernel on the first must not hold
    up a small kernel on the second. HIP maps a process's streams onto a few hardware queues, so two
    pool streams may share one (then the second waits behind the first)."""
    cands = [torch.cuda.Stream() for _ in range(tries)]
    x = torch.zeros(1, device="cuda")
    for i in range(tries):
        for j in range(tries):
            if i == j:
                continue
            torch.cuda.synchronize()
            with torch.cuda.stream(cands[i]):
                torch.cuda._sleep(100_000_000)  # tens of ms
            t0 = time.perf_counter()
            with torch.cuda.stream(cands[j]):
                x.add_(1)
            cands[j].synchronize()
            quick = time.perf_counter() - t0 < 0.005
            cands[i].synchronize()
            if quick:
                return cands[i], cands[j]
    return None


def test_pipeline_wait_fault_reported():
    """Failure path of the transfer's in-kernel wait for its prediction: with the bound set to 64
    polls and a stalled prediction stream (a bounded torch sleep kernel queued ahead of it), the
    staging kernel gives up, every kernel still ends, and oasis_pipeline_check reports the fault;
    a normal step before it reports none. The prediction and transfer streams are chosen on
    different hardware queues, so that the transfer's kernel runs while the prediction sleeps."""
    pair = _independent_stream_pair()
    assert pair is not None, "no two of 8 streams run independently"
    w = make_workload("c2", num_reqs=2, ctx_args=(900, 1500), budget=16 * 8, ar_queries=True)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    d = _dims(w)
    k = c.K
    ctx_d = dev_i32(w.ctx_len(0))
    qs = [dev_bf16(x) for x in w.layer_queries(0, 3)]
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=3, streams=pair)
    st = LayerState(d, c.T, k)
    path.build_summaries(st, ctx_d)
    path.predict(st, qs[0], ctx_d)
    path.stage(st, ctx_d, 0, fetch_cap=k)
    note("wait fault: normal pipelined step")
    path.step_pipelined(st, qs[1], ctx_d, 1)
    path.join()
    path.check()
    P.oasis_pipeline_set_wait_limit(path._pipe, 64)
    note("wait fault: stalled prediction stream, wait bound 64 polls")
    with torch.cuda.stream(path.side):
        torch.cuda._sleep(200_000_000)  # a bounded spin ahead of the prediction's kernels
    path.step_pipelined(st, qs[2], ctx_d, 2)
    path.join()
    with pytest.raises(P.OasisError, match="gave up waiting"):
        path.check()
    with pytest.raises(P.OasisError, match="gave up waiting"):
        path.close()  # reports it again and still releases the issuer
    assert path._pipe is None


@pytest.mark.parametrize("plan_pred", [False, True])
def test_pipelined_large_k_b32(plan_pred):
    """The pipelined step at block size 32 with k = 1,024 (one (request, KV head) pair per plan pass,
    72 query rows per KV head) and a binding fetch cap, the transfer planned on either stream;
    slot maps, stamps, pools and the last attention equal the oracle chain."""
    rounds, cap = 3, 48
    w = make_workload("c5", num_reqs=2, ctx_args=(40000,), budget=32 * 1024, ar_queries=True)
    c = w.cfg
    k = c.K
    hk_t, hv_t = pinned_pages(w)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    d = _dims(w)
    ctx = w.ctx_len(0)
    ctx_d = dev_i32(ctx)
    qs = w.layer_queries(0, rounds + 1)
    kmax, kmin = O.block_summaries(hk, w.block_table, ctx, c.block_size, w.NBmax)
    path = DecodePath(d, c.T, k, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap, plan_on_prediction=plan_pred)
    st = LayerState(d, c.T, k)
    path.build_summaries(st, ctx_d)
    path.predict(st, dev_bf16(qs[0]), ctx_d)
    path.stage(st, ctx_d, 0, fetch_cap=k)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    sc = O.block_scores(qs[0], kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel, cnt = O.select_topk(sc, ctx, k, c.block_size)
    O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
    q_dev = [dev_bf16(x) for x in qs]
    note(f"pipelined k=1024 B=32 (plan on prediction: {plan_pred}): issuing")
    for s in range(1, rounds + 1):
        path.step_pipelined(st, q_dev[s], ctx_d, s)
    path.join()
    torch.cuda.synchronize()
    moved_total = 0
    for s in range(1, rounds + 1):
        q = qs[s]
        if s == rounds:
            ref_o, ref_l = O.sparse_attend(q, pk, pv, smap, ctx, c.block_size)
        sc = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
        sel, cnt = O.select_topk(sc, ctx, k, c.block_size)
        moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, s, pk, pv, ctx, c.block_size,
                               copy_local=False, scores=sc, fetch_cap=cap)
        assert moved.max() <= cap
        moved_total += int(moved.sum())
    assert moved_total > 0
    assert_attn_close(host_bits(st.out), ref_o, "k=1024 out")
    assert_lse_close(st.lse.cpu().numpy(), ref_l)
    assert not selection_diff(st.sel.cpu().numpy(), st.sel_count.cpu().numpy(), sel, cnt, sc)
    assert np.array_equal(st.moved.cpu().numpy(), moved)
    assert np.array_equal(st.slot_map.cpu().numpy(), smap)
    assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp)
    assert np.array_equal(host_bits(st.pool_k), pk)
    assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv)
    path.close()


def test_pipeline_profile():
    """The native issuer's kernel timing records one span per kernel kind per step."""
    w = make_workload("c2", num_reqs=2, ctx_args=(3000, 5000), budget=16 * 32, ar_queries=True)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    d = _dims(w)
    ctx_d = dev_i32(w.ctx_len(0))
    qs = [dev_bf16(x) for x in w.layer_queries(0, 5)]
    path = DecodePath(d, c.T, c.K, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=4)
    st = LayerState(d, c.T, c.K)
    path.build_summaries(st, ctx_d)
    note("pipeline profile")
    path.step_pipelined(st, qs[0], ctx_d, 0)
    path.profile_begin(3)
    for s in range(1, 5):                      # one step more than profiled
        path.step_pipelined(st, qs[s], ctx_d, s)
    path.join()
    torch.cuda.synchronize()
    us, n, per_step = path.profile_end(per_step=True)
    assert n == 3 and per_step.shape == (3, 4)
    assert all(0.0 < us[k_] < 1e5 for k_ in ("attn", "score", "topk", "stage")), us
    np.testing.assert_allclose(per_step.mean(axis=0), [us[k_] for k_ in P._lib.PROFILE_KINDS], rtol=1e-4)
    with pytest.raises(P.OasisError):
        path.profile_end()
    path.close()


def test_pipeline_abi_errors_on_device():
    w = make_workload("c2", num_reqs=1, ctx_args=(500, 500), budget=16 * 8)
    c = w.cfg
    hk_t, hv_t = pinned_pages(w)
    d = _dims(w)
    bt = dev_i32(w.block_table)
    with pytest.raises(P.OasisError) as e:      # fetch cap below 1
        P.oasis_pipeline_create(d, c.T, 1, c.num_draft, c.K, 0, None, hk_t, hv_t, bt, 4)
    assert e.value.status == 1
    with pytest.raises(ValueError):             # host tier neither pinned nor on the device
        P.oasis_pipeline_create(d, c.T, 1, c.num_draft, c.K, c.K, None, hk_t.clone(), hv_t.clone(), bt, 4)
    h = P.oasis_pipeline_create(d, c.T, 1, c.num_draft, c.K, c.K, None, hk_t, hv_t, bt, 4)
    try:
        q = torch.zeros((1, c.T, c.num_q_heads, c.head_dim), dtype=torch.bfloat16, device="cuda")
        ctx = dev_i32(w.ctx_len(0))
        with pytest.raises(P.OasisError) as e:  # layer never registered
            P.oasis_pipeline_step(h, 0, q, ctx, 0, False)
        assert e.value.status == 1 and "set_layer" in str(e.value)
        st = LayerState(d, c.T, c.K)
        small_ws = torch.zeros(4, dtype=torch.uint8, device="cuda")
        P.oasis_pipeline_set_layer(h, 0, d, c.T, c.K, st.kmax, st.kmin, st.scores, st.sel, st.sel_count,
                                   st.slot_map, st.slot_stamp, st.pool_k, st.pool_v, st.moved, st.out, st.lse,
                                   small_ws)
        with pytest.raises(P.OasisError) as e:  # workspace too small, caught by the per-step checks
            P.oasis_pipeline_step(h, 0, q, ctx, 0, False)
        assert e.value.status == 4
        with pytest.raises(P.OasisError) as e:  # a summary update with no room for a new block
            P.oasis_pipeline_step(h, 0, q, ctx, 0, True, prev_ctx_len=ctx, max_new_blocks=0)
        assert e.value.status == 1 and "max_new_blocks" in str(e.value)
        # a local-block source needs all three of k_pages, v_pages and block_table
        assert P._lib.lib().oasis_pipeline_set_local_source(h, hk_t.data_ptr(), None, 1, None) == 1
        with pytest.raises(P.OasisError) as e:  # neither plan stream
            P.oasis_pipeline_set_plan_stream(h, 2)
        assert e.value.status == 1 and "where" in str(e.value)
        with pytest.raises(P.OasisError) as e:
            P.oasis_pipeline_set_layer(h, 4, d, c.T, c.K, st.kmax, st.kmin, st.scores, st.sel, st.sel_count,
                                       st.slot_map, st.slot_stamp, st.pool_k, st.pool_v, st.moved, st.out,
                                       st.lse, st.ws_attn)
        assert e.value.status == 1
    finally:
        torch.cuda.synchronize()
        P.oasis_pipeline_destroy(h)


# ---------------------------------------------------------------------------
# host-side errors through the C ABI with a GPU present
# ---------------------------------------------------------------------------

def test_abi_errors_on_device():
    d = P.dims(1, 32, 8, 128, 16, 16)
    T, k = 5, 128                       # 8 pairs over 16 splits: partials need a workspace
    q = torch.zeros((1, T, 32, 128), dtype=torch.bfloat16, device="cuda")
    pool = torch.zeros((1, k + 1, 8, 16, 128), dtype=torch.bfloat16, device="cuda")
    smap = torch.full((1, 8, k), -1, dtype=torch.int32, device="cuda")
    ctx = torch.ones(1, dtype=torch.int32, device="cuda")
    out = torch.zeros((1, T, 32, 128), dtype=torch.bfloat16, device="cuda")
    small = torch.empty(8, dtype=torch.uint8, device="cuda")
    assert P.oasis_attn_workspace_bytes(d, T, k) > 8
    with pytest.raises(P.OasisError) as e:
        P.oasis_sparse_decode_attn(d, q, T, pool, pool, smap, k, ctx, None, out, None, small)
    assert e.value.status == 4
    # a single split per pair needs no workspace: an empty one is accepted
    k1 = 4
    assert P.oasis_attn_workspace_bytes(d, T, k1) == 0
    P.oasis_sparse_decode_attn(d, q, T, pool[:, :k1 + 1].contiguous(), pool[:, :k1 + 1].contiguous(),
                               smap[:, :, :k1].contiguous(), k1, ctx, None, out, None,
                               torch.empty(0, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    host = torch.zeros((4, 8, 16, 128), dtype=torch.bfloat16)  # not pinned
    with pytest.raises(ValueError):
        P.oasis_build_summaries(d, host, torch.zeros((1, 16), dtype=torch.int32, device="cuda"), ctx,
                                pool, pool)
    with pytest.raises(P.OasisError) as e:
        P.oasis_stage_blocks(d, host.pin_memory(), host.pin_memory(), torch.zeros((1, 16), dtype=torch.int32,
                             device="cuda"), ctx, smap, torch.zeros((1, 8), dtype=torch.int32, device="cuda"), None,
                             k, smap, smap.clone(), 0, k - 1, True, pool, pool, None)
    assert e.value.status == 1 and "scores" in str(e.value)  # a binding cap ranks misses by score


# ---------------------------------------------------------------------------
# per-layer union of the per-head sets (paper §4.4.1)
# ---------------------------------------------------------------------------

UNION_CASES = [
    # (seed, R, H, NB, k)
    (1, 4, 8, 8192, 128),
    (2, 3, 8, 700, 1024),      # k above the candidates of some rows
    (3, 2, 1, 33, 5),          # one head, a ragged bitmap word
    (4, 5, 16, 100000, 64),    # many words per thread
]


@pytest.mark.parametrize("seed,R,H,NB,k", UNION_CASES)
def test_union_selection_exact(seed, R, H, NB, k):
    rng = np.random.default_rng(900 + seed)
    n_cand = rng.integers(0, NB, size=R)
    n_cand[0] = 0                                     # an empty request
    sel, cnt = random_selection_h(910 + seed, n_cand, H, k)
    if H > 1:
        sel[-1, 1] = sel[-1, 0]                       # two heads with the same set
        cnt[-1, 1] = cnt[-1, 0]
    ref_ids, ref_cnt = O.union_selection(sel, cnt)
    note(f"union seed={seed} R={R} H={H} NB={NB} k={k}")
    d = P.dims(R, 8 * H, H, 128, 16, NB)
    ids = torch.full((R, H * k), 77, dtype=torch.int32, device="cuda")
    n = torch.full((R,), -5, dtype=torch.int32, device="cuda")
    P.oasis_union_selection(d, dev_i32(sel), dev_i32(cnt), k, ids, n)
    torch.cuda.synchronize()
    assert np.array_equal(n.cpu().numpy(), ref_cnt)
    assert np.array_equal(ids.cpu().numpy(), ref_ids)
