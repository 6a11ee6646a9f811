"""Pins of the CPU oracle against what the paper and the mathematics fix (CPU only).

Each check is independent of the oracle's own formulas: brute force over the
bounding box of a block, exhaustive subset search, textbook attention from
torch in float64, the paper's stated counts (129 blocks / 2,064 tokens), and
invariants (idempotent delta staging, softmax normalisation, planted
heavy hitters selected).
"""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import oasis_oracle as O
from workloads import Config, Workload, f32_to_bf16_bits, make_workload, random_scores, random_selection_h


def tiny_cfg(**kw):
    base = dict(name="tiny", index=90, num_reqs=3, num_q_heads=4, num_kv_heads=2, head_dim=6,
                block_size=4, num_draft=2, budget=12, ctx_kind="uniform", ctx_args=(1, 45),
                key_dist="planted", n_planted=2)
    base.update(kw)
    return Config(**base)


def _summaries(w: Workload, step=0):
    hk, hv = w.fill_paged(threads=1)
    ctx = w.ctx_len(step)
    kmax, kmin = O.block_summaries(hk, w.block_table, ctx, w.cfg.block_size, w.NBmax)
    return hk, hv, ctx, kmax, kmin


# ---------------------------------------------------------------------------
# block counts (local block reading)
# ---------------------------------------------------------------------------

def test_block_counts():
    assert O.block_counts(8192, 16) == (512, 511, 16)      # c1: 511 candidates + local
    assert O.block_counts(131072, 16) == (8192, 8191, 16)  # c4
    assert O.block_counts(65536, 32) == (2048, 2047, 32)   # c5
    assert O.block_counts(17, 16) == (2, 1, 1)
    assert O.block_counts(1, 16) == (1, 0, 1)
    assert O.block_counts(0, 16) == (0, 0, 0)


# ---------------------------------------------------------------------------
# O0 summaries: brute force from the unpaged per-request keys
# ---------------------------------------------------------------------------

def test_summaries_bruteforce_through_pages():
    w = Workload(tiny_cfg())
    _, _, ctx, kmax, kmin = _summaries(w)
    c = w.cfg
    for r in range(c.num_reqs):
        k_r, _ = w.request_kv(r)                          # [Hkv][L][d], not paged
        kf = O.bf16_to_f64(k_r)
        _, n_cand, _ = O.block_counts(ctx[r], c.block_size)
        for h in range(c.num_kv_heads):
            for b in range(n_cand):
                for j in range(c.head_dim):
                    col = [kf[h, b * c.block_size + p, j] for p in range(c.block_size)]
                    assert kmax[r, h, b, j] == max(col)
                    assert kmin[r, h, b, j] == min(col)
            assert np.all(np.isnan(kmax[r, h, n_cand:]))


def test_summaries_identical_keys():
    B, d = 4, 5
    key = np.array([1.5, -2.0, 0.0, 3.25, -0.125], np.float32)
    host_k = np.tile(f32_to_bf16_bits(key), (3, 1, B, 1)).reshape(3, 1, B, d)
    kmax, kmin = O.block_summaries(host_k, np.array([[2, 0, 1]]), np.array([12]), B, 3)
    assert np.array_equal(kmax[0, 0, :2], np.tile(key.astype(np.float64), (2, 1)))
    assert np.array_equal(kmin[0, 0, :2], np.tile(key.astype(np.float64), (2, 1)))


# ---------------------------------------------------------------------------
# O1 scores
# ---------------------------------------------------------------------------

def _box_max(q, lo, hi):
    """max over the 2^d corners of the box [lo, hi] of q . x (brute force)."""
    best = -np.inf
    for corner in itertools.product(*[(lo[j], hi[j]) for j in range(len(q))]):
        best = max(best, float(np.dot(q, np.array(corner))))
    return best


def test_score_is_max_over_bounding_box():
    """The block score of one row is the largest q . x over the box spanned by the block's keys."""
    w = Workload(tiny_cfg(num_draft=1, num_q_heads=2, num_kv_heads=2))   # G = D = 1: one row per head
    hk, _, ctx, kmax, kmin = _summaries(w)
    q = w.queries(0)
    s = O.block_scores(q, kmax, kmin, ctx, w.cfg.num_kv_heads, w.cfg.block_size)
    qf = O.bf16_to_f64(q)
    for r in range(w.cfg.num_reqs):
        _, n_cand, _ = O.block_counts(ctx[r], w.cfg.block_size)
        for h in range(2):
            for b in range(n_cand):
                want = _box_max(qf[r, 1, h], kmin[r, h, b], kmax[r, h, b])
                assert math.isclose(s[r, h, b], want, rel_tol=1e-12, abs_tol=1e-12)
            assert np.all(s[r, h, n_cand:] == -np.inf)


def test_score_upper_bounds_every_key_and_every_row():
    w = Workload(tiny_cfg())
    c = w.cfg
    hk, _, ctx, kmax, kmin = _summaries(w)
    q = w.queries(0)
    s = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    qf = O.bf16_to_f64(q)
    for r in range(c.num_reqs):
        kf = O.bf16_to_f64(w.request_kv(r)[0])
        _, n_cand, _ = O.block_counts(ctx[r], c.block_size)
        for h in range(c.num_kv_heads):
            for b in range(n_cand):
                keys = kf[h, b * c.block_size:(b + 1) * c.block_size]
                best_dot = -np.inf
                for t in range(1, c.T):
                    for g in range(c.G):
                        dots = keys @ qf[r, t, h * c.G + g]
                        assert np.all(dots <= s[r, h, b] + 1e-9)
                        best_dot = max(best_dot, dots.max())
                # the bound is attained when the block is reduced to one key; here it is at least the best dot
                assert s[r, h, b] >= best_dot - 1e-9


def test_score_degenerate_block_is_dot_product():
    """All keys of a block equal -> the score is max over draft rows of the plain dot product."""
    B, d, G, D = 4, 8, 2, 3
    rng = np.random.default_rng(3)
    key = f32_to_bf16_bits(rng.standard_normal(d).astype(np.float32))
    host_k = np.tile(key, (2, 1, B, 1)).reshape(2, 1, B, d)
    q = f32_to_bf16_bits(rng.standard_normal((1, 1 + D, G, d)).astype(np.float32))
    ctx = np.array([8])
    kmax, kmin = O.block_summaries(host_k, np.array([[0, 1]]), ctx, B, 2)
    s = O.block_scores(q, kmax, kmin, ctx, 1, B)
    kf, qf = O.bf16_to_f64(key), O.bf16_to_f64(q)
    want = max(float(np.dot(qf[0, t, g], kf)) for t in range(1, 1 + D) for g in range(G))
    assert math.isclose(s[0, 0, 0], want, rel_tol=1e-13)


def test_score_rows_verify_excluded_and_gqa_grouping():
    w = Workload(tiny_cfg())
    c = w.cfg
    _, _, ctx, kmax, kmin = _summaries(w)
    q = w.queries(0).copy()
    s0 = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    # the verify row (t = 0) does not score
    q1 = q.copy()
    q1[:, 0] = f32_to_bf16_bits(np.full(q1[:, 0].shape, 7.0, np.float32))
    assert np.array_equal(O.block_scores(q1, kmax, kmin, ctx, c.num_kv_heads, c.block_size), s0)
    # a draft row of query head qh changes only KV head qh // G
    for qh in range(c.num_q_heads):
        q2 = q.copy()
        q2[:, 1, qh] = f32_to_bf16_bits(np.full(q2[:, 1, qh].shape, 5.0, np.float32))
        s2 = O.block_scores(q2, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
        for h in range(c.num_kv_heads):
            same = np.array_equal(s2[:, h], s0[:, h])
            assert same == (h != qh // c.G)


def test_score_aggregates_by_max_over_rows():
    """The head score equals the max of single-row scores and is invariant to row order."""
    w = Workload(tiny_cfg(num_reqs=1, ctx_kind="fixed", ctx_args=(40,)))
    c = w.cfg
    _, _, ctx, kmax, kmin = _summaries(w)
    q = w.queries(0)
    s = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    singles = []
    for t in range(1, c.T):
        for g in range(c.G):
            qs = np.zeros((1, 2, c.num_kv_heads, c.head_dim), np.uint16)
            for h in range(c.num_kv_heads):
                qs[0, 1, h] = q[0, t, h * c.G + g]
            singles.append(O.block_scores(qs, kmax, kmin, ctx, c.num_kv_heads, c.block_size))
    assert np.array_equal(s, np.max(np.stack(singles), axis=0))
    qp = q.copy()
    qp[:, 1:] = q[:, 1:][:, ::-1]
    assert np.array_equal(O.block_scores(qp, kmax, kmin, ctx, c.num_kv_heads, c.block_size), s)


# ---------------------------------------------------------------------------
# O2 selection: exhaustive subset search
# ---------------------------------------------------------------------------

def _valid_subset(S, scores):
    n = len(scores)
    for i in S:
        for j in range(n):
            if j in S:
                continue
            if not (scores[i] > scores[j] or (scores[i] == scores[j] and i < j)):
                return False
    return True


@pytest.mark.parametrize("seed", range(12))
def test_select_matches_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    B = 16
    n_cand = int(rng.integers(1, 10))
    scores = random_scores(1000 + seed, (1, 1, n_cand + 3), n_distinct=int(rng.integers(1, 5)))
    ctx = np.array([(n_cand + 1) * B - int(rng.integers(0, B))], np.int32)
    for k in range(1, 11):
        sel, cnt = O.select_topk(scores, ctx, k, B)
        m = min(k, n_cand)
        cand = [float(x) for x in scores[0, 0, :n_cand]]
        valid = [set(S) for S in itertools.combinations(range(n_cand), m) if _valid_subset(set(S), cand)]
        assert len(valid) == 1
        assert cnt[0, 0] == m
        assert list(sel[0, 0, :m]) == sorted(valid[0])
        assert np.all(sel[0, 0, m:] == -1)


def test_select_all_when_candidates_fit_budget():
    B = 16
    scores = random_scores(5, (2, 3, 50))
    ctx = np.array([16 * 20 + 3, 16 * 9], np.int32)   # 20 and 8 candidates
    sel, cnt = O.select_topk(scores, ctx, 20, B)
    assert list(cnt[0]) == [20] * 3 and list(cnt[1]) == [8] * 3
    assert np.array_equal(sel[0, 0], np.arange(20))
    assert np.array_equal(sel[1, 2, :8], np.arange(8)) and np.all(sel[1, 2, 8:] == -1)


# ---------------------------------------------------------------------------
# O3 staging
# ---------------------------------------------------------------------------

def _empty_state(R, Hkv, K, B, d):
    return (np.full((R, Hkv, K), -1, np.int32), np.zeros((R, Hkv, K), np.int32),
            np.zeros((R, K + 1, Hkv, B, d), np.uint16), np.zeros((R, K + 1, Hkv, B, d), np.uint16))


def _check_pool_matches_host(w, hk, hv, smap, pool_k, pool_v, ctx):
    c = w.cfg
    for r in range(c.num_reqs):
        nb, _, _ = O.block_counts(ctx[r], c.block_size)
        for h in range(c.num_kv_heads):
            for s in range(smap.shape[2]):
                b = smap[r, h, s]
                if b >= 0:
                    page = w.block_table[r, b]
                    assert np.array_equal(pool_k[r, s, h], hk[page, h])
                    assert np.array_equal(pool_v[r, s, h], hv[page, h])
            if nb:
                page = w.block_table[r, nb - 1]
                assert np.array_equal(pool_k[r, -1, h], hk[page, h])


def test_stage_cold_idempotent_and_lru():
    w = Workload(tiny_cfg(num_reqs=3, ctx_args=(30, 90)))
    c = w.cfg
    hk, hv, ctx, kmax, kmin = _summaries(w)
    K = c.K
    smap, stamp, pk, pv = _empty_state(c.num_reqs, c.num_kv_heads, K, c.block_size, c.head_dim)
    s = O.block_scores(w.queries(0), kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel, cnt = O.select_topk(s, ctx, K, c.block_size)
    moved = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 1, pk, pv, ctx, c.block_size)
    assert np.array_equal(moved, cnt)                                      # cold: every selected block moves
    for r in range(c.num_reqs):
        for h in range(c.num_kv_heads):
            assert set(sel[r, h, :cnt[r, h]]) <= set(smap[r, h])
    _check_pool_matches_host(w, hk, hv, smap, pk, pv, ctx)
    # the same selection again moves nothing and changes nothing but stamps
    snap = (smap.copy(), pk.copy(), pv.copy())
    moved2 = O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 2, pk, pv, ctx, c.block_size)
    assert moved2.sum() == 0
    assert np.array_equal(smap, snap[0]) and np.array_equal(pk, snap[1]) and np.array_equal(pv, snap[2])
    # a different selection evicts least-recently-selected slots first
    rng = np.random.default_rng(11)
    for r in range(c.num_reqs):
        for h in range(c.num_kv_heads):
            stamp[r, h] = rng.permutation(K).astype(np.int32)              # distinct stamps
    before_map, before_stamp = smap.copy(), stamp.copy()
    s2 = O.block_scores(w.queries(0)[:, ::-1].copy(), kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel2, cnt2 = O.select_topk(s2, ctx, K, c.block_size)
    moved3 = O.stage_blocks(hk, hv, w.block_table, sel2, cnt2, smap, stamp, 100, pk, pv, ctx, c.block_size)
    for r in range(c.num_reqs):
        for h in range(c.num_kv_heads):
            chosen = set(sel2[r, h, :cnt2[r, h]])
            assert chosen <= set(smap[r, h])
            evicted = [s for s in range(K) if before_map[r, h, s] != smap[r, h, s]]
            assert len(evicted) == moved3[r, h]
            free_before = [s for s in range(K) if before_map[r, h, s] < 0]
            stale_kept = [s for s in range(K) if before_map[r, h, s] >= 0 and before_map[r, h, s] not in chosen
                          and s not in evicted]
            for e in evicted:
                if before_map[r, h, e] >= 0:
                    # a stale slot is evicted only once every free slot has been filled
                    assert all(smap[r, h, f] >= 0 for f in free_before)
                    for k_ in stale_kept:
                        assert before_stamp[r, h, e] < before_stamp[r, h, k_]
            for s_ in range(K):
                if smap[r, h, s_] in chosen:
                    assert stamp[r, h, s_] == 100
    _check_pool_matches_host(w, hk, hv, smap, pk, pv, ctx)


def _random_stage_state(rng, R, H, K, nc):
    """Slot maps with distinct resident blocks per head, some free slots, random stamps."""
    smap = np.full((R, H, K), -1, np.int32)
    for r in range(R):
        for h in range(H):
            n_res = int(rng.integers(0, K + 1))
            slots = rng.choice(K, size=n_res, replace=False)
            smap[r, h, slots] = rng.choice(nc, size=n_res, replace=False)
    stamp = rng.integers(0, 6, size=(R, H, K)).astype(np.int32)     # many equal stamps
    return smap, stamp


@pytest.mark.parametrize("cap", [1, 2, 3, 7])
def test_stage_capped_properties(cap):
    """Paper §4.2.3 / §5.5.1: at most C pairs per head per step, the rest unchanged.

    Checked against the statement itself, head by head: the admitted misses are
    exactly the top-C misses by (score, -id) (brute force over all misses), the
    slots that change are exactly the first victims in LRU order, every other
    slot keeps its block and stamp, and a cap that does not bind reproduces the
    uncapped plan bit for bit.
    """
    rng = np.random.default_rng(100 + cap)
    R, H, K, B, d, nc = 3, 4, 8, 2, 4, 24
    hk = rng.integers(0, 2 ** 16, size=(nc + 1, H, B, d), dtype=np.uint16)
    hv = rng.integers(0, 2 ** 16, size=(nc + 1, H, B, d), dtype=np.uint16)
    bt = np.stack([rng.permutation(nc + 1) for _ in range(R)]).astype(np.int32)
    ctx = np.full(R, (nc + 1) * B, np.int32)
    scores = random_scores(31 + cap, (R, H, nc + 1), n_distinct=6)     # many exact ties
    for trial in range(4):
        smap, stamp = _random_stage_state(rng, R, H, K, nc)
        sel, cnt = random_selection_h(1000 * cap + trial, np.full(R, nc), H, K)
        pk = np.zeros((R, K + 1, H, B, d), np.uint16)
        pv = np.zeros_like(pk)
        m0, s0 = smap.copy(), stamp.copy()
        um, us = smap.copy(), stamp.copy()
        upk, upv = pk.copy(), pv.copy()
        O.stage_blocks(hk, hv, bt, sel, cnt, um, us, 9, upk, upv, ctx, B, copy_local=False)
        moved = O.stage_blocks(hk, hv, bt, sel, cnt, smap, stamp, 9, pk, pv, ctx, B, copy_local=False,
                               scores=scores, fetch_cap=cap)
        for r in range(R):
            for h in range(H):
                chosen = [int(b) for b in sel[r, h, :cnt[r, h]]]
                resident = {int(b) for b in m0[r, h] if b >= 0}
                misses = [b for b in chosen if b not in resident]
                n_adm = min(cap, len(misses))
                assert moved[r, h] == n_adm
                admitted = {int(smap[r, h, s]) for s in range(K) if smap[r, h, s] != m0[r, h, s]}
                assert len(admitted) == n_adm and admitted <= set(misses)
                key = lambda b: (float(scores[r, h, b]), -b)
                for b in set(misses) - admitted:                    # nothing left out beats anything admitted
                    assert all(key(b) < key(a) for a in admitted)
                free = [s for s in range(K) if m0[r, h, s] < 0]
                stale = sorted((int(s0[r, h, s]), s) for s in range(K)
                               if m0[r, h, s] >= 0 and m0[r, h, s] not in chosen)
                victims = free + [s for _, s in stale]
                changed = sorted(s for s in range(K) if smap[r, h, s] != m0[r, h, s])
                assert changed == sorted(victims[:n_adm])
                for s in range(K):
                    b = int(smap[r, h, s])
                    if b in chosen:
                        assert stamp[r, h, s] == 9
                    else:
                        assert b == m0[r, h, s] and stamp[r, h, s] == s0[r, h, s]
                    if s in changed:
                        assert np.array_equal(pk[r, s, h], hk[bt[r, b], h])
                        assert np.array_equal(pv[r, s, h], hv[bt[r, b], h])
                if len(misses) <= cap:
                    assert np.array_equal(smap[r, h], um[r, h]) and np.array_equal(stamp[r, h], us[r, h])


def test_stage_capped_converges():
    """With a fixed selection, a cap of C fills n misses in ceil(n / C) steps (§4.2.3)."""
    rng = np.random.default_rng(5)
    R, H, K, B, d, nc = 2, 2, 12, 2, 4, 40
    hk = rng.integers(0, 2 ** 16, size=(nc, H, B, d), dtype=np.uint16)
    hv = rng.integers(0, 2 ** 16, size=(nc, H, B, d), dtype=np.uint16)
    bt = np.stack([rng.permutation(nc) for _ in range(R)]).astype(np.int32)
    ctx = np.full(R, nc * B + 1, np.int32)                     # block nc is the local block
    scores = random_scores(8, (R, H, nc + 1))
    sel, cnt = random_selection_h(9, np.full(R, nc), H, K)
    for cap in (1, 5, 12):
        smap, stamp, pk, pv = (np.full((R, H, K), -1, np.int32), np.zeros((R, H, K), np.int32),
                               np.zeros((R, K + 1, H, B, d), np.uint16), np.zeros((R, K + 1, H, B, d), np.uint16))
        steps = math.ceil(K / cap)
        total = 0
        for t in range(steps):
            moved = O.stage_blocks(hk, hv, bt, sel, cnt, smap, stamp, t, pk, pv, ctx, B, copy_local=False,
                                   scores=scores, fetch_cap=cap)
            total += moved
            if t < steps - 1:
                assert (smap < 0).any(axis=2).all()
        assert np.array_equal(total, np.full((R, H), K))
        for r in range(R):
            for h in range(H):
                assert sorted(smap[r, h]) == sorted(sel[r, h, :cnt[r, h]])


def test_union_selection_against_numpy_and_properties():
    """§4.4.1: a block is in the layer's set if at least one head selected it."""
    rng = np.random.default_rng(17)
    for trial in range(20):
        R, H, K, NB = 3, int(rng.integers(1, 9)), int(rng.integers(1, 20)), int(rng.integers(1, 60))
        sel = np.full((R, H, K), -1, np.int32)
        cnt = rng.integers(0, min(K, NB) + 1, size=(R, H)).astype(np.int32)
        for r in range(R):
            for h in range(H):
                sel[r, h, :cnt[r, h]] = np.sort(rng.choice(NB, size=cnt[r, h], replace=False))
        ids, n = O.union_selection(sel, cnt)
        for r in range(R):
            ref = np.unique(np.concatenate([sel[r, h, :cnt[r, h]] for h in range(H)] + [np.zeros(0, np.int32)]))
            assert n[r] == len(ref) and np.array_equal(ids[r, :n[r]], ref)
            assert (ids[r, n[r]:] == -1).all()
            assert max(cnt[r], default=0) <= n[r] <= cnt[r].sum()
            for h in range(H):                         # every head's set is inside the union
                assert set(sel[r, h, :cnt[r, h]]) <= set(ids[r, :n[r]])


# ---------------------------------------------------------------------------
# Growth of the context: summary updates and block copies between tiers
# ---------------------------------------------------------------------------

def test_update_summaries_matches_full_build_along_growth():
    """Updating on every append reproduces the full build (§4.2.1 summaries, §5.1 updates)."""
    rng = np.random.default_rng(21)
    R, H, B, d, NB = 3, 2, 4, 8, 40
    keys = rng.integers(0, 2 ** 16, size=(R * NB, H, B, d), dtype=np.uint16) & np.uint16(0x7F7F)  # finite bf16
    bt = rng.permutation(R * NB).reshape(R, NB).astype(np.int32)
    kmax = np.full((R, H, NB, d), np.nan)
    kmin = np.full((R, H, NB, d), np.nan)
    ctx = np.zeros(R, np.int32)
    for step in range(25):
        prev = ctx.copy()
        ctx = np.minimum(ctx + rng.integers(0, 3 * B, size=R), NB * B).astype(np.int32)
        n = O.update_summaries(keys, bt, prev, ctx, B, kmax, kmin)
        ref_max, ref_min = O.block_summaries(keys, bt, ctx, B, NB)
        for r in range(R):
            nc = O.block_counts(ctx[r], B)[1]
            assert n[r] == nc - O.block_counts(prev[r], B)[1]
            assert np.array_equal(kmax[r, :, :nc], ref_max[r, :, :nc])
            assert np.array_equal(kmin[r, :, :nc], ref_min[r, :, :nc])
            assert np.isnan(kmax[r, :, nc:]).all()        # the local block and beyond: not yet summarised
    # a bound below the growth writes only the first rows
    kmax2 = np.full_like(kmax, np.nan)
    kmin2 = np.full_like(kmin, np.nan)
    n = O.update_summaries(keys, bt, np.zeros(R, np.int32), np.full(R, 10 * B + 1, np.int32), B, kmax2, kmin2,
                           max_new_blocks=3)
    assert list(n) == [3] * R
    assert not np.isnan(kmax2[:, :, :3]).any() and np.isnan(kmax2[:, :, 3:]).all()


@pytest.mark.parametrize("prev,cur,expect", [(0, 1, [0]), (0, 33, [0, 1, 2]), (32, 33, [2]), (31, 33, [1, 2]),
                                             (16, 16, []), (20, 19, []), (5, 48, [0, 1, 2])])
def test_copy_blocks_touched_range(prev, cur, expect):
    """Blocks copied = those holding tokens [prev, cur): ceil(cur/B) - floor(prev/B) of them (§4.3)."""
    B, H, d, NB = 16, 2, 4, 8
    rng = np.random.default_rng(prev * 100 + cur)
    src_k = rng.integers(0, 2 ** 16, size=(NB, H, B, d), dtype=np.uint16)
    src_v = rng.integers(0, 2 ** 16, size=(NB, H, B, d), dtype=np.uint16)
    st = rng.permutation(NB).astype(np.int32)[None]
    dt = rng.permutation(NB).astype(np.int32)[None]
    dst_k = np.zeros_like(src_k)
    dst_v = np.zeros_like(src_v)
    n = O.copy_blocks(src_k, src_v, st, dst_k, dst_v, dt, np.array([prev]), np.array([cur]), B)
    assert n[0] == len(expect)
    for b in range(NB):
        if b in expect:
            assert np.array_equal(dst_k[dt[0, b]], src_k[st[0, b]]) and np.array_equal(dst_v[dt[0, b]], src_v[st[0, b]])
        else:
            assert not dst_k[dt[0, b]].any() and not dst_v[dt[0, b]].any()


def test_copy_blocks_skips_blocks_without_pages():
    """A block with no page (-1) in either table is not copied, and nothing else is touched."""
    B, H, d = 4, 1, 2
    src_k = np.arange(6 * H * B * d, dtype=np.uint16).reshape(6, H, B, d)
    src_v = src_k + np.uint16(1000)
    st = np.array([[0, 1, -1, 3, 4, 5]], np.int32)
    dt = np.array([[5, -1, 3, 2, 1, 0]], np.int32)
    dst_k = np.zeros_like(src_k)
    dst_v = np.zeros_like(src_v)
    n = O.copy_blocks(src_k, src_v, st, dst_k, dst_v, dt, np.array([0]), np.array([6 * B]), B)
    assert n[0] == 4                                   # blocks 1 (no destination) and 2 (no source) skipped
    for b, (s_, t_) in enumerate(zip(st[0], dt[0])):
        if s_ >= 0 and t_ >= 0:
            assert np.array_equal(dst_k[t_], src_k[s_]) and np.array_equal(dst_v[t_], src_v[s_])
    assert not dst_k[3].any()                          # block 2's destination page stays untouched


def test_transition_then_staging_equals_staging_from_the_device_tier():
    """Dense -> sparse (§4.3): after copying the whole context to the host tier, staging the
    selection from it gives the same working set as staging from the device pages."""
    w = Workload(tiny_cfg(num_reqs=2, ctx_args=(40, 90)))
    c = w.cfg
    hk, hv, ctx, kmax, kmin = _summaries(w)
    K = c.K
    dev_bt = w.block_table
    n_host = c.num_reqs * w.NBmax                     # a host tier of its own, pages in another order
    host_bt = np.random.default_rng(3).permutation(n_host).reshape(c.num_reqs, w.NBmax).astype(np.int32)
    host_k = np.zeros((n_host,) + hk.shape[1:], hk.dtype)
    host_v = np.zeros_like(host_k)
    n = O.copy_blocks(hk, hv, dev_bt, host_k, host_v, host_bt, np.zeros(c.num_reqs, np.int32), ctx, c.block_size)
    assert list(n) == [O.block_counts(L, c.block_size)[0] for L in ctx]
    s = O.block_scores(w.queries(0), kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel, cnt = O.select_topk(s, ctx, K, c.block_size)
    pools = []
    for src_k, src_v, bt in ((hk, hv, dev_bt), (host_k, host_v, host_bt)):
        smap, stamp, pk, pv = _empty_state(c.num_reqs, c.num_kv_heads, K, c.block_size, c.head_dim)
        O.stage_blocks(src_k, src_v, bt, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
        pools.append((smap, pk, pv))
    assert all(np.array_equal(a, b) for a, b in zip(pools[0], pools[1]))


# ---------------------------------------------------------------------------
# O4 attention
# ---------------------------------------------------------------------------

def _torch_dense(w, hk, hv, ctx, scale=None):
    """Textbook GQA attention with torch in float64 on the CPU (library routine)."""
    c = w.cfg
    qf = torch.from_numpy(O.bf16_to_f64(w.queries(0)))
    out = np.zeros((c.num_reqs, c.T, c.num_q_heads, c.head_dim))
    for r in range(c.num_reqs):
        L = int(ctx[r])
        k_r, v_r = w.request_kv(r)
        kf = torch.from_numpy(O.bf16_to_f64(k_r[:, :L]))               # [Hkv][L][d]
        vf = torch.from_numpy(O.bf16_to_f64(v_r[:, :L]))
        kq = kf.repeat_interleave(c.G, dim=0)                            # [Hq][L][d]
        vq = vf.repeat_interleave(c.G, dim=0)
        qq = qf[r].permute(1, 0, 2)                                      # [Hq][T][d]
        o = torch.nn.functional.scaled_dot_product_attention(qq, kq, vq, scale=scale)
        out[r] = o.permute(1, 0, 2).numpy()
    return out


def _stage_all(w, hk, hv, ctx, K):
    c = w.cfg
    smap, stamp, pk, pv = _empty_state(c.num_reqs, c.num_kv_heads, K, c.block_size, c.head_dim)
    scores = np.zeros((c.num_reqs, c.num_kv_heads, w.NBmax))
    sel, cnt = O.select_topk(scores, ctx, K, c.block_size)
    O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
    return smap, pk, pv


def test_attend_dense_equivalence_vs_torch():
    """Budget covering every block: sparse attention == textbook dense attention."""
    w = Workload(tiny_cfg(num_reqs=4, ctx_args=(1, 60)))
    hk, hv = w.fill_paged(threads=1)
    ctx = w.ctx_len(0)
    K = int(w.NBmax)
    smap, pk, pv = _stage_all(w, hk, hv, ctx, K)
    o, lse = O.sparse_attend(w.queries(0), pk, pv, smap, ctx, w.cfg.block_size)
    ref = _torch_dense(w, hk, hv, ctx)
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-12)
    od, lsed = O.dense_attend(w.queries(0), hk, hv, w.block_table, ctx, w.cfg.block_size)
    assert np.allclose(od, ref, rtol=1e-12, atol=1e-12)
    assert np.allclose(lse, lsed, rtol=1e-12, atol=1e-12)


def test_attend_lse_normalises_weights():
    w = Workload(tiny_cfg(num_reqs=2, ctx_args=(20, 60)))
    c = w.cfg
    hk, hv = w.fill_paged(threads=1)
    ctx = w.ctx_len(0)
    _, lse = O.dense_attend(w.queries(0), hk, hv, w.block_table, ctx, c.block_size)
    qf = O.bf16_to_f64(w.queries(0))
    for r in range(c.num_reqs):
        kf = O.bf16_to_f64(w.request_kv(r)[0][:, :ctx[r]])
        for t in range(c.T):
            for qh in range(c.num_q_heads):
                z = kf[qh // c.G] @ qf[r, t, qh] / math.sqrt(c.head_dim)
                assert math.isclose(np.exp(z - lse[r, t, qh]).sum(), 1.0, rel_tol=1e-12)


def test_attend_single_token_and_equal_keys():
    c = tiny_cfg(num_reqs=1, ctx_kind="fixed", ctx_args=(1,), key_dist="zipf")
    w = Workload(c)
    hk, hv = w.fill_paged(threads=1)
    ctx = w.ctx_len(0)
    smap, pk, pv = _stage_all(w, hk, hv, ctx, 3)
    o, _ = O.sparse_attend(w.queries(0), pk, pv, smap, ctx, c.block_size)
    v0 = O.bf16_to_f64(w.request_kv(0)[1][:, 0])                        # [Hkv][d]
    for qh in range(c.num_q_heads):
        assert np.array_equal(o[0, :, qh], np.tile(v0[qh // c.G], (c.T, 1)))
    # all keys equal -> uniform weights -> mean of the values
    L = 37
    w = Workload(c.replace(ctx_args=(L,)))
    hk, hv = w.fill_paged(threads=1)
    hk[:] = hk[w.block_table[0, 0], :, 0:1, :]
    ctx = w.ctx_len(0)
    smap, pk, pv = _stage_all(w, hk, hv, ctx, 16)
    o, _ = O.sparse_attend(w.queries(0), pk, pv, smap, ctx, c.block_size)
    vf = O.bf16_to_f64(w.request_kv(0)[1][:, :L])
    for qh in range(c.num_q_heads):
        assert np.allclose(o[0, :, qh], vf[qh // c.G].mean(axis=0), rtol=1e-12, atol=1e-12)


def test_attend_skips_free_slots_even_with_garbage():
    w = Workload(tiny_cfg(num_reqs=2, ctx_args=(30, 60)))
    c = w.cfg
    hk, hv = w.fill_paged(threads=1)
    ctx = w.ctx_len(0)
    smap, pk, pv = _stage_all(w, hk, hv, ctx, w.NBmax)
    o, l = O.sparse_attend(w.queries(0), pk, pv, smap, ctx, c.block_size)
    smap2 = np.concatenate([smap, np.full(smap.shape[:2] + (3,), -1, np.int32)], axis=2)
    nan = f32_to_bf16_bits(np.zeros(1, np.float32))[0] | np.uint16(0x7FC0)
    garbage = np.full((c.num_reqs, 3, c.num_kv_heads, c.block_size, c.head_dim), nan, np.uint16)
    pk2 = np.concatenate([pk[:, :-1], garbage, pk[:, -1:]], axis=1)
    pv2 = np.concatenate([pv[:, :-1], garbage, pv[:, -1:]], axis=1)
    o2, l2 = O.sparse_attend(w.queries(0), pk2, pv2, smap2, ctx, c.block_size)
    assert np.array_equal(o, o2) and np.array_equal(l, l2)


def test_empty_context():
    c = tiny_cfg(num_reqs=1, ctx_kind="fixed", ctx_args=(1,))
    w = Workload(c)
    hk, hv = w.fill_paged(threads=1)
    smap, _, pk, pv = _empty_state(1, c.num_kv_heads, 2, c.block_size, c.head_dim)
    o, l = O.sparse_attend(w.queries(0), pk, pv, smap, np.array([0]), c.block_size)
    assert np.all(o == 0) and np.all(l == -np.inf)


# ---------------------------------------------------------------------------
# The paper's configuration: 129 blocks / 2,064 tokens, planted heavy hitters selected
# ---------------------------------------------------------------------------

def test_c1_pipeline_counts_and_planted_blocks():
    w = make_workload("c1")
    c = w.cfg
    hk, hv, ctx, kmax, kmin = _summaries(w)
    s = O.block_scores(w.queries(0), kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel, cnt = O.select_topk(s, ctx, c.K, c.block_size)
    assert c.K == 128 and np.all(cnt == 128)
    for h in range(c.num_kv_heads):
        planted = set(w.planted_ids(0, h))
        assert len(planted) == 8 and planted <= set(sel[0, h])
    smap, stamp, pk, pv = _empty_state(1, c.num_kv_heads, c.K, c.block_size, c.head_dim)
    O.stage_blocks(hk, hv, w.block_table, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
    # attended set per head: 128 selected blocks + the local block = 129 blocks, 2,064 tokens (paper §5.2)
    nb, n_cand, local_len = O.block_counts(ctx[0], c.block_size)
    for h in range(c.num_kv_heads):
        blocks = [b for b in smap[0, h] if b >= 0]
        assert len(blocks) == 128 and len(set(blocks)) == 128
        assert (len(blocks) + 1) * c.block_size == 2064 and local_len == 16
    # sparse output == dense attention restricted to exactly those 2,064 tokens (torch, float64)
    o, _ = O.sparse_attend(w.queries(0), pk, pv, smap, ctx, c.block_size)
    qf = torch.from_numpy(O.bf16_to_f64(w.queries(0)[0]))
    k_r, v_r = w.request_kv(0)
    for h in range(c.num_kv_heads):
        toks = np.concatenate([np.arange(b * 16, b * 16 + 16) for b in sorted(smap[0, h])] +
                              [np.arange(n_cand * 16, ctx[0])])
        assert toks.size == 2064
        kf = torch.from_numpy(O.bf16_to_f64(k_r[h, toks]))
        vf = torch.from_numpy(O.bf16_to_f64(v_r[h, toks]))
        for g in range(c.G):
            qh = h * c.G + g
            ref = torch.nn.functional.scaled_dot_product_attention(qf[:, qh][None], kf[None], vf[None])[0]
            assert np.allclose(o[0, :, qh], ref.numpy(), rtol=1e-12, atol=1e-12)


def test_c4_planted_fraction():
    c = make_workload("c4").cfg
    w = Workload(c.replace(num_reqs=1))
    assert w.n_cand0(0) == 8191 and len(w.planted_ids(0, 0)) == 82
