"""Oracle vs hand-worked examples stored under tests/golden (CPU only).

Each fixture cites the paper passage it follows and spells out its arithmetic.
"""
import json
import math
import os

import numpy as np

from oracle import oasis_oracle as O
from workloads import f32_to_bf16_bits


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _f(x):
    return float(x) if not isinstance(x, str) else float(x)


def _quest_inputs(g, G, D):
    """One request, one KV head; the two draft rows are laid out as (G heads x D drafts)."""
    d, B, L = g["head_dim"], g["block_size"], g["ctx_len"]
    keys = np.array(g["keys"], dtype=np.float32)
    nb = (L + B - 1) // B
    host_k = np.zeros((nb, 1, B, d), dtype=np.uint16)
    for p in range(L):
        host_k[p // B, 0, p % B] = f32_to_bf16_bits(keys[p])
    bt = np.arange(nb, dtype=np.int32)[None, :]
    T = 1 + D
    q = np.zeros((1, T, G, d), dtype=np.float32)
    q[0, 0, :, :] = np.array(g["verify_row"], dtype=np.float32)
    rows = [np.array(r, dtype=np.float32) for r in g["draft_rows"]]
    i = 0
    for t in range(1, T):
        for gg in range(G):
            q[0, t, gg] = rows[i % len(rows)]
            i += 1
    return host_k, bt, f32_to_bf16_bits(q), np.array([L], dtype=np.int32)


def test_quest_summaries_and_scores(golden_dir):
    g = _load(golden_dir, "quest_score_d4.json")
    for G, D in [(2, 1), (1, 2)]:
        host_k, bt, q, ctx = _quest_inputs(g, G, D)
        kmax, kmin = O.block_summaries(host_k, bt, ctx, g["block_size"], bt.shape[1])
        assert np.array_equal(kmax[0, 0, :2], np.array(g["expected_kmax"], dtype=np.float64))
        assert np.array_equal(kmin[0, 0, :2], np.array(g["expected_kmin"], dtype=np.float64))
        assert np.all(np.isnan(kmax[0, 0, 2:]))  # local block is not summarised
        s = O.block_scores(q, kmax, kmin, ctx, num_kv_heads=1, block_size=g["block_size"])
        assert np.array_equal(s[0, 0, :2], np.array(g["expected_scores"], dtype=np.float64))
        assert s[0, 0, 2] == -np.inf
        for k, want in g["expected_selection"].items():
            sel, cnt = O.select_topk(s, ctx, int(k), g["block_size"])
            assert cnt[0, 0] == len(want)
            assert list(sel[0, 0, :len(want)]) == want


def test_quest_row_scores(golden_dir):
    g = _load(golden_dir, "quest_score_d4.json")
    for i, row in enumerate(g["draft_rows"]):
        one = dict(g, draft_rows=[row])
        host_k, bt, q, ctx = _quest_inputs(one, 1, 1)
        kmax, kmin = O.block_summaries(host_k, bt, ctx, g["block_size"], bt.shape[1])
        s = O.block_scores(q, kmax, kmin, ctx, num_kv_heads=1, block_size=g["block_size"])
        assert np.array_equal(s[0, 0, :2], np.array(g["expected_row_scores"][i], dtype=np.float64))


def test_topk_ties(golden_dir):
    g = _load(golden_dir, "topk_ties.json")
    scores = np.array(g["scores"], dtype=np.float64)[None, None, :]
    ctx = np.array([g["ctx_len"]], dtype=np.int32)
    for c in g["cases"]:
        sel, cnt = O.select_topk(scores, ctx, c["k"], g["block_size"])
        assert list(sel[0, 0]) == c["sel"][:c["k"]]
        assert cnt[0, 0] == c["count"]
    for c in g["zero_cases"]:
        s = np.array([_f(x) for x in c["scores"]], dtype=np.float64)[None, None, :]
        sel, cnt = O.select_topk(s, np.array([c["ctx_len"]], np.int32), c["k"], g["block_size"])
        assert list(sel[0, 0]) == c["sel"]


def test_stage_lru(golden_dir):
    g = _load(golden_dir, "stage_lru.json")
    B, d = 2, 4
    for c in g["cases"]:
        K = len(c["slot_map"])
        nblocks = 32
        rng = np.random.default_rng(7)
        host_k = rng.integers(0, 2 ** 16, size=(nblocks, 1, B, d), dtype=np.uint16)
        host_v = rng.integers(0, 2 ** 16, size=(nblocks, 1, B, d), dtype=np.uint16)
        bt = np.arange(nblocks, dtype=np.int32)[::-1].copy()[None, :]   # non-identity pages
        ctx = np.array([nblocks * B], dtype=np.int32)
        sel = np.full((1, 1, K), -1, np.int32)
        sel[0, 0, :len(c["sel"])] = c["sel"]
        cnt = np.array([[len(c["sel"])]], np.int32)
        smap = np.array(c["slot_map"], np.int32)[None, None, :]
        stamp = np.array(c["slot_stamp"], np.int32)[None, None, :]
        pool_k = np.zeros((1, K + 1, 1, B, d), np.uint16)
        pool_v = np.zeros((1, K + 1, 1, B, d), np.uint16)
        moved = O.stage_blocks(host_k, host_v, bt, sel, cnt, smap, stamp, c["step"], pool_k, pool_v,
                               ctx, B, copy_local=True)
        assert list(smap[0, 0]) == c["expected_slot_map"]
        assert list(stamp[0, 0]) == c["expected_slot_stamp"]
        assert moved[0, 0] == c["expected_moved"]
        before = set(c["slot_map"])
        for s in range(K):
            b = int(smap[0, 0, s])
            if b not in before:          # newly staged: bytes equal the host page of block b
                assert np.array_equal(pool_k[0, s, 0], host_k[bt[0, b], 0])
                assert np.array_equal(pool_v[0, s, 0], host_v[bt[0, b], 0])
        assert np.array_equal(pool_k[0, K, 0], host_k[bt[0, nblocks - 1], 0])


def test_stage_capped(golden_dir):
    g = _load(golden_dir, "stage_capped.json")
    B, d, nblocks = 2, 4, 32
    for c in g["cases"]:
        K = len(c["slot_map"])
        rng = np.random.default_rng(11)
        host_k = rng.integers(0, 2 ** 16, size=(nblocks, 1, B, d), dtype=np.uint16)
        host_v = rng.integers(0, 2 ** 16, size=(nblocks, 1, B, d), dtype=np.uint16)
        bt = np.arange(nblocks, dtype=np.int32)[::-1].copy()[None, :]
        ctx = np.array([nblocks * B], dtype=np.int32)
        sel = np.full((1, 1, K), -1, np.int32)
        sel[0, 0, :len(c["sel"])] = c["sel"]
        cnt = np.array([[len(c["sel"])]], np.int32)
        scores = np.full((1, 1, nblocks), -np.inf)
        for b, v in c["scores"].items():
            scores[0, 0, int(b)] = v
        smap = np.array(c["slot_map"], np.int32)[None, None, :]
        stamp = np.array(c["slot_stamp"], np.int32)[None, None, :]
        pool_k = np.zeros((1, K + 1, 1, B, d), np.uint16)
        pool_v = np.zeros((1, K + 1, 1, B, d), np.uint16)
        moved = O.stage_blocks(host_k, host_v, bt, sel, cnt, smap, stamp, c["step"], pool_k, pool_v,
                               ctx, B, copy_local=False, scores=scores, fetch_cap=c["fetch_cap"])
        assert list(smap[0, 0]) == c["expected_slot_map"]
        assert list(stamp[0, 0]) == c["expected_slot_stamp"]
        assert moved[0, 0] == c["expected_moved"]
        before = c["slot_map"]
        for s in range(K):
            b = int(smap[0, 0, s])
            if b != before[s]:
                assert np.array_equal(pool_k[0, s, 0], host_k[bt[0, b], 0])
                assert np.array_equal(pool_v[0, s, 0], host_v[bt[0, b], 0])
            else:
                assert not pool_k[0, s, 0].any() and not pool_v[0, s, 0].any()
        assert not pool_k[0, K].any()


def test_attend_sigmoid(golden_dir):
    g = _load(golden_dir, "attend_sigmoid.json")
    keys = f32_to_bf16_bits(np.array(g["keys"], np.float32))
    vals = f32_to_bf16_bits(np.array(g["values"], np.float32))
    q = f32_to_bf16_bits(np.array(g["q"], np.float32))[None, None, None, :]
    want_o = np.array(g["expected_out"])
    want_l = g["expected_lse"]
    # layout A: B = 2, both tokens local
    pool_k = np.zeros((1, 2, 1, 2, 2), np.uint16)
    pool_v = np.zeros((1, 2, 1, 2, 2), np.uint16)
    pool_k[0, 1, 0] = keys
    pool_v[0, 1, 0] = vals
    smap = np.full((1, 1, 1), -1, np.int32)
    o, l = O.sparse_attend(q, pool_k, pool_v, smap, np.array([2], np.int32), 2, scale=g["scale"])
    assert np.allclose(o[0, 0, 0], want_o, rtol=0, atol=1e-15)
    assert math.isclose(l[0, 0, 0], want_l, rel_tol=0, abs_tol=1e-15)
    # layout B: B = 1, token 0 in slot 0, token 1 local
    pool_k = np.zeros((1, 2, 1, 1, 2), np.uint16)
    pool_v = np.zeros((1, 2, 1, 1, 2), np.uint16)
    pool_k[0, 0, 0, 0], pool_k[0, 1, 0, 0] = keys[0], keys[1]
    pool_v[0, 0, 0, 0], pool_v[0, 1, 0, 0] = vals[0], vals[1]
    smap = np.zeros((1, 1, 1), np.int32)
    o, l = O.sparse_attend(q, pool_k, pool_v, smap, np.array([2], np.int32), 1, scale=g["scale"])
    assert np.allclose(o[0, 0, 0], want_o, rtol=0, atol=1e-15)
    assert math.isclose(l[0, 0, 0], want_l, rel_tol=0, abs_tol=1e-15)
