"""Parity at the configured full sizes, on sampled requests.

The GPU runs every request of the batch in the configuration bench.py times
(one serial step per configuration; the pipelined, capped loop at 8 x 131,072
tokens; the growing reasoning loop at 64 requests); the oracle recomputes the
sampled requests one by one from the same seeded inputs, and their scores,
selections, working sets and attention outputs are compared.
"""
import numpy as np
import pytest
import torch

from oracle import oasis_oracle as O
from paper_2608_08097_amd.path import DecodePath, LayerState, dense_working_set
import paper_2608_08097_amd as P
from tests.gpu_util import (adjudicate_capped, assert_attn_close, assert_lse_close, assert_scores_close, as_np_bits,
                            dev_bf16, dev_i32, host_bits, note, pinned_pages, pool_v_from_htd, selection_diff)
from workloads import config, Workload

pytestmark = pytest.mark.gpu

_TIERS = {}


def _tier(name, **overrides):
    key = (name, tuple(sorted(overrides.items())))
    if key not in _TIERS:
        _TIERS.clear()                                    # one full-size host tier at a time
        note(f"full-size inputs {name} {overrides}")
        w = Workload(config(name, **overrides))
        hk_t, hv_t = pinned_pages(w)
        _TIERS[key] = (w, hk_t, hv_t)
    return _TIERS[key]


def _dims(w):
    c = w.cfg
    return P.dims(c.num_reqs, c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size, w.NBmax)


def _oracle_request(w, hk, hv, r, ctx, q, K):
    """The oracle's step for request r alone, from a cold working set."""
    c = w.cfg
    B, H = c.block_size, c.num_kv_heads
    bt, cr, qr = w.block_table[r:r + 1], ctx[r:r + 1], q[r:r + 1]
    kmax, kmin = O.block_summaries(hk, bt, cr, B, w.NBmax)
    s = O.block_scores(qr, kmax, kmin, cr, H, B)
    sel, cnt = O.select_topk(s, cr, K, B)
    smap = np.full((1, H, K), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((1, K + 1, H, B, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    moved = O.stage_blocks(hk, hv, bt, sel, cnt, smap, stamp, 0, pk, pv, cr, B)
    out, lse = O.sparse_attend(qr, pk, pv, smap, cr, B)
    return dict(s=s, sel=sel, cnt=cnt, smap=smap, moved=moved, out=out, lse=lse)


@pytest.mark.parametrize("name,budget", [("c1", None), ("c2", None), ("c4", 1024), ("c4", 2048), ("c4", 4096),
                                         ("c5", None)])
def test_fullsize_serial_step(name, budget):
    """One serial step of each configuration; c4 at each budget of its sweep (1,024 / 2,048 / 4,096 tokens:
    K = 64 / 128 / 256 blocks, §5.2: the budget is the sparsification threshold)."""
    w, hk_t, hv_t = _tier(name, ar_queries=True)
    c = w.cfg
    K = c.K if budget is None else budget // c.block_size
    d = _dims(w)
    ctx = w.ctx_len(0)
    q = w.queries(0)
    path = DecodePath(d, c.T, K, hk_t, hv_t, dev_i32(w.block_table))
    st = LayerState(d, c.T, K)
    ctx_d = dev_i32(ctx)
    note(f"full-size serial step {name}: R={c.num_reqs} L={int(ctx.max())} K={K}")
    path.build_summaries(st, ctx_d)
    path.step_serial(st, dev_bf16(q), ctx_d, 0)
    torch.cuda.synchronize()
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    scores, sel, cnt = st.scores.cpu().numpy(), st.sel.cpu().numpy(), st.sel_count.cpu().numpy()
    smap, moved = st.slot_map.cpu().numpy(), st.moved.cpu().numpy()
    out, lse = host_bits(st.out), st.lse.cpu().numpy()
    for r in sorted({0, c.num_reqs // 2, c.num_reqs - 1}):
        ref = _oracle_request(w, hk, hv, r, ctx, q, K)
        assert_scores_close(scores[r:r + 1], ref["s"])
        assert not selection_diff(sel[r:r + 1], cnt[r:r + 1], ref["sel"], ref["cnt"], ref["s"]), (name, r)
        assert np.array_equal(smap[r:r + 1], ref["smap"]) and np.array_equal(moved[r:r + 1], ref["moved"])
        assert_attn_close(out[r:r + 1], ref["out"], f"{name} request {r}")
        assert_lse_close(lse[r:r + 1], ref["lse"])


def test_fullsize_dense_c4():
    """The benchmark's dense comparison exactly as bench.py runs it: 8 x 131,072 tokens resident in HBM, every
    block in the slot of its own id, k_slots = 8,191 (4,096 units of 32 tokens per KV head, about 256 per
    wave, so the lazily rescaled online softmax runs its longest loop), against the oracle's dense
    attention over the paged host tier for sampled (request, KV head) pairs."""
    w, hk_t, hv_t = _tier("c4", ar_queries=True)
    c = w.cfg
    d = _dims(w)
    G = c.G
    ctx = w.ctx_len(0)
    q = w.queries(0)
    pool_k, pool_v, smap, ks = dense_working_set(hk_t, hv_t, w.block_table, ctx)
    assert ks == w.NBmax - 1 == 8191
    out = torch.empty((c.num_reqs, c.T, c.num_q_heads, c.head_dim), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((c.num_reqs, c.T, c.num_q_heads), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.oasis_attn_workspace_bytes(d, c.T, ks), dtype=torch.uint8, device="cuda")
    note(f"full-size dense c4: R={c.num_reqs} L={int(ctx[0])} k_slots={ks}")
    P.oasis_sparse_decode_attn(d, dev_bf16(q), c.T, pool_k, pool_v, smap, ks, dev_i32(ctx), None, out, lse, ws)
    torch.cuda.synchronize()
    out_np, lse_np = host_bits(out), lse.cpu().numpy()
    del pool_k, pool_v
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    for r, h in [(0, 0), (3, 5), (7, 7)]:
        ref_o, ref_l = O.dense_attend(q[r:r + 1, :, h * G:(h + 1) * G], hk[:, h:h + 1], hv[:, h:h + 1],
                                      w.block_table[r:r + 1], ctx[r:r + 1], c.block_size)
        assert_attn_close(out_np[r:r + 1, :, h * G:(h + 1) * G], ref_o, f"dense c4 request {r} KV head {h}")
        assert_lse_close(lse_np[r:r + 1, :, h * G:(h + 1) * G], ref_l)


def test_fullsize_pipelined_capped_c4():
    """The benchmark's loop: 8 x 131,072 tokens, budget 2,048, fetch cap 6, two layer states, issued through
    the native pipeline and read back after every step. A sampled request follows its oracle chain step by
    step; near ties at the selection cut or at the cap's admission cut are adjudicated by the tie rule and
    the oracle then continues from the GPU's choice (reading R22)."""
    NL, S, cap = 2, 4, 6
    w, hk_t, hv_t = _tier("c4", ar_queries=True)
    c = w.cfg
    B, H, K = c.block_size, c.num_kv_heads, c.K
    d = _dims(w)
    ctx = w.ctx_len(0)
    ctx_d = dev_i32(ctx)
    qs = [w.layer_queries(l, S) for l in range(NL)]
    path = DecodePath(d, c.T, K, hk_t, hv_t, dev_i32(w.block_table), fetch_cap=cap)
    layers = [path.new_layer() for _ in range(NL)]
    path.build_summaries(layers[0], ctx_d)
    layers[1].kmax.copy_(layers[0].kmax)
    layers[1].kmin.copy_(layers[0].kmin)
    q_dev = [[dev_bf16(x) for x in qs[l]] for l in range(NL)]
    for l, st in enumerate(layers):
        path.predict(st, q_dev[l][0], ctx_d)
        path.stage(st, ctx_d, 0, fetch_cap=K)
    torch.cuda.synchronize()
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    r = 5
    bt, cr = w.block_table[r:r + 1], ctx[r:r + 1]
    kmax, kmin = O.block_summaries(hk, bt, cr, B, w.NBmax)
    ref = []
    for l, st in enumerate(layers):   # the uncapped fill, on the GPU's selection (adjudicated)
        smap = np.full((1, H, K), -1, np.int32)
        stamp = np.zeros_like(smap)
        pk = np.zeros((1, K + 1, H, B, c.head_dim), np.uint16)
        pv = np.zeros_like(pk)
        s0 = O.block_scores(qs[l][0][r:r + 1], kmax, kmin, cr, H, B)
        sel, cnt = O.select_topk(s0, cr, K, B)
        sel_g, cnt_g = st.sel.cpu().numpy()[r:r + 1], st.sel_count.cpu().numpy()[r:r + 1]
        selection_diff(sel_g, cnt_g, sel, cnt, s0)
        O.stage_blocks(hk, hv, bt, sel_g, cnt_g, smap, stamp, 0, pk, pv, cr, B)
        assert np.array_equal(st.slot_map.cpu().numpy()[r:r + 1], smap), l
        ref.append(dict(smap=smap, stamp=stamp, pk=pk, pv=pv))
    for i in range(NL * S):
        l = i % NL
        st, o = layers[l], ref[l]
        note(f"full-size pipelined c4: step {i} (layer {l})")
        path.step_pipelined(st, q_dev[l][i // NL], ctx_d, i)
        path.join()
        torch.cuda.synchronize()
        qr = qs[l][i // NL][r:r + 1]
        ref_o, ref_l = O.sparse_attend(qr, o["pk"], o["pv"], o["smap"], cr, B)
        assert_attn_close(host_bits(st.out)[r:r + 1], ref_o, f"step {i} layer {l}")
        assert_lse_close(st.lse.cpu().numpy()[r:r + 1], ref_l)
        sc = O.block_scores(qr, kmax, kmin, cr, H, B)
        sel, cnt = O.select_topk(sc, cr, K, B)
        sel_g, cnt_g = st.sel.cpu().numpy()[r:r + 1], st.sel_count.cpu().numpy()[r:r + 1]
        smap_g = st.slot_map.cpu().numpy()[r:r + 1]
        use = adjudicate_capped(sel_g, cnt_g, o["smap"], smap_g, sc, sel, cnt, cap)
        O.stage_blocks(hk, hv, bt, sel_g, cnt_g, o["smap"], o["stamp"], i, o["pk"], o["pv"], cr, B, scores=use,
                       fetch_cap=cap)
        assert np.array_equal(smap_g, o["smap"]), (i, l)
        assert np.array_equal(st.slot_stamp.cpu().numpy()[r:r + 1], o["stamp"]), (i, l)
    for l, st in enumerate(layers):
        assert np.array_equal(host_bits(st.pool_k)[r:r + 1, :K], ref[l]["pk"][:, :K]), l
        assert np.array_equal(host_bits(st.pool_v)[r:r + 1, :K], pool_v_from_htd(ref[l]["pv"])[:, :K]), l
    path.close()


@pytest.mark.parametrize("plan_pred", [False, True])
def test_fullsize_growing_c3(plan_pred):
    """The reasoning loop: 64 requests (1K prompt + 4K-16K generated), one token per step, summary
    updates on block completion, two layer states; read back after every step, a sampled request follows
    its oracle chain under the tie rule (reading R22). The benchmark plans this loop's transfers on the
    prediction stream (``plan_pred``); with 512 (request, KV head) pairs the prediction runs as the fused
    score + select (+ plan) kernel."""
    NL, S, cap = 2, 20, 6
    w, hk_t, hv_t = _tier("c3", steps=S)
    c = w.cfg
    B, H, K = c.block_size, c.num_kv_heads, c.K
    d = _dims(w)
    bt = dev_i32(w.block_table)
    ctx_dev = [dev_i32(w.ctx_len(s)) for s in range(S)]
    qs = [w.layer_queries(l, S) for l in range(NL)]
    q_dev = [[dev_bf16(x) for x in qs[l]] for l in range(NL)]
    path = DecodePath(d, c.T, K, hk_t, hv_t, bt, fetch_cap=cap, plan_on_prediction=plan_pred)
    layers = [path.new_layer() for _ in range(NL)]
    for st in layers:
        path.build_summaries(st, ctx_dev[0])
    torch.cuda.synchronize()
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    r = int(np.argmax(w.ctx0 % B))                     # a request whose local block is far from full
    brow = w.block_table[r:r + 1]
    none_sel = np.full((1, H, K), -1, np.int32)
    zero_cnt = np.zeros((1, H), np.int32)
    c0 = w.ctx_len(0)[r:r + 1]
    ref = []
    for l in range(NL):
        kmax, kmin = O.block_summaries(hk, brow, c0, B, w.NBmax)
        smap = np.full((1, H, K), -1, np.int32)
        ref.append(dict(kmax=kmax, kmin=kmin, smap=smap, stamp=np.zeros_like(smap),
                        pk=np.zeros((1, K + 1, H, B, c.head_dim), np.uint16),
                        pv=np.zeros((1, K + 1, H, B, c.head_dim), np.uint16)))
    note(f"full-size growing c3 (plan on prediction: {plan_pred}): issuing")
    for s in range(S):
        cr = w.ctx_len(s)[r:r + 1]
        for l, st in enumerate(layers):
            o = ref[l]
            if s:
                P.oasis_update_summaries(d, hk_t, bt, ctx_dev[s - 1], ctx_dev[s], 1, st.kmax, st.kmin)
                O.update_summaries(hk, brow, w.ctx_len(s - 1)[r:r + 1], cr, B, o["kmax"], o["kmin"], 1)
            path.step_pipelined(st, q_dev[l][s], ctx_dev[s], s, growing=True)
            path.join()
            torch.cuda.synchronize()
            O.stage_blocks(hk, hv, brow, none_sel, zero_cnt, o["smap"], o["stamp"], s, o["pk"], o["pv"], cr, B)
            qr = qs[l][s][r:r + 1]
            ref_o, ref_l = O.sparse_attend(qr, o["pk"], o["pv"], o["smap"], cr, B)
            assert_attn_close(host_bits(st.out)[r:r + 1], ref_o, f"step {s} layer {l}")
            assert_lse_close(st.lse.cpu().numpy()[r:r + 1], ref_l)
            sc = O.block_scores(qr, o["kmax"], o["kmin"], cr, H, B)
            sel, cnt = O.select_topk(sc, cr, K, B)
            sel_g, cnt_g = st.sel.cpu().numpy()[r:r + 1], st.sel_count.cpu().numpy()[r:r + 1]
            smap_g = st.slot_map.cpu().numpy()[r:r + 1]
            use = adjudicate_capped(sel_g, cnt_g, o["smap"], smap_g, sc, sel, cnt, cap)
            O.stage_blocks(hk, hv, brow, sel_g, cnt_g, o["smap"], o["stamp"], s, o["pk"], o["pv"], cr, B,
                           copy_local=False, scores=use, fetch_cap=cap)
            assert np.array_equal(smap_g, o["smap"]), (s, l)
            assert np.array_equal(st.slot_stamp.cpu().numpy()[r:r + 1], o["stamp"]), (s, l)
    path.close()
