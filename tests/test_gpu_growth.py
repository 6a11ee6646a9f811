"""GPU parity of the operations around the path as a context grows: compressed-key
updates on append (paper §5.1), block copies between the GPU pages and the full
host tier, and the dense-to-sparse transition (§4.3), against the CPU oracle."""
import numpy as np
import pytest
import torch

import paper_2608_08097_amd as P
from oracle import oasis_oracle as O
from paper_2608_08097_amd.path import DecodePath, LayerState
from tests.gpu_util import (as_np_bits, assert_attn_close, assert_lse_close, dev_bf16, dev_i32, device_local_pages,
                            host_bits, note, pinned_pages, pool_v_to_htd, selection_diff)
from workloads import make_workload

pytestmark = pytest.mark.gpu


def _dims(w):
    c = w.cfg
    return P.dims(c.num_reqs, c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size, w.NBmax)


@pytest.mark.parametrize("block_size,bound", [(16, None), (32, None), (16, 1)])
def test_update_summaries_along_growth(block_size, bound):
    """Rows of the blocks completed since the previous length, bit-exact; no other row written."""
    w = make_workload("c3", num_reqs=4, ctx_args=(100, 30, 900), steps=9, grow_per_step=3 * block_size,
                      block_size=block_size)
    c = w.cfg
    B = c.block_size
    hk_t, _ = pinned_pages(w)
    hk = as_np_bits(hk_t)
    d = _dims(w)
    bt = dev_i32(w.block_table)
    rng = np.random.default_rng(44 + B)
    ctx = w.ctx_len(0)
    ref_max, ref_min = O.block_summaries(hk, w.block_table, ctx, B, w.NBmax)
    kmax = torch.zeros((c.num_reqs, c.num_kv_heads, w.NBmax, c.head_dim), dtype=torch.bfloat16, device="cuda")
    kmin = torch.zeros_like(kmax)
    P.oasis_build_summaries(d, hk_t, bt, dev_i32(ctx), kmax, kmin)
    for step in range(12):
        prev = ctx.copy()
        ctx = np.minimum(prev + rng.integers(0, 3 * B, size=c.num_reqs), w.alloc_len).astype(np.int32)
        grown = [O.block_counts(b, B)[1] - O.block_counts(a, B)[1] for a, b in zip(prev, ctx)]
        max_new = bound if bound is not None else max(1, max(grown))
        O.update_summaries(hk, w.block_table, prev, ctx, B, ref_max, ref_min, max_new)
        note(f"update summaries B={B} step={step} max_new={max_new}")
        P.oasis_update_summaries(d, hk_t, bt, dev_i32(prev), dev_i32(ctx), max_new, kmax, kmin)
        torch.cuda.synchronize()
        gmax, gmin = O.bf16_to_f64(host_bits(kmax)), O.bf16_to_f64(host_bits(kmin))
        written = ~np.isnan(ref_max)
        assert np.array_equal(gmax[written], ref_max[written]) and np.array_equal(gmin[written], ref_min[written])
        assert not gmax[~written].any() and not gmin[~written].any(), "a row was written that should not be"


def test_copy_blocks_between_tiers():
    """Device pages -> pinned host tier (whole context, then appends), and back to the device."""
    w = make_workload("c2", num_reqs=3, ctx_args=(200, 700), budget=128)
    c = w.cfg
    B, H = c.block_size, c.num_kv_heads
    src_k, src_v = pinned_pages(w)
    dev_k, dev_v = src_k.cuda(), src_v.cuda()
    d = _dims(w)
    n_host = c.num_reqs * w.NBmax
    host_bt = np.random.default_rng(5).permutation(n_host).reshape(c.num_reqs, w.NBmax).astype(np.int32)
    shape = (n_host, H, B, c.head_dim)
    host_k = torch.zeros(shape, dtype=torch.bfloat16).pin_memory()
    host_v = torch.zeros(shape, dtype=torch.bfloat16).pin_memory()
    ref_k = np.zeros(shape, np.uint16)
    ref_v = np.zeros(shape, np.uint16)
    sk, sv = as_np_bits(src_k), as_np_bits(src_v)
    ctx = w.ctx_len(0)
    note("copy blocks: transition (whole context) device -> host")
    O.copy_blocks(sk, sv, w.block_table, ref_k, ref_v, host_bt, np.zeros_like(ctx), ctx, B)
    P.oasis_copy_blocks(d, dev_k, dev_v, dev_i32(w.block_table), host_k, host_v, dev_i32(host_bt), None,
                        dev_i32(ctx), w.NBmax)
    torch.cuda.synchronize()
    assert np.array_equal(as_np_bits(host_k), ref_k) and np.array_equal(as_np_bits(host_v), ref_v)
    # appends: new tokens land in the device pages; only the touched blocks are copied
    rng = np.random.default_rng(6)
    for step in range(4):
        prev = ctx.copy()
        ctx = np.minimum(prev + rng.integers(0, 2 * B, size=c.num_reqs), w.NBmax * B).astype(np.int32)
        for r in range(c.num_reqs):   # overwrite the pages of the touched blocks with fresh values
            for b in range(prev[r] // B, (ctx[r] + B - 1) // B):
                pg = w.block_table[r, b]
                if pg >= 0:
                    sk[pg] = rng.integers(0, 2 ** 16, size=sk[pg].shape, dtype=np.uint16)
                    sv[pg] = rng.integers(0, 2 ** 16, size=sv[pg].shape, dtype=np.uint16)
        dev_k.copy_(src_k)
        dev_v.copy_(src_v)
        O.copy_blocks(sk, sv, w.block_table, ref_k, ref_v, host_bt, prev, ctx, B, max_blocks=3)
        note(f"copy blocks: append step {step}")
        P.oasis_copy_blocks(d, dev_k, dev_v, dev_i32(w.block_table), host_k, host_v, dev_i32(host_bt),
                            dev_i32(prev), dev_i32(ctx), 3)
        torch.cuda.synchronize()
        assert np.array_equal(as_np_bits(host_k), ref_k) and np.array_equal(as_np_bits(host_v), ref_v), step
    # host -> device, into a device tier of the host's layout
    back_k = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    back_v = torch.zeros_like(back_k)
    note("copy blocks: host -> device")
    P.oasis_copy_blocks(d, host_k, host_v, dev_i32(host_bt), back_k, back_v, dev_i32(host_bt), None, dev_i32(ctx),
                        w.NBmax)
    torch.cuda.synchronize()
    assert np.array_equal(host_bits(back_k), ref_k) and np.array_equal(host_bits(back_v), ref_v)


def test_dense_to_sparse_transition():
    """§4.3: the whole KV goes to the host tier, the GPU keeps the selection (staged from the
    still-resident device pages) and the local block; the next step reads the host tier."""
    w = make_workload("c2", num_reqs=3, ctx_args=(1000, 3000), budget=16 * 24, ar_queries=True)
    c = w.cfg
    B, H, K = c.block_size, c.num_kv_heads, c.K
    src_k, src_v = pinned_pages(w)
    sk, sv = as_np_bits(src_k), as_np_bits(src_v)
    dev_k, dev_v = src_k.cuda(), src_v.cuda()     # the dense request's pages in HBM
    d = _dims(w)
    n_host = c.num_reqs * w.NBmax
    host_bt = np.random.default_rng(9).permutation(n_host).reshape(c.num_reqs, w.NBmax).astype(np.int32)
    shape = (n_host, H, B, c.head_dim)
    host_k = torch.zeros(shape, dtype=torch.bfloat16).pin_memory()
    host_v = torch.zeros(shape, dtype=torch.bfloat16).pin_memory()
    ctx = w.ctx_len(0)
    ctx_d, dev_bt, host_bt_d = dev_i32(ctx), dev_i32(w.block_table), dev_i32(host_bt)
    q0, q1 = w.layer_queries(0, 2)

    # oracle: copy, predict from the device pages, stage (cold), then one decode step on the host tier
    ref_k = np.zeros(shape, np.uint16)
    ref_v = np.zeros(shape, np.uint16)
    O.copy_blocks(sk, sv, w.block_table, ref_k, ref_v, host_bt, np.zeros_like(ctx), ctx, B)
    kmax, kmin = O.block_summaries(sk, w.block_table, ctx, B, w.NBmax)
    s0 = O.block_scores(q0, kmax, kmin, ctx, H, B)
    sel0, cnt0 = O.select_topk(s0, ctx, K, B)
    smap = np.full((c.num_reqs, H, K), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, K + 1, H, B, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    O.stage_blocks(sk, sv, w.block_table, sel0, cnt0, smap, stamp, 0, pk, pv, ctx, B)
    s1 = O.block_scores(q1, kmax, kmin, ctx, H, B)
    sel1, cnt1 = O.select_topk(s1, ctx, K, B)
    O.stage_blocks(ref_k, ref_v, host_bt, sel1, cnt1, smap, stamp, 1, pk, pv, ctx, B, scores=s1, fetch_cap=4)
    ref_o, ref_l = O.sparse_attend(q1, pk, pv, smap, ctx, B)

    note("transition: copy to the host tier, stage from the device pages")
    path = DecodePath(d, c.T, K, host_k, host_v, host_bt_d, fetch_cap=4)
    st = LayerState(d, c.T, K)
    P.oasis_copy_blocks(d, dev_k, dev_v, dev_bt, host_k, host_v, host_bt_d, None, ctx_d, w.NBmax)
    P.oasis_build_summaries(d, dev_k, dev_bt, ctx_d, st.kmax, st.kmin)
    path.predict(st, dev_bf16(q0), ctx_d)
    P.oasis_stage_blocks(d, dev_k, dev_v, dev_bt, ctx_d, st.sel, st.sel_count, st.scores, K, st.slot_map,
                         st.slot_stamp, 0, K, True, st.pool_k, st.pool_v, st.moved)
    note("transition: first sparse step from the host tier")
    path.step_serial(st, dev_bf16(q1), ctx_d, 1)
    torch.cuda.synchronize()
    assert np.array_equal(as_np_bits(host_k), ref_k) and np.array_equal(as_np_bits(host_v), ref_v)
    assert not selection_diff(st.sel.cpu().numpy(), st.sel_count.cpu().numpy(), sel1, cnt1, s1)
    assert np.array_equal(st.slot_map.cpu().numpy(), smap)
    assert np.array_equal(st.slot_stamp.cpu().numpy(), stamp)
    assert np.array_equal(host_bits(st.pool_k), pk)
    assert np.array_equal(pool_v_to_htd(host_bits(st.pool_v)), pv)
    assert_attn_close(host_bits(st.out), ref_o)
    assert_lse_close(st.lse.cpu().numpy(), ref_l)


@pytest.mark.parametrize("local_source", ["host", "device"])
def test_growing_layers_pipelined(local_source):
    """The reasoning loop of §4.2.2 on the native issuer: several layers, one token appended per
    step, each layer's compressed keys updated when a block completes, capped staging; every
    layer's output and working set equal its own oracle chain. The local block is refreshed from
    the host tier with the compressed keys updated by the caller, or from device copies of the
    active blocks (where a model writes new tokens) with the update issued by the step itself."""
    n_layers, steps, cap = 3, 40, 3
    w = make_workload("c3", num_reqs=3, ctx_args=(100, 30, 400), steps=steps, budget=16 * 12, ar_queries=True)
    c = w.cfg
    B, H, K = c.block_size, c.num_kv_heads, c.K
    hk_t, hv_t = pinned_pages(w)
    hk, hv = as_np_bits(hk_t), as_np_bits(hv_t)
    d = _dims(w)
    bt = dev_i32(w.block_table)
    path = DecodePath(d, c.T, K, hk_t, hv_t, bt, fetch_cap=cap)
    if local_source == "device":
        path.set_local_source(*device_local_pages(w, hk_t, hv_t, steps))
    layers = [LayerState(d, c.T, K) for _ in range(n_layers)]
    qs = [w.layer_queries(l, steps) for l in range(n_layers)]
    q_dev = [[dev_bf16(x) for x in qs[l]] for l in range(n_layers)]
    ctx0 = w.ctx_len(0)
    ctx_dev = [dev_i32(w.ctx_len(s)) for s in range(steps)]
    ref = []
    for l, st in enumerate(layers):
        path.build_summaries(st, ctx_dev[0])
        kmax, kmin = O.block_summaries(hk, w.block_table, ctx0, B, w.NBmax)
        ref.append(dict(kmax=kmax, kmin=kmin, smap=np.full((c.num_reqs, H, K), -1, np.int32),
                        stamp=np.zeros((c.num_reqs, H, K), np.int32),
                        pk=np.zeros((c.num_reqs, K + 1, H, B, c.head_dim), np.uint16),
                        pv=np.zeros((c.num_reqs, K + 1, H, B, c.head_dim), np.uint16)))
    note("growing layers: issuing all steps")
    for s in range(steps):
        for l, st in enumerate(layers):
            if local_source == "host":   # compressed keys updated by the caller, on the foreground
                if s > 0:
                    P.oasis_update_summaries(d, hk_t, bt, ctx_dev[s - 1], ctx_dev[s], 1, st.kmax, st.kmin)
                path.step_pipelined(st, q_dev[l][s], ctx_dev[s], s, growing=True)
            else:                        # by the step, on the prediction stream, from the device pages
                path.step_pipelined(st, q_dev[l][s], ctx_dev[s], s, growing=True,
                                    prev_ctx_len=ctx_dev[s - 1] if s > 0 else None)
    path.join()
    torch.cuda.synchronize()
    none_sel = np.full((c.num_reqs, H, K), -1, np.int32)
    zero_cnt = np.zeros((c.num_reqs, H), np.int32)
    for l, st in enumerate(layers):
        r_ = ref[l]
        for s in range(steps):
            ctx = w.ctx_len(s)
            if s > 0:
                O.update_summaries(hk, w.block_table, w.ctx_len(s - 1), ctx, B, r_["kmax"], r_["kmin"], 1)
            O.stage_blocks(hk, hv, w.block_table, none_sel, zero_cnt, r_["smap"], r_["stamp"], s, r_["pk"], r_["pv"],
                           ctx, B)
            ref_o, ref_l = O.sparse_attend(qs[l][s], r_["pk"], r_["pv"], r_["smap"], ctx, B)
            sc = O.block_scores(qs[l][s], r_["kmax"], r_["kmin"], ctx, H, B)
            sel, cnt = O.select_topk(sc, ctx, K, B)
            O.stage_blocks(hk, hv, w.block_table, sel, cnt, r_["smap"], r_["stamp"], s, r_["pk"], r_["pv"], ctx, B,
                           copy_local=False, scores=sc, fetch_cap=cap)
        assert not selection_diff(st.sel.cpu().numpy(), st.sel_count.cpu().numpy(), sel, cnt, sc)
        assert np.array_equal(st.slot_map.cpu().numpy(), r_["smap"]), l
        assert np.array_equal(st.slot_stamp.cpu().numpy(), r_["stamp"]), l
        assert_attn_close(host_bits(st.out), ref_o, f"layer {l} out")
        assert_lse_close(st.lse.cpu().numpy(), ref_l)
        ok = ~np.isnan(r_["kmax"])                    # rows the oracle wrote; the rest was never initialised
        assert np.array_equal(O.bf16_to_f64(host_bits(st.kmax)[ok]), r_["kmax"][ok])
    path.close()
