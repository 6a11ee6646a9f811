"""Helpers for the GPU parity tests: moving seeded inputs to the device, reading
results back, and the comparison rules of the parity contract."""
from __future__ import annotations

import math
import os
import sys

import numpy as np
import torch

from oracle import oasis_oracle as O
from workloads import Workload

# attention outputs, bf16 GPU vs float64 oracle: |x - ref| <= ATOL + RTOL * |ref|
ATTN_ATOL, ATTN_RTOL = 2e-2, 1e-2
# log-sum-exp (fp32 logits and sums vs float64)
LSE_ATOL = 2e-3
# selection: a swapped pair is allowed only if both oracle scores are this close to the cut
TIE_REL = 1e-3
# block scores (diagnostic): fp32 MFMA accumulation of exact bf16 products
SCORE_RTOL, SCORE_ATOL = 1e-5, 1e-3


def note(msg: str) -> None:
    """Print and flush what names the case before a GPU step runs."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def dev_i32(x: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(device)


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def pinned_pages(w: Workload):
    """Fill the workload's K/V pages straight into pinned host memory."""
    c = w.cfg
    shape = (w.NPhys, c.num_kv_heads, c.block_size, c.head_dim)
    hk = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    hv = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    w.fill_paged(hk.numpy().view(np.uint16), hv.numpy().view(np.uint16))
    return hk.view(torch.bfloat16), hv.view(torch.bfloat16)


def as_np_bits(t: torch.Tensor) -> np.ndarray:
    """uint16 view of a CPU bf16/int16 tensor (no copy)."""
    return t.view(torch.int16).numpy().view(np.uint16)


def pool_v_to_htd(pool_v_t: np.ndarray) -> np.ndarray:
    """GPU pool_v [R][K+1][Hkv][d][B] -> oracle layout [R][K+1][Hkv][B][d]."""
    return np.ascontiguousarray(np.swapaxes(pool_v_t, -1, -2))


def pool_v_from_htd(pool_v: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(np.swapaxes(pool_v, -1, -2))


def assert_attn_close(out_gpu_bits: np.ndarray, ref: np.ndarray, what: str = "out") -> None:
    got = O.bf16_to_f64(out_gpu_bits)
    err = np.abs(got - ref)
    lim = ATTN_ATOL + ATTN_RTOL * np.abs(ref)
    bad = err > lim
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} elements outside 2e-2 + 1e-2|ref|; "
                             f"max err {err.max():.4g}; first {idx.tolist()}")


def assert_lse_close(lse_gpu: np.ndarray, ref: np.ndarray) -> None:
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(lse_gpu), fin), "lse: -inf pattern differs"
    if fin.any():
        err = np.abs(lse_gpu[fin] - ref[fin])
        assert err.max() <= LSE_ATOL, f"lse: max err {err.max():.4g}"


def assert_scores_close(gpu: np.ndarray, ref: np.ndarray) -> None:
    ninf = ref == -np.inf
    assert np.array_equal(gpu == -np.inf, ninf), "scores: -inf padding differs"
    fin = ~ninf
    err = np.abs(gpu[fin].astype(np.float64) - ref[fin])
    lim = SCORE_ATOL + SCORE_RTOL * np.abs(ref[fin])
    assert np.all(err <= lim), f"scores: max err {err.max():.4g}"


def selection_diff(sel_gpu, cnt_gpu, sel_ref, cnt_ref, scores_ref):
    """Compare selections per (r, h) under the near-tie rule.

    Returns the list of (r, h) whose sets differ by allowed swaps; raises on a
    disallowed difference. tau is the oracle's m-th best score; a block in one
    set and not the other must score within TIE_REL * max(|tau|, 1) of tau.
    """
    R, H = cnt_ref.shape
    swapped = []
    assert np.array_equal(cnt_gpu, cnt_ref), "sel_count differs"
    for r in range(R):
        for h in range(H):
            m = int(cnt_ref[r, h])
            a = sel_gpu[r, h, :m]
            b = sel_ref[r, h, :m]
            assert np.all(sel_gpu[r, h, m:] == -1), f"({r},{h}) padding"
            assert np.all(np.diff(a) > 0), f"({r},{h}) not strictly ascending"
            if np.array_equal(a, b):
                continue
            s = scores_ref[r, h]
            tau = np.sort(s[b])[0]
            tol = TIE_REL * max(abs(tau), 1.0)
            for x in set(a.tolist()) ^ set(b.tolist()):
                assert abs(s[x] - tau) <= tol, f"({r},{h}) block {x}: score {s[x]} vs cut {tau}"
            swapped.append((r, h))
    return swapped


def adjudicate_capped(sel_g, cnt_g, smap_before, smap_after_g, scores_ref, sel_ref, cnt_ref, cap):
    """The near-tie rule of a capped delta step (reading R22), applied to one GPU step.

    The GPU ranks by its fp32 scores, the oracle by float64 ones. The GPU's
    selection must match the oracle's under the selection rule (swaps only
    within TIE_REL of the cut). Its admission under the cap (the blocks newly
    resident in ``smap_after_g`` compared with ``smap_before``) must equal the
    ``cap`` highest-scoring misses of that selection, except for blocks whose
    oracle score is within TIE_REL * max(|tau_C|, 1) of tau_C, the oracle's
    C-th admitted score. Returns the scores with which the oracle, given the
    GPU's selection, admits exactly the GPU's choice (the oracle's own scores
    wherever the two agree), so that the rest of the step (victims, slot map,
    stamps, pools) is then compared bit for bit.
    """
    selection_diff(sel_g, cnt_g, sel_ref, cnt_ref, scores_ref)
    use = np.array(scores_ref, dtype=np.float64, copy=True)
    R, H, _ = smap_before.shape
    for r in range(R):
        for h in range(H):
            m = int(cnt_g[r, h])
            resident = {int(b) for b in smap_before[r, h] if b >= 0}
            misses = [int(b) for b in sel_g[r, h, :m] if int(b) not in resident]
            if cap is None or len(misses) <= cap:
                continue
            s = use[r, h]
            ranked = sorted(misses, key=lambda b: (-s[b], b))
            adm_ref = set(ranked[:cap])
            tau = s[ranked[cap - 1]]
            adm_g = {int(b) for b in smap_after_g[r, h] if b >= 0} - resident
            assert len(adm_g) == cap, f"({r},{h}): {len(adm_g)} admitted under a cap of {cap}"
            tol = TIE_REL * max(abs(tau), 1.0)
            for x in adm_g ^ adm_ref:
                assert abs(s[x] - tau) <= tol, f"({r},{h}) block {x}: score {s[x]} vs admission cut {tau}"
            if adm_g != adm_ref:
                top = np.max(s[np.isfinite(s)]) + 1.0
                for x in adm_g:
                    s[x] = top
    return use


def oracle_layer(w: Workload, host_k: np.ndarray, host_v: np.ndarray, ctx: np.ndarray, q: np.ndarray, k: int):
    """Oracle pipeline for one step from a cold working set: summaries, scores, selection, staging, attention."""
    c = w.cfg
    kmax, kmin = O.block_summaries(host_k, w.block_table, ctx, c.block_size, w.NBmax)
    s = O.block_scores(q, kmax, kmin, ctx, c.num_kv_heads, c.block_size)
    sel, cnt = O.select_topk(s, ctx, k, c.block_size)
    smap = np.full((c.num_reqs, c.num_kv_heads, k), -1, np.int32)
    stamp = np.zeros_like(smap)
    pk = np.zeros((c.num_reqs, k + 1, c.num_kv_heads, c.block_size, c.head_dim), np.uint16)
    pv = np.zeros_like(pk)
    moved = O.stage_blocks(host_k, host_v, w.block_table, sel, cnt, smap, stamp, 0, pk, pv, ctx, c.block_size)
    out, lse = O.sparse_attend(q, pk, pv, smap, ctx, c.block_size)
    return dict(kmax=kmax, kmin=kmin, scores=s, sel=sel, cnt=cnt, slot_map=smap, stamp=stamp, pool_k=pk,
                pool_v=pv, moved=moved, out=out, lse=lse)


def gpu_available() -> bool:
    return torch.cuda.is_available() and os.path.exists(
        os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2608_08097_amd",
                     "liboasis.so"))


def sqrt_d(d: int) -> float:
    return 1.0 / math.sqrt(d)


def device_local_pages(w, hk_t, hv_t, steps):
    """Device copies of the pages that hold a local block during the first ``steps`` steps, and
    their block table (the active blocks a model would keep on the GPU)."""
    pages, table = w.local_block_pages(steps)
    idx = torch.from_numpy(pages)
    dk = hk_t[idx].cuda() if len(pages) else torch.zeros((1,) + tuple(hk_t.shape[1:]), dtype=hk_t.dtype, device="cuda")
    dv = hv_t[idx].cuda() if len(pages) else torch.zeros_like(dk)
    return dk, dv, dev_i32(table)

