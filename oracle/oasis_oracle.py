"""CPU oracle for OasisKV's decode-time hot path.

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module. The
library in ``paper_2608_08097_amd`` never does; it shares no code with this
file, and this file imports nothing from it.

Plain, slow, float64 NumPy written from the paper (arXiv 2608.08097,
"OasisKV: Scaling In-Decode KV Cache Beyond HBM with Lookahead Sparse
Prefetching"). Every input tensor arrives as raw bf16 bits (``uint16``) and is
decoded exactly to float64 here, so all arithmetic below is exact products and
float64 sums. Each function names the passage it follows and the readings taken
where the paper is silent (readings R1..R20, listed with their reasons in the
design notes of this repository).

Shapes (R requests, Hq query heads, Hkv KV heads, G = Hq / Hkv, d head dim,
B block size, T = 1 + D query rows per head, K resident slots per KV head):

* ``q``            bf16 bits ``[R][T][Hq][d]``; row 0 verifies, rows 1..D draft.
* ``host_k/host_v`` bf16 bits ``[NPhys][Hkv][B][d]`` (Head-Token-Dimension pages).
* ``block_table``  int ``[R][NBmax]``: logical block -> physical page.
* ``kmax/kmin``    float64 ``[R][Hkv][NBmax][d]`` (NaN where undefined).
* ``scores``       float64 ``[R][Hkv][NBmax]``, ``-inf`` past the candidates.
* ``sel``          int32 ``[R][Hkv][K]`` ascending, ``-1`` padded; ``sel_count``.
* ``slot_map``     int32 ``[R][Hkv][K]``: resident logical block per slot or -1.
* ``slot_stamp``   int32 ``[R][Hkv][K]``: step at which the slot was last selected.
* ``pool_k/pool_v`` bf16 bits ``[R][K+1][Hkv][B][d]``; slot K holds the local block.

Parity pins: every function here is checked by ``tests/test_oracle_pins.py``
and ``tests/test_golden.py`` against values and properties the paper and the
mathematics fix (hand-worked examples, brute force over a bounding box,
exhaustive subset search, textbook attention from ``torch`` in float64, and
invariants). No function is "parity unpinned".
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "bf16_to_f64", "block_counts", "block_summaries", "update_summaries", "copy_blocks", "block_scores",
    "select_topk", "union_selection", "stage_blocks", "sparse_attend", "dense_attend",
]


def bf16_to_f64(bits) -> np.ndarray:
    """Exact value of bf16 bit patterns: the 16 bits are the high half of a float32."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def block_counts(L: int, B: int) -> tuple[int, int, int]:
    """(blocks, candidate blocks, tokens in the local block) of a context of L tokens.

    Paper §5.2: each head keeps the active local block in addition to the K
    selected blocks. Reading R4: the last logical block (index nb - 1, possibly
    partial) is that local block; it is always attended and never ranked, so
    the candidates are blocks 0 .. nb - 2.
    """
    L = int(L)
    if L <= 0:
        return 0, 0, 0
    nb = (L + B - 1) // B
    n_cand = nb - 1
    return nb, n_cand, L - B * n_cand


# ---------------------------------------------------------------------------
# O0: compressed keys (per-block min/max pooling)
# ---------------------------------------------------------------------------

def block_summaries(host_k, block_table, ctx_len, block_size: int, nb_max: int):
    """Coordinate-wise maximum and minimum of the keys of each candidate block.

    Paper §4.2.1 and the "Look-ahead attention" figure: the compressed keys keep,
    per logical block and KV head, the coordinate-wise minimum and maximum of
    the block's keys (Quest-style summaries, two rows per block; §5.2 puts them
    at 1/16 of the KV cache for B = 16). The keys of logical block b of request
    r live in physical page ``block_table[r][b]`` (§4.3, unchanged page tables).
    Only candidate blocks are summarised (reading R4).
    """
    host_k = np.asarray(host_k)
    _, Hkv, B, d = host_k.shape
    assert B == block_size
    R = len(ctx_len)
    kmax = np.full((R, Hkv, nb_max, d), np.nan)
    kmin = np.full((R, Hkv, nb_max, d), np.nan)
    for r in range(R):
        _, n_cand, _ = block_counts(ctx_len[r], B)
        for b in range(n_cand):
            page = int(block_table[r][b])
            keys = bf16_to_f64(host_k[page])          # [Hkv][B][d]
            kmax[r, :, b, :] = keys.max(axis=1)       # over the B tokens
            kmin[r, :, b, :] = keys.min(axis=1)
    return kmax, kmin


def update_summaries(host_k, block_table, prev_ctx_len, ctx_len, block_size: int, kmax, kmin,
                     max_new_blocks: int | None = None):
    """Compressed keys of the blocks completed since ``prev_ctx_len``; in place.

    Paper §5.1 lists compressed-key updates among the native operations: as the
    context grows, each logical block that fills up gets its min/max rows
    (§4.2.1), and earlier rows stay as they are. Here, per request, the rows of
    candidate blocks [n_cand(prev), n_cand(cur)) are written, at most
    ``max_new_blocks`` of them from the first; every other row is untouched.
    Returns the number of rows written per request.
    """
    host_k = np.asarray(host_k)
    _, Hkv, B, d = host_k.shape
    assert B == block_size
    written = np.zeros(len(ctx_len), np.int32)
    for r in range(len(ctx_len)):
        _, lo, _ = block_counts(prev_ctx_len[r], B)
        _, hi, _ = block_counts(ctx_len[r], B)
        if max_new_blocks is not None:
            hi = min(hi, lo + max_new_blocks)
        for b in range(lo, hi):
            keys = bf16_to_f64(host_k[int(block_table[r][b])])   # [Hkv][B][d]
            kmax[r, :, b, :] = keys.max(axis=1)
            kmin[r, :, b, :] = keys.min(axis=1)
            written[r] += 1
    return written


def copy_blocks(src_k, src_v, src_table, dst_k, dst_v, dst_table, prev_ctx_len, ctx_len, block_size: int,
                max_blocks: int | None = None):
    """Copy the logical blocks touched by tokens [prev, cur) between two paged tiers; in place.

    Paper §4.3: once a request's context passes the sparsification threshold,
    its whole KV cache is copied to CPU memory (the full tier) and only the
    selected blocks and the local window stay on the GPU; after that, newly
    written tokens must reach the full tier as well. Both are this copy: with
    prev = 0 every block of the context (the partial local block included); with
    the previous length, the blocks that received new tokens. Pages hold every
    KV head of a block ([Hkv][B][d], §4.3 Head-Token-Dimension order); at most
    ``max_blocks`` blocks are copied per request, from the first. A block whose
    page id in either table is negative (no page) is skipped (reading R24).
    Returns the number of blocks copied per request.
    """
    B = block_size
    copied = np.zeros(len(ctx_len), np.int32)
    for r in range(len(ctx_len)):
        prev, cur = int(prev_ctx_len[r]), int(ctx_len[r])
        if cur <= prev:
            continue
        lo, hi = prev // B, (cur + B - 1) // B
        if max_blocks is not None:
            hi = min(hi, lo + max_blocks)
        for b in range(lo, min(hi, len(src_table[r]))):
            s, t = int(src_table[r][b]), int(dst_table[r][b])
            if s < 0 or t < 0:
                continue
            dst_k[t] = src_k[s]
            dst_v[t] = src_v[s]
            copied[r] += 1
    return copied


# ---------------------------------------------------------------------------
# O1: block importance from the draft queries
# ---------------------------------------------------------------------------

def block_scores(q, kmax, kmin, ctx_len, num_kv_heads: int, block_size: int,
                 first_draft: int = 1, num_draft: int | None = None):
    """Importance of every candidate block for every (request, KV head).

    Paper §4.2.1: the prediction reads only the compressed keys, so every
    logical block of the context gets a rank, separately per KV head, and no
    full key is brought back for it. The importance of a block to one query row is
    the Quest upper bound on that row's dot product with any key of the block
    (reading R1): for every coordinate take the larger of q_d * kmin_d and
    q_d * kmax_d, and add the coordinates up (no 1/sqrt(d): the ranking does
    not depend on it). A KV head serves G query heads (GQA, query head qh
    belongs to KV head qh // G, reading R9) and each of them has D draft rows;
    the block's score for the head is the largest of those G * D row scores
    (reading R2). Only the draft rows score (reading R3); the verify row does
    not. Blocks past the candidates score -inf.
    """
    qf = bf16_to_f64(q)                               # [R][T][Hq][d]
    R, T, Hq, d = qf.shape
    Hkv = num_kv_heads
    G = Hq // Hkv
    if num_draft is None:
        num_draft = T - first_draft
    nb_max = kmax.shape[2]
    scores = np.full((R, Hkv, nb_max), -np.inf)
    for r in range(R):
        _, n_cand, _ = block_counts(ctx_len[r], block_size)
        if n_cand == 0:
            continue
        for h in range(Hkv):
            lo = kmin[r, h, :n_cand, :]               # [n_cand][d]
            hi = kmax[r, h, :n_cand, :]
            best = np.full(n_cand, -np.inf)
            for t in range(first_draft, first_draft + num_draft):
                for g in range(G):
                    row = qf[r, t, h * G + g, :]      # [d]
                    per_coord = np.maximum(row * lo, row * hi)
                    best = np.maximum(best, per_coord.sum(axis=1))
            scores[r, h, :n_cand] = best
    return scores


# ---------------------------------------------------------------------------
# O2: top-K selection
# ---------------------------------------------------------------------------

def select_topk(scores, ctx_len, k: int, block_size: int):
    """The m = min(k, n_cand) best candidate blocks of every (request, KV head).

    Paper §4.2.1/§4.2.2 (top-K prediction per KV head; K = 128 blocks of 16
    tokens is the 2,048-token budget of §5.2). Readings: a larger score wins
    and equal scores go to the lower block id (R7); when the candidates fit
    the budget all of them are taken (R6, §5.2: the budget is the
    sparsification threshold); the result is listed in ascending block id,
    padded with -1, with a count (R8).
    """
    s = np.asarray(scores, dtype=np.float64)
    R, Hkv, _ = s.shape
    sel = np.full((R, Hkv, k), -1, dtype=np.int32)
    cnt = np.zeros((R, Hkv), dtype=np.int32)
    for r in range(R):
        _, n_cand, _ = block_counts(ctx_len[r], block_size)
        m = min(k, n_cand)
        for h in range(Hkv):
            cand = s[r, h, :n_cand]
            assert np.all(np.isfinite(cand)), "candidate scores must be finite"
            ids = np.arange(n_cand)
            order = np.lexsort((ids, -cand))          # score descending, then id ascending
            chosen = np.sort(order[:m])
            sel[r, h, :m] = chosen
            cnt[r, h] = m
    return sel, cnt


def union_selection(sel, sel_count):
    """Per-layer union of the per-head top-K sets (paper §4.4.1, partial transfer).

    For each request, the blocks whose token range at least one KV head
    selected, in ascending block id. Returns (ids [R][Hkv*K], -1 padded;
    count [R]).
    """
    R, H, K = sel.shape
    ids = np.full((R, H * K), -1, np.int32)
    cnt = np.zeros(R, np.int32)
    for r in range(R):
        u = set()
        for h in range(H):
            u.update(int(b) for b in sel[r, h, :sel_count[r, h]])
        u = sorted(u)
        ids[r, :len(u)] = u
        cnt[r] = len(u)
    return ids, cnt


# ---------------------------------------------------------------------------
# O3: delta selection + staging from the host tier
# ---------------------------------------------------------------------------

def stage_blocks(host_k, host_v, block_table, sel, sel_count, slot_map, slot_stamp,
                 step: int, pool_k, pool_v, ctx_len, block_size: int, copy_local: bool = True,
                 scores=None, fetch_cap: int | None = None):
    """Bring the selected blocks into the HBM working set; updates in place.

    Paper §4.2.3 (KV selection): the predicted set is intersected with the
    resident set and resident hits stay where they are, moving no bytes; the
    resident blocks outside the prediction are ranked by the step at which they
    were last selected and the least recently selected ones become eviction
    targets; each admitted missing block is paired with one target, and the
    pairs (CPU source, GPU destination) are the transfer plan. §4.3: a per-KV-
    head table records which CPU logical block each GPU slot holds (the slot
    map); §5.1: the transfer copies block-head entries (K and V of B tokens of
    one head) from the host pages into the resident GPU pages.

    Readings (R14): free slots (-1) are used first in ascending slot order,
    then non-selected residents by (last-selected step, slot); admitted misses
    are paired with the targets in ascending block id; every slot that holds a
    selected block afterwards gets ``step`` as its stamp. ``copy_local`` also
    refreshes slot K of every head with the local block (reading R4: the local
    block is always attended).

    Fetch cap (§4.2.3, §5.5.1): each KV head admits at most ``fetch_cap``
    pairs per step and leaves every other slot as it is, so a selected block
    that is not admitted is simply absent this step while the stale residents
    that were not evicted keep being attended. Reading R15: the admitted misses
    are the ``fetch_cap`` ones with the highest score in ``scores`` [R][Hkv][NB]
    (ties: lowest block id). ``fetch_cap=None`` (or >= K) admits every miss.

    Returns the number of block-head entries moved per (request, KV head),
    excluding the local block.
    """
    B = block_size
    R, Hkv, K = slot_map.shape
    moved = np.zeros((R, Hkv), dtype=np.int32)
    for r in range(R):
        nb, _, _ = block_counts(ctx_len[r], B)
        for h in range(Hkv):
            m = int(sel_count[r, h])
            chosen = [int(b) for b in sel[r, h, :m]]
            chosen_set = set(chosen)
            resident = {int(slot_map[r, h, s]) for s in range(K) if slot_map[r, h, s] >= 0}
            misses = [b for b in chosen if b not in resident]
            free = [s for s in range(K) if slot_map[r, h, s] < 0]
            stale = sorted((int(slot_stamp[r, h, s]), s) for s in range(K)
                           if slot_map[r, h, s] >= 0 and int(slot_map[r, h, s]) not in chosen_set)
            victims = free + [s for _, s in stale]
            assert len(victims) >= len(misses)
            assert fetch_cap is None or fetch_cap >= 1
            if fetch_cap is not None and len(misses) > fetch_cap:
                by_score = sorted(misses, key=lambda b: (-float(scores[r, h, b]), b))
                misses = sorted(by_score[:fetch_cap])
            for b, s in zip(misses, victims):
                slot_map[r, h, s] = b
                page = int(block_table[r][b])
                pool_k[r, s, h] = host_k[page, h]
                pool_v[r, s, h] = host_v[page, h]
            for s in range(K):
                if int(slot_map[r, h, s]) in chosen_set:
                    slot_stamp[r, h, s] = step
            moved[r, h] = len(misses)
            if copy_local and nb > 0:
                page = int(block_table[r][nb - 1])
                pool_k[r, K, h] = host_k[page, h]
                pool_v[r, K, h] = host_v[page, h]
    return moved


# ---------------------------------------------------------------------------
# O4: attention over the resident working set
# ---------------------------------------------------------------------------

def _softmax_attend(qrows, keys, vals, scale):
    """softmax(scale * q . k) weighted sum of v, plus log-sum-exp, per query row."""
    z = scale * (qrows @ keys.T)                      # [rows][S]
    zmax = z.max(axis=1, keepdims=True)
    e = np.exp(z - zmax)
    den = e.sum(axis=1, keepdims=True)
    out = (e / den) @ vals
    lse = zmax[:, 0] + np.log(den[:, 0])
    return out, lse


def sparse_attend(q, pool_k, pool_v, slot_map, ctx_len, block_size: int, scale: float | None = None):
    """Block-sparse GQA decode attention over the staged slots and the local block.

    Paper §4.2.1: the normal and the draft queries are stacked and attend the
    same resident KV working set in one call, which returns both outputs.
    §5.2: a head attends its K selected blocks plus the active local block
    (129 blocks = 2,064 tokens at K = 128, B = 16). The attended set of KV head
    h is the B tokens of every slot whose map entry is not -1, plus the first
    local_len tokens of slot K (readings R4, R10: no mask among the T rows).
    Scale 1/sqrt(d), no sinks or soft-capping (R11). An empty set gives a zero
    output and lse = -inf.
    """
    qf = bf16_to_f64(q)
    R, T, Hq, d = qf.shape
    _, Kp1, Hkv, B, _ = pool_k.shape
    K = Kp1 - 1
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((R, T, Hq, d))
    lse = np.full((R, T, Hq), -np.inf)
    for r in range(R):
        _, _, local_len = block_counts(ctx_len[r], B)
        for h in range(Hkv):
            slots = [s for s in range(K) if slot_map[r, h, s] >= 0]
            kparts = [bf16_to_f64(pool_k[r, s, h]) for s in slots]
            vparts = [bf16_to_f64(pool_v[r, s, h]) for s in slots]
            if local_len > 0:
                kparts.append(bf16_to_f64(pool_k[r, K, h, :local_len]))
                vparts.append(bf16_to_f64(pool_v[r, K, h, :local_len]))
            if not kparts:
                continue
            keys = np.concatenate(kparts)             # [S][d]
            vals = np.concatenate(vparts)
            qrows = qf[r, :, h * G:(h + 1) * G, :].reshape(T * G, d)
            o, l = _softmax_attend(qrows, keys, vals, scale)
            out[r, :, h * G:(h + 1) * G, :] = o.reshape(T, G, d)
            lse[r, :, h * G:(h + 1) * G] = l.reshape(T, G)
    return out, lse


def dense_attend(q, host_k, host_v, block_table, ctx_len, block_size: int, scale: float | None = None):
    """Full-context GQA decode attention over the paged host KV (the dense reference)."""
    qf = bf16_to_f64(q)
    R, T, Hq, d = qf.shape
    Hkv = host_k.shape[1]
    G = Hq // Hkv
    B = block_size
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((R, T, Hq, d))
    lse = np.full((R, T, Hq), -np.inf)
    for r in range(R):
        L = int(ctx_len[r])
        if L <= 0:
            continue
        nb = (L + B - 1) // B
        pages = [int(p) for p in block_table[r][:nb]]
        for h in range(Hkv):
            keys = np.concatenate([bf16_to_f64(host_k[p, h]) for p in pages])[:L]
            vals = np.concatenate([bf16_to_f64(host_v[p, h]) for p in pages])[:L]
            qrows = qf[r, :, h * G:(h + 1) * G, :].reshape(T * G, d)
            o, l = _softmax_attend(qrows, keys, vals, scale)
            out[r, :, h * G:(h + 1) * G, :] = o.reshape(T, G, d)
            lse[r, :, h * G:(h + 1) * G] = l.reshape(T, G)
    return out, lse
