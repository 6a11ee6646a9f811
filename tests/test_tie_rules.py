"""The comparison rules the GPU parity tests apply at near ties (CPU only): a swapped pair at the selection
cut, and a different admission at the fetch cap's cut, are accepted only within the tie tolerance, and the
admission rule hands the oracle the scores that make it follow the GPU's choice."""
import numpy as np
import pytest

from oracle import oasis_oracle as O
from tests.gpu_util import TIE_REL, adjudicate_capped, selection_diff


def _case():
    # one request, one head, K = 4 slots, 10 candidate blocks; blocks 0-3 resident
    s = np.array([[[9.0, 8.0, 1.0, 0.5, 7.0, 6.0, 5.0, 5.0 + 1e-4, 2.0, 1.5]]])
    smap = np.array([[[0, 1, 2, 3]]], np.int32)
    ctx = np.array([16 * 11], np.int32)
    sel, cnt = O.select_topk(s, ctx, 4, 16)
    return s, smap, ctx, sel, cnt


def test_selection_swap_within_tolerance_only():
    s = np.array([[[3.0, 2.0, 1.0 + 1e-5, 1.0, 0.0]]])
    ctx = np.array([16 * 6], np.int32)
    sel, cnt = O.select_topk(s, ctx, 3, 16)               # blocks 0, 1, 2
    assert sel[0, 0].tolist() == [0, 1, 2]
    assert selection_diff(np.array([[[0, 1, 3]]]), cnt, sel, cnt, s) == [(0, 0)]  # 2 <-> 3 within 1e-3
    with pytest.raises(AssertionError):
        selection_diff(np.array([[[0, 2, 3]]]), cnt, sel, cnt, s)               # drops block 1 (2.0)


def test_admission_tie_at_the_cap():
    s, smap, ctx, _, _ = _case()
    # selection: blocks 0, 4, 6, 7; misses 4, 6, 7 against residents 0-3
    sel = np.array([[[0, 4, 6, 7]]], np.int32)
    cnt = np.array([[4]], np.int32)
    scores = s.copy()
    scores[0, 0, [1, 2, 3, 5, 8, 9]] = -1.0              # make that selection the oracle's own top 4
    sel_o, cnt_o = O.select_topk(scores, ctx, 4, 16)
    assert sel_o[0, 0].tolist() == [0, 4, 6, 7]
    cap = 2
    # the oracle admits 4 (7.0) and 7 (5.0001); 6 (5.0) is within 1e-3 of the cut 5.0001, and the GPU
    # admitted 4 and 6 (victims: slots 1 and 2)
    after_gpu = np.array([[[0, 4, 6, 3]]], np.int32)
    use = adjudicate_capped(sel, cnt, smap, after_gpu, scores, sel_o, cnt_o, cap)
    smap_o = smap.copy()
    stamp = np.zeros_like(smap)
    hk = np.zeros((16, 1, 16, 4), np.uint16)
    pk = np.zeros((1, 5, 1, 16, 4), np.uint16)
    table = np.arange(11, dtype=np.int32)[None]
    O.stage_blocks(hk, hk, table, sel, cnt, smap_o, stamp, 1, pk, pk.copy(), ctx, 16, scores=use, fetch_cap=cap)
    assert sorted(set(smap_o[0, 0].tolist()) - {0, 1, 2, 3}) == [4, 6]
    # a GPU admission of a block far below the cut is refused
    scores2 = scores.copy()
    scores2[0, 0, 6] = 4.0                                 # 6 now 1.0001 below the cut
    with pytest.raises(AssertionError):
        adjudicate_capped(sel, cnt, smap, after_gpu, scores2, sel_o, cnt_o, cap)
    assert TIE_REL == 1e-3
