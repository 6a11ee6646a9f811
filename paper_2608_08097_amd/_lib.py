"""ctypes binding of liboasis.so: the C ABI declared in include/oasis.h, one
Python function per entry point, with the same names.

Marshalling only: the functions check that tensors sit where the C ABI expects
them (device or pinned host), have the right dtype and are contiguous, then
pass raw pointers and the current HIP stream. Every step of the path runs in
the library's kernels; there is no fallback. If the library is not built, the
first call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liboasis.so")

STATUS = {0: "OASIS_OK", 1: "OASIS_ERR_INVALID_ARG", 2: "OASIS_ERR_UNSUPPORTED",
          3: "OASIS_ERR_HIP", 4: "OASIS_ERR_WORKSPACE"}

EXPORTS = (
    "oasis_last_error", "oasis_abi_version", "oasis_build_summaries", "oasis_update_summaries",
    "oasis_copy_blocks", "oasis_score_blocks", "oasis_score_select",
    "oasis_select_topk", "oasis_stage_blocks",
    "oasis_attn_workspace_bytes", "oasis_sparse_decode_attn", "oasis_sparse_decode_attn_noalloc",
    "oasis_union_selection",
    "oasis_pipeline_create", "oasis_pipeline_set_layer", "oasis_pipeline_set_local_source",
    "oasis_pipeline_set_plan_stream", "oasis_pipeline_set_fused_prediction", "oasis_pipeline_step",
    "oasis_pipeline_join", "oasis_pipeline_check", "oasis_pipeline_set_wait_limit",
    "oasis_pipeline_set_prediction_order",
    "oasis_pipeline_destroy", "oasis_pipeline_profile_begin", "oasis_pipeline_profile_end",
)


class OasisError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: {STATUS.get(status, status)}: {msg}")
        self.status = status


class OasisDims(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("max_blocks", ctypes.c_int32)]

    def __repr__(self):
        return "OasisDims(" + ", ".join(f"{n}={getattr(self, n)}" for n, _ in self._fields_) + ")"


class OasisLayerBuffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("kmax", "kmin", "scores", "sel", "sel_count", "slot_map",
                                               "slot_stamp", "pool_k", "pool_v", "moved", "out", "lse",
                                               "workspace")] + [("workspace_bytes", ctypes.c_size_t)]


def dims(num_reqs, num_q_heads, num_kv_heads, head_dim, block_size, max_blocks) -> OasisDims:
    return OasisDims(int(num_reqs), int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size),
                     int(max_blocks))


_lib = None
ABI_VERSION = 7  # OASIS_ABI_VERSION of include/oasis.h

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_DIMS = ctypes.POINTER(OasisDims)


def lib() -> ctypes.CDLL:
    """Load liboasis.so (once); raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "or python -m paper_2608_08097_amd.build_lib")
        L = ctypes.CDLL(LIB_PATH)
        L.oasis_last_error.restype = ctypes.c_char_p
        L.oasis_last_error.argtypes = []
        L.oasis_abi_version.restype = _I32
        L.oasis_abi_version.argtypes = []
        if L.oasis_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {L.oasis_abi_version()}, this binding expects "
                               f"{ABI_VERSION}: rebuild it")
        L.oasis_build_summaries.restype = _I32
        L.oasis_build_summaries.argtypes = [_DIMS, _P, _I64, _P, _P, _P, _P, _P]
        L.oasis_update_summaries.restype = _I32
        L.oasis_update_summaries.argtypes = [_DIMS, _P, _I64, _P, _P, _P, _I32, _P, _P, _P]
        L.oasis_copy_blocks.restype = _I32
        L.oasis_copy_blocks.argtypes = [_DIMS, _P, _P, _I64, _P, _P, _P, _I64, _P, _P, _P, _I32, _P]
        L.oasis_score_blocks.restype = _I32
        L.oasis_score_blocks.argtypes = [_DIMS, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P]
        L.oasis_select_topk.restype = _I32
        L.oasis_select_topk.argtypes = [_DIMS, _P, _P, _I32, _P, _P, _P]
        L.oasis_stage_blocks.restype = _I32
        L.oasis_stage_blocks.argtypes = [_DIMS, _P, _P, _I64, _P, _P, _P, _P, _P, _I32, _P, _P, _I32, _I32, _I32,
                                         _P, _P, _P, _P]
        L.oasis_score_select.restype = _I32
        L.oasis_score_select.argtypes = [_DIMS, _P, _I32, _I32, _I32, _P, _P, _P, _I32, _P, _P, _P, _P]
        L.oasis_union_selection.restype = _I32
        L.oasis_union_selection.argtypes = [_DIMS, _P, _P, _I32, _P, _P, _P]
        L.oasis_attn_workspace_bytes.restype = _SZ
        L.oasis_attn_workspace_bytes.argtypes = [_DIMS, _I32, _I32]
        L.oasis_sparse_decode_attn.restype = _I32
        L.oasis_sparse_decode_attn.argtypes = [_DIMS, _P, _I32, _P, _P, _P, _I32, _P, ctypes.c_float, _P, _P,
                                               _P, _SZ, _P]
        L.oasis_sparse_decode_attn_noalloc.restype = _I32
        L.oasis_sparse_decode_attn_noalloc.argtypes = [_DIMS, _P, _I32, _P, _P, _P, _I32, _P, ctypes.c_float, _P,
                                                       _P, _P]
        L.oasis_pipeline_create.restype = _I32
        L.oasis_pipeline_create.argtypes = [_DIMS, _I32, _I32, _I32, _I32, _I32, ctypes.c_float, _P, _P, _I64, _P,
                                            _I32, _P, _P, ctypes.POINTER(_P)]
        L.oasis_pipeline_set_fused_prediction.restype = _I32
        L.oasis_pipeline_set_fused_prediction.argtypes = [_P, _I32]
        L.oasis_pipeline_set_layer.restype = _I32
        L.oasis_pipeline_set_layer.argtypes = [_P, _I32, ctypes.POINTER(OasisLayerBuffers)]
        L.oasis_pipeline_set_local_source.restype = _I32
        L.oasis_pipeline_set_local_source.argtypes = [_P, _P, _P, _I64, _P]
        L.oasis_pipeline_set_plan_stream.restype = _I32
        L.oasis_pipeline_set_plan_stream.argtypes = [_P, _I32]
        L.oasis_pipeline_step.restype = _I32
        L.oasis_pipeline_step.argtypes = [_P, _I32, _P, _P, _P, _I32, _I32, _I32, _P, _P]
        L.oasis_pipeline_join.restype = _I32
        L.oasis_pipeline_join.argtypes = [_P, _P]
        L.oasis_pipeline_check.restype = _I32
        L.oasis_pipeline_check.argtypes = [_P]
        L.oasis_pipeline_set_prediction_order.restype = _I32
        L.oasis_pipeline_set_prediction_order.argtypes = [_P, _I32]
        L.oasis_pipeline_set_wait_limit.restype = _I32
        L.oasis_pipeline_set_wait_limit.argtypes = [_P, ctypes.c_uint32]
        L.oasis_pipeline_destroy.restype = None
        L.oasis_pipeline_destroy.argtypes = [_P]
        L.oasis_pipeline_profile_begin.restype = _I32
        L.oasis_pipeline_profile_begin.argtypes = [_P, _I32]
        L.oasis_pipeline_profile_end.restype = _I32
        L.oasis_pipeline_profile_end.argtypes = [_P, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float),
                                                   ctypes.POINTER(_I32)]
        _lib = L
    return _lib


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise OasisError(fn, status, lib().oasis_last_error().decode())


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev(t: torch.Tensor | None, name: str, dtypes, nullable: bool = False):
    if t is None:
        if nullable:
            return None
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _host_or_dev(t: torch.Tensor, name: str, dtypes):
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if not t.is_cuda and not t.is_pinned():
        raise ValueError(f"{name} must be pinned host memory or a device tensor")
    return t.data_ptr()


def _need(t: torch.Tensor | None, numel: int, name: str) -> None:
    """Element count the C ABI will address for this argument (no kernel may go past it)."""
    if t is not None and t.numel() != numel:
        raise ValueError(f"{name}: {t.numel()} elements, {numel} expected")


_BF16 = (torch.bfloat16, torch.uint16, torch.int16)
_I32T = (torch.int32,)
_F32 = (torch.float32,)


def oasis_abi_version() -> int:
    return int(lib().oasis_abi_version())


def oasis_last_error() -> str:
    return lib().oasis_last_error().decode()


def oasis_build_summaries(d: OasisDims, k_pages, block_table, ctx_len, kmax, kmin, stream=None) -> None:
    R, H, NB, D = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim
    _need(k_pages, k_pages.shape[0] * H * d.block_size * D, "k_pages")
    _need(block_table, R * NB, "block_table")
    _need(ctx_len, R, "ctx_len")
    _need(kmax, R * H * NB * D, "kmax")
    _need(kmin, R * H * NB * D, "kmin")
    _check("oasis_build_summaries", lib().oasis_build_summaries(
        ctypes.byref(d), _host_or_dev(k_pages, "k_pages", _BF16), int(k_pages.shape[0]),
        _dev(block_table, "block_table", _I32T), _dev(ctx_len, "ctx_len", _I32T),
        _dev(kmax, "kmax", _BF16), _dev(kmin, "kmin", _BF16), _stream(stream)))


def oasis_update_summaries(d: OasisDims, k_pages, block_table, prev_ctx_len, ctx_len, max_new_blocks: int,
                           kmax, kmin, stream=None) -> None:
    R, H, NB, D = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim
    _need(k_pages, k_pages.shape[0] * H * d.block_size * D, "k_pages")
    _need(block_table, R * NB, "block_table")
    _need(prev_ctx_len, R, "prev_ctx_len")
    _need(ctx_len, R, "ctx_len")
    _need(kmax, R * H * NB * D, "kmax")
    _need(kmin, R * H * NB * D, "kmin")
    _check("oasis_update_summaries", lib().oasis_update_summaries(
        ctypes.byref(d), _host_or_dev(k_pages, "k_pages", _BF16), int(k_pages.shape[0]),
        _dev(block_table, "block_table", _I32T), _dev(prev_ctx_len, "prev_ctx_len", _I32T),
        _dev(ctx_len, "ctx_len", _I32T), int(max_new_blocks), _dev(kmax, "kmax", _BF16), _dev(kmin, "kmin", _BF16),
        _stream(stream)))


def oasis_copy_blocks(d: OasisDims, src_k, src_v, src_block_table, dst_k, dst_v, dst_block_table, prev_ctx_len,
                      ctx_len, max_blocks: int, stream=None) -> None:
    R, H, NB, D, B = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim, d.block_size
    for t, name in ((src_k, "src_k"), (src_v, "src_v"), (dst_k, "dst_k"), (dst_v, "dst_v")):
        if t.dim() < 1 or t.numel() % (H * B * D):
            raise ValueError(f"{name}: not whole pages of [Hkv][B][d]")
    if src_k.shape != src_v.shape or dst_k.shape != dst_v.shape:
        raise ValueError("K and V tiers differ in shape")
    _need(src_block_table, R * NB, "src_block_table")
    _need(dst_block_table, R * NB, "dst_block_table")
    _need(prev_ctx_len, R, "prev_ctx_len")
    _need(ctx_len, R, "ctx_len")
    _check("oasis_copy_blocks", lib().oasis_copy_blocks(
        ctypes.byref(d), _host_or_dev(src_k, "src_k", _BF16), _host_or_dev(src_v, "src_v", _BF16),
        src_k.numel() // (H * B * D), _dev(src_block_table, "src_block_table", _I32T),
        _host_or_dev(dst_k, "dst_k", _BF16), _host_or_dev(dst_v, "dst_v", _BF16), dst_k.numel() // (H * B * D),
        _dev(dst_block_table, "dst_block_table", _I32T), _dev(prev_ctx_len, "prev_ctx_len", _I32T, nullable=True),
        _dev(ctx_len, "ctx_len", _I32T), int(max_blocks), _stream(stream)))


def oasis_score_blocks(d: OasisDims, q, num_q_tokens: int, first_draft: int, num_draft: int,
                       kmax, kmin, ctx_len, scores, stream=None) -> None:
    R, H, NB, D = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim
    _need(q, R * num_q_tokens * d.num_q_heads * D, "q")
    _need(kmax, R * H * NB * D, "kmax")
    _need(kmin, R * H * NB * D, "kmin")
    _need(ctx_len, R, "ctx_len")
    _need(scores, R * H * NB, "scores")
    _check("oasis_score_blocks", lib().oasis_score_blocks(
        ctypes.byref(d), _dev(q, "q", _BF16), int(num_q_tokens), int(first_draft), int(num_draft),
        _dev(kmax, "kmax", _BF16), _dev(kmin, "kmin", _BF16), _dev(ctx_len, "ctx_len", _I32T),
        _dev(scores, "scores", _F32), _stream(stream)))


def oasis_select_topk(d: OasisDims, scores, ctx_len, k: int, sel, sel_count, stream=None) -> None:
    R, H = d.num_reqs, d.num_kv_heads
    _need(scores, R * H * d.max_blocks, "scores")
    _need(ctx_len, R, "ctx_len")
    _need(sel, R * H * k, "sel")
    _need(sel_count, R * H, "sel_count")
    _check("oasis_select_topk", lib().oasis_select_topk(
        ctypes.byref(d), _dev(scores, "scores", _F32), _dev(ctx_len, "ctx_len", _I32T), int(k),
        _dev(sel, "sel", _I32T), _dev(sel_count, "sel_count", _I32T), _stream(stream)))


def oasis_score_select(d: OasisDims, q, num_q_tokens: int, first_draft: int, num_draft: int, kmax, kmin, ctx_len,
                       k: int, scores, sel, sel_count, stream=None) -> None:
    """Scores and top-K in one kernel (the same results as oasis_score_blocks + oasis_select_topk)."""
    R, H, NB, D = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim
    _need(q, R * num_q_tokens * d.num_q_heads * D, "q")
    _need(kmax, R * H * NB * D, "kmax")
    _need(kmin, R * H * NB * D, "kmin")
    _need(ctx_len, R, "ctx_len")
    _need(scores, R * H * NB, "scores")
    _need(sel, R * H * k, "sel")
    _need(sel_count, R * H, "sel_count")
    _check("oasis_score_select", lib().oasis_score_select(
        ctypes.byref(d), _dev(q, "q", _BF16), int(num_q_tokens), int(first_draft), int(num_draft),
        _dev(kmax, "kmax", _BF16), _dev(kmin, "kmin", _BF16), _dev(ctx_len, "ctx_len", _I32T), int(k),
        _dev(scores, "scores", _F32), _dev(sel, "sel", _I32T), _dev(sel_count, "sel_count", _I32T),
        _stream(stream)))


def oasis_stage_blocks(d: OasisDims, host_k, host_v, host_block_table, ctx_len, sel, sel_count, scores, k: int,
                       slot_map, slot_stamp, step: int, fetch_cap: int, copy_local: bool, pool_k, pool_v,
                       moved, stream=None) -> None:
    if host_k.shape != host_v.shape:
        raise ValueError("host_k and host_v differ in shape")
    R, H, B, D = d.num_reqs, d.num_kv_heads, d.block_size, d.head_dim
    _need(host_k, host_k.shape[0] * H * B * D, "host_k")
    _need(host_block_table, R * d.max_blocks, "host_block_table")
    _need(ctx_len, R, "ctx_len")
    for t, n in ((sel, "sel"), (slot_map, "slot_map"), (slot_stamp, "slot_stamp")):
        _need(t, R * H * k, n)
    _need(sel_count, R * H, "sel_count")
    _need(scores, R * H * d.max_blocks, "scores")
    _need(moved, R * H, "moved")
    _need(pool_k, R * (k + 1) * H * B * D, "pool_k")
    _need(pool_v, R * (k + 1) * H * B * D, "pool_v")
    _check("oasis_stage_blocks", lib().oasis_stage_blocks(
        ctypes.byref(d), _host_or_dev(host_k, "host_k", _BF16), _host_or_dev(host_v, "host_v", _BF16),
        int(host_k.shape[0]), _dev(host_block_table, "host_block_table", _I32T), _dev(ctx_len, "ctx_len", _I32T),
        _dev(sel, "sel", _I32T, nullable=True), _dev(sel_count, "sel_count", _I32T, nullable=True),
        _dev(scores, "scores", (torch.float32,), nullable=True), int(k),
        _dev(slot_map, "slot_map", _I32T, nullable=True), _dev(slot_stamp, "slot_stamp", _I32T, nullable=True),
        int(step), int(fetch_cap), 1 if copy_local else 0, _dev(pool_k, "pool_k", _BF16),
        _dev(pool_v, "pool_v", _BF16), _dev(moved, "moved", _I32T, nullable=True), _stream(stream)))


def oasis_union_selection(d: OasisDims, sel, sel_count, k: int, union_ids, union_count, stream=None) -> None:
    R, H = d.num_reqs, d.num_kv_heads
    _need(sel, R * H * k, "sel")
    _need(sel_count, R * H, "sel_count")
    _need(union_ids, R * H * k, "union_ids")
    _need(union_count, R, "union_count")
    _check("oasis_union_selection", lib().oasis_union_selection(
        ctypes.byref(d), _dev(sel, "sel", _I32T), _dev(sel_count, "sel_count", _I32T), int(k),
        _dev(union_ids, "union_ids", _I32T), _dev(union_count, "union_count", _I32T), _stream(stream)))


def oasis_attn_workspace_bytes(d: OasisDims, num_q_tokens: int, k_slots: int) -> int:
    return int(lib().oasis_attn_workspace_bytes(ctypes.byref(d), int(num_q_tokens), int(k_slots)))


def oasis_sparse_decode_attn(d: OasisDims, q, num_q_tokens: int, pool_k, pool_v, slot_map, k_slots: int,
                             ctx_len, scale: float | None, out, lse, workspace, stream=None) -> None:
    if scale is None:
        scale = 1.0 / math.sqrt(d.head_dim)
    R, H, B, D = d.num_reqs, d.num_kv_heads, d.block_size, d.head_dim
    _need(q, R * num_q_tokens * d.num_q_heads * D, "q")
    _need(out, R * num_q_tokens * d.num_q_heads * D, "out")
    _need(lse, R * num_q_tokens * d.num_q_heads, "lse")
    _need(pool_k, R * (k_slots + 1) * H * B * D, "pool_k")
    _need(pool_v, R * (k_slots + 1) * H * B * D, "pool_v")
    _need(slot_map, R * H * k_slots, "slot_map")
    _need(ctx_len, R, "ctx_len")
    _check("oasis_sparse_decode_attn", lib().oasis_sparse_decode_attn(
        ctypes.byref(d), _dev(q, "q", _BF16), int(num_q_tokens), _dev(pool_k, "pool_k", _BF16),
        _dev(pool_v, "pool_v", _BF16), _dev(slot_map, "slot_map", _I32T, nullable=k_slots == 0), int(k_slots),
        _dev(ctx_len, "ctx_len", _I32T), float(scale), _dev(out, "out", _BF16),
        _dev(lse, "lse", _F32, nullable=True),
        _dev(workspace, "workspace", (torch.uint8,), nullable=workspace is None or workspace.numel() == 0),
        int(workspace.numel()) if workspace is not None else 0, _stream(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20  # OASIS_NOALLOC_SCRATCH_BYTES of include/oasis.h


def oasis_sparse_decode_attn_noalloc(d: OasisDims, q, num_q_tokens: int, pool_k, pool_v, slot_map, k_slots: int,
                                     ctx_len, scale: float | None, out, lse, stream=None) -> None:
    """oasis_sparse_decode_attn with the library's own scratch instead of a workspace (allocates nothing)."""
    if scale is None:
        scale = 1.0 / math.sqrt(d.head_dim)
    R, H, B, D = d.num_reqs, d.num_kv_heads, d.block_size, d.head_dim
    _need(q, R * num_q_tokens * d.num_q_heads * D, "q")
    _need(out, R * num_q_tokens * d.num_q_heads * D, "out")
    _need(lse, R * num_q_tokens * d.num_q_heads, "lse")
    _need(pool_k, R * (k_slots + 1) * H * B * D, "pool_k")
    _need(pool_v, R * (k_slots + 1) * H * B * D, "pool_v")
    _need(slot_map, R * H * k_slots, "slot_map")
    _need(ctx_len, R, "ctx_len")
    _check("oasis_sparse_decode_attn_noalloc", lib().oasis_sparse_decode_attn_noalloc(
        ctypes.byref(d), _dev(q, "q", _BF16), int(num_q_tokens), _dev(pool_k, "pool_k", _BF16),
        _dev(pool_v, "pool_v", _BF16), _dev(slot_map, "slot_map", _I32T, nullable=k_slots == 0), int(k_slots),
        _dev(ctx_len, "ctx_len", _I32T), float(scale), _dev(out, "out", _BF16),
        _dev(lse, "lse", _F32, nullable=True), _stream(stream)))


# --- native step issuer --------------------------------------------------------

_PIPE_SIZES: dict[int, tuple[int, int, int]] = {}  # handle -> element counts of q, ctx_len, moved

def oasis_pipeline_create(d: OasisDims, num_q_tokens: int, first_draft: int, num_draft: int, k: int,
                          fetch_cap: int, scale: float | None, host_k, host_v, host_block_table, max_layers: int,
                          pred_stream=None, xfer_stream=None) -> int:
    """Returns the pipeline handle (an address); release it with oasis_pipeline_destroy."""
    if scale is None:
        scale = 1.0 / math.sqrt(d.head_dim)
    if host_k.shape != host_v.shape:
        raise ValueError("host_k and host_v differ in shape")
    _need(host_k, host_k.shape[0] * d.num_kv_heads * d.block_size * d.head_dim, "host_k")
    _need(host_block_table, d.num_reqs * d.max_blocks, "host_block_table")
    h = ctypes.c_void_p()
    _check("oasis_pipeline_create", lib().oasis_pipeline_create(
        ctypes.byref(d), int(num_q_tokens), int(first_draft), int(num_draft), int(k), int(fetch_cap), float(scale),
        _host_or_dev(host_k, "host_k", _BF16), _host_or_dev(host_v, "host_v", _BF16), int(host_k.shape[0]),
        _dev(host_block_table, "host_block_table", _I32T),
        int(max_layers), None if pred_stream is None else _stream(pred_stream),
        None if xfer_stream is None else _stream(xfer_stream), ctypes.byref(h)))
    _PIPE_SIZES[h.value] = (d.num_reqs * int(num_q_tokens) * d.num_q_heads * d.head_dim, d.num_reqs,
                            d.num_reqs * d.num_kv_heads)
    return h.value


PLAN_ON_TRANSFER = 0    # OASIS_PLAN_ON_TRANSFER
PLAN_ON_PREDICTION = 1  # OASIS_PLAN_ON_PREDICTION


def oasis_pipeline_set_plan_stream(handle: int, where: int) -> None:
    """Plan each step's transfer on the transfer stream (PLAN_ON_TRANSFER) or in the top-K kernel
    on the prediction stream (PLAN_ON_PREDICTION)."""
    _check("oasis_pipeline_set_plan_stream", lib().oasis_pipeline_set_plan_stream(handle, int(where)))


FUSED_PREDICTION_AUTO = 0  # OASIS_FUSED_PREDICTION_AUTO
FUSED_PREDICTION_OFF = 1   # OASIS_FUSED_PREDICTION_OFF
FUSED_PREDICTION_ON = 2    # OASIS_FUSED_PREDICTION_ON


def oasis_pipeline_set_fused_prediction(handle: int, mode: int) -> None:
    """Score and select (and plan) in one kernel per step: AUTO (many short rows), OFF or ON."""
    _check("oasis_pipeline_set_fused_prediction", lib().oasis_pipeline_set_fused_prediction(handle, int(mode)))


def oasis_pipeline_set_local_source(handle: int, d: OasisDims, k_pages, v_pages, block_table) -> None:
    """Pages a growing step refreshes the local block from (all None: the host tier)."""
    if k_pages is None and v_pages is None and block_table is None:
        _check("oasis_pipeline_set_local_source", lib().oasis_pipeline_set_local_source(handle, None, None, 0, None))
        return
    if k_pages is None or v_pages is None or block_table is None:
        raise ValueError("k_pages, v_pages and block_table must all be given or all be None")
    if k_pages.shape != v_pages.shape:
        raise ValueError("k_pages and v_pages differ in shape")
    _need(k_pages, k_pages.shape[0] * d.num_kv_heads * d.block_size * d.head_dim, "k_pages")
    _need(block_table, d.num_reqs * d.max_blocks, "block_table")
    _check("oasis_pipeline_set_local_source", lib().oasis_pipeline_set_local_source(
        handle, _host_or_dev(k_pages, "k_pages", _BF16), _host_or_dev(v_pages, "v_pages", _BF16),
        int(k_pages.shape[0]), _dev(block_table, "block_table", _I32T)))


def oasis_pipeline_set_layer(handle: int, layer: int, d: OasisDims, num_q_tokens: int, k: int, kmax, kmin, scores,
                             sel, sel_count, slot_map, slot_stamp, pool_k, pool_v, moved, out, lse,
                             workspace) -> None:
    R, H, NB, D, B = d.num_reqs, d.num_kv_heads, d.max_blocks, d.head_dim, d.block_size
    T, Hq = int(num_q_tokens), d.num_q_heads
    for t, n, name in ((kmax, R * H * NB * D, "kmax"), (kmin, R * H * NB * D, "kmin"), (scores, R * H * NB, "scores"),
                       (sel, R * H * k, "sel"), (sel_count, R * H, "sel_count"), (slot_map, R * H * k, "slot_map"),
                       (slot_stamp, R * H * k, "slot_stamp"), (pool_k, R * (k + 1) * H * B * D, "pool_k"),
                       (pool_v, R * (k + 1) * H * B * D, "pool_v"), (moved, R * H, "moved"),
                       (out, R * T * Hq * D, "out"), (lse, R * T * Hq, "lse")):
        _need(t, n, name)
    b = OasisLayerBuffers(
        _dev(kmax, "kmax", _BF16), _dev(kmin, "kmin", _BF16), _dev(scores, "scores", _F32),
        _dev(sel, "sel", _I32T), _dev(sel_count, "sel_count", _I32T), _dev(slot_map, "slot_map", _I32T),
        _dev(slot_stamp, "slot_stamp", _I32T), _dev(pool_k, "pool_k", _BF16), _dev(pool_v, "pool_v", _BF16),
        _dev(moved, "moved", _I32T, nullable=True), _dev(out, "out", _BF16), _dev(lse, "lse", _F32, nullable=True),
        _dev(workspace, "workspace", (torch.uint8,), nullable=True),
        0 if workspace is None else workspace.numel() * workspace.element_size())
    _check("oasis_pipeline_set_layer", lib().oasis_pipeline_set_layer(handle, int(layer), ctypes.byref(b)))


def oasis_pipeline_step(handle: int, layer: int, q, ctx_len, step: int, growing: bool, moved=None,
                        stream=None, prev_ctx_len=None, max_new_blocks: int = 1) -> None:
    """One layer's pipelined step (q, ctx_len, prev_ctx_len, moved: device tensors of the pipeline's
    shapes); with prev_ctx_len the compressed keys of newly completed blocks are added first."""
    nq, nr, nm = _PIPE_SIZES[handle]
    _need(q, nq, "q")
    _need(ctx_len, nr, "ctx_len")
    _need(prev_ctx_len, nr, "prev_ctx_len")
    _need(moved, nm, "moved")
    _check("oasis_pipeline_step", lib().oasis_pipeline_step(
        handle, int(layer), _dev(q, "q", _BF16), _dev(ctx_len, "ctx_len", _I32T),
        _dev(prev_ctx_len, "prev_ctx_len", _I32T, nullable=True), int(max_new_blocks), int(step),
        1 if growing else 0, _dev(moved, "moved", _I32T, nullable=True), _stream(stream)))


def oasis_pipeline_join(handle: int, stream=None) -> None:
    _check("oasis_pipeline_join", lib().oasis_pipeline_join(handle, _stream(stream)))


def oasis_pipeline_check(handle: int) -> None:
    """Synchronize the device; raise if a transfer of the pipeline gave up waiting for its prediction."""
    _check("oasis_pipeline_check", lib().oasis_pipeline_check(handle))


PREDICT_AUTO = 0              # OASIS_PREDICT_AUTO
PREDICT_BESIDE_ATTENTION = 1  # OASIS_PREDICT_BESIDE_ATTENTION
PREDICT_AFTER_ATTENTION = 2   # OASIS_PREDICT_AFTER_ATTENTION


def oasis_pipeline_set_prediction_order(handle: int, order: int) -> None:
    """Start each step's prediction beside or after its attention (PREDICT_AUTO: by the pair count)."""
    _check("oasis_pipeline_set_prediction_order", lib().oasis_pipeline_set_prediction_order(handle, int(order)))


def oasis_pipeline_set_wait_limit(handle: int, polls: int) -> None:
    """Bound (in polls, about 1 us each) of the staging kernel's wait for its prediction."""
    _check("oasis_pipeline_set_wait_limit", lib().oasis_pipeline_set_wait_limit(handle, int(polls)))


def oasis_pipeline_destroy(handle: int | None) -> None:
    if handle:
        _PIPE_SIZES.pop(handle, None)
        lib().oasis_pipeline_destroy(handle)


PROFILE_KINDS = ("attn", "score", "topk", "stage")


_PROF_CAP: dict[int, int] = {}


def oasis_pipeline_profile_begin(handle: int, max_steps: int) -> None:
    _check("oasis_pipeline_profile_begin", lib().oasis_pipeline_profile_begin(handle, int(max_steps)))
    _PROF_CAP[handle] = int(max_steps)


def oasis_pipeline_profile_end(handle: int, per_step: bool = False):
    """Mean kernel durations (us) over the profiled steps and the number of steps; with
    ``per_step`` also a [steps, 4] array of each step's durations (columns: PROFILE_KINDS)."""
    avg = (ctypes.c_float * 4)()
    n = _I32()
    cap = _PROF_CAP.pop(handle, 0)
    steps = (ctypes.c_float * (4 * max(cap, 1)))() if per_step else None
    _check("oasis_pipeline_profile_end", lib().oasis_pipeline_profile_end(handle, avg, steps, ctypes.byref(n)))
    means = {k: float(avg[i]) for i, k in enumerate(PROFILE_KINDS)}
    if not per_step:
        return means, int(n.value)
    import numpy as np
    return means, int(n.value), np.ctypeslib.as_array(steps)[: 4 * int(n.value)].reshape(-1, 4).copy()
