"""One layer of the OasisKV decode path: device buffers and the stream schedule.

Paper §4.2.2: at every decode step the foreground runs attention of the stacked
queries over the current working set while a background stream turns the draft
queries into the next working set (top-K prediction -> KV selection -> KV
transfer); events keep the dependencies of each layer. This module owns the
buffers of one layer and issues the library calls in that order; every
computation happens in liboasis.so (through ``_lib``). PyTorch provides device
memory, pinned host memory, streams and events.
"""
from __future__ import annotations

import math

import torch

from . import _lib as L


class LayerState:
    """HBM state of one layer: compressed keys, scores, selection, slot map, pools."""

    def __init__(self, d: L.OasisDims, num_q_tokens: int, k: int, device: str | torch.device = "cuda",
                 ws_attn: torch.Tensor | None = None):
        R, Hq, Hkv, D, B, NB = (d.num_reqs, d.num_q_heads, d.num_kv_heads, d.head_dim, d.block_size,
                               d.max_blocks)
        self.dims, self.T, self.k = d, int(num_q_tokens), int(k)
        dev = torch.device(device)
        bf = torch.bfloat16
        i32 = torch.int32
        self.kmax = torch.empty((R, Hkv, NB, D), dtype=bf, device=dev)
        self.kmin = torch.empty((R, Hkv, NB, D), dtype=bf, device=dev)
        self.scores = torch.empty((R, Hkv, NB), dtype=torch.float32, device=dev)
        self.sel = torch.empty((R, Hkv, k), dtype=i32, device=dev)
        self.sel_count = torch.empty((R, Hkv), dtype=i32, device=dev)
        self.slot_map = torch.full((R, Hkv, k), -1, dtype=i32, device=dev)
        self.slot_stamp = torch.zeros((R, Hkv, k), dtype=i32, device=dev)
        self.pool_k = torch.zeros((R, k + 1, Hkv, B, D), dtype=bf, device=dev)
        self.pool_v = torch.zeros((R, k + 1, Hkv, D, B), dtype=bf, device=dev)
        self.moved = torch.zeros((R, Hkv), dtype=i32, device=dev)
        self.out = torch.empty((R, self.T, Hq, D), dtype=bf, device=dev)
        self.lse = torch.empty((R, self.T, Hq), dtype=torch.float32, device=dev)
        # the attention's split partials: scratch of one call, so layers whose attention
        # runs in order on one stream can share it (ws_attn, at least
        # oasis_attn_workspace_bytes long)
        need = max(1, L.oasis_attn_workspace_bytes(d, self.T, k))
        if ws_attn is None:
            ws_attn = torch.zeros(need, dtype=torch.uint8, device=dev)
        elif ws_attn.numel() * ws_attn.element_size() < need:
            raise ValueError(f"ws_attn holds {ws_attn.numel() * ws_attn.element_size()} bytes, {need} needed")
        self.ws_attn = ws_attn
        self.ev_staged = None   # recorded after the last stage of this layer
        self.ev_attended = None  # recorded after the last attention of this layer
        self.layer_id = None    # id in the native issuer of the DecodePath that runs it
        self.pipe_token = None  # the native issuer this layer is registered with

    def reset(self):
        self.slot_map.fill_(-1)
        self.slot_stamp.zero_()


def dense_working_set(host_k: torch.Tensor, host_v: torch.Tensor, block_table, ctx_len, device="cuda"):
    """Working set that holds every block of every request: the dense comparison of the budget sweep
    (§5.2: the budget is the sparsification threshold; a budget that covers the context is dense
    attention), run through the same attention entry point as the sparse path.

    ``block_table`` / ``ctx_len`` are host int arrays ([R][NBmax], [R]). Returns (pool_k, pool_v,
    slot_map, k_slots) with k_slots = NBmax - 1: slot s of request r holds logical block s for every
    candidate block s < n_cand_r (slot_map = s, later slots free: -1), and slot k_slots holds the
    request's local block nb_r - 1, as the sparse pools do. Only page copies happen here (torch
    indexing, host to device); pool_v is transposed per head as the attention kernel reads it.
    """
    import numpy as np
    host_k, host_v = host_k.view(torch.bfloat16), host_v.view(torch.bfloat16)  # bf16 bits in any 16-bit dtype
    bt = np.asarray(block_table)
    lens = np.asarray(ctx_len)
    R, NB = bt.shape
    _, H, B, D = host_k.shape
    ks = NB - 1
    pool_k = torch.zeros((R, NB, H, B, D), dtype=torch.bfloat16, device=device)
    pool_v = torch.zeros((R, NB, H, D, B), dtype=torch.bfloat16, device=device)
    smap = torch.full((R, H, max(ks, 1)), -1, dtype=torch.int32)
    for r in range(R):
        L_r = max(0, min(int(lens[r]), NB * B))
        nb = (L_r + B - 1) // B
        n_cand = max(nb - 1, 0)
        if n_cand:
            pages = torch.from_numpy(bt[r, :n_cand].astype(np.int64))
            pool_k[r, :n_cand].copy_(host_k[pages].to(device))
            pool_v[r, :n_cand].copy_(host_v[pages].to(device).transpose(-1, -2))
            smap[r, :, :n_cand] = torch.arange(n_cand, dtype=torch.int32)
        if nb:
            page = int(bt[r, nb - 1])
            pool_k[r, ks].copy_(host_k[page].to(device))
            pool_v[r, ks].copy_(host_v[page].to(device).transpose(-1, -2))
    return pool_k, pool_v, smap.to(device), ks


class KernelTimer:
    """HIP events around library calls, recorded on the stream each call runs on."""

    def __init__(self):
        self.pairs: dict[str, list] = {}
        self.enabled = True

    def begin(self, name: str, stream):
        if not self.enabled:
            return None
        ev = torch.cuda.Event(enable_timing=True)
        ev.record(stream)
        return ev

    def end(self, name: str, stream, ev0):
        if ev0 is None:
            return
        ev1 = torch.cuda.Event(enable_timing=True)
        ev1.record(stream)
        self.pairs.setdefault(name, []).append((ev0, ev1))

    def mean_us(self, name: str) -> float:
        ps = self.pairs.get(name, [])
        return 1000.0 * sum(a.elapsed_time(b) for a, b in ps) / max(1, len(ps))

    def reset(self):
        self.pairs.clear()


class DecodePath:
    """Issues score -> select -> stage -> attend for one layer on HIP streams.

    ``host_k``/``host_v`` are the pinned host tier (bf16 pages
    ``[NPhys][Hkv][B][d]``), ``block_table`` the device page table
    ``[R][NBmax]``. The layers from ``new_layer`` share one attention
    workspace, so their attention calls must run in order (the schedules
    below issue them all on the caller's current stream).
    """

    def __init__(self, d: L.OasisDims, num_q_tokens: int, k: int, host_k: torch.Tensor, host_v: torch.Tensor,
                 block_table: torch.Tensor, first_draft: int = 1, num_draft: int | None = None,
                 scale: float | None = None, fetch_cap: int | None = None, native: bool = True,
                 max_layers: int = 256, streams: tuple | None = None, plan_on_prediction: bool = False,
                 fused_prediction: int | None = None, prediction_order: int | None = None):
        self.dims, self.T, self.k = d, int(num_q_tokens), int(k)
        # native issuer: plan each step's transfer in the top-K kernel on the
        # prediction stream instead of in the staging kernel on the transfer stream
        self.plan_on_prediction = bool(plan_on_prediction)
        # native issuer: score and select (and plan) in one kernel per step (L.FUSED_PREDICTION_*;
        # None keeps the library's default, AUTO)
        self.fused_prediction = fused_prediction
        # native issuer: where each step's prediction starts (L.PREDICT_*; None keeps AUTO)
        self.prediction_order = prediction_order
        # step_pipelined issues through the library's native step issuer unless a timer is given
        self.native = bool(native)
        self.max_layers = int(max_layers)
        self._pipe = None
        self._pipe_token = None
        self._n_layers = 0
        # admitted misses per (request, KV head) and step; k admits every miss
        self.fetch_cap = self.k if fetch_cap is None else int(fetch_cap)
        self.first_draft = int(first_draft)
        self.num_draft = int(num_draft if num_draft is not None else self.T - self.first_draft)
        self.host_k, self.host_v, self.block_table = host_k, host_v, block_table
        self.scale = scale if scale is not None else 1.0 / math.sqrt(d.head_dim)
        # background streams (default priority): top-K prediction, KV transfer; paths
        # created one after another can pass the same pair, which keeps the streams
        # on the hardware queues they were first given
        self.side, self.xfer = streams if streams is not None else (torch.cuda.Stream(), torch.cuda.Stream())
        # pages a growing step refreshes the local block from (None: the host tier)
        self.local_source = None
        self._ws_attn = None  # the attention workspace of every layer (new_layer)

    def new_layer(self) -> LayerState:
        # One attention workspace for all layers of the path: it is scratch of a
        # single call, their attention calls run in order on the foreground stream,
        # and a workspace that every call reuses can stay in the caches (8 x 9.4 MB
        # fewer at 16 x 65,536 tokens and 72 rows over eight layers).
        if self._ws_attn is None:
            self._ws_attn = torch.zeros(max(1, L.oasis_attn_workspace_bytes(self.dims, self.T, self.k)),
                                        dtype=torch.uint8, device=self.block_table.device)
        return LayerState(self.dims, self.T, self.k, self.block_table.device, ws_attn=self._ws_attn)

    def _native_layer(self, st: LayerState) -> int:
        """Handle of the native issuer and the layer id of ``st`` (registered on first use)."""
        if self._pipe is None:
            self._pipe = L.oasis_pipeline_create(self.dims, self.T, self.first_draft, self.num_draft, self.k,
                                                 self.fetch_cap, self.scale, self.host_k, self.host_v,
                                                 self.block_table, self.max_layers, self.side, self.xfer)
            if self.local_source is not None:
                L.oasis_pipeline_set_local_source(self._pipe, self.dims, *self.local_source)
            if self.plan_on_prediction:
                L.oasis_pipeline_set_plan_stream(self._pipe, L.PLAN_ON_PREDICTION)
            if self.fused_prediction is not None:
                L.oasis_pipeline_set_fused_prediction(self._pipe, self.fused_prediction)
            if self.prediction_order is not None:
                L.oasis_pipeline_set_prediction_order(self._pipe, self.prediction_order)
            # identifies this issuer: a later one may be created at the same address
            self._pipe_token = object()
        lid = getattr(st, "layer_id", None)
        if lid is None or getattr(st, "pipe_token", None) is not self._pipe_token:
            if self._n_layers >= self.max_layers:
                raise RuntimeError(f"more than {self.max_layers} layers on one DecodePath")
            lid = self._n_layers
            self._n_layers += 1
            L.oasis_pipeline_set_layer(self._pipe, lid, self.dims, self.T, self.k, st.kmax, st.kmin, st.scores,
                                       st.sel, st.sel_count, st.slot_map, st.slot_stamp, st.pool_k, st.pool_v,
                                       st.moved, st.out, st.lse, st.ws_attn)
            st.layer_id, st.pipe_token = lid, self._pipe_token
        return lid

    def set_plan_on_prediction(self, on: bool):
        """Plan the native issuer's transfers in the top-K kernel (True) or the staging kernel
        (False), from the next step on."""
        self.plan_on_prediction = bool(on)
        if self._pipe is not None:
            L.oasis_pipeline_set_plan_stream(self._pipe, L.PLAN_ON_PREDICTION if on else L.PLAN_ON_TRANSFER)

    def set_local_source(self, k_pages: torch.Tensor | None, v_pages: torch.Tensor | None,
                         block_table: torch.Tensor | None):
        """Refresh the local block of growing steps from these pages (bf16 [N][Hkv][B][d], device or
        pinned, with their own [R][NBmax] block table) instead of the host tier; all None: the host tier.
        A model writes its newest tokens on the GPU, so keeping the active blocks in device pages keeps
        the refresh off the PCIe link."""
        self.local_source = None if k_pages is None else (k_pages, v_pages, block_table)
        if self._pipe is not None:
            L.oasis_pipeline_set_local_source(self._pipe, self.dims, k_pages, v_pages, block_table)

    def profile_begin(self, max_steps: int):
        """Time every kernel of the next ``max_steps`` native steps on its own stream."""
        if self._pipe is None:
            raise RuntimeError("no native step has been issued yet")
        L.oasis_pipeline_profile_begin(self._pipe, max_steps)

    def profile_end(self, per_step: bool = False):
        """Mean durations (us) of attention, scoring, top-K and staging, and the step count
        (with ``per_step``, also each step's four durations as a [steps, 4] array)."""
        return L.oasis_pipeline_profile_end(self._pipe, per_step)

    def check(self):
        """Synchronize the device and raise if a pipelined transfer gave up waiting for its prediction."""
        if self._pipe is not None:
            L.oasis_pipeline_check(self._pipe)

    def close(self):
        """Wait for the background streams, check the native issuer's transfers and release it."""
        if self._pipe is not None:
            self.side.synchronize()
            self.xfer.synchronize()
            try:
                L.oasis_pipeline_check(self._pipe)
            finally:
                L.oasis_pipeline_destroy(self._pipe)
                self._pipe = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- individual steps (all asynchronous on `stream`) ----------------------
    def build_summaries(self, st: LayerState, ctx_len: torch.Tensor, k_pages: torch.Tensor | None = None,
                        stream=None):
        L.oasis_build_summaries(self.dims, self.host_k if k_pages is None else k_pages, self.block_table,
                                ctx_len, st.kmax, st.kmin, stream)

    def predict(self, st: LayerState, q: torch.Tensor, ctx_len: torch.Tensor, stream=None):
        L.oasis_score_blocks(self.dims, q, self.T, self.first_draft, self.num_draft, st.kmax, st.kmin, ctx_len,
                             st.scores, stream)
        L.oasis_select_topk(self.dims, st.scores, ctx_len, self.k, st.sel, st.sel_count, stream)

    def stage(self, st: LayerState, ctx_len: torch.Tensor, step: int, stream=None, fetch_cap: int | None = None,
              copy_local: bool = True):
        L.oasis_stage_blocks(self.dims, self.host_k, self.host_v, self.block_table, ctx_len, st.sel, st.sel_count,
                             st.scores, self.k, st.slot_map, st.slot_stamp, step,
                             self.fetch_cap if fetch_cap is None else fetch_cap, copy_local, st.pool_k, st.pool_v,
                             st.moved, stream)

    def refresh_local(self, st: LayerState, ctx_len: torch.Tensor, stream=None):
        """Write the active local block into slot k (stands in for the model's KV write)."""
        hk, hv, bt = self.local_source if self.local_source is not None else (self.host_k, self.host_v,
                                                                               self.block_table)
        L.oasis_stage_blocks(self.dims, hk, hv, bt, ctx_len, None, None, None,
                             self.k, None, None, 0, self.k, True, st.pool_k, st.pool_v, None, stream)

    def attend(self, st: LayerState, q: torch.Tensor, ctx_len: torch.Tensor, stream=None):
        L.oasis_sparse_decode_attn(self.dims, q, self.T, st.pool_k, st.pool_v, st.slot_map, self.k, ctx_len,
                                   self.scale, st.out, st.lse, st.ws_attn, stream)

    # -- schedules --------------------------------------------------------------
    def step_serial(self, st: LayerState, q: torch.Tensor, ctx_len: torch.Tensor, step: int):
        """predict -> stage -> attend on the current stream: attention uses this step's selection."""
        self.predict(st, q, ctx_len)
        self.stage(st, ctx_len, step)
        self.attend(st, q, ctx_len)

    def step_pipelined(self, st: LayerState, q: torch.Tensor, ctx_len: torch.Tensor, step: int,
                       growing: bool = False, timer: KernelTimer | None = None, moved: torch.Tensor | None = None,
                       prev_ctx_len: torch.Tensor | None = None, max_new_blocks: int = 1):
        """One steady-state step of one layer (paper §4.2.2 pipeline).

        Foreground (current stream): wait for this layer's previous transfer,
        then attention of all T rows over the working set it produced.
        Prediction stream: score + select from the draft rows of ``q``,
        concurrently with the attention. Transfer stream: once the selection
        is ready and the attention no longer reads the pools, stage the new
        selection for this layer's next step. Consecutive calls for different
        layers therefore overlap one layer's transfer with the next layer's
        attention and prediction.
        With ``growing`` (one token appended per step) the local block is
        rewritten on the foreground before the attention, since it changes
        every step; otherwise it is unchanged since it was last staged (the
        initial fill stages it) and nothing moves it.
        ``timer`` records HIP events around each call on its own stream;
        ``moved`` (int32 [R][Hkv]) receives the entries this step copies.
        With ``prev_ctx_len`` (the lengths at this layer's previous step) the
        compressed keys of the blocks completed since then are added on the
        prediction stream before the scoring, read from the local-block source.
        Without a timer the step goes through the library's native issuer (one
        C call); with one it is issued call by call from here. Switching between
        the two for one layer needs a device synchronization in between.
        """
        if timer is None and self.native:
            lid = self._native_layer(st)
            L.oasis_pipeline_step(self._pipe, lid, q, ctx_len, step, growing, moved, torch.cuda.current_stream(),
                                  prev_ctx_len, max_new_blocks)
            return
        tm = timer if timer is not None else _NO_TIMER
        fg = torch.cuda.current_stream()
        pred, xfer = self.side, self.xfer
        ev_q = torch.cuda.Event()
        ev_q.record(fg)  # q and ctx_len are ready on the foreground
        pred.wait_event(ev_q)
        if st.ev_staged is not None:
            fg.wait_event(st.ev_staged)
            pred.wait_event(st.ev_staged)  # the previous transfer of this layer read sel and scores
        if growing:
            self.refresh_local(st, ctx_len, fg)
        e = tm.begin("attn", fg)
        self.attend(st, q, ctx_len, fg)
        tm.end("attn", fg, e)
        ev_attn = torch.cuda.Event()
        ev_attn.record(fg)
        if prev_ctx_len is not None:
            hk, _, bt = self.local_source if self.local_source is not None else (self.host_k, self.host_v,
                                                                                 self.block_table)
            L.oasis_update_summaries(self.dims, hk, bt, prev_ctx_len, ctx_len, max_new_blocks, st.kmax, st.kmin,
                                     pred)
        e = tm.begin("score", pred)
        L.oasis_score_blocks(self.dims, q, self.T, self.first_draft, self.num_draft, st.kmax, st.kmin, ctx_len,
                             st.scores, pred)
        tm.end("score", pred, e)
        e = tm.begin("topk", pred)
        L.oasis_select_topk(self.dims, st.scores, ctx_len, self.k, st.sel, st.sel_count, pred)
        tm.end("topk", pred, e)
        ev_pred = torch.cuda.Event()
        ev_pred.record(pred)
        xfer.wait_event(ev_pred)
        xfer.wait_event(ev_attn)  # the gather overwrites slots the attention reads
        e = tm.begin("stage", xfer)
        L.oasis_stage_blocks(self.dims, self.host_k, self.host_v, self.block_table, ctx_len, st.sel, st.sel_count,
                             st.scores, self.k, st.slot_map, st.slot_stamp, step, self.fetch_cap, False,
                             st.pool_k, st.pool_v, st.moved if moved is None else moved, xfer)
        tm.end("stage", xfer, e)
        ev_staged = torch.cuda.Event()
        ev_staged.record(xfer)
        st.ev_staged, st.ev_attended = ev_staged, ev_attn

    def join(self):
        fg = torch.cuda.current_stream()
        fg.wait_stream(self.side)
        fg.wait_stream(self.xfer)


class _NullTimer(KernelTimer):
    def __init__(self):
        super().__init__()
        self.enabled = False


_NO_TIMER = _NullTimer()
