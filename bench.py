"""Benchmark of the OasisKV decode-time hot path on one MI355X.

One step = one pass of the whole path for one layer of a batch: attention of
the stacked (verify + draft) queries over the HBM working set, and, on
background streams, block scoring from the draft queries, top-K selection and
the delta staging of the selected blocks from the pinned host tier under the
fetch cap (paper §4.2.2 schedule for one layer, §5.5.1 default fetch ratio
0.05). The value is decode steps per second per layer with every input
resident in HBM (or in pinned host memory for the host tier) when the timed
region starts.

Timed regions: (1) the step rate, steps issued through the native step issuer
with nothing else on the streams; (2) the same steps again with dispatch-timed
events on every kernel (durations inside the running pipeline); (3) each
kernel alone, back to back, for the roofline of the dominant kernel (the
scorer) and the attention.

Workload (default): long-context serving, 8 requests x 131,072 tokens, GQA
32 query / 8 KV heads, head_dim 128, block 16 (8,192 blocks), 4 draft tokens,
2,048-token budget (K = 128 blocks + the local block), 1 % planted heavy-hitter
blocks, queries following AR(1) over steps. Eight layer states rotate so that
the working set of consecutive steps does not sit in the 256 MB Infinity Cache
(the host K/V tier is shared by the layers; each layer has its own query
stream, summaries, slot map and pools).

The transfer of each step is planned (delta selection, paper §4.2.3) in the
staging kernel on the transfer stream, or with `--plan-stream prediction` in
the top-K kernel on the prediction stream; `auto` takes the prediction stream
for the 32-layer reasoning loop (`--workload c3`), where the transfer stream
sets the rate, and the transfer stream otherwise.

Output: one JSON line (see the fields at the end of main()).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

# The pipelined step keeps three streams busy at once (foreground, prediction,
# transfer). A kernel trace at HIP's default of 4 hardware queues per process
# shows them on three distinct queues, and the step rate is the same at 4 and
# at 16 queues (c4: 10,490 / 10,463 / 10,492 against 10,524 / 10,450 / 10,514
# steps/s, three processes each); the run takes whatever the environment sets
# and records it.
HW_QUEUES = os.environ.get("GPU_MAX_HW_QUEUES")

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
TRAFFIC_NOTE = os.path.join(ROOT, "profiles", "c4_score_attention_hbm_traffic.md")


def measured_traffic(kind):
    """HBM bytes per launch ("score": the scorer; "attention": split + merge of one call) from the
    committed FETCH_SIZE / WRITE_SIZE passes, or None if the sources they name have changed since
    (their sha256 differs) or the note is missing."""
    import hashlib
    import re
    key = {"score": ("score_kernel_traffic_bytes", "score_sources_sha256"),
           "attention": ("attention_traffic_bytes", "attn_sources_sha256")}[kind]
    files = {"score": ("score.hip", "score_core.h", "oasis_internal.h"),
             "attention": ("attn.hip", "oasis_internal.h")}[kind]
    try:
        note = open(TRAFFIC_NOTE).read()
        h = hashlib.sha256()
        for f in files:
            h.update(open(os.path.join(ROOT, "paper_2608_08097_amd", "csrc", f), "rb").read())
    except OSError:
        return None
    m = re.search(key[0] + r"=(\d+) " + key[1] + r"=([0-9a-f]{64})", note)
    if not m or m.group(2) != h.hexdigest():
        return None
    return int(m.group(1))


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=40)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--budget", type=int, default=2048)
    ap.add_argument("--layers", type=int, default=8, help="layer states rotated through (Infinity Cache defeat)")
    ap.add_argument("--fetch-ratio", type=float, default=0.05,
                    help="per-step fetch cap as a fraction of K (paper default 0.05); >= 1 admits every miss")
    ap.add_argument("--plan-stream", choices=("auto", "transfer", "prediction"), default="auto",
                    help="stream that plans each step's transfer (auto: prediction for c3, transfer otherwise)")
    ap.add_argument("--fused-prediction", choices=("auto", "off", "on"), default="auto",
                    help="score and select (and plan) in one kernel per step: auto = with >= 256 (request, KV head) "
                         "pairs")
    ap.add_argument("--prediction-order", choices=("auto", "beside", "after"), default="auto",
                    help="start each step's prediction beside its attention or after it (auto: after for at most "
                         "64 (request, KV head) pairs)")
    ap.add_argument("--tp-share", type=int, default=1,
                    help="one GPU's share of an N-way tensor-parallel deployment: KV and query heads divided by N "
                         "(a shape probe of the same kernels; design only beyond one GPU)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle sample")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-attention comparison")
    ap.add_argument("--fetch-sweep", action="store_true",
                    help="step rate and bytes per step for fetch ratios 0.01 .. 0.2 and uncapped (Tab. eviction)")
    ap.add_argument("--budget-sweep", action="store_true",
                    help="step rate and attention for token budgets 1,024 / 2,048 / 4,096 against dense attention")
    ap.add_argument("--kernels-only", action="store_true",
                    help="only time the kernels alone on one stream (for hardware-counter passes)")
    ap.add_argument("--copy-calib", action="store_true",
                    help="only run a plain 1 GiB device copy (for scaling FETCH_SIZE/WRITE_SIZE counters)")
    return ap.parse_args()


def plan_on_prediction(args) -> bool:
    """Plan the transfer in the top-K kernel (prediction stream) or in the staging kernel (transfer
    stream). Measured on MI355X: the prediction stream is faster for the 32-layer reasoning loop
    (+4 %), the transfer stream for the single-layer workloads (13-23 %)."""
    if args.plan_stream == "auto":
        return args.workload == "c3"
    return args.plan_stream == "prediction"


def prediction_order(args) -> int:
    from paper_2608_08097_amd import _lib as L
    return {"auto": L.PREDICT_AUTO, "beside": L.PREDICT_BESIDE_ATTENTION,
            "after": L.PREDICT_AFTER_ATTENTION}[args.prediction_order]


def fused_mode(args) -> int:
    from paper_2608_08097_amd import _lib as L
    return {"auto": L.FUSED_PREDICTION_AUTO, "off": L.FUSED_PREDICTION_OFF,
            "on": L.FUSED_PREDICTION_ON}[args.fused_prediction]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def copy_calibration():
    import torch
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "dispatches": 3}), flush=True)


def measured_peaks(torch, reps=10):
    """Rates measured on this GPU for reference: a 1 GiB read (torch's row sums
    over rows of 4,096 floats, its fastest read-only op here), a
    1 GiB device-to-device copy (HBM read + write bytes per second) and a
    256 MiB pinned host-to-device copy (the runtime's own copy path)."""
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    hsrc = torch.ones(256 << 20, dtype=torch.uint8, pin_memory=True)
    hdst = torch.empty(hsrc.shape, dtype=torch.uint8, device="cuda")

    def rate(fn, nbytes):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return nbytes * reps / (e0.elapsed_time(e1) * 1e6)

    xf = src.view(torch.float32)
    out = {"hbm_read_GBs": round(rate(lambda: xf.view(-1, 4096).sum(1), n), 1),
           "hbm_copy_GBs": round(rate(lambda: dst.copy_(src), 2 * n), 1),
           "h2d_memcpy_GBs": round(rate(lambda: hdst.copy_(hsrc, non_blocking=True), hsrc.numel()), 2),
           "pcie_nominal_GBs": 64.0}
    del src, dst, hsrc, hdst
    torch.cuda.empty_cache()
    return out


def pctl(x):
    """p10 / median / p90 of a sample, rounded."""
    return [round(float(v), 2) for v in np.percentile(np.asarray(x, dtype=np.float64), [10, 50, 90])]


def algorithmic_bytes(c, w, ctx, K):
    """Algorithmic HBM bytes of one scorer launch and one attention call over all requests."""
    n_cand = np.array([max(0, (int(L) + c.block_size - 1) // c.block_size - 1) for L in ctx])
    bh = int(n_cand.sum()) * c.num_kv_heads                      # candidate block-heads per step
    score_bytes = bh * (2 * c.head_dim * 2) + c.num_reqs * c.num_kv_heads * w.NBmax * 4 \
        + c.num_reqs * c.T * c.num_q_heads * c.head_dim * 2
    tok_per_head = np.minimum(K, n_cand) * c.block_size + np.array([L - c.block_size * nc
                                                                    for L, nc in zip(ctx, n_cand)])
    attn_bytes = int(tok_per_head.sum()) * c.num_kv_heads * (2 * c.head_dim * 2) \
        + 2 * c.num_reqs * c.T * c.num_q_heads * c.head_dim * 2
    return score_bytes, attn_bytes


def cold_fill(torch, path, layers, ctx_d, c):
    """Staging of a whole working set into empty slot maps (every selected block a miss, no cap):
    the host-to-device gather at full size, back to back over the layer states."""
    for st in layers:
        st.reset()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for st in layers:
        path.stage(st, ctx_d, 0, fetch_cap=path.k)
    e1.record()
    torch.cuda.synchronize()
    us = 1000.0 * e0.elapsed_time(e1) / len(layers)
    entries = sum(int(st.moved.sum().item()) for st in layers) / len(layers)
    nbytes = entries * 2 * c.block_size * c.head_dim * 2
    return {"avg_us": round(us, 1), "entries": round(entries, 1), "h2d_bytes": round(nbytes),
            "h2d_GBs": round(nbytes / (us * 1e3), 2)}


def describe(c, ctx, budget, K, fetch_cap, NL):
    kinds = {"c1": "parity case", "c2": "batched serving", "c4": "long-context serving", "c5": "large-GQA stress"}
    lens = f"{int(ctx[0])} tokens" if int(ctx.min()) == int(ctx.max()) else f"{int(ctx.min())}-{int(ctx.max())} tokens"
    return (f"{c.name}: {kinds.get(c.name, c.name)}, {c.num_reqs} requests x {lens}, GQA "
            f"{c.num_q_heads}q/{c.num_kv_heads}kv, head_dim {c.head_dim}, block {c.block_size}, "
            f"{c.num_draft} draft tokens, budget {budget} (K={K}), fetch cap {fetch_cap} "
            f"per KV head per step, AR(1) queries, {NL} rotating layer states")


def host_cores() -> int:
    """CPU cores this process may run on (its affinity set)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def blas_threads():
    """Threads of the BLAS library NumPy calls (threadpoolctl), or None if it cannot be asked."""
    try:
        from threadpoolctl import threadpool_info
    except ImportError:  # pragma: no cover
        return None
    n = [i.get("num_threads") for i in threadpool_info() if i.get("user_api") == "blas"]
    return n[0] if n else None


def cpu_baseline(w, hk, hv, queries, k, fetch_cap, budget_s):
    """Time the oracle on a bounded sample of the same step, on the host's own cores.

    Every request's working set is first filled from its step-0 prediction
    (untimed, as on the GPU); then whole-batch decode steps are timed, each
    one scoring, top-K, capped delta staging and attention per request. The
    requests of a step are independent, so they run on a pool of worker
    threads, one per host core up to the batch size, with the BLAS library
    held to one thread per worker; a first, shorter sample runs the same
    steps on a single thread. ``queries`` are the bf16 queries of
    consecutive steps.
    """
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oasis_oracle as O
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    import contextlib
    c = w.cfg
    ctx = w.ctx_len(0)
    B, H, d = c.block_size, c.num_kv_heads, c.head_dim
    cap = None if fetch_cap >= k else fetch_cap
    cores = host_cores()
    blas_default = blas_threads()
    workers = max(1, min(c.num_reqs, cores))

    def fill(r):
        bt, cr = w.block_table[r:r + 1], ctx[r:r + 1]
        kmax, kmin = O.block_summaries(hk, bt, cr, B, w.NBmax)
        s = O.block_scores(queries[0][r:r + 1], kmax, kmin, cr, H, B)
        sel, cnt = O.select_topk(s, cr, k, B)
        smap = np.full((1, H, k), -1, np.int32)
        stamp = np.zeros_like(smap)
        pk = np.zeros((1, k + 1, H, B, d), np.uint16)
        pv = np.zeros_like(pk)
        O.stage_blocks(hk, hv, bt, sel, cnt, smap, stamp, 0, pk, pv, cr, B)
        return (bt, cr, kmax, kmin, smap, stamp, pk, pv)

    def one(r, st, step):
        bt, cr, kmax, kmin, smap, stamp, pk, pv = st
        qr = queries[step][r:r + 1]
        s = O.block_scores(qr, kmax, kmin, cr, H, B)
        sel, cnt = O.select_topk(s, cr, k, B)
        O.stage_blocks(hk, hv, bt, sel, cnt, smap, stamp, step, pk, pv, cr, B, scores=s, fetch_cap=cap)
        O.sparse_attend(qr, pk, pv, smap, cr, B)

    limit = threadpool_limits(limits=1) if threadpool_limits is not None else contextlib.nullcontext()
    with limit, ThreadPoolExecutor(max_workers=workers) as ex:
        state = list(ex.map(fill, range(c.num_reqs)))   # setup, not timed
        step = 0

        def sample(seconds, pool, last):
            nonlocal step
            steps, spent = 0, 0.0
            while spent < seconds and step < last:
                step += 1
                t0 = time.perf_counter()
                if pool is None:
                    for r, st in enumerate(state):
                        one(r, st, step)
                else:
                    list(pool.map(lambda r: one(r, state[r], step), range(c.num_reqs)))
                spent += time.perf_counter() - t0
                steps += 1
            return steps, spent

        # steps 1 .. len(queries) - 1: at most half of them on one thread, the rest on the workers
        n_steps = len(queries) - 1
        n1, t1 = sample(budget_s / 3, None, n_steps // 2)
        nw, tw = sample(2 * budget_s / 3, ex, n_steps)
    # the faster of the two arrangements is the baseline (for many small requests the worker
    # threads mostly contend for the interpreter)
    r_w, r_1 = nw / tw, n1 / t1
    return {"value": max(r_w, r_1), "unit": "steps/s", "cores": workers if r_w >= r_1 else 1, "kind": "oracle",
            "host_cores": cores, "blas_threads_per_worker": 1, "blas_threads_default": blas_default,
            "value_workers": r_w, "value_1_thread": r_1,
            "sample": f"whole decode steps of all {c.num_reqs} requests (scores, top-K, delta staging with fetch "
                      f"cap {fetch_cap}, attention; after an untimed initial fill) in float64 NumPy: {nw} steps in "
                      f"{tw:.1f} s with the requests on {workers} worker threads (host has {cores} cores), then "
                      f"the rate of {n1} earlier steps on 1 thread ({t1:.1f} s)"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: measures one GPU only; --gpus N with N > 1 is not supported (the path has no "
              "cross-GPU step: requests and KV heads would be split over GPUs, each running this path alone)",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calib:
        copy_calibration()
        return

    import torch

    import paper_2608_08097_amd as P
    from paper_2608_08097_amd.path import DecodePath
    from workloads import config, Workload

    if not os.path.exists(P._lib.LIB_PATH):
        from paper_2608_08097_amd.build_lib import build
        build()
    torch.cuda.set_device(0)

    if args.workload == "c3":
        run_reasoning(args, P, torch, DecodePath)
        return

    total_steps = args.warmup + args.steps
    NL = max(1, args.layers)
    per_layer_steps = (total_steps + args.steps + NL - 1) // NL  # queries of both timed regions
    base = config(args.workload)
    if args.tp_share < 1 or base.num_kv_heads % args.tp_share:
        raise SystemExit(f"--tp-share {args.tp_share} must divide the {base.num_kv_heads} KV heads")
    heads = {} if args.tp_share == 1 else dict(num_kv_heads=base.num_kv_heads // args.tp_share,
                                               num_q_heads=base.num_q_heads // args.tp_share)
    cfg = config(args.workload, budget=args.budget, ar_queries=True, steps=per_layer_steps, grow_per_step=0,
                 **heads)
    w = Workload(cfg)
    c = w.cfg
    K = c.K
    t0 = time.perf_counter()
    shape = (w.NPhys, c.num_kv_heads, c.block_size, c.head_dim)
    hk_t = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    hv_t = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    hk, hv = hk_t.numpy().view(np.uint16), hv_t.numpy().view(np.uint16)
    w.fill_paged(hk, hv)
    log(f"inputs: {c.name} R={c.num_reqs} L={list(w.ctx0[:2])}.. host KV {2 * hk.nbytes / 1e9:.2f} GB "
        f"generated in {time.perf_counter() - t0:.1f} s")

    d = P.dims(c.num_reqs, c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size, w.NBmax)
    bt = torch.from_numpy(w.block_table).cuda()
    ctx = w.ctx_len(0)
    ctx_d = torch.from_numpy(ctx).cuda()
    fetch_cap = K if args.fetch_ratio >= 1.0 else max(1, int(math.floor(args.fetch_ratio * K)))
    path = DecodePath(d, c.T, K, hk_t.view(torch.bfloat16), hv_t.view(torch.bfloat16), bt, fetch_cap=fetch_cap,
                      plan_on_prediction=plan_on_prediction(args),
                      fused_prediction=fused_mode(args), prediction_order=prediction_order(args))
    layers = [path.new_layer() for _ in range(NL)]
    path.build_summaries(layers[0], ctx_d)
    for st in layers[1:]:
        st.kmax.copy_(layers[0].kmax)
        st.kmin.copy_(layers[0].kmin)
    qs = [[torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16) for x in w.layer_queries(l, per_layer_steps)]
          for l in range(NL)]
    if args.budget_sweep:
        path.close()
        sweep = budget_sweep(P, torch, DecodePath, d, c, w, hk_t, hv_t, bt, layers, qs, ctx_d, ctx, args,
                             (path.side, path.xfer))
        dense = dense_attention(P, torch, w, hk_t, hv_t, ctx_d, d, c) if not args.no_dense else None
        print(json.dumps({"budget_sweep": sweep, "dense_attention": dense}), flush=True)
        return
    if args.fetch_sweep:
        path.close()
        print(json.dumps({"fetch_sweep": fetch_sweep(P, torch, DecodePath, d, c, K, hk_t, hv_t, bt, layers, qs,
                                                     ctx_d, args, (path.side, path.xfer))}), flush=True)
        return
    # The working set a layer holds when decoding starts: one uncapped fill from
    # its first prediction (untimed; decode steps are then capped).
    for l, st in enumerate(layers):
        path.predict(st, qs[l][0], ctx_d)
        path.stage(st, ctx_d, 0, fetch_cap=K)
    moved_log = torch.zeros((args.steps, c.num_reqs, c.num_kv_heads), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    if args.kernels_only:
        # For hardware-counter passes, which serialize dispatches: no cross-stream
        # waits may be in flight, so only the single-stream region 3 runs.
        iso = isolated(P, torch, path, layers, qs, ctx_d)
        torch.cuda.synchronize()
        print(json.dumps({"kernels_only": {k_: round(v, 2) for k_, v in iso.items()}}), flush=True)
        return

    def run(i, log_moved):
        # The warm-up steps log their moved counts too, so that they take the
        # timed steps' exact call path (the timed steps overwrite every row).
        l, s = i % NL, i // NL
        path.step_pipelined(layers[l], qs[l][s], ctx_d, i, growing=False,
                            moved=moved_log[(i - args.warmup) % args.steps] if log_moved else None)

    for i in range(args.warmup):
        run(i, True)
    path.join()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")
    # Timed region 1: the step rate (no events between kernels).
    t_start = time.perf_counter()
    for i in range(args.warmup, total_steps):
        run(i, True)
    path.join()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = 1000.0 * elapsed / args.steps
    log(f"timed {args.steps} steps in {elapsed:.3f} s")
    # Timed region 2: the same pipelined steps again with HIP timing events
    # recorded by the native issuer around every kernel, on the stream the
    # kernel runs on (per-kernel durations inside the running pipeline).
    moved_rate = moved_log.cpu().numpy().copy()
    path.profile_begin(args.steps)
    for i in range(total_steps, total_steps + args.steps):
        run(i, False)
    path.join()
    torch.cuda.synchronize()
    us, n_prof, per_step = path.profile_end(per_step=True)
    assert n_prof == args.steps
    score_bytes, attn_bytes = algorithmic_bytes(c, w, ctx, K)
    entry_bytes = 2 * c.block_size * c.head_dim * 2
    moved = moved_rate
    h2d_per_step = float(moved.sum()) / args.steps * entry_bytes
    # Timed region 3: each kernel alone, back to back on the current stream over
    # the rotating layer states between one pair of HIP events (the per-launch
    # event cost vanishes; this is the duration a kernel trace reports).
    iso = isolated(P, torch, path, layers, qs, ctx_d)
    score_gbs = score_bytes / (iso["score"] * 1e3)
    attn_gbs = attn_bytes / (iso["attn"] * 1e3)
    # The same launches on one layer state only: its summaries and pools stay
    # partly in the Infinity Cache (a warm reference, not the reported rate).
    warm = isolated(P, torch, path, layers[:1], qs[:1], ctx_d)
    path.join()
    torch.cuda.synchronize()
    cold = cold_fill(torch, path, layers, ctx_d, c)
    peaks = measured_peaks(torch)

    dense = None
    if not args.no_dense and args.workload == "c4":
        dense = dense_attention(P, torch, w, hk_t, hv_t, ctx_d, d, c)

    result = {
        "metric": "sparse decode attn steps/s per layer + achieved HBM GB/s (% of peak) @2048 budget",
        "value": round(1000.0 / ms_per_step, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": describe(c, ctx, args.budget, K, fetch_cap, NL),
            "global_batch": c.num_reqs, "seq_len": int(ctx.max()), "budget": args.budget,
            "fetch_ratio": args.fetch_ratio if fetch_cap < K else "all", "fetch_cap": fetch_cap,
            "parallelism": "single GPU", "plan_stream": "prediction" if plan_on_prediction(args) else "transfer",
            "fused_prediction": args.fused_prediction,
            "prediction_order": args.prediction_order,
            "gpu_max_hw_queues": HW_QUEUES if HW_QUEUES is not None else "unset (HIP default, 4)",
            "tp_share": args.tp_share,
        },
        "roofline": {
            "bound": "hbm", "kernel": "score_kernel (oasis_score_blocks)",
            "achieved": round(score_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(score_gbs / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic("score") if args.workload == "c4" else None,
            "algorithmic_bytes": score_bytes, "avg_us": round(iso["score"], 2),
            "timing": "64 back-to-back launches over the rotating layer states, one event pair",
        },
        "attention": {"avg_us": round(iso["attn"], 2), "algorithmic_bytes": attn_bytes,
                      "traffic": measured_traffic("attention") if args.workload == "c4" else None,
                      "achieved_GBs": round(attn_gbs, 1), "frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                      "frac_of_measured_read": round(attn_gbs / peaks["hbm_read_GBs"], 4)},
        "score_frac_of_measured_read": round(score_gbs / peaks["hbm_read_GBs"], 4),
        "topk_us": round(iso["topk"], 2),
        "staging": {"avg_us_in_pipeline": round(us["stage"], 2), "h2d_bytes_per_step": round(h2d_per_step),
                    "entries_per_step": round(float(moved.sum()) / args.steps, 1),
                    "h2d_GBs": round(h2d_per_step / (us["stage"] * 1e3), 2) if us["stage"] > 0 else None,
                    "cold_fill": cold,
                    "cold_fill_frac_of_memcpy": round(cold["h2d_GBs"] / peaks["h2d_memcpy_GBs"], 4)},
        "measured_peaks": peaks,
        "warm_single_layer_us": {k_: round(v, 2) for k_, v in warm.items()},
        # region 2: dispatch-timed events per kernel inside the running pipeline; they include the
        # slowdown from concurrent kernels and host reads, and a few us of event latency each
        "pipeline_kernel_us": {k_: round(v, 2) for k_, v in us.items()},
        "pipeline_kernel_p10_p50_p90_us": {k_: pctl(per_step[:, i]) for i, k_ in enumerate(P._lib.PROFILE_KINDS)},
        "dense_attention": dense,
    }
    if not args.no_cpu_baseline:
        log("timing the oracle sample")
        result["cpu_baseline"] = cpu_baseline(w, hk, hv, w.layer_queries(0, 64), K, fetch_cap, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def run_reasoning(args, P, torch, DecodePath):
    """Reasoning-style decode on the layer-pipelined path (§4.2.2, Eq. "prefetch-rate").

    32 layers, 64 requests with a 1K prompt plus 4K-16K generated tokens, block
    16, 4 draft tokens, budget 2,048; 64 consecutive decode steps, one token
    appended per request per step. Per step and layer, one pipelined step: the
    local block is refreshed and attended on the foreground; the compressed keys
    of a block that just completed are added, then scoring and top-K run on the
    prediction stream; capped staging follows on the transfer stream. The host
    K/V tier is shared by the layers; each layer has its own summaries, working
    set and query stream. The active (local) blocks are device-resident,
    standing in for the model's own KV writes, so only the delta transfer
    crosses PCIe. Queries follow the AR(1) recipe, drawn on the GPU from a
    seeded generator (2.7 G values would take a minute to draw on the host).
    Reports tokens/s, layer-steps/s, and T_pipe against Delta_prefetch =
    T_step / N_layer.
    """
    from workloads import config, Workload
    cfg = config("c3", budget=args.budget, ar_queries=True)
    w = Workload(cfg)
    c = w.cfg
    K, NL, S = c.K, c.layers, c.steps
    fetch_cap = K if args.fetch_ratio >= 1.0 else max(1, int(math.floor(args.fetch_ratio * K)))
    t0 = time.perf_counter()
    shape = (w.NPhys, c.num_kv_heads, c.block_size, c.head_dim)
    hk_t = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    hv_t = torch.empty(shape, dtype=torch.int16, pin_memory=True)
    hk, hv = hk_t.numpy().view(np.uint16), hv_t.numpy().view(np.uint16)
    w.fill_paged(hk, hv)
    log(f"inputs: c3 R={c.num_reqs} L0 in [{int(w.ctx0.min())}, {int(w.ctx0.max())}] host KV "
        f"{2 * hk.nbytes / 1e9:.2f} GB in {time.perf_counter() - t0:.1f} s")
    d = P.dims(c.num_reqs, c.num_q_heads, c.num_kv_heads, c.head_dim, c.block_size, w.NBmax)
    bt = torch.from_numpy(w.block_table).cuda()
    ctx_d = [torch.from_numpy(w.ctx_len(s_)).cuda() for s_ in range(S)]
    path = DecodePath(d, c.T, K, hk_t.view(torch.bfloat16), hv_t.view(torch.bfloat16), bt, fetch_cap=fetch_cap,
                      max_layers=NL, plan_on_prediction=plan_on_prediction(args),
                      fused_prediction=fused_mode(args), prediction_order=prediction_order(args))
    # The blocks that are a request's local block during the run live in device
    # pages, as a model writes its newest tokens on the GPU: the local refresh
    # and the compressed-key update of a completed block read them there, and
    # only the delta transfer reads the host tier.
    lpages, ltable = w.local_block_pages(S)
    lidx = torch.from_numpy(lpages)
    dev_k = hk_t[lidx].cuda().view(torch.bfloat16)
    dev_v = hv_t[lidx].cuda().view(torch.bfloat16)
    dev_bt = torch.from_numpy(ltable).cuda()
    path.set_local_source(dev_k, dev_v, dev_bt)
    layers = [path.new_layer() for _ in range(NL)]
    path.build_summaries(layers[0], ctx_d[0])
    gen = torch.Generator(device="cuda")
    qs = []
    for l in range(NL):
        gen.manual_seed(c.base_seed + 2 + 1000 * (l + 1))
        state = torch.randn((c.num_reqs, c.T, c.num_q_heads, c.head_dim), generator=gen, device="cuda")
        ql = [state.to(torch.bfloat16)]
        for _ in range(1, S):
            eps = torch.randn(state.shape, generator=gen, device="cuda")
            state = 0.9 * state + 0.436 * eps
            ql.append(state.to(torch.bfloat16))
        qs.append(ql)
    torch.cuda.synchronize()

    def prime():
        for l, st in enumerate(layers):
            if l:
                st.kmax.copy_(layers[0].kmax)
                st.kmin.copy_(layers[0].kmin)
            st.reset()
            path.predict(st, qs[l][0], ctx_d[0])
            path.stage(st, ctx_d[0], 0, fetch_cap=K)
        torch.cuda.synchronize()

    moved_log = torch.zeros((S, NL, c.num_reqs, c.num_kv_heads), dtype=torch.int32, device="cuda")

    def decode():
        for s_ in range(S):
            for l, st in enumerate(layers):
                # the step adds the compressed keys of a block that just completed (prediction stream)
                path.step_pipelined(st, qs[l][s_], ctx_d[s_], s_, growing=True, moved=moved_log[s_, l],
                                    prev_ctx_len=ctx_d[s_ - 1] if s_ else None)
        path.join()
        torch.cuda.synchronize()

    prime()
    decode()                      # warm-up pass over the 64 steps
    path.build_summaries(layers[0], ctx_d[0])
    prime()
    t0 = time.perf_counter()
    decode()
    elapsed = time.perf_counter() - t0
    entries = float(moved_log.sum().item()) / (S * NL)   # per layer-step, this timed pass
    entry_bytes = 2 * c.block_size * c.head_dim * 2
    # same pass again with per-kernel dispatch timing
    path.build_summaries(layers[0], ctx_d[0])
    prime()
    path.profile_begin(NL * S)
    decode()
    prof, n_prof = path.profile_end()
    t_step_us = 1e6 * elapsed / S
    delta = t_step_us / NL
    t_pipe = max(prof["score"] + prof["topk"], prof["stage"])
    result = {
        "metric": "sparse decode attn steps/s per layer + achieved HBM GB/s (% of peak) @2048 budget",
        "value": round(NL * S / elapsed, 2), "unit": "layer-steps/s", "n_gpus": 1, "steps": S, "warmup": S,
        "ms_per_step": round(t_step_us / 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"c3: reasoning decode, {NL} layers x {c.num_reqs} requests, prompt 1,024 + "
                               f"U[4,096, 16,384] generated tokens, block 16, {c.num_draft} draft tokens, budget "
                               f"{args.budget} (K={K}), fetch cap {fetch_cap}, {S} steps of one token",
                   "global_batch": c.num_reqs, "layers": NL, "fetch_cap": fetch_cap,
                   "plan_stream": "prediction" if plan_on_prediction(args) else "transfer",
                   "fused_prediction": args.fused_prediction,
                   "prediction_order": args.prediction_order,
                   "gpu_max_hw_queues": HW_QUEUES if HW_QUEUES is not None else "unset (HIP default, 4)"},
        "tokens_per_s": round(c.num_reqs * S / elapsed, 1),
        "decode_step_ms_all_layers": round(t_step_us / 1e3, 3),
        "prefetch_rate": {"delta_prefetch_us": round(delta, 2), "t_pred_us": round(prof["score"] + prof["topk"], 2),
                          "t_transfer_us": round(prof["stage"], 2), "t_pipe_us": round(t_pipe, 2),
                          "t_pipe_le_delta": bool(t_pipe <= delta)},
        "staging": {"entries_per_layer_step": round(entries, 1),
                    "h2d_bytes_per_layer_step": round(entries * entry_bytes),
                    "h2d_GBs_in_transfer": round(entries * entry_bytes / (prof["stage"] * 1e3), 2),
                    "h2d_GBs_at_step_rate": round(entries * entry_bytes * NL * S / elapsed / 1e9, 2)},
        "pipeline_kernel_us": {k_: round(v, 2) for k_, v in prof.items()},
    }
    path.close()
    if not args.no_cpu_baseline:
        log("timing the oracle sample")
        result["cpu_baseline"] = cpu_baseline(w, hk, hv, w.layer_queries(0, 8), K, fetch_cap, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def budget_sweep(P, torch, DecodePath, d, c, w, hk_t, hv_t, bt, layers, qs, ctx_d, ctx, args, streams):
    """Token budgets 1,024 / 2,048 / 4,096 on the same inputs: for each, the step rate
    (fetch cap = ratio x K), the attention alone over the working set, and the scorer."""
    from paper_2608_08097_amd.path import LayerState
    NL = len(layers)
    out = []
    for budget in (1024, 2048, 4096):
        K = budget // c.block_size
        cap = K if args.fetch_ratio >= 1.0 else max(1, int(math.floor(args.fetch_ratio * K)))
        path = DecodePath(d, c.T, K, hk_t.view(torch.bfloat16), hv_t.view(torch.bfloat16), bt, fetch_cap=cap,
                          streams=streams, prediction_order=prediction_order(args))
        sts = []
        for l in range(NL):
            st = LayerState(d, c.T, K)
            st.kmax, st.kmin = layers[l].kmax, layers[l].kmin      # summaries are read-only here
            path.predict(st, qs[l][0], ctx_d)
            path.stage(st, ctx_d, 0, fetch_cap=K)
            sts.append(st)
        torch.cuda.synchronize()
        for i in range(args.warmup):
            path.step_pipelined(sts[i % NL], qs[i % NL][i // NL], ctx_d, i)
        path.join()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.warmup, args.warmup + args.steps):
            path.step_pipelined(sts[i % NL], qs[i % NL][i // NL], ctx_d, i)
        path.join()
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        iso = isolated(P, torch, path, sts, qs, ctx_d)
        path.close()
        score_bytes, attn_bytes = algorithmic_bytes(c, w, ctx, K)
        row = {"budget": budget, "K": K, "fetch_cap": cap, "steps_per_s": round(args.steps / el, 1),
               "attn_us": round(iso["attn"], 2), "attn_bytes": attn_bytes,
               "attn_GBs": round(attn_bytes / (iso["attn"] * 1e3), 1),
               "score_us": round(iso["score"], 2), "score_GBs": round(score_bytes / (iso["score"] * 1e3), 1),
               "topk_us": round(iso["topk"], 2)}
        log(f"budget sweep {row}")
        out.append(row)
        del sts
        torch.cuda.empty_cache()
    return out


def fetch_sweep(P, torch, DecodePath, d, c, K, hk_t, hv_t, bt, layers, qs, ctx_d, args, streams):
    """The fetch-cap ablation of §5.5.1 on this workload: for each ratio, the same
    steps from the same initial fill; entries and bytes moved per step, the step
    rate, and the host-to-device rate the staging sustains at that step rate."""
    NL = len(layers)
    entry_bytes = 2 * c.block_size * c.head_dim * 2
    out = []
    for ratio in (0.01, 0.02, 0.05, 0.10, 0.20, 1.0):
        cap = K if ratio >= 1.0 else max(1, int(math.floor(ratio * K)))
        path = DecodePath(d, c.T, K, hk_t.view(torch.bfloat16), hv_t.view(torch.bfloat16), bt, fetch_cap=cap,
                          streams=streams, prediction_order=prediction_order(args))
        for l, st in enumerate(layers):
            st.reset()
            path.predict(st, qs[l][0], ctx_d)
            path.stage(st, ctx_d, 0, fetch_cap=K)
        moved = torch.zeros((args.steps, c.num_reqs, c.num_kv_heads), dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        for i in range(args.warmup):
            path.step_pipelined(layers[i % NL], qs[i % NL][i // NL], ctx_d, i)
        path.join()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.warmup, args.warmup + args.steps):
            path.step_pipelined(layers[i % NL], qs[i % NL][i // NL], ctx_d, i, moved=moved[i - args.warmup])
        path.join()
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        n_prof = min(64, args.steps)
        path.profile_begin(n_prof)
        for i in range(args.warmup + args.steps, args.warmup + args.steps + n_prof):
            path.step_pipelined(layers[i % NL], qs[i % NL][i // NL], ctx_d, i)
        path.join()
        torch.cuda.synchronize()
        prof, _ = path.profile_end()
        path.close()
        entries = float(moved.sum().item()) / args.steps
        rate = args.steps / el
        row = {"fetch_ratio": ratio if cap < K else "all", "fetch_cap": cap, "entries_per_step": round(entries, 1),
               "MB_per_step": round(entries * entry_bytes / 1e6, 3), "steps_per_s": round(rate, 1),
               "h2d_GBs_at_step_rate": round(entries * entry_bytes * rate / 1e9, 2),
               "pipeline_kernel_us": {k_: round(v, 1) for k_, v in prof.items()}}
        log(f"fetch sweep {row}")
        out.append(row)
    return out


def isolated(P, torch, path, layers, qs, ctx_d, iters=64):
    """Mean duration (us) of each kernel alone on the current stream, rotating over the layer states."""
    d, T, K = path.dims, path.T, path.k
    NL = len(layers)
    res = {}

    def timeit(fn):
        for i in range(8):
            fn(layers[i % NL], qs[i % NL][0])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(iters):
            fn(layers[i % NL], qs[i % NL][0])
        e1.record()
        torch.cuda.synchronize()
        return 1000.0 * e0.elapsed_time(e1) / iters

    res["score"] = timeit(lambda st, q: P.oasis_score_blocks(d, q, T, 1, T - 1, st.kmax, st.kmin, ctx_d,
                                                            st.scores))
    res["topk"] = timeit(lambda st, q: P.oasis_select_topk(d, st.scores, ctx_d, K, st.sel, st.sel_count))
    res["attn"] = timeit(lambda st, q: P.oasis_sparse_decode_attn(d, q, T, st.pool_k, st.pool_v, st.slot_map, K,
                                                                  ctx_d, None, st.out, st.lse, st.ws_attn))
    return res


def dense_attention(P, torch, w, hk_t, hv_t, ctx_d, d, c, iters=20):
    """Same attention kernel over the whole context resident in HBM (every candidate block in the
    slot of its own id, the local block in the last slot; `tests/test_gpu_fullsize.py` checks this
    exact call against the oracle's dense attention)."""
    from paper_2608_08097_amd.path import dense_working_set
    D = c.head_dim
    pool_k, pool_v, smap, ks = dense_working_set(hk_t, hv_t, w.block_table, w.ctx_len(0))
    out = torch.empty((c.num_reqs, c.T, c.num_q_heads, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((c.num_reqs, c.T, c.num_q_heads), dtype=torch.float32, device="cuda")
    ws = torch.zeros(P.oasis_attn_workspace_bytes(d, c.T, ks), dtype=torch.uint8, device="cuda")
    q = torch.from_numpy(w.queries(0).view(np.int16)).cuda().view(torch.bfloat16)
    for _ in range(3):
        P.oasis_sparse_decode_attn(d, q, c.T, pool_k, pool_v, smap, ks, ctx_d, None, out, lse, ws)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        P.oasis_sparse_decode_attn(d, q, c.T, pool_k, pool_v, smap, ks, ctx_d, None, out, lse, ws)
    e1.record()
    torch.cuda.synchronize()
    us = 1000.0 * e0.elapsed_time(e1) / iters
    tokens = int(w.ctx_len(0).sum())
    nbytes = c.num_kv_heads * tokens * 2 * D * 2
    del pool_k, pool_v
    return {"avg_us": round(us, 2), "algorithmic_bytes": nbytes, "achieved_GBs": round(nbytes / (us * 1e3), 1),
            "frac": round(nbytes / (us * 1e3) / HBM_PEAK_GBS, 4), "tokens_per_head": int(w.ctx_len(0).max()),
            "parity": "tests/test_gpu_fullsize.py::test_fullsize_dense_c4"}


if __name__ == "__main__":
    main()
