// Native issuer of the layer-pipelined decode step (paper §4.2.2: prediction,
// selection and transfer run on background streams, each layer's chain is
// ordered across streams, and the foreground waits only for its own layer's
// transfer; §5.1: the same on the engine's streams).
//
// Host code only: every step builds the kernel arguments with the checks the
// single-call entry points use and launches the same kernels, so a pipelined
// step computes exactly what the sequence of entry-point calls computes.
//
// Cross-stream edges are monotone 32-bit counters in a small device array
// (hipStreamWriteValue32 after the producer's work, hipStreamWaitValue32 >=
// before the consumer's; the transfer's wait for the prediction is made by
// the staging kernel itself, a bounded poll). Measured on MI355X, one edge costs about 4.4 us of
// host time and 8 us of GPU latency this way, against 8-10 us (p90 above 20)
// and 15 us with event record + stream wait. Each counter has its own 256-byte
// line; the host keeps the value last written and drains and resets everything
// long before a counter could wrap.
#include <new>

#include "oasis_internal.h"

namespace {
constexpr int kFlagStride = 64;  // uint32 per counter (256 bytes)
constexpr int kQ = 0, kPred = 1, kAttn = 2, kJoinPred = 3, kJoinXfer = 4, kStaged0 = 5;  // counter slots
constexpr uint32_t kWrapGuard = 1u << 30;
constexpr int kProfKinds = 4;  // attention (split + merge), scoring, top-K, staging
// (request, KV head) pairs from which OASIS_FUSED_PREDICTION_AUTO scores and
// selects in one kernel (one 1024-thread workgroup per pair: a full chip)
constexpr long long kFusedMinPairs = 256;
// (request, KV head) pairs up to which OASIS_PREDICT_AUTO starts the prediction
// after the attention (measured on MI355X, steps/s beside / after: 1 pair x
// 8,192 tokens 30,311 / 32,119; 64 pairs x 131,072 tokens 10,922 / 11,212;
// 128 pairs x 65,536 tokens 3,971 / 3,188; 256 pairs 9,543 / 9,116; the
// 32-layer loop of 512 pairs 3,543 / 3,466 layer-steps/s)
constexpr long long kAfterMaxPairs = 64;
}  // namespace

struct oasis_pipeline {
  oasis_dims dims;
  int32_t T, first_draft, num_draft, k, fetch_cap;
  float scale;
  const uint16_t* host_k;  // device-visible addresses
  const uint16_t* host_v;
  int64_t num_pages;
  const int32_t* block_table;
  // where a growing step refreshes the local block from (the host tier unless set)
  const uint16_t* local_k;
  const uint16_t* local_v;
  int64_t local_num_pages;
  const int32_t* local_block_table;
  int32_t max_layers;
  hipStream_t pred, xfer;
  bool own_streams;
  uint32_t* flags;              // device [(kStaged0 + max_layers) * kFlagStride]
  uint32_t count[kStaged0];     // last value written to each shared counter
  oasis_layer_buffers* layers;  // [max_layers]
  uint32_t* staged;             // [max_layers]: transfers issued per layer (its counter's last value)
  bool* is_set;                 // [max_layers]
  int32_t** plan_ws;            // [max_layers]: device staging-plan workspace of each layer (set_layer)
  bool plan_on_pred;            // OASIS_PLAN_ON_PREDICTION
  int32_t fused_pred;           // OASIS_FUSED_PREDICTION_*: score and top-K (+ plan) in one kernel
  uint32_t wait_polls;          // bound of the staging kernel's wait for its prediction
  int32_t pred_order;           // OASIS_PREDICT_*: where a step's prediction starts
  // optional profile: timing events around each kernel of the next prof_cap steps
  int32_t prof_cap, prof_n;
  hipEvent_t* prof_ev;          // [prof_cap][kProfKinds][2]
};

namespace {

using oasis::fail;
using oasis::hip_status;
using oasis::ok;

#define HIP_TRY(call, fn)                          \
  do {                                             \
    const hipError_t e_ = (call);                  \
    if (e_ != hipSuccess) return hip_status(e_, fn); \
  } while (0)

uint32_t* slot(oasis_pipeline* p, int i) { return p->flags + (size_t)i * kFlagStride; }
// the fault mark of the staging kernel's counter wait: the line after the
// counters, which reset_counters leaves alone
uint32_t* fault_word(oasis_pipeline* p) { return slot(p, kStaged0 + p->max_layers); }

hipError_t signal(oasis_pipeline* p, hipStream_t s, int i, uint32_t v) {
  return hipStreamWriteValue32(s, slot(p, i), v, 0);
}

// Write counter value last + 1 on stream s and record it in *last only once the
// write is enqueued: a failed enqueue leaves the host's value as it was, so no
// later wait is issued for a value that nothing will write.
hipError_t signal_next(oasis_pipeline* p, hipStream_t s, int i, uint32_t* last) {
  const uint32_t v = *last + 1;
  const hipError_t e = signal(p, s, i, v);
  if (e == hipSuccess) *last = v;
  return e;
}

hipError_t wait_for(oasis_pipeline* p, hipStream_t s, int i, uint32_t v) {
  return hipStreamWaitValue32(s, slot(p, i), v, hipStreamWaitValueGte, 0xFFFFFFFFu);
}

// Drain every stream that can wait on a counter, then zero all counters.
hipError_t reset_counters(oasis_pipeline* p, hipStream_t fg) {
  hipError_t e = hipStreamSynchronize(fg);
  if (e == hipSuccess) e = hipStreamSynchronize(p->pred);
  if (e == hipSuccess) e = hipStreamSynchronize(p->xfer);
  if (e == hipSuccess) e = hipMemset(p->flags, 0, sizeof(uint32_t) * kFlagStride * (kStaged0 + p->max_layers));
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) return e;
  for (uint32_t& c : p->count) c = 0;
  for (int l = 0; l < p->max_layers; ++l) p->staged[l] = 0;
  return hipSuccess;
}

void drop_profile(oasis_pipeline* p) {
  if (p->prof_ev) {
    for (int i = 0; i < p->prof_cap * kProfKinds * 2; ++i)
      if (p->prof_ev[i]) (void)hipEventDestroy(p->prof_ev[i]);
    delete[] p->prof_ev;
  }
  p->prof_ev = nullptr;
  p->prof_cap = p->prof_n = 0;
}

// Dispatch timing of kernel kind `kind` in the current profiled step (none when not profiling).
oasis::LaunchTiming prof_timing(oasis_pipeline* p, int kind) {
  if (!p->prof_ev || p->prof_n >= p->prof_cap) return {};
  hipEvent_t* e = p->prof_ev + (p->prof_n * kProfKinds + kind) * 2;
  return oasis::LaunchTiming{e[0], e[1]};
}

void release(oasis_pipeline* p) {
  if (!p) return;
  if (p->flags) {
    (void)hipDeviceSynchronize();  // no stream may still wait on a counter
    (void)hipFree(p->flags);
  }
  drop_profile(p);
  if (p->own_streams) {
    if (p->pred) (void)hipStreamDestroy(p->pred);
    if (p->xfer) (void)hipStreamDestroy(p->xfer);
  }
  if (p->plan_ws) {
    for (int l = 0; l < p->max_layers; ++l)
      if (p->plan_ws[l]) (void)hipFree(p->plan_ws[l]);
  }
  delete[] p->plan_ws;
  delete[] p->layers;
  delete[] p->staged;
  delete[] p->is_set;
  delete p;
}

// The staging-plan workspace of a layer (OASIS_PLAN_ON_PREDICTION hands each
// step's plan from the prediction to the transfer stream through it); made
// once per layer, kept until destroy.
hipError_t alloc_plan_ws(oasis_pipeline* p, int layer) {
  if (p->plan_ws[layer]) return hipSuccess;
  const size_t bytes = sizeof(int32_t) * oasis::stage_ws_ints((long long)p->dims.num_reqs * p->dims.num_kv_heads, p->k);
  const hipError_t e = hipMalloc(&p->plan_ws[layer], bytes > 0 ? bytes : sizeof(int32_t));
  if (e != hipSuccess) p->plan_ws[layer] = nullptr;
  return e;
}

}  // namespace

extern "C" {

oasis_status oasis_pipeline_create(const oasis_dims* dims, int32_t num_q_tokens, int32_t first_draft,
                                   int32_t num_draft, int32_t k, int32_t fetch_cap, float scale,
                                   const uint16_t* host_k, const uint16_t* host_v, int64_t num_pages,
                                   const int32_t* host_block_table, int32_t max_layers, void* pred_stream,
                                   void* xfer_stream, oasis_pipeline** pipeline) {
  static const char* fn = "oasis_pipeline_create";
  if (!pipeline) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  *pipeline = nullptr;
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (max_layers < 1 || max_layers > 65536)
    return fail(OASIS_ERR_INVALID_ARG, "%s: max_layers = %d outside [1, 65536]", fn, max_layers);
  if ((pred_stream == nullptr) != (xfer_stream == nullptr))
    return fail(OASIS_ERR_INVALID_ARG, "%s: pass both background streams or neither", fn);
  if (pred_stream && pred_stream == xfer_stream)
    return fail(OASIS_ERR_INVALID_ARG, "%s: the two background streams must differ", fn);
  if (!host_k || !host_v || !host_block_table)
    return fail(OASIS_ERR_INVALID_ARG, "%s: host_k, host_v and host_block_table are required", fn);
  // The scalar arguments of the operations are checked here through the same
  // builders each step uses (placeholder pointers stand in for the per-step
  // buffers), so a bad configuration fails at create rather than at the first step.
  {
    oasis::ScoreArgs sa{};
    oasis::TopkArgs ta{};
    oasis::StageArgs ga{};
    const uint16_t* dummy16 = host_k;
    int32_t dummy32 = 0;
    float dummyf = 0.f;
    if ((st = oasis::make_score_args(dims, dummy16, num_q_tokens, first_draft, num_draft, dummy16, dummy16,
                                     &dummy32, &dummyf, &sa, fn)) != OASIS_OK)
      return st;
    if ((st = oasis::make_topk_args(dims, &dummyf, &dummy32, k, &dummy32, &dummy32, &ta, fn)) != OASIS_OK)
      return st;
    if ((st = oasis::make_stage_args(dims, host_k, host_v, num_pages, host_block_table, &dummy32, &dummy32,
                                     &dummy32, &dummyf, k, &dummy32, &dummy32, 0, fetch_cap, 1,
                                     const_cast<uint16_t*>(dummy16), const_cast<uint16_t*>(dummy16), nullptr, &ga,
                                     fn)) != OASIS_OK)
      return st;
  }
  const void *hk = nullptr, *hv = nullptr;
  if ((st = oasis::device_view(host_k, &hk, "host_k", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(host_v, &hv, "host_v", fn)) != OASIS_OK) return st;

  oasis_pipeline* p = new (std::nothrow) oasis_pipeline();
  if (!p) return fail(OASIS_ERR_HIP, "%s: out of host memory", fn);
  p->dims = *dims;
  p->T = num_q_tokens;
  p->first_draft = first_draft;
  p->num_draft = num_draft;
  p->k = k;
  p->fetch_cap = fetch_cap;
  p->scale = scale;
  p->host_k = static_cast<const uint16_t*>(hk);
  p->host_v = static_cast<const uint16_t*>(hv);
  p->num_pages = num_pages;
  p->block_table = host_block_table;
  p->local_k = p->host_k;
  p->local_v = p->host_v;
  p->local_num_pages = num_pages;
  p->local_block_table = host_block_table;
  p->max_layers = max_layers;
  p->wait_polls = oasis::kStageWaitSpins;
  p->pred_order = OASIS_PREDICT_AUTO;
  p->layers = new (std::nothrow) oasis_layer_buffers[max_layers]();
  p->staged = new (std::nothrow) uint32_t[max_layers]();
  p->is_set = new (std::nothrow) bool[max_layers]();
  p->plan_ws = new (std::nothrow) int32_t*[max_layers]();
  if (!p->layers || !p->staged || !p->is_set || !p->plan_ws) {
    release(p);
    return fail(OASIS_ERR_HIP, "%s: out of host memory", fn);
  }
  hipError_t e = hipSuccess;
  if (pred_stream) {
    p->pred = static_cast<hipStream_t>(pred_stream);
    p->xfer = static_cast<hipStream_t>(xfer_stream);
  } else {
    p->own_streams = true;
    e = hipStreamCreateWithFlags(&p->pred, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->xfer, hipStreamNonBlocking);
  }
  const size_t flag_bytes = sizeof(uint32_t) * kFlagStride * (kStaged0 + max_layers + 1);
  if (e == hipSuccess) e = hipMalloc(&p->flags, flag_bytes);
  if (e == hipSuccess) e = hipMemset(p->flags, 0, flag_bytes);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    release(p);
    return hip_status(e, fn);
  }
  *pipeline = p;
  return ok();
}

oasis_status oasis_pipeline_set_local_source(oasis_pipeline* p, const uint16_t* k_pages, const uint16_t* v_pages,
                                             int64_t num_pages, const int32_t* block_table) {
  static const char* fn = "oasis_pipeline_set_local_source";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (!k_pages && !v_pages && !block_table) {  // back to the host tier
    p->local_k = p->host_k;
    p->local_v = p->host_v;
    p->local_num_pages = p->num_pages;
    p->local_block_table = p->block_table;
    return ok();
  }
  if (!k_pages || !v_pages || !block_table)
    return fail(OASIS_ERR_INVALID_ARG, "%s: k_pages, v_pages and block_table must all be set or all be NULL", fn);
  if (num_pages < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_pages < 1", fn);
  const void *kv = nullptr, *vv = nullptr;
  oasis_status st;
  if ((st = oasis::device_view(k_pages, &kv, "k_pages", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(v_pages, &vv, "v_pages", fn)) != OASIS_OK) return st;
  p->local_k = static_cast<const uint16_t*>(kv);
  p->local_v = static_cast<const uint16_t*>(vv);
  p->local_num_pages = num_pages;
  p->local_block_table = block_table;
  return ok();
}

oasis_status oasis_pipeline_set_layer(oasis_pipeline* p, int32_t layer, const oasis_layer_buffers* b) {
  static const char* fn = "oasis_pipeline_set_layer";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (!b) return fail(OASIS_ERR_INVALID_ARG, "%s: buffers is NULL", fn);
  if (layer < 0 || layer >= p->max_layers)
    return fail(OASIS_ERR_INVALID_ARG, "%s: layer %d outside [0, %d)", fn, layer, p->max_layers);
  if (p->plan_on_pred) {
    const hipError_t e = alloc_plan_ws(p, layer);
    if (e != hipSuccess) return hip_status(e, fn);
  }
  p->layers[layer] = *b;
  p->is_set[layer] = true;  // a transfer still pending for this layer is waited on at its next step
  return ok();
}

oasis_status oasis_pipeline_set_plan_stream(oasis_pipeline* p, int32_t where) {
  static const char* fn = "oasis_pipeline_set_plan_stream";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (where != OASIS_PLAN_ON_TRANSFER && where != OASIS_PLAN_ON_PREDICTION)
    return fail(OASIS_ERR_INVALID_ARG, "%s: where = %d is neither OASIS_PLAN_ON_TRANSFER nor OASIS_PLAN_ON_PREDICTION",
                fn, where);
  if (where == OASIS_PLAN_ON_PREDICTION) {
    for (int l = 0; l < p->max_layers; ++l) {
      if (!p->is_set[l]) continue;
      const hipError_t e = alloc_plan_ws(p, l);
      if (e != hipSuccess) return hip_status(e, fn);
    }
  }
  p->plan_on_pred = where == OASIS_PLAN_ON_PREDICTION;
  return ok();
}

oasis_status oasis_pipeline_set_fused_prediction(oasis_pipeline* p, int32_t mode) {
  static const char* fn = "oasis_pipeline_set_fused_prediction";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (mode != OASIS_FUSED_PREDICTION_AUTO && mode != OASIS_FUSED_PREDICTION_OFF && mode != OASIS_FUSED_PREDICTION_ON)
    return fail(OASIS_ERR_INVALID_ARG, "%s: mode = %d is not an OASIS_FUSED_PREDICTION_* value", fn, mode);
  p->fused_pred = mode;
  return ok();
}

oasis_status oasis_pipeline_set_wait_limit(oasis_pipeline* p, uint32_t polls) {
  static const char* fn = "oasis_pipeline_set_wait_limit";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (polls == 0) return fail(OASIS_ERR_INVALID_ARG, "%s: polls must be at least 1", fn);
  p->wait_polls = polls;
  return ok();
}

oasis_status oasis_pipeline_set_prediction_order(oasis_pipeline* p, int32_t order) {
  static const char* fn = "oasis_pipeline_set_prediction_order";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (order != OASIS_PREDICT_AUTO && order != OASIS_PREDICT_BESIDE_ATTENTION && order != OASIS_PREDICT_AFTER_ATTENTION)
    return fail(OASIS_ERR_INVALID_ARG, "%s: order = %d is not an OASIS_PREDICT_* value", fn, order);
  p->pred_order = order;
  return ok();
}

oasis_status oasis_pipeline_step(oasis_pipeline* p, int32_t layer, const uint16_t* q, const int32_t* ctx_len,
                                 const int32_t* prev_ctx_len, int32_t max_new_blocks, int32_t step, int32_t growing,
                                 int32_t* moved, void* stream) {
  static const char* fn = "oasis_pipeline_step";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (layer < 0 || layer >= p->max_layers || !p->is_set[layer])
    return fail(OASIS_ERR_INVALID_ARG, "%s: layer %d has no buffers (oasis_pipeline_set_layer)", fn, layer);
  if (growing != 0 && growing != 1) return fail(OASIS_ERR_INVALID_ARG, "%s: growing must be 0 or 1", fn);
  if (prev_ctx_len && max_new_blocks < 1)
    return fail(OASIS_ERR_INVALID_ARG, "%s: max_new_blocks = %d < 1", fn, max_new_blocks);
  const oasis_layer_buffers& b = p->layers[layer];
  const oasis_dims* d = &p->dims;
  oasis::AttnArgs aa{};
  oasis::ScoreArgs sa{};
  oasis::TopkArgs ta{};
  oasis::StageArgs ga{}, la{};
  oasis_status st;
  if ((st = oasis::make_attn_args(d, q, p->T, b.pool_k, b.pool_v, b.slot_map, p->k, ctx_len, p->scale, b.out,
                                  b.lse, b.workspace, b.workspace_bytes, &aa, fn)) != OASIS_OK)
    return st;
  if ((st = oasis::make_score_args(d, q, p->T, p->first_draft, p->num_draft, b.kmax, b.kmin, ctx_len, b.scores,
                                   &sa, fn)) != OASIS_OK)
    return st;
  if ((st = oasis::make_topk_args(d, b.scores, ctx_len, p->k, b.sel, b.sel_count, &ta, fn)) != OASIS_OK) return st;
  if ((st = oasis::make_stage_args(d, p->host_k, p->host_v, p->num_pages, p->block_table, ctx_len, b.sel,
                                   b.sel_count, b.scores, p->k, b.slot_map, b.slot_stamp, step, p->fetch_cap,
                                   0, b.pool_k, b.pool_v, moved ? moved : b.moved, &ga, fn)) != OASIS_OK)
    return st;
  if (growing &&
      (st = oasis::make_stage_args(d, p->local_k, p->local_v, p->local_num_pages, p->local_block_table, ctx_len,
                                   nullptr, nullptr, nullptr, p->k, nullptr, nullptr, 0, p->k, 1, b.pool_k, b.pool_v,
                                   nullptr, &la, fn)) != OASIS_OK)
    return st;
  if (d->num_reqs == 0) return ok();
  // OASIS_PLAN_ON_PREDICTION: the plan runs in the top-K kernel, into the
  // layer's workspace (the slot map stays as the attention reads it); the
  // transfer stream then only copies and commits the planned rows.
  oasis::StageArgs gp = ga;
  if (p->plan_on_pred && !p->plan_ws[layer])  // made by set_layer / set_plan_stream
    return fail(OASIS_ERR_INVALID_ARG, "%s: layer %d has no plan workspace", fn, layer);
  if (p->plan_on_pred) {
    gp.mode = oasis::kStagePlanOnly;
    gp.ws = p->plan_ws[layer];
    ga.mode = oasis::kStageCopyOnly;
    ga.ws = p->plan_ws[layer];
  }
  // compressed keys of the blocks completed since prev_ctx_len, read from the
  // local-block source (where the newest tokens are), before the scoring
  const oasis::SummaryArgs ua{p->local_k, p->local_num_pages, p->local_block_table, ctx_len, b.kmax, b.kmin,
                              d->num_reqs, d->num_kv_heads, d->block_size, d->max_blocks, prev_ctx_len,
                              max_new_blocks};

  hipStream_t fg = static_cast<hipStream_t>(stream);
  bool near_wrap = p->staged[layer] >= kWrapGuard;
  for (uint32_t c : p->count) near_wrap |= c >= kWrapGuard;
  if (near_wrap) HIP_TRY(reset_counters(p, fg), fn);
  uint32_t* cnt = p->count;
  const int sl = kStaged0 + layer;
  // foreground: this layer's previous transfer must have landed before its attention
  if (p->staged[layer]) HIP_TRY(wait_for(p, fg, sl, p->staged[layer]), fn);
  // kQ: q and ctx_len are ready on the foreground; past the wait above this
  // also means the previous transfer has finished reading sel and scores (which
  // the prediction rewrites). kAttn: the attention is done with the pool slots
  // this step's gather overwrites. Beside the attention, the prediction starts
  // at kQ and the transfer waits for both counters; after it, one counter
  // raised after the attention serves as both (the transfer waits for the
  // prediction, which waited for the attention).
  const bool beside = p->pred_order == OASIS_PREDICT_BESIDE_ATTENTION ||
                      (p->pred_order == OASIS_PREDICT_AUTO && (long long)d->num_reqs * d->num_kv_heads > kAfterMaxPairs);
  if (beside) {
    HIP_TRY(signal_next(p, fg, kQ, &cnt[kQ]), fn);
    HIP_TRY(wait_for(p, p->pred, kQ, cnt[kQ]), fn);
  }
  if (growing) HIP_TRY(oasis::launch_stage(la, fg), fn);
  HIP_TRY(oasis::launch_attn(aa, fg, prof_timing(p, 0)), fn);
  if (beside) {
    HIP_TRY(signal_next(p, fg, kAttn, &cnt[kAttn]), fn);
  } else {
    HIP_TRY(signal_next(p, fg, kQ, &cnt[kQ]), fn);
    HIP_TRY(wait_for(p, p->pred, kQ, cnt[kQ]), fn);
  }
  if (prev_ctx_len) HIP_TRY(oasis::launch_summaries(ua, p->pred), fn);
  // one workgroup per (request, KV head) scores and selects (and plans) when
  // the rows are many and short enough to fill the chip that way
  const bool fused = oasis::score_select_supported(sa) &&
                     (p->fused_pred == OASIS_FUSED_PREDICTION_ON ||
                      (p->fused_pred == OASIS_FUSED_PREDICTION_AUTO &&
                       (long long)d->num_reqs * d->num_kv_heads >= kFusedMinPairs));
  if (fused) {
    // profiled as scoring; the top-K span is left empty
    HIP_TRY(oasis::launch_score_select(sa, ta, p->plan_on_pred ? &gp : nullptr, p->pred, prof_timing(p, 1)), fn);
    const oasis::LaunchTiming tk = prof_timing(p, 2);
    if (tk.start) HIP_TRY(hipEventRecord(tk.start, p->pred), fn);
    if (tk.stop) HIP_TRY(hipEventRecord(tk.stop, p->pred), fn);
  } else {
    HIP_TRY(oasis::launch_score(sa, p->pred, prof_timing(p, 1)), fn);
    if (p->plan_on_pred)
      HIP_TRY(oasis::launch_topk_plan(ta, gp, p->pred, prof_timing(p, 2)), fn);
    else
      HIP_TRY(oasis::launch_topk(ta, p->pred, prof_timing(p, 2)), fn);
  }
  HIP_TRY(signal_next(p, p->pred, kPred, &cnt[kPred]), fn);
  // the transfer waits for the prediction and for the attention inside its own
  // kernel (no stream-wait dispatch on the stream that paces the step)
  ga.wait_flag[0] = slot(p, kPred);
  ga.wait_value[0] = cnt[kPred];
  ga.wait_flag[1] = beside ? slot(p, kAttn) : nullptr;
  ga.wait_value[1] = beside ? cnt[kAttn] : 0;
  ga.wait_fault = fault_word(p);
  ga.wait_polls = p->wait_polls;
  HIP_TRY(oasis::launch_stage(ga, p->xfer, prof_timing(p, 3)), fn);
  HIP_TRY(signal_next(p, p->xfer, sl, &p->staged[layer]), fn);
  if (p->prof_ev && p->prof_n < p->prof_cap) ++p->prof_n;
  return ok();
}

oasis_status oasis_pipeline_join(oasis_pipeline* p, void* stream) {
  static const char* fn = "oasis_pipeline_join";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  hipStream_t fg = static_cast<hipStream_t>(stream);
  uint32_t* cnt = p->count;
  if (cnt[kJoinPred] >= kWrapGuard || cnt[kJoinXfer] >= kWrapGuard) HIP_TRY(reset_counters(p, fg), fn);
  HIP_TRY(signal_next(p, p->pred, kJoinPred, &cnt[kJoinPred]), fn);
  HIP_TRY(wait_for(p, fg, kJoinPred, cnt[kJoinPred]), fn);
  HIP_TRY(signal_next(p, p->xfer, kJoinXfer, &cnt[kJoinXfer]), fn);
  HIP_TRY(wait_for(p, fg, kJoinXfer, cnt[kJoinXfer]), fn);
  return ok();
}

oasis_status oasis_pipeline_profile_begin(oasis_pipeline* p, int32_t max_steps) {
  static const char* fn = "oasis_pipeline_profile_begin";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (max_steps < 1 || max_steps > 65536)
    return fail(OASIS_ERR_INVALID_ARG, "%s: max_steps = %d outside [1, 65536]", fn, max_steps);
  drop_profile(p);
  const int n = max_steps * kProfKinds * 2;
  p->prof_ev = new (std::nothrow) hipEvent_t[n]();
  if (!p->prof_ev) return fail(OASIS_ERR_HIP, "%s: out of host memory", fn);
  p->prof_cap = max_steps;
  for (int i = 0; i < n; ++i) {
    const hipError_t e = hipEventCreate(&p->prof_ev[i]);
    if (e != hipSuccess) {
      drop_profile(p);
      return hip_status(e, fn);
    }
  }
  return ok();
}

oasis_status oasis_pipeline_profile_end(oasis_pipeline* p, float* avg_us, float* step_us, int32_t* steps) {
  static const char* fn = "oasis_pipeline_profile_end";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  if (!avg_us) return fail(OASIS_ERR_INVALID_ARG, "%s: avg_us is NULL", fn);
  if (!p->prof_ev) return fail(OASIS_ERR_INVALID_ARG, "%s: no profile was begun", fn);
  const int n = p->prof_n;
  double sum[kProfKinds] = {0, 0, 0, 0};
  hipError_t e = hipSuccess;
  for (int i = 0; i < n && e == hipSuccess; ++i) {
    for (int kind = 0; kind < kProfKinds && e == hipSuccess; ++kind) {
      hipEvent_t a = p->prof_ev[(i * kProfKinds + kind) * 2], b = p->prof_ev[(i * kProfKinds + kind) * 2 + 1];
      e = hipEventSynchronize(b);
      float ms = 0.f;
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
      sum[kind] += ms;
      if (step_us) step_us[i * kProfKinds + kind] = 1000.f * ms;
    }
  }
  drop_profile(p);
  if (e != hipSuccess) return hip_status(e, fn);
  for (int kind = 0; kind < kProfKinds; ++kind) avg_us[kind] = n ? (float)(1000.0 * sum[kind] / n) : 0.f;
  if (steps) *steps = n;
  return ok();
}

oasis_status oasis_pipeline_check(oasis_pipeline* p) {
  static const char* fn = "oasis_pipeline_check";
  if (!p) return fail(OASIS_ERR_INVALID_ARG, "%s: pipeline is NULL", fn);
  uint32_t v = 0;
  HIP_TRY(hipDeviceSynchronize(), fn);
  HIP_TRY(hipMemcpy(&v, fault_word(p), sizeof(v), hipMemcpyDeviceToHost), fn);
  if (v) return fail(OASIS_ERR_HIP, "%s: a transfer gave up waiting for its prediction", fn);
  return ok();
}

void oasis_pipeline_destroy(oasis_pipeline* p) { release(p); }

}  // extern "C"
