// C ABI of the OasisKV decode path: argument checks, workspace carving and
// kernel launches. Nothing here allocates memory or throws.
//
// Every entry point is "check and build the kernel arguments" followed by one
// launch; the builders are shared with the native step issuer (pipeline.hip),
// so both forms accept and reject exactly the same arguments.
#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "oasis_internal.h"

namespace oasis {

namespace {
thread_local char g_err[512] = "";
}  // namespace

oasis_status fail(oasis_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

oasis_status ok() {
  g_err[0] = '\0';
  return OASIS_OK;
}

const char* last_error() { return g_err; }

oasis_status hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return ok();
  return fail(OASIS_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

oasis_status check_dims(const oasis_dims* d, const char* fn) {
  if (!d) return fail(OASIS_ERR_INVALID_ARG, "%s: dims is NULL", fn);
  if (d->num_reqs < 0) return fail(OASIS_ERR_INVALID_ARG, "%s: num_reqs < 0", fn);
  if (d->num_kv_heads < 1 || d->num_q_heads < 1)
    return fail(OASIS_ERR_INVALID_ARG, "%s: num_q_heads and num_kv_heads must be >= 1", fn);
  if (d->num_q_heads % d->num_kv_heads)
    return fail(OASIS_ERR_INVALID_ARG, "%s: num_q_heads (%d) is not a multiple of num_kv_heads (%d)", fn,
                d->num_q_heads, d->num_kv_heads);
  if (d->head_dim != kHeadDim)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: head_dim %d (only 128 is supported)", fn, d->head_dim);
  if (d->block_size != 16 && d->block_size != 32)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: block_size %d (16 or 32 are supported)", fn, d->block_size);
  if (d->max_blocks < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: max_blocks < 1", fn);
  if ((long long)d->num_reqs * d->num_kv_heads > 65535)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: num_reqs * num_kv_heads > 65535", fn);
  return OASIS_OK;
}

#define REQUIRE_PTR(p, fn)                                                   \
  do {                                                                       \
    if (!(p)) return fail(OASIS_ERR_INVALID_ARG, "%s: " #p " is NULL", fn); \
  } while (0)

oasis_status device_view(const void* p, const void** out, const char* what, const char* fn) {
  hipPointerAttribute_t attr;
  const hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(OASIS_ERR_INVALID_ARG, "%s: %s is neither pinned host memory nor device memory", fn, what);
  }
  if (attr.type == hipMemoryTypeDevice || attr.type == hipMemoryTypeManaged || attr.type == hipMemoryTypeUnified) {
    *out = p;
    return OASIS_OK;
  }
  if (attr.type == hipMemoryTypeHost && attr.devicePointer) {
    const char* host_base = static_cast<const char*>(attr.hostPointer ? attr.hostPointer : p);
    *out = static_cast<const char*>(attr.devicePointer) + (static_cast<const char*>(p) - host_base);
    return OASIS_OK;
  }
  return fail(OASIS_ERR_INVALID_ARG, "%s: %s is host memory that is not pinned and mapped", fn, what);
}

oasis_status make_score_args(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens, int32_t first_draft,
                             int32_t num_draft, const uint16_t* kmax, const uint16_t* kmin, const int32_t* ctx_len,
                             float* scores, ScoreArgs* a, const char* fn) {
  oasis_status st = check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (num_q_tokens < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_q_tokens < 1", fn);
  if (first_draft < 0 || num_draft < 1 || (long long)first_draft + num_draft > num_q_tokens)
    return fail(OASIS_ERR_INVALID_ARG, "%s: draft rows [%d, %d) outside [0, %d)", fn, first_draft,
                first_draft + num_draft, num_q_tokens);
  const int G = dims->num_q_heads / dims->num_kv_heads;
  if ((long long)num_draft * G > 64)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: num_draft * G = %lld scoring rows (at most 64)", fn,
                (long long)num_draft * G);
  if (dims->num_reqs == 0) return OASIS_OK;
  REQUIRE_PTR(q, fn);
  REQUIRE_PTR(kmax, fn);
  REQUIRE_PTR(kmin, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(scores, fn);
  *a = ScoreArgs{q, kmax, kmin, ctx_len, scores, dims->num_reqs, dims->num_q_heads, dims->num_kv_heads, G,
                 num_q_tokens, first_draft, num_draft, dims->block_size, dims->max_blocks};
  return OASIS_OK;
}

oasis_status make_topk_args(const oasis_dims* dims, const float* scores, const int32_t* ctx_len, int32_t k,
                            int32_t* sel, int32_t* sel_count, TopkArgs* a, const char* fn) {
  oasis_status st = check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (k < 1 || k > 65536) return fail(OASIS_ERR_INVALID_ARG, "%s: k = %d outside [1, 65536]", fn, k);
  if (dims->num_reqs == 0) return OASIS_OK;
  REQUIRE_PTR(scores, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(sel, fn);
  REQUIRE_PTR(sel_count, fn);
  *a = TopkArgs{scores, ctx_len, sel, sel_count, dims->num_reqs, dims->num_kv_heads, dims->block_size,
                dims->max_blocks, k};
  return OASIS_OK;
}

// host_k / host_v are stored as given: the caller passes device-visible addresses
// (device_view) before launching.
oasis_status make_stage_args(const oasis_dims* dims, const uint16_t* host_k, const uint16_t* host_v,
                             int64_t num_pages, const int32_t* host_block_table, const int32_t* ctx_len,
                             const int32_t* sel, const int32_t* sel_count, const float* scores, int32_t k,
                             int32_t* slot_map, int32_t* slot_stamp, int32_t step, int32_t fetch_cap,
                             int32_t copy_local, uint16_t* pool_k, uint16_t* pool_v, int32_t* moved, StageArgs* a,
                             const char* fn) {
  oasis_status st = check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (k < 1 || k > 1024) return fail(OASIS_ERR_INVALID_ARG, "%s: k = %d outside [1, 1024]", fn, k);
  if (fetch_cap < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: fetch_cap = %d < 1", fn, fetch_cap);
  if (copy_local != 0 && copy_local != 1) return fail(OASIS_ERR_INVALID_ARG, "%s: copy_local must be 0 or 1", fn);
  if (num_pages < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_pages < 1", fn);
  if ((sel == nullptr) != (sel_count == nullptr))
    return fail(OASIS_ERR_INVALID_ARG, "%s: sel and sel_count must both be set or both be NULL", fn);
  const bool local_only = sel == nullptr;
  if (local_only && !copy_local)
    return fail(OASIS_ERR_INVALID_ARG, "%s: no selection and copy_local = 0: nothing to do", fn);
  if (dims->num_reqs == 0) return OASIS_OK;
  REQUIRE_PTR(host_k, fn);
  REQUIRE_PTR(host_v, fn);
  REQUIRE_PTR(host_block_table, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(pool_k, fn);
  REQUIRE_PTR(pool_v, fn);
  if (!local_only) {
    REQUIRE_PTR(slot_map, fn);
    REQUIRE_PTR(slot_stamp, fn);
    if (fetch_cap < k) REQUIRE_PTR(scores, fn);
  }
  StageArgs s{};
  s.host_k = host_k;
  s.host_v = host_v;
  s.num_pages = num_pages;
  s.block_table = host_block_table;
  s.ctx_len = ctx_len;
  s.sel = sel;
  s.sel_count = sel_count;
  s.scores = scores;
  s.slot_map = slot_map;
  s.slot_stamp = slot_stamp;
  s.pool_k = pool_k;
  s.pool_v = pool_v;
  s.moved = moved;
  s.local_only = local_only ? 1 : 0;
  s.R = dims->num_reqs;
  s.Hkv = dims->num_kv_heads;
  s.B = dims->block_size;
  s.NBmax = dims->max_blocks;
  s.k = k;
  s.step = step;
  s.copy_local = copy_local;
  s.fetch_cap = fetch_cap < k ? fetch_cap : k;
  *a = s;
  return OASIS_OK;
}

oasis_status make_attn_args(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens, const uint16_t* pool_k,
                            const uint16_t* pool_v, const int32_t* slot_map, int32_t k_slots, const int32_t* ctx_len,
                            float scale, uint16_t* out, float* lse, void* workspace, size_t workspace_bytes,
                            AttnArgs* a, const char* fn) {
  oasis_status st = check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (num_q_tokens < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_q_tokens < 1", fn);
  if (k_slots < 0) return fail(OASIS_ERR_INVALID_ARG, "%s: k_slots < 0", fn);
  if (!std::isfinite(scale)) return fail(OASIS_ERR_INVALID_ARG, "%s: scale is not finite", fn);
  const int G = dims->num_q_heads / dims->num_kv_heads;
  if ((long long)G * num_q_tokens > 80)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: G * num_q_tokens = %lld rows per KV head (at most 80)", fn,
                (long long)G * num_q_tokens);
  if (dims->num_reqs == 0) return OASIS_OK;
  REQUIRE_PTR(q, fn);
  REQUIRE_PTR(pool_k, fn);
  REQUIRE_PTR(pool_v, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(out, fn);
  if (k_slots > 0) REQUIRE_PTR(slot_map, fn);
  const AttnPlan p = attn_plan(dims->num_reqs, dims->num_q_heads, dims->num_kv_heads, num_q_tokens,
                               dims->block_size, k_slots);
  if (p.bytes > 0 && (!workspace || workspace_bytes < p.bytes))
    return fail(OASIS_ERR_WORKSPACE, "%s: workspace of %zu bytes, %zu needed", fn, workspace_bytes, p.bytes);
  AttnArgs t{};
  t.q = q;
  t.pool_k = pool_k;
  t.pool_v = pool_v;
  t.slot_map = slot_map;
  t.ctx_len = ctx_len;
  t.out = out;
  t.lse = lse;
  t.part_o = static_cast<float*>(workspace);
  t.part_ml = static_cast<float*>(workspace) + p.part_o_floats;
  t.R = dims->num_reqs;
  t.Hq = dims->num_q_heads;
  t.Hkv = dims->num_kv_heads;
  t.G = G;
  t.T = num_q_tokens;
  t.B = dims->block_size;
  t.NBmax = dims->max_blocks;
  t.k_slots = k_slots;
  t.scale_log2 = scale * 1.4426950408889634f;
  t.rows = p.rows;
  t.n_units = p.n_units;
  t.nsplit = p.nsplit;
  t.units_per_split = p.units_per_split;
  *a = t;
  return OASIS_OK;
}

}  // namespace oasis

using oasis::fail;
using oasis::hip_status;
using oasis::ok;

extern "C" {

const char* oasis_last_error(void) { return oasis::last_error(); }

int32_t oasis_abi_version(void) { return OASIS_ABI_VERSION; }

oasis_status oasis_build_summaries(const oasis_dims* dims, const uint16_t* k_pages, int64_t num_pages,
                                   const int32_t* block_table, const int32_t* ctx_len, uint16_t* kmax,
                                   uint16_t* kmin, void* stream) {
  static const char* fn = "oasis_build_summaries";
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  REQUIRE_PTR(k_pages, fn);
  REQUIRE_PTR(block_table, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(kmax, fn);
  REQUIRE_PTR(kmin, fn);
  if (num_pages < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_pages < 1", fn);
  const void* kp = nullptr;
  st = oasis::device_view(k_pages, &kp, "k_pages", fn);
  if (st != OASIS_OK) return st;
  oasis::SummaryArgs a{static_cast<const uint16_t*>(kp), num_pages, block_table, ctx_len, kmax, kmin,
                       dims->num_reqs, dims->num_kv_heads, dims->block_size, dims->max_blocks, nullptr, 0};
  return hip_status(oasis::launch_summaries(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_update_summaries(const oasis_dims* dims, const uint16_t* k_pages, int64_t num_pages,
                                    const int32_t* block_table, const int32_t* prev_ctx_len, const int32_t* ctx_len,
                                    int32_t max_new_blocks, uint16_t* kmax, uint16_t* kmin, void* stream) {
  static const char* fn = "oasis_update_summaries";
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (max_new_blocks < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: max_new_blocks = %d < 1", fn, max_new_blocks);
  if (num_pages < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_pages < 1", fn);
  if (dims->num_reqs == 0) return ok();
  REQUIRE_PTR(k_pages, fn);
  REQUIRE_PTR(block_table, fn);
  REQUIRE_PTR(prev_ctx_len, fn);
  REQUIRE_PTR(ctx_len, fn);
  REQUIRE_PTR(kmax, fn);
  REQUIRE_PTR(kmin, fn);
  const void* kp = nullptr;
  st = oasis::device_view(k_pages, &kp, "k_pages", fn);
  if (st != OASIS_OK) return st;
  oasis::SummaryArgs a{static_cast<const uint16_t*>(kp), num_pages, block_table, ctx_len, kmax, kmin,
                       dims->num_reqs, dims->num_kv_heads, dims->block_size, dims->max_blocks, prev_ctx_len,
                       max_new_blocks};
  return hip_status(oasis::launch_summaries(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_copy_blocks(const oasis_dims* dims, const uint16_t* src_k, const uint16_t* src_v,
                               int64_t num_src_pages, const int32_t* src_block_table, uint16_t* dst_k, uint16_t* dst_v,
                               int64_t num_dst_pages, const int32_t* dst_block_table, const int32_t* prev_ctx_len,
                               const int32_t* ctx_len, int32_t max_blocks, void* stream) {
  static const char* fn = "oasis_copy_blocks";
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (max_blocks < 1 || max_blocks > 65535)
    return fail(OASIS_ERR_INVALID_ARG, "%s: max_blocks = %d outside [1, 65535]", fn, max_blocks);
  if (num_src_pages < 1 || num_dst_pages < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: a tier has no pages", fn);
  if (dims->num_reqs == 0) return ok();
  REQUIRE_PTR(src_k, fn);
  REQUIRE_PTR(src_v, fn);
  REQUIRE_PTR(src_block_table, fn);
  REQUIRE_PTR(dst_k, fn);
  REQUIRE_PTR(dst_v, fn);
  REQUIRE_PTR(dst_block_table, fn);
  REQUIRE_PTR(ctx_len, fn);
  const void *sk = nullptr, *sv = nullptr, *dk = nullptr, *dv = nullptr;
  if ((st = oasis::device_view(src_k, &sk, "src_k", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(src_v, &sv, "src_v", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(dst_k, &dk, "dst_k", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(dst_v, &dv, "dst_v", fn)) != OASIS_OK) return st;
  oasis::CopyArgs a{};
  a.src_k = static_cast<const uint16_t*>(sk);
  a.src_v = static_cast<const uint16_t*>(sv);
  a.num_src_pages = num_src_pages;
  a.src_table = src_block_table;
  a.dst_k = static_cast<uint16_t*>(const_cast<void*>(dk));
  a.dst_v = static_cast<uint16_t*>(const_cast<void*>(dv));
  a.num_dst_pages = num_dst_pages;
  a.dst_table = dst_block_table;
  a.prev_ctx_len = prev_ctx_len;
  a.ctx_len = ctx_len;
  a.R = dims->num_reqs;
  a.Hkv = dims->num_kv_heads;
  a.B = dims->block_size;
  a.NBmax = dims->max_blocks;
  a.max_blocks = max_blocks;
  return hip_status(oasis::launch_copy_blocks(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_score_blocks(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                int32_t first_draft, int32_t num_draft, const uint16_t* kmax,
                                const uint16_t* kmin, const int32_t* ctx_len, float* scores, void* stream) {
  static const char* fn = "oasis_score_blocks";
  oasis::ScoreArgs a{};
  const oasis_status st =
      oasis::make_score_args(dims, q, num_q_tokens, first_draft, num_draft, kmax, kmin, ctx_len, scores, &a, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  return hip_status(oasis::launch_score(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_select_topk(const oasis_dims* dims, const float* scores, const int32_t* ctx_len, int32_t k,
                               int32_t* sel, int32_t* sel_count, void* stream) {
  static const char* fn = "oasis_select_topk";
  oasis::TopkArgs a{};
  const oasis_status st = oasis::make_topk_args(dims, scores, ctx_len, k, sel, sel_count, &a, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  return hip_status(oasis::launch_topk(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_score_select(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                int32_t first_draft, int32_t num_draft, const uint16_t* kmax,
                                const uint16_t* kmin, const int32_t* ctx_len, int32_t k, float* scores,
                                int32_t* sel, int32_t* sel_count, void* stream) {
  static const char* fn = "oasis_score_select";
  oasis::ScoreArgs sa{};
  oasis::TopkArgs ta{};
  oasis_status st =
      oasis::make_score_args(dims, q, num_q_tokens, first_draft, num_draft, kmax, kmin, ctx_len, scores, &sa, fn);
  if (st != OASIS_OK) return st;
  if ((st = oasis::make_topk_args(dims, scores, ctx_len, k, sel, sel_count, &ta, fn)) != OASIS_OK) return st;
  const int rows = num_draft * (dims->num_q_heads / dims->num_kv_heads);
  if (rows <= oasis::kScoreValuMaxRows || rows > oasis::kScoreSelectMaxRows)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: %d scoring rows (%d to %d are supported)", fn, rows,
                oasis::kScoreValuMaxRows + 1, oasis::kScoreSelectMaxRows);
  if (dims->max_blocks > oasis::kScoreSelectMaxBlocks)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: max_blocks %d > %d", fn, dims->max_blocks, oasis::kScoreSelectMaxBlocks);
  if (dims->num_reqs == 0) return ok();
  return hip_status(oasis::launch_score_select(sa, ta, nullptr, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_stage_blocks(const oasis_dims* dims, const uint16_t* host_k, const uint16_t* host_v,
                                int64_t num_pages, const int32_t* host_block_table, const int32_t* ctx_len,
                                const int32_t* sel, const int32_t* sel_count, const float* scores, int32_t k,
                                int32_t* slot_map, int32_t* slot_stamp, int32_t step, int32_t fetch_cap,
                                int32_t copy_local, uint16_t* pool_k, uint16_t* pool_v, int32_t* moved,
                                void* stream) {
  static const char* fn = "oasis_stage_blocks";
  oasis::StageArgs a{};
  // the host tier's device-visible addresses are resolved after every cheap check
  oasis_status st = oasis::make_stage_args(dims, host_k, host_v, num_pages, host_block_table, ctx_len, sel,
                                           sel_count, scores, k, slot_map, slot_stamp, step, fetch_cap, copy_local,
                                           pool_k, pool_v, moved, &a, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  const void *hk = nullptr, *hv = nullptr;
  if ((st = oasis::device_view(host_k, &hk, "host_k", fn)) != OASIS_OK) return st;
  if ((st = oasis::device_view(host_v, &hv, "host_v", fn)) != OASIS_OK) return st;
  a.host_k = static_cast<const uint16_t*>(hk);
  a.host_v = static_cast<const uint16_t*>(hv);
  return hip_status(oasis::launch_stage(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_union_selection(const oasis_dims* dims, const int32_t* sel, const int32_t* sel_count, int32_t k,
                                   int32_t* union_ids, int32_t* union_count, void* stream) {
  static const char* fn = "oasis_union_selection";
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (k < 1 || k > 65536) return fail(OASIS_ERR_INVALID_ARG, "%s: k = %d outside [1, 65536]", fn, k);
  if (dims->max_blocks > oasis::kUnionMaxBlocks)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: max_blocks %d > %d", fn, dims->max_blocks, oasis::kUnionMaxBlocks);
  if ((long long)dims->num_kv_heads * k > (1LL << 30))
    return fail(OASIS_ERR_UNSUPPORTED, "%s: num_kv_heads * k too large", fn);
  if (dims->num_reqs == 0) return ok();
  REQUIRE_PTR(sel, fn);
  REQUIRE_PTR(sel_count, fn);
  REQUIRE_PTR(union_ids, fn);
  REQUIRE_PTR(union_count, fn);
  oasis::UnionArgs a{sel, sel_count, union_ids, union_count, dims->num_reqs, dims->num_kv_heads, dims->max_blocks, k};
  return hip_status(oasis::launch_union(a, static_cast<hipStream_t>(stream)), fn);
}

size_t oasis_attn_workspace_bytes(const oasis_dims* dims, int32_t num_q_tokens, int32_t k_slots) {
  if (oasis::check_dims(dims, "oasis_attn_workspace_bytes") != OASIS_OK || num_q_tokens < 1 || k_slots < 0)
    return 0;
  return oasis::attn_plan(dims->num_reqs, dims->num_q_heads, dims->num_kv_heads, num_q_tokens, dims->block_size,
                          k_slots)
      .bytes;
}

oasis_status oasis_sparse_decode_attn(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                      const uint16_t* pool_k, const uint16_t* pool_v, const int32_t* slot_map,
                                      int32_t k_slots, const int32_t* ctx_len, float scale, uint16_t* out,
                                      float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  static const char* fn = "oasis_sparse_decode_attn";
  oasis::AttnArgs a{};
  const oasis_status st = oasis::make_attn_args(dims, q, num_q_tokens, pool_k, pool_v, slot_map, k_slots, ctx_len,
                                                scale, out, lse, workspace, workspace_bytes, &a, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  return hip_status(oasis::launch_attn(a, static_cast<hipStream_t>(stream)), fn);
}

oasis_status oasis_sparse_decode_attn_noalloc(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                              const uint16_t* pool_k, const uint16_t* pool_v,
                                              const int32_t* slot_map, int32_t k_slots, const int32_t* ctx_len,
                                              float scale, uint16_t* out, float* lse, void* stream) {
  static const char* fn = "oasis_sparse_decode_attn_noalloc";
  oasis_status st = oasis::check_dims(dims, fn);
  if (st != OASIS_OK) return st;
  if (num_q_tokens < 1) return fail(OASIS_ERR_INVALID_ARG, "%s: num_q_tokens < 1", fn);
  if (k_slots < 0) return fail(OASIS_ERR_INVALID_ARG, "%s: k_slots < 0", fn);
  const size_t need = oasis::attn_plan(dims->num_reqs, dims->num_q_heads, dims->num_kv_heads, num_q_tokens,
                                       dims->block_size, k_slots)
                          .bytes;
  if (need > oasis::kNoAllocScratchBytes)
    return fail(OASIS_ERR_UNSUPPORTED, "%s: these sizes need %zu bytes of scratch, more than the %zu it holds", fn,
                need, oasis::kNoAllocScratchBytes);
  // every argument is checked before the first runtime call (the scratch
  // address is not needed for that), then the arguments are built on it
  oasis::AttnArgs a{};
  static int sentinel;
  st = oasis::make_attn_args(dims, q, num_q_tokens, pool_k, pool_v, slot_map, k_slots, ctx_len, scale, out, lse,
                             &sentinel, oasis::kNoAllocScratchBytes, &a, fn);
  if (st != OASIS_OK) return st;
  if (dims->num_reqs == 0) return ok();
  void* scratch = nullptr;
  const hipError_t e = oasis::noalloc_scratch(&scratch);
  if (e != hipSuccess) return hip_status(e, fn);
  st = oasis::make_attn_args(dims, q, num_q_tokens, pool_k, pool_v, slot_map, k_slots, ctx_len, scale, out, lse,
                             scratch, oasis::kNoAllocScratchBytes, &a, fn);
  if (st != OASIS_OK) return st;
  return hip_status(oasis::launch_attn(a, static_cast<hipStream_t>(stream)), fn);
}

}  // extern "C"
