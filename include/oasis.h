/*
 * oasis.h -- C ABI of the OasisKV decode-time hot path on AMD Instinct MI355X (gfx950).
 *
 * Paper: "OasisKV: Scaling In-Decode KV Cache Beyond HBM with Lookahead Sparse
 * Prefetching" (arXiv 2608.08097). One decode step of one layer is
 *
 *   oasis_score_blocks       rank every KV block from the draft queries     (paper §4.2.1)
 *   oasis_select_topk        keep the K best blocks per (request, KV head)   (§4.2.1, §4.2.2, §5.2)
 *   oasis_stage_blocks       delta-select and gather them from pinned host   (§4.2.3, §4.3, §5.1)
 *   oasis_sparse_decode_attn attention of the stacked queries over them      (§4.2.1, §4.3, §5.2)
 *
 * plus oasis_build_summaries / oasis_update_summaries, which make the
 * compressed keys the scorer reads (§4.2.1, "Look-ahead attention" figure; §5.1)
 * for the whole context or for the blocks completed since the last call;
 * oasis_copy_blocks, which moves blocks between the GPU pages and the full host
 * tier (§4.3, dense-to-sparse transition and appends); and oasis_pipeline_*,
 * the native issuer of the layer-pipelined step (§4.2.2).
 *
 * General conventions
 * -------------------
 * - Every pointer is owned by the caller. The single-call entry points
 *   (oasis_build_summaries ... oasis_sparse_decode_attn) allocate no memory;
 *   the scratch the attention call needs is a caller-provided workspace whose
 *   size comes from oasis_attn_workspace_bytes. The step issuer does allocate,
 *   outside its steps: oasis_pipeline_create (its counter array, and the two
 *   background streams unless the caller passes them), oasis_pipeline_set_layer
 *   and oasis_pipeline_set_plan_stream (a plan workspace per layer when the plan
 *   runs on the prediction stream) and oasis_pipeline_profile_begin (timing
 *   events); oasis_pipeline_destroy frees all of it. oasis_pipeline_step and
 *   oasis_pipeline_join allocate nothing.
 * - Calls are asynchronous on `stream` (a hipStream_t passed as void*, NULL =
 *   the null stream). They return once the kernels are enqueued.
 * - Host-side checks (null pointers, supported sizes, workspace size) return
 *   OASIS_ERR_INVALID_ARG or OASIS_ERR_UNSUPPORTED and launch nothing.
 *   oasis_last_error() then describes the problem (thread-local string).
 * - A failed kernel launch returns OASIS_ERR_HIP. A fault inside a kernel is
 *   reported by HIP at the caller's next synchronisation.
 * - Values that live on the device (context lengths, counts, block ids, page
 *   ids) are clamped or skipped by the kernels, never trusted for addressing:
 *   ctx_len is clamped to [0, max_blocks * block_size]; a page id outside
 *   [0, num_pages) is not read; a selection count is clamped to [0, k].
 * - No C++ exception crosses this interface.
 * - bf16 tensors are raw bfloat16 bit patterns (uint16_t).
 *
 * Notation: R requests, Hq query heads, Hkv KV heads, G = Hq / Hkv query heads
 * per KV head (query head qh belongs to KV head qh / G), d = head_dim = 128,
 * B = block_size, T = num_q_tokens query rows per head (row 0 is the token
 * being verified, the following rows are draft / lookahead tokens),
 * NBmax = max_blocks, L_r = ctx_len[r], nb_r = ceil(L_r / B) logical blocks,
 * n_cand_r = max(nb_r - 1, 0) candidate blocks (the last block, possibly
 * partial, is the active local block: always attended, never ranked),
 * local_len_r = L_r - B * n_cand_r tokens in the local block.
 *
 * Layouts (row-major, innermost last):
 *   q            bf16 [R][T][Hq][d]
 *   host pages   bf16 [NPhys][Hkv][B][d]   Head-Token-Dimension pages (§4.3)
 *   block table  int32 [R][NBmax]           logical block -> physical page (§4.3)
 *   kmax, kmin   bf16 [R][Hkv][NBmax][d]
 *   scores       fp32 [R][Hkv][NBmax]
 *   sel          int32 [R][Hkv][k]          ascending block ids, -1 padded
 *   sel_count    int32 [R][Hkv]
 *   slot_map     int32 [R][Hkv][k]          resident logical block per slot, -1 = free (§4.3)
 *   slot_stamp   int32 [R][Hkv][k]          decode step at which the slot was last selected (§4.2.3)
 *   pool_k       bf16 [R][k+1][Hkv][B][d]   HBM working set, keys, token-major per head
 *   pool_v       bf16 [R][k+1][Hkv][d][B]   HBM working set, values, TRANSPOSED per head:
 *                d x B, unlike the token-major K pool and the host pages (the
 *                staging kernel transposes while it copies); slot k of both
 *                pools holds the active local block
 *   out          bf16 [R][T][Hq][d]
 *   lse          fp32 [R][T][Hq]            natural-log log-sum-exp of the scaled logits
 */
#ifndef OASIS_H
#define OASIS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OASIS_ABI_VERSION 7

/* Only the entry points below are exported from liboasis.so. */
#if defined(__GNUC__) || defined(__clang__)
#define OASIS_API __attribute__((visibility("default")))
#else
#define OASIS_API
#endif

typedef enum {
  OASIS_OK = 0,
  OASIS_ERR_INVALID_ARG = 1,  /* null pointer, inconsistent or out-of-range argument */
  OASIS_ERR_UNSUPPORTED = 2,  /* valid but not implemented (head_dim != 128, B not 16/32, ...) */
  OASIS_ERR_HIP = 3,          /* a HIP runtime call or kernel launch failed */
  OASIS_ERR_WORKSPACE = 4     /* workspace missing or smaller than *_workspace_bytes */
} oasis_status;

typedef struct {
  int32_t num_reqs;      /* R   >= 0 (0: every call is a no-op)       */
  int32_t num_q_heads;   /* Hq  >= 1, multiple of num_kv_heads          */
  int32_t num_kv_heads;  /* Hkv >= 1                                    */
  int32_t head_dim;      /* d, must be 128                              */
  int32_t block_size;    /* B, 16 or 32                                 */
  int32_t max_blocks;    /* NBmax >= 1: row stride of block table, summaries and scores */
} oasis_dims;

/* Message for the last non-OK status returned on this thread ("" if none). */
OASIS_API const char* oasis_last_error(void);

/* OASIS_ABI_VERSION of the loaded library. */
OASIS_API int32_t oasis_abi_version(void);

/*
 * Compressed keys (paper §4.2.1 and the "Look-ahead attention" figure: Quest-
 * style per-block min/max pooling; §5.2: two summary rows per block, 1/16 of
 * the KV size at B = 16). For every request r, KV head h and candidate block
 * b < n_cand_r: kmax[r][h][b][:] / kmin[r][h][b][:] = coordinate-wise max /
 * min of the B keys of logical block b, read from page block_table[r][b].
 * Rows b >= n_cand_r are not written. The result is exact (bf16 min/max).
 *
 * k_pages: device-accessible pages (device memory, or pinned host memory
 * from hipHostMalloc) [num_pages][Hkv][B][d]. block_table, ctx_len: device.
 */
OASIS_API oasis_status oasis_build_summaries(const oasis_dims* dims, const uint16_t* k_pages, int64_t num_pages,
                                   const int32_t* block_table, const int32_t* ctx_len,
                                   uint16_t* kmax, uint16_t* kmin, void* stream);

/*
 * Compressed-key update on append (paper §5.1 lists compressed-key updates
 * among the native operations; §4.2.1 defines the rows). For every request r:
 * the rows of the candidate blocks completed since prev_ctx_len[r], i.e.
 * b in [n_cand(prev_ctx_len[r]), n_cand(ctx_len[r])), at most max_new_blocks
 * of them from the first, are written as oasis_build_summaries writes them;
 * every other row is untouched. ctx_len[r] <= prev_ctx_len[r] writes nothing.
 * A caller appending one token per step passes max_new_blocks = 1; a bound
 * below a request's growth leaves its later rows unwritten.
 * k_pages: device memory or pinned host memory; everything else: device.
 */
OASIS_API oasis_status oasis_update_summaries(const oasis_dims* dims, const uint16_t* k_pages, int64_t num_pages,
                                    const int32_t* block_table, const int32_t* prev_ctx_len,
                                    const int32_t* ctx_len, int32_t max_new_blocks,
                                    uint16_t* kmax, uint16_t* kmin, void* stream);

/*
 * Block copy between two paged KV tiers (paper §4.3: once a request's context
 * passes the sparsification threshold, its whole KV cache is copied to CPU
 * memory while the GPU keeps only the selected blocks and the local window;
 * blocks that receive new tokens afterwards must reach the full tier as well).
 * For every request r, the logical blocks holding tokens
 * [prev_ctx_len[r], ctx_len[r]) (prev_ctx_len NULL: from 0) are copied, at most
 * max_blocks of them from the first: page src_block_table[r][b] of src_k/src_v
 * to page dst_block_table[r][b] of dst_k/dst_v, all KV heads of the page
 * ([Hkv][B][d] each). Blocks past max_blocks of the table, or pages outside
 * [0, num_*_pages), are skipped. The dense-to-sparse transition is one call
 * with prev_ctx_len = NULL from the device pages to the pinned host tier,
 * followed by oasis_stage_blocks from the device pages (still resident) into
 * empty slots. src/dst: device memory or pinned host memory (device-visible;
 * the library resolves the address); block tables and lengths: device.
 * 1 <= max_blocks <= 65535.
 */
OASIS_API oasis_status oasis_copy_blocks(const oasis_dims* dims, const uint16_t* src_k, const uint16_t* src_v,
                               int64_t num_src_pages, const int32_t* src_block_table,
                               uint16_t* dst_k, uint16_t* dst_v, int64_t num_dst_pages,
                               const int32_t* dst_block_table, const int32_t* prev_ctx_len,
                               const int32_t* ctx_len, int32_t max_blocks, void* stream);

/*
 * Block importance from the lookahead (draft) queries (paper §4.2.1: the
 * prediction reads only the compressed keys and ranks every logical block,
 * separately per KV head). For row q of query head qh, the Quest upper
 * bound of block b is  sum_d max(q_d * kmin_d, q_d * kmax_d); the score of
 * (r, h, b) is the maximum of that bound over the rows t in [first_draft,
 * first_draft + num_draft) and the G query heads of KV head h. Scores of
 * b in [n_cand_r, NBmax) are -inf. No 1/sqrt(d) factor (ranking only).
 *
 * Requires kmin <= kmax coordinate-wise (as built by oasis_build_summaries).
 * Arithmetic: bf16 products, fp32 accumulation (MFMA for 5 to 64 rows; up to
 * 4 rows, a quarter of an MFMA tile, v_dot2 on the vector ALUs).
 * num_draft * G <= 64.
 * All pointers are device pointers.
 */
OASIS_API oasis_status oasis_score_blocks(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                int32_t first_draft, int32_t num_draft,
                                const uint16_t* kmax, const uint16_t* kmin, const int32_t* ctx_len,
                                float* scores, void* stream);

/*
 * Top-K selection (paper §4.2.1-§4.2.2: top-K prediction per KV head; §5.2:
 * K = 128 blocks of 16 tokens = the 2,048-token budget, which is also the
 * sparsification threshold). For every (r, h): the m = min(k, n_cand_r)
 * candidates with the largest score, equal scores going to the lower block
 * id (-0.0 equals +0.0). sel[r][h][0..m) lists them in ascending block id,
 * sel[r][h][m..k) = -1, sel_count[r][h] = m. Deterministic and exact.
 * Candidate scores must be finite. 1 <= k <= 65536. Device pointers.
 */
OASIS_API oasis_status oasis_select_topk(const oasis_dims* dims, const float* scores, const int32_t* ctx_len,
                               int32_t k, int32_t* sel, int32_t* sel_count, void* stream);

/*
 * oasis_score_blocks followed by oasis_select_topk in one kernel: one workgroup
 * per (request, KV head) scores the head's candidate blocks and selects its
 * top k from them (paper §4.2.1-§4.2.2), so the scores make no round trip
 * between two launches. Results (scores, sel, sel_count) are bit-identical to
 * the two calls. Worth it when the rows are many and short (hundreds of
 * (request, KV head) pairs with a few thousand blocks each); with few long rows
 * the two calls spread each row over many workgroups. Supported for
 * 5 <= num_draft * G <= 32 scoring rows and max_blocks <= 16,384
 * (OASIS_ERR_UNSUPPORTED otherwise); arguments as in the two calls. Device
 * pointers.
 */
OASIS_API oasis_status oasis_score_select(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                int32_t first_draft, int32_t num_draft, const uint16_t* kmax,
                                const uint16_t* kmin, const int32_t* ctx_len, int32_t k, float* scores,
                                int32_t* sel, int32_t* sel_count, void* stream);

/*
 * Delta selection + KV transfer into the HBM working set (paper §4.2.3: resident
 * hits stay and move no bytes; non-selected residents are evicted least-recently-
 * selected first; each admitted miss is paired with one eviction target; §4.3:
 * the head-wise slot map records which logical block every slot holds; §5.1:
 * the copy is a GPU kernel that pulls each admitted (block, KV head) entry out
 * of pinned host memory across PCIe into its pool slot).
 *
 * For every (r, h), with S = sel[r][h][0..sel_count) (ascending, as produced by
 * oasis_select_topk): misses = S minus the resident blocks; admitted = all
 * misses, or, when there are more than fetch_cap, the fetch_cap misses with the
 * highest scores[r][h][block] (equal scores: lower block id; §4.2.3 caps the
 * pairs per KV head and step, §5.5.1 sets the cap as a fraction of K); victims =
 * free slots (ascending), then resident non-selected slots by (slot_stamp, slot);
 * the i-th admitted miss in ascending block id goes to the i-th victim; slots
 * that receive nothing keep their block and stamp (a non-admitted miss is absent
 * for this step, and stale residents keep being attended). Each admitted block's
 * K entry (B x d) is copied from
 * host_k page host_block_table[r][block] head h into pool_k[r][slot][h], its V
 * entry into pool_v[r][slot][h] (transposed to d x B). slot_map is updated and
 * every slot that holds a selected block afterwards gets slot_stamp = step.
 * If copy_local != 0, slot k of every head is refreshed from the local block
 * (logical block nb_r - 1). moved[r][h] (nullable) = entries copied, local
 * block excluded. A miss whose page id is outside [0, num_pages) is not copied
 * and its victim slot is left free (-1).
 *
 * Local-only form: with sel == NULL and sel_count == NULL (and copy_local = 1)
 * only slot k is refreshed; slot_map, slot_stamp and moved may then be NULL. This stands in for the model writing the newest token's K/V
 * into the resident local block before attention.
 *
 * fetch_cap: most misses admitted per (r, h) per call, >= 1 (a fetch ratio rho
 * gives max(1, floor(rho * k))); fetch_cap >= k means uncapped. scores: the
 * [R][Hkv][max_blocks] fp32 output of oasis_score_blocks for this selection,
 * read only when fetch_cap < k (may be NULL otherwise); any value ranks
 * (order-preserving integer keys), so exactly min(fetch_cap, misses) are admitted.
 * host_k/host_v: pinned host memory (hipHostMalloc) or device memory; the
 * library resolves the device-visible address. Everything else: device.
 * sel must be strictly ascending within [0, sel_count); 1 <= k <= 1024.
 * slot_map must not hold one block twice. Calls that share slot_map/pools
 * must be ordered on one stream (or by events).
 */
OASIS_API oasis_status oasis_stage_blocks(const oasis_dims* dims, const uint16_t* host_k, const uint16_t* host_v,
                                int64_t num_pages, const int32_t* host_block_table, const int32_t* ctx_len,
                                const int32_t* sel, const int32_t* sel_count, const float* scores, int32_t k,
                                int32_t* slot_map, int32_t* slot_stamp, int32_t step, int32_t fetch_cap,
                                int32_t copy_local, uint16_t* pool_k, uint16_t* pool_v, int32_t* moved,
                                void* stream);

/*
 * Per-layer union of the per-head top-K sets (paper §4.4.1: for disaggregated
 * admission the prefill node sends, per layer, every block whose token range
 * at least one KV head selected, with its index). For every request r:
 * union_ids[r][0..union_count[r]) = the distinct ids of sel[r][h][0..sel_count)
 * over all heads h, ascending; union_ids[r][union_count[r]..Hkv*k) = -1. Ids
 * outside [0, max_blocks) are ignored; counts are clamped to [0, k].
 * union_ids: device [R][Hkv * k]; union_count: device [R]; sel, sel_count as
 * produced by oasis_select_topk. max_blocks <= 524,288; 1 <= k <= 65536.
 */
OASIS_API oasis_status oasis_union_selection(const oasis_dims* dims, const int32_t* sel, const int32_t* sel_count,
                                   int32_t k, int32_t* union_ids, int32_t* union_count, void* stream);

/* Bytes of workspace oasis_sparse_decode_attn needs for these sizes: the split
 * partials (fp32 output, maximum and sum per split and row), 0 when a single
 * split per (request, KV head) suffices (then the workspace may be NULL) or
 * when the sizes are invalid. Calls that run at the same time need separate
 * workspaces. */
OASIS_API size_t oasis_attn_workspace_bytes(const oasis_dims* dims, int32_t num_q_tokens, int32_t k_slots);

/*
 * Block-sparse GQA decode attention over the working set (paper §4.2.1: the
 * normal and draft queries are stacked and attend one resident KV set in one
 * call that returns both outputs; §5.2: each head attends its K selected
 * blocks plus the active local block -- 129 blocks, 2,064 tokens at K = 128,
 * B = 16). For every request r, query row t and query head qh (KV head
 * h = qh / G), the attended set is the B tokens of every slot s < k_slots with
 * slot_map[r][h][s] >= 0, plus the first local_len_r tokens of slot k_slots:
 *   out = softmax(scale * q . K^T) V,  lse = log sum exp(scale * q . K^T).
 * No mask among the T rows; an empty set gives out = 0, lse = -inf.
 * Arithmetic: bf16 inputs, fp32 logits / softmax / accumulation (MFMA), the
 * probabilities rounded to bf16 for the PV product, bf16 output.
 * G * T <= 80. lse is nullable. Device pointers.
 */
OASIS_API oasis_status oasis_sparse_decode_attn(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens,
                                      const uint16_t* pool_k, const uint16_t* pool_v,
                                      const int32_t* slot_map, int32_t k_slots, const int32_t* ctx_len,
                                      float scale, uint16_t* out, float* lse,
                                      void* workspace, size_t workspace_bytes, void* stream);

/*
 * oasis_sparse_decode_attn without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * that must not call the allocator, harnesses that forbid it). Same operation,
 * arguments, layouts and checks as oasis_sparse_decode_attn; the split partials
 * go to a scratch array of the library in device memory: OASIS_NOALLOC_SCRATCH_BYTES
 * (16 MiB) per GPU, held from the library's load until the process ends. Sizes
 * whose oasis_attn_workspace_bytes exceeds it return OASIS_ERR_UNSUPPORTED
 * without launching. Nothing is allocated, on the host or the device; the first
 * call on a device looks up the scratch array's address there (one runtime
 * query, not an allocation). Every call on one GPU shares that GPU's scratch:
 * calls that overlap in time on one GPU (different streams, or a graph replayed
 * beside another call) race and may corrupt each other's results; order them on
 * one stream. The scratch needs no clearing between calls (each call writes the
 * partials it reads).
 */
#define OASIS_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
OASIS_API oasis_status oasis_sparse_decode_attn_noalloc(const oasis_dims* dims, const uint16_t* q,
                                              int32_t num_q_tokens, const uint16_t* pool_k,
                                              const uint16_t* pool_v, const int32_t* slot_map, int32_t k_slots,
                                              const int32_t* ctx_len, float scale, uint16_t* out, float* lse,
                                              void* stream);

/*
 * Native step issuer for the layer-pipelined schedule (paper §4.2.2, the
 * asynchronous prefetch pipeline figure and Eq. "prefetch-rate"; §5.1: the
 * stages run on background streams and events order each layer's chain).
 * One oasis_pipeline_step call issues one layer's decode step on three HIP
 * streams:
 *   foreground (`stream`): wait for this layer's transfer issued at its
 *     previous step (a layer-local wait, not a wait for every layer), refresh
 *     the local block if `growing`, then oasis_sparse_decode_attn over the
 *     working set;
 *   prediction stream: once q is ready and the layer's previous transfer has
 *     read sel and scores, oasis_score_blocks on the draft rows of q and
 *     oasis_select_topk (the prediction for the layer's next step; both in one
 *     kernel under oasis_pipeline_set_fused_prediction);
 *   transfer stream: once the prediction is ready and this step's attention
 *     has read the pools, oasis_stage_blocks (delta selection with the fetch
 *     cap, then the gather; the paper's selection and transfer stages are one
 *     kernel here), with copy_local = 0. The local block is rewritten on
 *     the foreground when `growing`; otherwise the context has not changed
 *     since the local block was last staged (the caller stages it once, e.g.
 *     in the initial fill) and it stays in place.
 * Consecutive calls for different layers overlap one layer's transfer with
 * the next layers' attention and prediction. The streams are ordered through
 * monotone counters in device memory, raised by a stream write-value after
 * the producer: the foreground waits for them with a stream wait-value, the
 * staging kernel polls its two itself (bounded, see
 * oasis_pipeline_set_wait_limit). Three or four such edges and four to seven
 * kernel launches per step (attention split and merge, scoring and top-K or
 * their fused kernel, staging; the local refresh and the compressed-key
 * update when growing), nothing allocated.
 *
 * Arguments are checked on every step exactly as the four entry points check
 * them. Ownership: every pointer stays the caller's and must outlive the
 * pipeline's use of it (tensors read by a step stay alive until the layer's
 * next step or a join); the pipeline owns its counter array (hipMalloc at
 * create, 256 bytes per counter, (5 + max_layers) counters), with the plan on
 * the prediction stream one staging-plan workspace per registered layer
 * (hipMalloc at set_plan_stream or set_layer, R * Hkv * (4 * k + 1) int32),
 * and the two background streams when it creates them; destroy frees them. host_k/host_v are resolved to
 * device-visible addresses once, at create. All calls for one pipeline must come
 * from one host thread with the creating device current.
 */
typedef struct oasis_pipeline oasis_pipeline;

/* Per-layer device buffers of the path (shapes as in the entry points above). */
typedef struct {
  uint16_t* kmax;          /* bf16 [R][Hkv][max_blocks][d] (oasis_build_summaries) */
  uint16_t* kmin;
  float* scores;           /* [R][Hkv][max_blocks] */
  int32_t* sel;            /* [R][Hkv][k] */
  int32_t* sel_count;      /* [R][Hkv] */
  int32_t* slot_map;       /* [R][Hkv][k], -1 = free */
  int32_t* slot_stamp;     /* [R][Hkv][k] */
  uint16_t* pool_k;        /* bf16 [R][k+1][Hkv][B][d] */
  uint16_t* pool_v;        /* bf16 [R][k+1][Hkv][d][B] */
  int32_t* moved;          /* [R][Hkv], nullable */
  uint16_t* out;           /* bf16 [R][T][Hq][d] */
  float* lse;              /* [R][T][Hq], nullable */
  void* workspace;         /* oasis_attn_workspace_bytes(dims, T, k) bytes */
  size_t workspace_bytes;
} oasis_layer_buffers;

/* pred_stream / xfer_stream: caller streams (non-blocking, default priority) or
 * NULL to let the pipeline create its own. max_layers >= 1 bounds the layer ids
 * of set_layer / step. fetch_cap as in oasis_stage_blocks (>= k: uncapped). */
OASIS_API oasis_status oasis_pipeline_create(const oasis_dims* dims, int32_t num_q_tokens, int32_t first_draft,
                                   int32_t num_draft, int32_t k, int32_t fetch_cap, float scale,
                                   const uint16_t* host_k, const uint16_t* host_v, int64_t num_pages,
                                   const int32_t* host_block_table, int32_t max_layers, void* pred_stream,
                                   void* xfer_stream, oasis_pipeline** pipeline);

/* Register (or replace) the buffers of layer `layer` (0 <= layer < max_layers). A
 * transfer already issued for the layer is still waited on at its next step.
 * Errors: INVALID_ARG for a NULL pipeline or buffers or a layer out of range;
 * HIP when the layer's plan workspace (OASIS_PLAN_ON_PREDICTION) cannot be
 * allocated. */
OASIS_API oasis_status oasis_pipeline_set_layer(oasis_pipeline* pipeline, int32_t layer,
                                      const oasis_layer_buffers* buffers);

/* Pages the local block is refreshed from when a step is `growing` (by default
 * the host tier given at create). A growing context's newest tokens are written
 * by the model on the GPU, so a caller that keeps the active blocks in device
 * pages passes them here and the refresh stays off the PCIe link. k_pages /
 * v_pages: bf16 [num_pages][Hkv][B][d], device memory or pinned host memory
 * (the library resolves the address); block_table: device [R][max_blocks],
 * -1 or out-of-range ids skipped. All three NULL restores the host tier. The
 * pointers stay the caller's and must outlive the steps that use them; steps
 * already issued keep the source they were issued with. */
OASIS_API oasis_status oasis_pipeline_set_local_source(oasis_pipeline* pipeline, const uint16_t* k_pages,
                                             const uint16_t* v_pages, int64_t num_pages,
                                             const int32_t* block_table);

/* Where a step plans its transfer (paper §4.2.3, the delta selection between the
 * prediction and the transfer of §4.2.2). OASIS_PLAN_ON_TRANSFER (the default):
 * the staging kernel on the transfer stream plans and then copies.
 * OASIS_PLAN_ON_PREDICTION: the top-K kernel on the prediction stream plans
 * right after it selects, into a workspace of the layer (the slot map the
 * attention reads stays untouched), and the transfer stream only copies and
 * commits. Moving the plan pays when the transfer stream is the longer one and
 * its workgroups would plan several passes of pairs each (measured on MI355X:
 * 32 layers x 64 requests +4 %; 8 x 131,072 tokens -16 %, 32 requests of
 * 16K-32K tokens -13 %, 16 x 65,536 tokens at B = 32 -23 %). Both give the same
 * slot maps, stamps, counts and pools. Takes effect from the next step issued;
 * OASIS_PLAN_ON_PREDICTION allocates the plan workspace of every registered
 * layer that has none. Errors: INVALID_ARG for a NULL pipeline or another
 * value; HIP when a workspace cannot be allocated (the setting is unchanged). */
#define OASIS_PLAN_ON_TRANSFER 0
#define OASIS_PLAN_ON_PREDICTION 1
OASIS_API oasis_status oasis_pipeline_set_plan_stream(oasis_pipeline* pipeline, int32_t where);

/* How a step predicts (paper §4.2.1-§4.2.2). OASIS_FUSED_PREDICTION_AUTO (the
 * default): scoring and top-K (and the plan, when it runs on the prediction
 * stream) in one kernel with one workgroup per (request, KV head), as
 * oasis_score_select does, when the step has at least 256 such pairs and
 * oasis_score_select supports the sizes; otherwise the separate kernels.
 * OASIS_FUSED_PREDICTION_OFF: always the separate kernels.
 * OASIS_FUSED_PREDICTION_ON: the fused kernel whenever the sizes are supported.
 * The results are the same either way. Takes effect from the next step.
 * Errors: INVALID_ARG for a NULL pipeline or another value. */
#define OASIS_FUSED_PREDICTION_AUTO 0
#define OASIS_FUSED_PREDICTION_OFF 1
#define OASIS_FUSED_PREDICTION_ON 2
OASIS_API oasis_status oasis_pipeline_set_fused_prediction(oasis_pipeline* pipeline, int32_t mode);

/* Where a step's prediction (scoring and top-K on the prediction stream)
 * starts. OASIS_PREDICT_BESIDE_ATTENTION (paper §4.2.2: the prediction runs
 * in the background beside the foreground's attention): once the step's
 * queries are ready, and the transfer waits for the prediction and for the
 * attention. OASIS_PREDICT_AFTER_ATTENTION: once the step's attention has
 * finished, and the transfer waits for the prediction alone; one
 * cross-stream edge fewer, and the bandwidth-bound scorer no longer shares
 * HBM with this attention (it still runs beside the next layers'). The
 * results are the same either way; which is faster depends on the shapes.
 * OASIS_PREDICT_AUTO (default): after the attention for at most 64
 * (request, KV head) pairs, beside it otherwise. Takes effect from the next
 * step. Errors: INVALID_ARG for a NULL pipeline or another value. */
#define OASIS_PREDICT_AUTO 0
#define OASIS_PREDICT_BESIDE_ATTENTION 1
#define OASIS_PREDICT_AFTER_ATTENTION 2
OASIS_API oasis_status oasis_pipeline_set_prediction_order(oasis_pipeline* pipeline, int32_t order);

/* Issue one decode step of `layer` (see above). q: bf16 device [R][T][Hq][d];
 * ctx_len: device [R]; prev_ctx_len (nullable, device [R]): the lengths at the
 * layer's previous step; when set, the compressed keys of the blocks completed
 * since then (at most max_new_blocks >= 1 per request) are added on the
 * prediction stream before the scoring (as oasis_update_summaries, reading the
 * local-block source, where the newest tokens are), so that this small kernel
 * does not wait behind the scan on the foreground; step: the stamp of this
 * step's selection; moved: where the transfer writes its per-(r, h) entry
 * counts (NULL: the layer's buffer). */
OASIS_API oasis_status oasis_pipeline_step(oasis_pipeline* pipeline, int32_t layer, const uint16_t* q,
                                 const int32_t* ctx_len, const int32_t* prev_ctx_len, int32_t max_new_blocks,
                                 int32_t step, int32_t growing, int32_t* moved, void* stream);

/* Make `stream` wait for all work issued so far on the two background streams. */
OASIS_API oasis_status oasis_pipeline_join(oasis_pipeline* pipeline, void* stream);

/* Profile the next max_steps steps: each kernel launch carries timing events
 * that take the start and end timestamps of its own dispatch, on the stream it
 * runs on (attention from its split kernel's start to its merge kernel's end on the foreground;
 * scoring and top-K on the prediction stream; staging on the transfer stream).
 * The events are created here, not in the steps. */
OASIS_API oasis_status oasis_pipeline_profile_begin(oasis_pipeline* pipeline, int32_t max_steps);

/* Wait for the profiled steps and write the mean duration in microseconds of
 * attention, scoring, top-K and staging to avg_us[0..3]. step_us (nullable,
 * caller-owned, room for max_steps x 4 floats as passed to profile_begin)
 * receives each profiled step's four durations, step-major in the same order;
 * steps (nullable) receives how many steps were profiled. Releases the
 * profile's events. */
OASIS_API oasis_status oasis_pipeline_profile_end(oasis_pipeline* pipeline, float* avg_us, float* step_us,
                                                  int32_t* steps);

/* Synchronize the device, then report whether any transfer of this pipeline
 * gave up waiting for its prediction. The staging kernel of a step waits for
 * the step's prediction itself, polling the counter the prediction stream
 * raises, for a bounded time (oasis_pipeline_set_wait_limit; a few seconds by
 * default); past that it marks a fault and proceeds (its
 * results are then undefined) instead of holding the GPU. OASIS_OK when no
 * fault was marked, OASIS_ERR_HIP when one was (or a HIP call failed). */
OASIS_API oasis_status oasis_pipeline_check(oasis_pipeline* pipeline);

/* Bound of the staging kernel's wait for its prediction, in polls (each about
 * a microsecond; default 2^21, a few seconds), from the next step on. A smaller
 * bound reports a stalled prediction sooner; a step whose prediction is merely
 * slower than the bound then marks a fault too. Errors: INVALID_ARG for a NULL
 * pipeline or polls = 0. */
OASIS_API oasis_status oasis_pipeline_set_wait_limit(oasis_pipeline* pipeline, uint32_t polls);

/* Synchronize the device, then release the counters (and owned streams). NULL is a no-op. */
OASIS_API void oasis_pipeline_destroy(oasis_pipeline* pipeline);

#ifdef __cplusplus
}
#endif

#endif /* OASIS_H */
