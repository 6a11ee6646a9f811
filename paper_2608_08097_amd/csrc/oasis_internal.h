// Internal declarations of the OasisKV HIP library (gfx950 / MI355X).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oasis.h"

namespace oasis {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kHeadDim = 128;
constexpr int kWave = 64;

// --- small device helpers ---------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Round-to-nearest-even float -> bf16 bits (inputs are finite here).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ u32x4 ldg16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Number of logical blocks, candidate blocks and local-block tokens of a context.
struct Ctx {
  int nb, n_cand, local_len;
};
__device__ __forceinline__ Ctx ctx_blocks(int L, int B, int max_blocks) {
  Ctx c;
  long long cap = (long long)max_blocks * B;
  if (L < 0) L = 0;
  if ((long long)L > cap) L = (int)cap;
  c.nb = (L + B - 1) / B;
  c.n_cand = c.nb > 0 ? c.nb - 1 : 0;
  c.local_len = L - B * c.n_cand;
  return c;
}

// --- host-side launchers (one per .hip translation unit) ---------------------

// Optional timing of one launch: when set, the events take the start / end
// timestamps of the kernel dispatch itself (not of a marker next to it).
struct LaunchTiming {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};

template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, hipStream_t s, const LaunchTiming& t, Args... args) {
  if (t.start || t.stop)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, t.start, t.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, args...);
}

struct SummaryArgs {
  const uint16_t* k_pages;
  int64_t num_pages;
  const int32_t* block_table;
  const int32_t* ctx_len;
  uint16_t* kmax;
  uint16_t* kmin;
  int R, Hkv, B, NBmax;
  const int32_t* prev_ctx_len;  // NULL: every candidate block; else blocks completed since this length
  int max_new;                  // with prev_ctx_len: at most this many rows per request
};
hipError_t launch_summaries(const SummaryArgs& a, hipStream_t s);

struct CopyArgs {
  const uint16_t* src_k;  // device-visible addresses, pages [num_pages][Hkv][B][d]
  const uint16_t* src_v;
  int64_t num_src_pages;
  const int32_t* src_table;
  uint16_t* dst_k;
  uint16_t* dst_v;
  int64_t num_dst_pages;
  const int32_t* dst_table;
  const int32_t* prev_ctx_len;  // NULL: from token 0
  const int32_t* ctx_len;
  int R, Hkv, B, NBmax, max_blocks;
};
hipError_t launch_copy_blocks(const CopyArgs& a, hipStream_t s);

struct UnionArgs {
  const int32_t* sel;       // [R][Hkv][k]
  const int32_t* sel_count; // [R][Hkv]
  int32_t* ids;             // [R][Hkv * k]
  int32_t* count;           // [R]
  int R, Hkv, NBmax, k;
};
constexpr int kUnionMaxBlocks = 1 << 19;  // LDS bitmap of 64 KiB (the default dynamic LDS limit)
hipError_t launch_union(const UnionArgs& a, hipStream_t s);

struct ScoreArgs {
  const uint16_t* q;
  const uint16_t* kmax;
  const uint16_t* kmin;
  const int32_t* ctx_len;
  float* scores;
  int R, Hq, Hkv, G, T, first_draft, num_draft, B, NBmax;
};
hipError_t launch_score(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t = {});
// Scorer on the vector ALUs for at most kScoreValuMaxRows rows (launch_score
// calls it for those row counts).
constexpr int kScoreValuMaxRows = 4;
hipError_t launch_score_valu(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t = {});

// Wave-wide inclusive prefix sum on the DPP network (no LDS round trips):
// row shifts by 1, 2, 4 and 8 give each 16-lane row its own prefix sums, then
// row broadcasts of lanes 15 and 31 carry the totals of the earlier rows.
__device__ __forceinline__ int wave_incl_sum(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, false);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1 and 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31 into rows 2 and 3
  return x;
}

// Split bf16 pairs into their non-negative and non-positive parts (bitwise, exact).
__device__ __forceinline__ void split_sign(u32x4 v, u32x4& pos, u32x4& neg) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t negmask = ((v[w] & 0x80008000u) >> 15) * 0xFFFFu;
    neg[w] = v[w] & negmask;
    pos[w] = v[w] & ~negmask;
  }
}

struct TopkArgs {
  const float* scores;
  const int32_t* ctx_len;
  int32_t* sel;
  int32_t* sel_count;
  int R, Hkv, B, NBmax, k;
};
hipError_t launch_topk(const TopkArgs& a, hipStream_t s, const LaunchTiming& t = {});

struct StageArgs {
  const uint16_t* host_k;   // device-visible addresses
  const uint16_t* host_v;
  int64_t num_pages;
  const int32_t* block_table;
  const int32_t* ctx_len;
  const int32_t* sel;
  const int32_t* sel_count;
  const float* scores;      // [R][Hkv][NBmax], read only under a binding cap
  int32_t* slot_map;
  int32_t* slot_stamp;
  uint16_t* pool_k;
  uint16_t* pool_v;
  int32_t* moved;
  int R, Hkv, B, NBmax, k, step, copy_local;
  int fetch_cap;            // admitted misses per (request, KV head), >= k: all
  int local_only;           // no selection: refresh the local block only
  // kStagePlanCopy: plan, update slot_map / slot_stamp, copy. kStagePlanOnly:
  // plan into `ws` (new map and stamp rows, admitted entries, their counts),
  // leaving slot_map / slot_stamp as they are; nothing is copied. kStageCopyOnly:
  // copy the entries in `ws` and commit its rows to slot_map / slot_stamp.
  int mode;
  int32_t* ws;              // stage_ws_ints(R * Hkv, k) ints (modes 1 and 2)
  // For each wait_flag[i] that is set, the staging kernel first waits until
  // *wait_flag[i] >= wait_value[i] (counters that other streams' work raises):
  // one thread of each workgroup polls them, at most wait_polls times in all;
  // past that the workgroup stores 1 to *wait_fault and goes on.
  const uint32_t* wait_flag[2];
  uint32_t wait_value[2];
  uint32_t* wait_fault;
  uint32_t wait_polls;
};
// default bound of the staging kernel's counter wait in the pipeline: each poll
// is a 128-clock sleep and an uncached load (about a microsecond), a few
// seconds in all
constexpr uint32_t kStageWaitSpins = 1u << 21;
constexpr int kStagePlanCopy = 0, kStagePlanOnly = 1, kStageCopyOnly = 2;
// Plan workspace: [nrh][k] map rows, [nrh][k] stamp rows, [nrh][k][2] entries (slot, page), [nrh] counts.
inline size_t stage_ws_ints(long long nrh, int k) { return (size_t)nrh * (4 * (size_t)k + 1); }
// Top-K (as launch_topk) and the staging plan of each (request, KV head) in one
// kernel; a.mode must be kStagePlanOnly (the plan goes to a.ws).
hipError_t launch_topk_plan(const TopkArgs& t, const StageArgs& a, hipStream_t s, const LaunchTiming& lt = {});
hipError_t launch_stage(const StageArgs& a, hipStream_t s, const LaunchTiming& t = {});
// Scoring and top-K of each (request, KV head) in one workgroup (stage.hip), with
// the transfer plan when `plan` is set (mode kStagePlanOnly, into plan->ws).
// Scores and selections are identical to launch_score followed by launch_topk.
// For 5 to kScoreSelectMaxRows scoring rows (more would not fit the registers of
// a 1024-thread workgroup) and at most kScoreSelectMaxBlocks blocks per row.
constexpr int kScoreSelectMaxRows = 32;
constexpr int kScoreSelectMaxBlocks = 16384;
bool score_select_supported(const ScoreArgs& sa);
hipError_t launch_score_select(const ScoreArgs& sa, const TopkArgs& t, const StageArgs* plan, hipStream_t s,
                               const LaunchTiming& lt = {});

struct AttnArgs {
  const uint16_t* q;
  const uint16_t* pool_k;
  const uint16_t* pool_v;
  const int32_t* slot_map;
  const int32_t* ctx_len;
  uint16_t* out;
  float* lse;
  float* part_o;            // workspace [R*Hkv][nsplit][rows][d]
  float* part_ml;           // workspace [R*Hkv][nsplit][rows][2]
  int R, Hq, Hkv, G, T, B, NBmax, k_slots;
  float scale_log2;         // scale * log2(e)
  int rows, n_units, nsplit, units_per_split;
};
struct AttnPlan {
  int rows, n_units, nsplit, units_per_split;
  size_t part_o_floats, part_ml_floats, bytes;
};
AttnPlan attn_plan(int R, int Hq, int Hkv, int T, int B, int k_slots);
hipError_t launch_attn(const AttnArgs& a, hipStream_t s, const LaunchTiming& t = {});
// Scratch of oasis_sparse_decode_attn_noalloc: a device array of this many bytes
// per GPU (attn.hip); noalloc_scratch returns its address on the current device.
constexpr size_t kNoAllocScratchBytes = OASIS_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch(void** ptr);

// --- argument checks shared by the entry points (api.hip) ---------------------
// Each builder validates like the entry point of the same operation (fn names
// it in the message) and fills the kernel arguments; with num_reqs == 0 it
// returns OASIS_OK without checking pointers and leaves *a untouched.

oasis_status fail(oasis_status st, const char* fmt, ...);
oasis_status ok();
const char* last_error();
oasis_status hip_status(hipError_t e, const char* where);
oasis_status check_dims(const oasis_dims* d, const char* fn);
// Device-visible address of pinned host memory (or of device memory as is).
oasis_status device_view(const void* p, const void** out, const char* what, const char* fn);

oasis_status make_score_args(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens, int32_t first_draft,
                             int32_t num_draft, const uint16_t* kmax, const uint16_t* kmin, const int32_t* ctx_len,
                             float* scores, ScoreArgs* a, const char* fn);
oasis_status make_topk_args(const oasis_dims* dims, const float* scores, const int32_t* ctx_len, int32_t k,
                            int32_t* sel, int32_t* sel_count, TopkArgs* a, const char* fn);
oasis_status make_stage_args(const oasis_dims* dims, const uint16_t* host_k, const uint16_t* host_v,
                             int64_t num_pages, const int32_t* host_block_table, const int32_t* ctx_len,
                             const int32_t* sel, const int32_t* sel_count, const float* scores, int32_t k,
                             int32_t* slot_map, int32_t* slot_stamp, int32_t step, int32_t fetch_cap,
                             int32_t copy_local, uint16_t* pool_k, uint16_t* pool_v, int32_t* moved, StageArgs* a,
                             const char* fn);
oasis_status make_attn_args(const oasis_dims* dims, const uint16_t* q, int32_t num_q_tokens, const uint16_t* pool_k,
                            const uint16_t* pool_v, const int32_t* slot_map, int32_t k_slots, const int32_t* ctx_len,
                            float scale, uint16_t* out, float* lse, void* workspace, size_t workspace_bytes,
                            AttnArgs* a, const char* fn);

}  // namespace oasis
