// Internal declarations of the OasisKV HIP library (gfx950 / MI355X).
#pragma once

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

struct SummaryArgs {
  const uint16_t* k_pages;
  int64_t num_pages;
  const int32_t* block_table;
  const int32_t* ctx_len;
  uint16_t* kmax;
  uint16_t* kmin;
  int R, Hkv, B, NBmax;
};
hipError_t launch_summaries(const SummaryArgs& a, hipStream_t s);

struct ScoreArgs {
  const uint16_t* q;
  const uint16_t* kmax;
  const uint16_t* kmin;
  const int32_t* ctx_len;
  float* scores;
  int R, Hq, Hkv, G, T, first_draft, num_draft, B, NBmax;
};
hipError_t launch_score(const ScoreArgs& a, hipStream_t s);

struct TopkArgs {
  const float* scores;
  const int32_t* ctx_len;
  int32_t* sel;
  int32_t* sel_count;
  int R, Hkv, B, NBmax, k;
};
hipError_t launch_topk(const TopkArgs& a, hipStream_t s);

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
};
hipError_t launch_stage(const StageArgs& a, hipStream_t s);

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
hipError_t launch_attn(const AttnArgs& a, hipStream_t s);

}  // namespace oasis
