// Block importance for a few draft rows (paper §4.2.1; the bound is the one
// of score.hip): up to 4 rows of a KV head, a quarter of a 16-row MFMA tile,
// are scored on the vector ALUs instead. Measured at 8 x 8 x 8,192 blocks:
// 47.5 us here against 48.2 us for the padded MFMA tile at 4 rows; at 8 rows
// the dot products and row sums make it slower (58 us against 49 us), so the
// MFMA kernel takes 5 rows and more.
//
// Layout: lane (j, c) of a wave holds the 8 dimensions 8c .. 8c+7 of block j
// of a group of 4 consecutive blocks, so one 16-byte load instruction reads 4
// whole summary rows (1 KiB contiguous); every lane loads the kmax and kmin
// slices of all kGroups groups before it computes. For each row, the lane's
// partial bound is two chains of v_dot2 over its 8 dimensions
// ([q+ | q-] . [kmax ; kmin], bf16 products, fp32 accumulation); four DPP
// adds inside the 16 lanes of a block (one DPP row) sum the partials over
// head_dim, and the maximum over the draft rows is kept in the lane. Lanes past the
// candidates re-read the last candidate block (a cache hit) and write -inf.
#include "oasis_internal.h"

namespace oasis {

namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kGroups = 8;  // groups of 4 blocks per wave: 32 blocks

__device__ __forceinline__ float dot2(uint32_t x, uint32_t y, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x), __builtin_bit_cast(bf16x2, y), acc, false);
}

// Value of another lane of the same 16-lane row, moved by a DPP control.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row, left in every lane: row mirror (lane i
// with 15 - i), half-row mirror (i with 7 - i within 8), then the two quad
// exchanges (i with i ^ 2, i with i ^ 1). After the two mirrors lanes 0..3
// hold the sums of {0,15,7,8}, {1,14,6,9}, {2,13,5,10}, {3,12,4,11}, and so on
// for every quad, so the quad exchanges complete the sum.
__device__ __forceinline__ float row16_sum(float s) {
  s += dpp<0x140>(s);  // row_mirror
  s += dpp<0x141>(s);  // row_half_mirror
  s += dpp<0x4E>(s);   // quad_perm [2, 3, 0, 1]
  s += dpp<0xB1>(s);   // quad_perm [1, 0, 3, 2]
  return s;
}

template <int ROWS>
__global__ __launch_bounds__(256) void score_valu_kernel(ScoreArgs a) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int j = lane >> 4;  // block within the group
  const int c = lane & 15;  // 8-dimension slice
  const int rh = blockIdx.y;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const Ctx cx = ctx_blocks(a.ctx_len[r], a.B, a.NBmax);
  // block groups rotated by the row, as in the MFMA scorer: every group spread over the XCDs
  const int group = (int)((blockIdx.x + blockIdx.y) % gridDim.x);
  const int blk0 = (group * 4 + wave) * (4 * kGroups);
  if (blk0 >= a.NBmax) return;

  float* srow = a.scores + (long long)rh * a.NBmax;
  const long long base = (long long)rh * a.NBmax * kHeadDim + c * 8;
  const int last = cx.n_cand > 0 ? cx.n_cand - 1 : 0;
  u32x4 vmax[kGroups], vmin[kGroups];
#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int blk = min(blk0 + 4 * gi + j, last);
    vmax[gi] = ldg16(a.kmax + base + (long long)blk * kHeadDim);
    vmin[gi] = ldg16(a.kmin + base + (long long)blk * kHeadDim);
  }

  // [q+ | q-] of this lane's slice for every row; rows past the last real row
  // repeat row 0, which leaves the maximum unchanged
  const int nrows = a.num_draft * a.G;
  u32x4 qp[ROWS], qn[ROWS];
#pragma unroll
  for (int v = 0; v < ROWS; ++v) {
    const int row = v < nrows ? v : 0;
    const int t = a.first_draft + row / a.G;
    const int qh = h * a.G + row % a.G;
    split_sign(ldg16(a.q + (((long long)r * a.T + t) * a.Hq + qh) * kHeadDim + c * 8), qp[v], qn[v]);
  }

#pragma unroll
  for (int gi = 0; gi < kGroups; ++gi) {
    const int g0 = blk0 + 4 * gi;
    if (g0 >= a.NBmax) break;
    float best = -INFINITY;
    if (g0 < cx.n_cand) {
#pragma unroll
      for (int v = 0; v < ROWS; ++v) {
        float pos = 0.f, neg = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          pos = dot2(qp[v][w], vmax[gi][w], pos);
          neg = dot2(qn[v][w], vmin[gi][w], neg);
        }
        best = fmaxf(best, row16_sum(pos + neg));
      }
    }
    const int blk = g0 + j;
    if (c == 0 && blk < a.NBmax) srow[blk] = blk < cx.n_cand ? best : -INFINITY;
  }
}

template <int ROWS>
hipError_t launch_rows(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t) {
  constexpr int kPerWorkgroup = 4 * 4 * kGroups;  // 4 waves x 32 blocks
  const dim3 grid((unsigned)((a.NBmax + kPerWorkgroup - 1) / kPerWorkgroup), (unsigned)(a.R * a.Hkv));
  launch_kernel(score_valu_kernel<ROWS>, grid, dim3(256), s, t, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_valu(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int rows = a.num_draft * a.G;
  if (rows <= 1) return launch_rows<1>(a, s, t);
  if (rows <= 2) return launch_rows<2>(a, s, t);
  if (rows <= kScoreValuMaxRows) return launch_rows<kScoreValuMaxRows>(a, s, t);
  return hipErrorInvalidValue;
}

}  // namespace oasis
