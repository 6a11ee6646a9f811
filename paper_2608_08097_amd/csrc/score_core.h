// Pieces of the MFMA block scorer (paper §4.2.1: Quest upper bound per draft row,
// maximum over the G x D rows of a KV head) shared by the scoring kernel and the
// fused score + select kernel, so that both compute bit-identical scores.
//
// For one row q and a block with per-coordinate bounds kmin <= kmax,
//   sum_d max(q_d kmin_d, q_d kmax_d) = sum_d (q+_d kmax_d + q-_d kmin_d)
// with q+ = max(q, 0), q- = min(q, 0): a dot product of [q+ | q-] with
// [kmax ; kmin], so 16 rows x a tile of 16 blocks is a [16 x 256] x [256 x 16]
// product on v_mfma_f32_16x16x32_bf16.
#pragma once

#include "oasis_internal.h"

namespace oasis {

// Query operands of a KV head's rows: [row tile][k-step][q+ / q-][lane], 16 bytes
// each, built once per workgroup in LDS so that every MFMA operand is one
// conflict-free 16-byte read.
template <int NRT>
using ScoreQOperands = u32x4[NRT][4][2][64];

// Raw query bytes of operand element e (row tile e >> 8, k-step (e >> 6) & 3,
// lane e & 63): 8 dims of one row. Rows past the last draft row repeat row 0,
// which leaves every maximum unchanged.
__device__ __forceinline__ u32x4 score_q_raw(const ScoreArgs& a, int r, int h, int e) {
  const int v = e >> 8;
  const int st = (e >> 6) & 3;
  const int el = e & 63;
  const int nrows = a.num_draft * a.G;
  int row = v * 16 + (el & 15);
  if (row >= nrows) row = 0;
  const int t = a.first_draft + row / a.G;
  const int qh = h * a.G + row % a.G;
  return ldg16(a.q + (((long long)r * a.T + t) * a.Hq + qh) * kHeadDim + st * 32 + (el >> 4) * 8);
}

template <int NRT>
__device__ __forceinline__ void score_q_store(ScoreQOperands<NRT>& s_q, int e, u32x4 raw) {
  u32x4 p, m;
  split_sign(raw, p, m);
  s_q[e >> 8][(e >> 6) & 3][0][e & 63] = p;
  s_q[e >> 8][(e >> 6) & 3][1][e & 63] = m;
}

// Summary rows of block tile*16 + n for lane (g, n): 16 bytes at 64*step + 16*g
// of the kmax row and of the kmin row (zero past the candidates).
__device__ __forceinline__ void score_tile_load(const uint16_t* kmx, const uint16_t* kmn, int tile, int n_cand,
                                                int g, int n, u32x4 (&vmax)[4], u32x4 (&vmin)[4]) {
  const int blk = tile * 16 + n;
  const bool live = blk < n_cand;
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const long long off = (long long)blk * kHeadDim + st * 32 + g * 8;
    vmax[st] = live ? ldg16(kmx + off) : u32x4{0, 0, 0, 0};
    vmin[st] = live ? ldg16(kmn + off) : u32x4{0, 0, 0, 0};
  }
}

// Operands of row tile v for this lane, from LDS into registers.
template <int NRT>
__device__ __forceinline__ void score_q_tile(const ScoreQOperands<NRT>& s_q, int v, int lane, bf16x8 (&ap)[4],
                                             bf16x8 (&an)[4]) {
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    ap[st] = as_bf16x8(s_q[v][st][0][lane]);
    an[st] = as_bf16x8(s_q[v][st][1][lane]);
  }
}

// Maximum over rows 4g .. 4g+3 of a row tile (operands ap / an) against block n
// of a tile (lane (g, n)), folded into `best`.
__device__ __forceinline__ float score_tile_fold(const bf16x8 (&ap)[4], const bf16x8 (&an)[4],
                                                 const u32x4 (&vmax)[4], const u32x4 (&vmin)[4], float best) {
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < 4; ++st)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ap[st], as_bf16x8(vmax[st]), acc, 0, 0, 0);
#pragma unroll
  for (int st = 0; st < 4; ++st)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(an[st], as_bf16x8(vmin[st]), acc, 0, 0, 0);
  return fmaxf(best, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
}

// The block's score in every lane: maximum over the four lane groups.
__device__ __forceinline__ float score_lane_reduce(float best) {
  const float b = fmaxf(best, __shfl_xor(best, 16));
  return fmaxf(b, __shfl_xor(b, 32));
}

}  // namespace oasis
