// Block importance from the lookahead queries (paper §4.2.1): Quest upper bound
// of every candidate block for every draft row, maximum over the G x D rows of
// a KV head.
//
// For one row q and a block with per-coordinate bounds kmin <= kmax,
//   sum_d max(q_d kmin_d, q_d kmax_d) = sum_d (q+_d kmax_d + q-_d kmin_d)
// with q+ = max(q, 0), q- = min(q, 0): exactly a dot product of [q+ | q-]
// (2d bf16 values, exact) with [kmax ; kmin]. The rows of one KV head (5 to
// 64 here; fewer go to the vector-ALU scorer of score_valu.hip) times a tile
// of 16 blocks is therefore a dense [rows x 256] x [256 x 16] product, done
// with v_mfma_f32_16x16x32_bf16 (fp32 accumulation), and the row maximum is
// taken in the epilogue with two cross-lane exchanges.
//
// Memory: every summary byte is read once. A wave owns TPW consecutive tiles
// of 16 blocks; for a tile, lane (g, n) loads 16 bytes of block n at byte
// offset 64*step + 16*g of its kmax row and of its kmin row, so four lanes
// read 64 contiguous bytes and the wave covers the tile's 2 x 4 KiB in 8
// load instructions. All loads of a wave are issued before its first MFMA.
#include "oasis_internal.h"

namespace oasis {

namespace {

template <int NRT, int TPW>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;   // k-group of the MFMA operands
  const int n = lane & 15;   // block within the tile (B operand) / row within the tile (A operand)
  const int rh = blockIdx.y;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const Ctx c = ctx_blocks(a.ctx_len[r], a.B, a.NBmax);
  const int ntiles = (a.NBmax + 15) >> 4;
  const int tile0 = (blockIdx.x * 4 + wave) * TPW;
  if (tile0 >= ntiles) return;

  float* srow = a.scores + (long long)rh * a.NBmax;
  const long long sum_base = (long long)rh * a.NBmax * kHeadDim;
  const uint16_t* kmx = a.kmax + sum_base;
  const uint16_t* kmn = a.kmin + sum_base;

  // Issue the summary loads of all TPW tiles first.
  u32x4 vmax[TPW][4], vmin[TPW][4];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int blk = (tile0 + t) * 16 + n;
    const bool live = blk < c.n_cand;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      const long long off = (long long)blk * kHeadDim + st * 32 + g * 8;
      vmax[t][st] = live ? ldg16(kmx + off) : u32x4{0, 0, 0, 0};
      vmin[t][st] = live ? ldg16(kmn + off) : u32x4{0, 0, 0, 0};
    }
  }

  // A operands: [q+ | q-] of the rows of this KV head. Rows past the last
  // real row repeat row 0, which leaves the maximum unchanged.
  const int nrows = a.num_draft * a.G;
  bf16x8 qpos[NRT][4], qneg[NRT][4];
#pragma unroll
  for (int v = 0; v < NRT; ++v) {
    int row = v * 16 + n;
    if (row >= nrows) row = 0;
    const int t = a.first_draft + row / a.G;
    const int qh = h * a.G + row % a.G;
    const uint16_t* qrow = a.q + (((long long)r * a.T + t) * a.Hq + qh) * kHeadDim;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      u32x4 p, m;
      split_sign(ldg16(qrow + st * 32 + g * 8), p, m);
      qpos[v][st] = as_bf16x8(p);
      qneg[v][st] = as_bf16x8(m);
    }
  }

#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int tile = tile0 + t;
    if (tile >= ntiles) break;
    const int b0 = tile * 16;
    float best = -INFINITY;
    if (b0 < c.n_cand) {
#pragma unroll
      for (int v = 0; v < NRT; ++v) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < 4; ++st)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qpos[v][st], as_bf16x8(vmax[t][st]), acc, 0, 0, 0);
#pragma unroll
        for (int st = 0; st < 4; ++st)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qneg[v][st], as_bf16x8(vmin[t][st]), acc, 0, 0, 0);
        // lane (g, n) holds rows 4g..4g+3 of the row tile for block n
        best = fmaxf(best, fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
      }
      best = fmaxf(best, __shfl_xor(best, 16));
      best = fmaxf(best, __shfl_xor(best, 32));
    }
    const int blk = b0 + n;
    if (g == 0 && blk < a.NBmax) srow[blk] = blk < c.n_cand ? best : -INFINITY;
  }
}

template <int NRT, int TPW>
hipError_t launch_t(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int ntiles = (a.NBmax + 15) / 16;
  const dim3 grid((unsigned)((ntiles + 4 * TPW - 1) / (4 * TPW)), (unsigned)(a.R * a.Hkv));
  launch_kernel(score_kernel<NRT, TPW>, grid, dim3(256), s, t, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const ScoreArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int rows = a.num_draft * a.G;
  // a quarter of a 16-row tile or less: no MFMA
  if (rows <= kScoreValuMaxRows) return launch_score_valu(a, s, t);
  switch ((rows + 15) / 16) {
    case 1: return launch_t<1, 4>(a, s, t);
    case 2: return launch_t<2, 4>(a, s, t);
    case 3: return launch_t<3, 2>(a, s, t);
    case 4: return launch_t<4, 2>(a, s, t);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oasis
