// Block importance from the lookahead queries (paper §4.2.1): Quest upper bound
// of every candidate block for every draft row, maximum over the G x D rows of
// a KV head.
//
// The bound is a dense [rows x 256] x [256 x 16] product per tile of 16 blocks
// (score_core.h: [q+ | q-] . [kmax ; kmin], exact bf16 operands, fp32
// accumulation on v_mfma_f32_16x16x32_bf16) for the 5 to 64 rows of a KV head
// (fewer go to the vector-ALU scorer of score_valu.hip), and the row maximum is
// taken in the epilogue with two cross-lane exchanges.
//
// Memory: every summary byte is read once. A wave owns TPW consecutive tiles
// of 16 blocks; for a tile, lane (g, n) loads 16 bytes of block n at byte
// offset 64*step + 16*g of its kmax row and of its kmin row, so four lanes
// read 64 contiguous bytes and the wave covers the tile's 2 x 4 KiB in 8
// load instructions. All loads of a wave are issued before its first MFMA.
//
// The operands of the rows go to LDS once per workgroup and each wave holds
// one row tile's operands at a time (4 summary tiles per wave with one row
// tile, 2 with more). Measured on MI355X against keeping all operands in
// every wave's registers: 64 rows (16 requests x 65,536 tokens, B = 32,
// 134 MB) 30.1 us against 38.5 us (4 waves per SIMD instead of 2); 16 rows
// (8 x 131,072 tokens, 268 MB) 48.6 us against 49.9 us (fewer query reads;
// 3, 5, 6 and 8 summary tiles per wave: 48.6, 50.8, 51.7 and 56.6 us).
#include "oasis_internal.h"
#include "score_core.h"

namespace oasis {

namespace {

// The [q+ | q-] operands of the KV head's rows are built once per workgroup in
// LDS, laid out per lane so that each MFMA operand is one conflict-free
// 16-byte LDS read, and a wave walks the row tiles in its outer loop. Only one
// row tile's operands are then live in registers, which leaves room for more
// summary tiles in flight per CU, and the queries are read once per workgroup
// rather than once per wave.
template <int NRT, int TPW>
__global__ __launch_bounds__(256) void score_kernel(ScoreArgs a) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int n = lane & 15;
  const int rh = blockIdx.y;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const Ctx c = ctx_blocks(a.ctx_len[r], a.B, a.NBmax);
  const int ntiles = (a.NBmax + 15) >> 4;
  // Workgroups are dealt to the 8 XCDs round-robin by linear id, so with a
  // grid 8 (or a multiple of 8) tile groups wide one XCD would always get the
  // same tile group of every row, and the tail groups of short rows (no live
  // blocks) would leave their XCDs idle; rotating the group by the row spreads
  // every group over all XCDs (ragged 16K-32K-token rows: 48.0 -> 47.0 us).
  const int group = (int)((blockIdx.x + blockIdx.y) % gridDim.x);
  const int tile0 = (group * 4 + wave) * TPW;
  __shared__ ScoreQOperands<NRT> s_q;

  // queries first (cache-resident, needed first), then the summaries of all TPW tiles
  u32x4 qraw[NRT];
#pragma unroll
  for (int j = 0; j < NRT; ++j) qraw[j] = score_q_raw(a, r, h, threadIdx.x + j * 256);
  const long long sum_base = (long long)rh * a.NBmax * kHeadDim;
  const uint16_t* kmx = a.kmax + sum_base;
  const uint16_t* kmn = a.kmin + sum_base;
  // (the loads are written out here rather than through score_tile_load: with
  // both helpers the compiler keeps far more registers live, 284 VGPRs instead
  // of 116 at four row tiles, one wave per SIMD instead of four)
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
#pragma unroll
  for (int j = 0; j < NRT; ++j) score_q_store<NRT>(s_q, threadIdx.x + j * 256, qraw[j]);
  __syncthreads();  // every wave reaches it: waves past the last tile return only below
  if (tile0 >= ntiles) return;

  float best[TPW];
#pragma unroll
  for (int t = 0; t < TPW; ++t) best[t] = -INFINITY;
  if (tile0 * 16 < c.n_cand) {
#pragma unroll
    for (int v = 0; v < NRT; ++v) {
      bf16x8 ap[4], an[4];
      score_q_tile<NRT>(s_q, v, lane, ap, an);
#pragma unroll
      for (int t = 0; t < TPW; ++t) best[t] = score_tile_fold(ap, an, vmax[t], vmin[t], best[t]);
    }
  }
  float* srow = a.scores + (long long)rh * a.NBmax;
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int tile = tile0 + t;
    if (tile >= ntiles) break;
    const float b = score_lane_reduce(best[t]);
    const int blk = tile * 16 + n;
    if (g == 0 && blk < a.NBmax) srow[blk] = blk < c.n_cand ? b : -INFINITY;
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
    case 2: return launch_t<2, 2>(a, s, t);
    case 3: return launch_t<3, 2>(a, s, t);
    case 4: return launch_t<4, 2>(a, s, t);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace oasis
