// Compressed keys: per-block coordinate-wise min/max of the keys (paper §4.2.1,
// "Look-ahead attention" figure; Quest-style summaries, two rows per block),
// built for every candidate block, or updated for the blocks completed since a
// previous context length (§5.1 compressed-key updates).
//
// One thread owns 8 consecutive dimensions of one (request, block, KV head) and
// reads the B tokens of the page with 16-byte loads, all issued before the
// first is used (B is a template parameter, so the token loop unrolls);
// neighbouring threads cover neighbouring dimensions, so a wave reads whole
// 256-byte key rows. The result is exact: min/max of bf16 values is a bf16
// value.
#include "oasis_internal.h"

namespace oasis {

namespace {

template <int BS>
__global__ __launch_bounds__(256) void summaries_kernel(SummaryArgs a) {
  const int r = blockIdx.y;
  const long long item = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int per_block = a.Hkv * (kHeadDim / 8);
  const int rem = (int)(item % per_block);
  const int h = rem / (kHeadDim / 8);
  const int d0 = (rem % (kHeadDim / 8)) * 8;
  const Ctx c = ctx_blocks(a.ctx_len[r], BS, a.NBmax);
  // update form: the grid covers max_new blocks per request, from the first one completed since prev
  const int lo = a.prev_ctx_len ? ctx_blocks(a.prev_ctx_len[r], BS, a.NBmax).n_cand : 0;
  const int b = lo + (int)(item / per_block);
  if (b >= c.n_cand || (a.prev_ctx_len && b >= lo + a.max_new)) return;
  const int page = a.block_table[(long long)r * a.NBmax + b];
  if (page < 0 || page >= a.num_pages) return;

  const uint16_t* src = a.k_pages + (((long long)page * a.Hkv + h) * BS) * kHeadDim + d0;
  float mx[8], mn[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    mx[j] = -INFINITY;
    mn[j] = INFINITY;
  }
  u32x4 rows[BS];
#pragma unroll
  for (int p = 0; p < BS; ++p) rows[p] = ldg16(src + (long long)p * kHeadDim);
#pragma unroll
  for (int p = 0; p < BS; ++p) {
    const u32x4 v = rows[p];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float lo = bf16_bits_to_f32(v[w] & 0xFFFFu);
      const float hi = bf16_bits_to_f32(v[w] >> 16);
      mx[2 * w] = fmaxf(mx[2 * w], lo);
      mn[2 * w] = fminf(mn[2 * w], lo);
      mx[2 * w + 1] = fmaxf(mx[2 * w + 1], hi);
      mn[2 * w + 1] = fminf(mn[2 * w + 1], hi);
    }
  }
  u32x4 omx, omn;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    // exact: the values are bf16, so the upper 16 bits of the float are the result
    omx[w] = (__float_as_uint(mx[2 * w]) >> 16) | (__float_as_uint(mx[2 * w + 1]) & 0xFFFF0000u);
    omn[w] = (__float_as_uint(mn[2 * w]) >> 16) | (__float_as_uint(mn[2 * w + 1]) & 0xFFFF0000u);
  }
  const long long o = (((long long)r * a.Hkv + h) * a.NBmax + b) * kHeadDim + d0;
  *reinterpret_cast<u32x4*>(a.kmax + o) = omx;
  *reinterpret_cast<u32x4*>(a.kmin + o) = omn;
}

}  // namespace

hipError_t launch_summaries(const SummaryArgs& a, hipStream_t s) {
  const long long blocks = a.prev_ctx_len ? (a.max_new < a.NBmax ? a.max_new : a.NBmax) : a.NBmax;
  const long long items = blocks * a.Hkv * (kHeadDim / 8);
  const dim3 grid((unsigned)((items + 255) / 256), (unsigned)a.R);
  if (a.B == 16)
    hipLaunchKernelGGL(summaries_kernel<16>, grid, dim3(256), 0, s, a);
  else if (a.B == 32)
    hipLaunchKernelGGL(summaries_kernel<32>, grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace oasis
