// Block copies between two paged KV tiers (paper §4.3: when a request passes
// the sparsification threshold its whole KV cache is copied to CPU memory and
// only the selected blocks and the local window stay on the GPU; afterwards the
// blocks that receive new tokens must reach the full tier too).
//
// Per request the logical blocks holding tokens [prev, cur) are copied, at most
// max_blocks of them from the first; a page holds every KV head of its block
// ([Hkv][B][d]), so each block is two contiguous runs (K and V). Either tier may
// be device memory or pinned host memory (device-visible): device-to-host
// copies are posted writes over PCIe, host-to-device ones reads. One thread
// moves 16 bytes; grid (chunks of K and V, block, request).
#include "oasis_internal.h"

namespace oasis {

namespace {

__global__ __launch_bounds__(256) void copy_blocks_kernel(CopyArgs a) {
  const int r = blockIdx.z;
  const int cur = a.ctx_len[r];
  const int prev = a.prev_ctx_len ? a.prev_ctx_len[r] : 0;
  if (cur <= prev) return;
  const int lo = prev / a.B;
  int hi = (cur + a.B - 1) / a.B;
  if (hi > a.NBmax) hi = a.NBmax;
  if (hi > lo + a.max_blocks) hi = lo + a.max_blocks;
  const int b = lo + (int)blockIdx.y;
  if (b >= hi) return;
  const int sp = a.src_table[(long long)r * a.NBmax + b];
  const int dp = a.dst_table[(long long)r * a.NBmax + b];
  if (sp < 0 || sp >= a.num_src_pages || dp < 0 || dp >= a.num_dst_pages) return;
  const long long chunks = (long long)a.Hkv * a.B * kHeadDim / 8;  // 16-byte chunks per page
  const long long c = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= 2 * chunks) return;
  const bool is_v = c >= chunks;
  const long long off = (is_v ? c - chunks : c) * 8;
  const uint16_t* src = (is_v ? a.src_v : a.src_k) + (long long)sp * chunks * 8 + off;
  uint16_t* dst = (is_v ? a.dst_v : a.dst_k) + (long long)dp * chunks * 8 + off;
  *reinterpret_cast<u32x4*>(dst) = ldg16(src);
}

}  // namespace

hipError_t launch_copy_blocks(const CopyArgs& a, hipStream_t s) {
  const long long chunks = (long long)a.Hkv * a.B * kHeadDim / 8;
  const dim3 grid((unsigned)((2 * chunks + 255) / 256), (unsigned)a.max_blocks, (unsigned)a.R);
  hipLaunchKernelGGL(copy_blocks_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace oasis
