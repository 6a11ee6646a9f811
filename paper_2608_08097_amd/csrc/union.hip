// Per-layer union of the per-head top-K sets (paper §4.4.1: at admission the
// prefill node sends, per layer, the blocks whose token range at least one KV
// head selected, with their indices).
//
// One workgroup per request: every selected id of every head sets its bit in
// an LDS bitmap over the max_blocks logical blocks; a workgroup scan over the
// per-thread popcounts of contiguous word ranges then writes the ids in
// ascending order, and the rest of the row is padded with -1.
#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void union_kernel(UnionArgs a) {
  extern __shared__ uint32_t bm[];
  __shared__ int s_wave[kThreads / 64 + 1];
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int words = (a.NBmax + 31) / 32;
  for (int w = tid; w < words; w += kThreads) bm[w] = 0u;
  __syncthreads();
  // (head, entry) pairs of the request, four per thread at a time; the count
  // and the id of an entry are loaded together, so the loads of a group are
  // all in flight before any is used
  const int pairs = a.Hkv * a.k;
  const long long row0 = (long long)r * a.Hkv;
  for (int base = 0; base < pairs; base += 4 * kThreads) {
    int b[4], m[4], i[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + u * kThreads + tid;
      const int h = idx < pairs ? idx / a.k : 0;
      i[u] = idx < pairs ? idx - h * a.k : a.k;
      m[u] = a.sel_count[row0 + h];
      b[u] = a.sel[(row0 + h) * a.k + (i[u] < a.k ? i[u] : 0)];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int mm = m[u] < 0 ? 0 : (m[u] > a.k ? a.k : m[u]);
      if (i[u] < mm && b[u] >= 0 && b[u] < a.NBmax) atomicOr(&bm[b[u] >> 5], 1u << (b[u] & 31));
    }
  }
  __syncthreads();
  // contiguous word range per thread, popcount, exclusive scan
  const int per = (words + kThreads - 1) / kThreads;
  const int w0 = tid * per;
  const int w1 = min(words, w0 + per);
  int n = 0;
  for (int w = w0; w < w1; ++w) n += __popc(bm[w]);
  const int lane = tid & 63, wave = tid >> 6;
  int x = n;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  int base = x - n;
  int total = 0;
  for (int v = 0; v < kThreads / 64; ++v) {
    if (v < wave) base += s_wave[v];
    total += s_wave[v];
  }
  const long long row = (long long)r * a.Hkv * a.k;
  int pos = base;
  for (int w = w0; w < w1; ++w) {
    uint32_t bits = bm[w];
    while (bits) {
      const int bit = __ffs(bits) - 1;
      bits &= bits - 1;
      a.ids[row + pos++] = w * 32 + bit;
    }
  }
  const int cap = a.Hkv * a.k;
  for (int i = total + tid; i < cap; i += kThreads) a.ids[row + i] = -1;
  if (tid == 0) a.count[r] = total;
}

}  // namespace

hipError_t launch_union(const UnionArgs& a, hipStream_t s) {
  const size_t lds = sizeof(uint32_t) * (size_t)((a.NBmax + 31) / 32);
  hipLaunchKernelGGL(union_kernel, dim3((unsigned)a.R), dim3(kThreads), lds, s, a);
  return hipGetLastError();
}

}  // namespace oasis
