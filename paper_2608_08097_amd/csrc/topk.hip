// Top-K selection per (request, KV head) (paper §4.2.1-§4.2.2; §5.2: K = 128
// blocks of 16 tokens, and the budget is the sparsification threshold): one
// 1024-thread workgroup per (request, KV head) runs the exact select of
// select.h over the candidates of its score row.
#include "oasis_internal.h"
#include "select.h"

namespace oasis {

namespace {

constexpr int kThreads = 1024;

template <int KPT>
__global__ __launch_bounds__(kThreads) void topk_kernel(TopkArgs a) {
  __shared__ SelectShared<kThreads, KPT> sh;
  const int rh = blockIdx.x;
  const int r = rh / a.Hkv;
  const Ctx c = ctx_blocks(a.ctx_len[r], a.B, a.NBmax);
  select_row<kThreads, KPT>(a.scores + (long long)rh * a.NBmax, c.n_cand, a.k, a.sel + (long long)rh * a.k,
                            a.sel_count + rh, sh);
}

}  // namespace

hipError_t launch_topk(const TopkArgs& a, hipStream_t s, const LaunchTiming& t) {
  // the candidate count of every request is at most NBmax - 1
  const int per = (a.NBmax + kThreads - 1) / kThreads;
  const dim3 grid((unsigned)(a.R * a.Hkv));
  if (per <= 8)
    launch_kernel(topk_kernel<8>, grid, dim3(kThreads), s, t, a);
  else if (per <= 16)
    launch_kernel(topk_kernel<16>, grid, dim3(kThreads), s, t, a);
  else if (per <= 32)
    launch_kernel(topk_kernel<32>, grid, dim3(kThreads), s, t, a);
  else
    launch_kernel(topk_kernel<0>, grid, dim3(kThreads), s, t, a);
  return hipGetLastError();
}

}  // namespace oasis
