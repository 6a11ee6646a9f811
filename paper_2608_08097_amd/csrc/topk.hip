// Top-K selection per (request, KV head) (paper §4.2.1-§4.2.2; §5.2: K = 128
// blocks of 16 tokens, and the budget is the sparsification threshold).
//
// One 1024-thread workgroup per (request, KV head). Scores are mapped to
// order-preserving uint32 keys (-0 folded into +0) and held in registers. A
// 4-pass, 8-bit radix
// select over an LDS histogram finds the exact key tau of the k-th largest
// score and how many of the keys equal to tau are needed. Each thread owns a
// contiguous range of block ids, so two block-wide exclusive scans give (1)
// the rank of every tau-valued key in id order, which resolves ties to the
// lowest ids, and (2) the output position of every selected block, which
// writes the selection in ascending id order without a sort. The result is
// exact and deterministic.
#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;

__device__ __forceinline__ uint32_t order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;  // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive scan of one int per thread over the 1024-thread workgroup.
__device__ int block_exclusive_scan(int v, int* s_wave) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kWaves ? s_wave[lane] : 0;
#pragma unroll
    for (int o = 1; o < kWaves; o <<= 1) {
      const int y = __shfl_up(w, o);
      if (lane >= o) w += y;
    }
    if (lane < kWaves) s_wave[kWaves + lane] = w - s_wave[lane];  // exclusive wave offsets
  }
  __syncthreads();
  const int res = s_wave[kWaves + wave] + x - v;
  __syncthreads();
  return res;
}

// Keys live in registers (KPT per thread, contiguous ids per thread); with
// KPT == 0 they are re-read from global memory (very long contexts).
template <int KPT>
__global__ __launch_bounds__(kThreads) void topk_kernel(TopkArgs a) {
  const int rh = blockIdx.x;
  const int r = rh / a.Hkv;
  const int tid = threadIdx.x;
  const Ctx c = ctx_blocks(a.ctx_len[r], a.B, a.NBmax);
  const int n = c.n_cand;
  const int k = a.k;
  int32_t* out = a.sel + (long long)rh * k;

  if (n <= k) {  // every candidate fits the budget
    for (int i = tid; i < k; i += kThreads) out[i] = i < n ? i : -1;
    if (tid == 0) a.sel_count[rh] = n;
    return;
  }

  __shared__ uint32_t hist[256];
  __shared__ int s_digit, s_rem;
  __shared__ int s_wave[2 * kWaves];

  const float* s = a.scores + (long long)rh * a.NBmax;
  const int per = (n + kThreads - 1) / kThreads;
  const int lo = min(n, tid * per);
  const int cnt_local = min(n, lo + per) - lo;

  constexpr int kRegs = KPT > 0 ? KPT : 1;
  uint32_t keys[kRegs];
  if (KPT > 0) {
#pragma unroll
    for (int j = 0; j < kRegs; ++j) keys[j] = j < cnt_local ? order_key(s[lo + j]) : 0u;
  }
  auto key_at = [&](int j) -> uint32_t { return KPT > 0 ? keys[j] : order_key(s[lo + j]); };
  const int jmax = KPT > 0 ? kRegs : cnt_local;

  if (tid == 0) {
    s_digit = 0;
    s_rem = 1;
  }
  uint32_t prefix = 0u, mask = 0u;
  int rem = k;  // rank (from the top) of the wanted key among keys matching the prefix
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    uint32_t cur = 0xFFFFFFFFu;
    uint32_t run = 0u;
#pragma unroll
    for (int j = 0; j < jmax; ++j) {
      if (j >= cnt_local) break;
      const uint32_t key = key_at(j);
      if ((key & mask) != prefix) continue;
      const uint32_t dg = (key >> shift) & 0xFFu;
      if (dg == cur) {
        ++run;
      } else {
        if (run) atomicAdd(&hist[cur], run);
        cur = dg;
        run = 1u;
      }
    }
    if (run) atomicAdd(&hist[cur], run);
    __syncthreads();
    if (tid < 64) {
      // lane L looks at bins 255-4L .. 252-4L (descending)
      uint32_t hb[4];
      int local = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        hb[j] = hist[255 - 4 * tid - j];
        local += (int)hb[j];
      }
      int incl = local;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (tid >= o) incl += y;
      }
      const int excl = incl - local;
      if (excl < rem && rem <= incl) {
        int acc = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (acc + (int)hb[j] >= rem) {
            s_digit = 255 - 4 * tid - j;
            s_rem = rem - acc;
            break;
          }
          acc += (int)hb[j];
        }
      }
    }
    __syncthreads();
    prefix |= (uint32_t)s_digit << shift;
    mask |= 0xFFu << shift;
    rem = s_rem;
    __syncthreads();
  }
  const uint32_t tau = prefix;
  const int need_eq = rem;  // how many tau-valued keys are taken, lowest ids first

  int n_eq = 0, n_gt = 0;
#pragma unroll
  for (int j = 0; j < jmax; ++j) {
    if (j >= cnt_local) break;
    const uint32_t key = key_at(j);
    n_eq += key == tau;
    n_gt += key > tau;
  }
  const int eq_base = block_exclusive_scan(n_eq, s_wave);
  const int n_sel = n_gt + max(0, min(n_eq, need_eq - eq_base));
  int pos = block_exclusive_scan(n_sel, s_wave);
  int eq_rank = eq_base;
#pragma unroll
  for (int j = 0; j < jmax; ++j) {
    if (j >= cnt_local) break;
    const uint32_t key = key_at(j);
    bool take = key > tau;
    if (key == tau) {
      take = eq_rank < need_eq;
      ++eq_rank;
    }
    if (take && pos < k) out[pos++] = lo + j;
  }
  if (tid == 0) a.sel_count[rh] = k;
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
