// Exact top-K of one (request, KV head) score row by a workgroup (paper
// §4.2.1-§4.2.2: top-K prediction per KV head; ties go to the lowest block id).
//
// Scores are mapped to order-preserving uint32 keys (-0 folded into +0); each
// thread owns a contiguous range of block ids (KPT keys in registers, or
// re-read from memory with KPT == 0). A 4-pass, 8-bit radix select over an LDS
// histogram finds the exact key tau of the k-th largest score and how many
// keys equal to tau are needed; two workgroup-wide exclusive scans then give
// the rank of every tau-valued key in id order (lowest ids win the ties) and
// the output position of every selected block, so the selection is written in
// ascending id order without a sort. The top-K kernel runs it with 1024
// threads per row; the thread count is a template parameter.
#pragma once

#include "oasis_internal.h"

namespace oasis {

__device__ __forceinline__ uint32_t select_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;  // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int NTHR>
struct SelectShared {
  uint32_t hist[256];
  int digit, rem;
  int wave[2 * (NTHR / 64)];
};

// Exclusive scan of one int per thread over the NTHR-thread workgroup.
template <int NTHR>
__device__ int select_exclusive_scan(int v, int* s_wave) {
  constexpr int kWaves = NTHR / 64;
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

// Select the top k of s[0..n) into out[0..k) (ascending ids, -1 padded when
// n < k) and set *count; every thread of the workgroup calls it.
template <int NTHR, int KPT>
__device__ void select_row(const float* s, int n, int k, int32_t* out, int32_t* count, SelectShared<NTHR>& sh) {
  const int tid = threadIdx.x;
  if (n <= k) {  // every candidate fits the budget
    for (int i = tid; i < k; i += NTHR) out[i] = i < n ? i : -1;
    if (tid == 0) *count = n;
    return;
  }

  uint32_t* hist = sh.hist;
  int& s_digit = sh.digit;
  int& s_rem = sh.rem;
  int* s_wave = sh.wave;

  const int per = (n + NTHR - 1) / NTHR;
  const int lo = min(n, tid * per);
  const int cnt_local = min(n, lo + per) - lo;

  constexpr int kRegs = KPT > 0 ? KPT : 1;
  uint32_t keys[kRegs];
  if (KPT > 0) {
    // every load is issued (index clamped into the row, n > k >= 1 here) before
    // any is used; keys past this thread's range are masked afterwards
#pragma unroll
    for (int j = 0; j < kRegs; ++j) {
      const uint32_t key = select_key(s[min(lo + j, n - 1)]);
      keys[j] = j < cnt_local ? key : 0u;
    }
  }
  auto key_at = [&](int j) -> uint32_t { return KPT > 0 ? keys[j] : select_key(s[lo + j]); };
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
  const int eq_base = select_exclusive_scan<NTHR>(n_eq, s_wave);
  const int n_sel = n_gt + max(0, min(n_eq, need_eq - eq_base));
  int pos = select_exclusive_scan<NTHR>(n_sel, s_wave);
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
  if (tid == 0) *count = k;
}

}  // namespace oasis
