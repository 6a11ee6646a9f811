// Exact top-K of one (request, KV head) score row by a workgroup (paper
// §4.2.1-§4.2.2: top-K prediction per KV head; ties go to the lowest block id).
//
// Scores are mapped to order-preserving uint32 keys (-0 folded into +0); each
// thread owns a contiguous range of block ids (KPT keys in registers, or
// re-read from memory with KPT == 0). A radix select over an LDS histogram
// finds the exact key tau of the k-th largest score and how many keys equal
// to tau are needed. It runs on the offsets of the keys from the row's
// smallest key, 8 bits per pass from the highest bit of the row's key range
// down: scores of one row share their sign and most exponent bits, which
// would put nearly every key in one bin of a first pass over the raw top
// byte (LDS atomics on one address), and a narrow range needs fewer passes.
// Workgroup-wide exclusive scans then give the rank of every tau-valued key
// in id order (lowest ids win the ties; one scan suffices when every
// tau-valued key is taken) and the output position of every selected block,
// so the selection is written in ascending id order without a sort. The
// top-K kernel runs it with 1024 threads per row; the thread count is a
// template parameter.
#pragma once

#include "oasis_internal.h"

namespace oasis {

__device__ __forceinline__ uint32_t select_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;  // -0.0 == +0.0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Wave-wide minimum and maximum of uint32 values, returned to every lane (the
// same DPP steps; lanes without a source keep the identity).
__device__ __forceinline__ void wave_min_max(uint32_t& mn, uint32_t& mx) {
  int a = (int)mn, b = (int)mx;
#define OASIS_DPP_MINMAX(CTRL, ROWS)                                                              \
  a = (int)min((uint32_t)a, (uint32_t)__builtin_amdgcn_update_dpp((int)0xFFFFFFFF, a, CTRL, ROWS, 0xF, false)); \
  b = (int)max((uint32_t)b, (uint32_t)__builtin_amdgcn_update_dpp(0, b, CTRL, ROWS, 0xF, false));
  OASIS_DPP_MINMAX(0x111, 0xF)
  OASIS_DPP_MINMAX(0x112, 0xF)
  OASIS_DPP_MINMAX(0x114, 0xF)
  OASIS_DPP_MINMAX(0x118, 0xF)
  OASIS_DPP_MINMAX(0x142, 0xA)
  OASIS_DPP_MINMAX(0x143, 0xC)
#undef OASIS_DPP_MINMAX
  mn = (uint32_t)__builtin_amdgcn_readlane(a, 63);
  mx = (uint32_t)__builtin_amdgcn_readlane(b, 63);
}

template <int NTHR, int KPT>
struct SelectShared {
  uint32_t keys[KPT > 0 ? NTHR * KPT : 1];  // the row's keys, staged (KPT > 0)
  uint32_t hist[2][256];  // one per pass, alternately: the next is cleared while the current fills
  int digit, rem, eq_total;
  int wave[2 * (NTHR / 64)];
  uint32_t wmin[NTHR / 64], wmax[NTHR / 64];
};

// Exclusive scan of one int per thread over the NTHR-thread workgroup.
template <int NTHR>
__device__ int select_exclusive_scan(int v, int* s_wave) {
  constexpr int kWaves = NTHR / 64;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int x = wave_incl_sum(v);
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  if (wave == 0) {
    const int t = lane < kWaves ? s_wave[lane] : 0;
    const int w = wave_incl_sum(t);
    if (lane < kWaves) s_wave[kWaves + lane] = w - t;  // exclusive wave offsets
  }
  __syncthreads();
  const int res = s_wave[kWaves + wave] + x - v;
  __syncthreads();
  return res;
}

// Select the top k of s[0..n) into out[0..k) (ascending ids, -1 padded when
// n < k) and set *count; every thread of the workgroup calls it. With lout
// (LDS, k entries) the selection is also left there for the workgroup.
template <int NTHR, int KPT>
__device__ void select_row(const float* s, int n, int k, int32_t* out, int32_t* count, SelectShared<NTHR, KPT>& sh,
                           int* lout = nullptr) {
  const int tid = threadIdx.x;
  if (n <= k) {  // every candidate fits the budget
    for (int i = tid; i < k; i += NTHR) {
      out[i] = i < n ? i : -1;
      if (lout) lout[i] = i < n ? i : -1;
    }
    if (tid == 0) *count = n;
    return;
  }

  int& s_digit = sh.digit;
  int& s_rem = sh.rem;
  int& s_eq = sh.eq_total;
  int* s_wave = sh.wave;

  const int per = (n + NTHR - 1) / NTHR;
  const int lo = min(n, tid * per);
  const int cnt_local = min(n, lo + per) - lo;

  constexpr int kRegs = KPT > 0 ? KPT : 1;
  uint32_t keys[kRegs];
  if (KPT > 0) {
    // Coalesced loads staged through LDS: thread t reads ids t, t + NTHR, ...
    // (every load issued, index clamped into the row, n > k >= 1 here, before
    // any is used), then takes its own contiguous range from LDS. Reading the
    // range straight from memory would spread each load instruction over 16
    // cache lines.
    float v[kRegs];
#pragma unroll
    for (int j = 0; j < kRegs; ++j) v[j] = s[min(tid + j * NTHR, n - 1)];
#pragma unroll
    for (int j = 0; j < kRegs; ++j) {
      const int i = tid + j * NTHR;
      if (i < n) sh.keys[i] = select_key(v[j]);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kRegs; ++j) keys[j] = j < cnt_local ? sh.keys[min(lo + j, n - 1)] : 0u;
  }
  auto key_at = [&](int j) -> uint32_t { return KPT > 0 ? keys[j] : select_key(s[lo + j]); };
  const int jmax = KPT > 0 ? kRegs : cnt_local;

  // range of the row's keys: wave minima / maxima, then over the waves
  constexpr int kWaves = NTHR / 64;
  uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
#pragma unroll
  for (int j = 0; j < jmax; ++j) {
    if (j >= cnt_local) break;
    const uint32_t key = key_at(j);
    kmin = min(kmin, key);
    kmax = max(kmax, key);
  }
  wave_min_max(kmin, kmax);
  if ((tid & 63) == 0) {
    sh.wmin[tid >> 6] = kmin;
    sh.wmax[tid >> 6] = kmax;
  }
  if (tid == 0) {
    s_digit = 0;
    s_rem = k;
    s_eq = 0;
  }
  if (tid < 256) sh.hist[0][tid] = 0u;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    kmin = min(kmin, sh.wmin[w]);
    kmax = max(kmax, sh.wmax[w]);
  }
  const uint32_t range = kmax - kmin;
  // offsets from kmin have `top` significant bits; passes resolve them 8 at a time
  int top = range ? 32 - __clz((int)range) : 0;
  uint32_t prefix = 0u;  // resolved high bits of the wanted offset (bits >= top)
  int rem = k;           // rank (from the top) of the wanted key among keys matching the prefix
  int eq_total = n;      // keys equal to tau (all of them when the range is empty)
  // Two barriers per pass: after the histogram is filled, and after the
  // digit is found (the next pass fills the other histogram, cleared here).
  for (int pass = 0; top > 0; ++pass) {
    const int shift = top > 8 ? top - 8 : 0;
    const uint32_t dmask = (1u << (top - shift)) - 1u;  // this pass resolves bits [shift, top)
    uint32_t* hist = sh.hist[pass & 1];
    if (tid < 256) sh.hist[(pass & 1) ^ 1][tid] = 0u;
    uint32_t cur = 0xFFFFFFFFu;
    uint32_t run = 0u;
#pragma unroll
    for (int j = 0; j < jmax; ++j) {
      if (j >= cnt_local) break;
      const uint32_t off = key_at(j) - kmin;
      if (top < 32 && (off >> top) != prefix) continue;
      const uint32_t dg = (off >> shift) & dmask;
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
      const int incl = wave_incl_sum(local);
      const int excl = incl - local;
      if (excl < rem && rem <= incl) {
        int acc = excl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (acc + (int)hb[j] >= rem) {
            s_digit = 255 - 4 * tid - j;
            s_rem = rem - acc;
            s_eq = (int)hb[j];
            break;
          }
          acc += (int)hb[j];
        }
      }
    }
    __syncthreads();
    prefix = (prefix << (top - shift)) | (uint32_t)s_digit;
    rem = s_rem;
    eq_total = s_eq;
    top = shift;
  }
  const uint32_t tau = kmin + prefix;
  const int need_eq = rem;  // how many tau-valued keys are taken, lowest ids first

  int n_eq = 0, n_gt = 0;
#pragma unroll
  for (int j = 0; j < jmax; ++j) {
    if (j >= cnt_local) break;
    const uint32_t key = key_at(j);
    n_eq += key == tau;
    n_gt += key > tau;
  }
  // every tau-valued key taken (no tie to break at the threshold): one scan
  const bool all_eq = need_eq == eq_total;
  const int eq_base = all_eq ? 0 : select_exclusive_scan<NTHR>(n_eq, s_wave);
  const int n_sel = all_eq ? n_gt + n_eq : n_gt + max(0, min(n_eq, need_eq - eq_base));
  int pos = select_exclusive_scan<NTHR>(n_sel, s_wave);
  int eq_rank = eq_base;
#pragma unroll
  for (int j = 0; j < jmax; ++j) {
    if (j >= cnt_local) break;
    const uint32_t key = key_at(j);
    bool take = key > tau;
    if (key == tau) {
      take = all_eq || eq_rank < need_eq;
      ++eq_rank;
    }
    if (take && pos < k) {
      out[pos] = lo + j;
      if (lout) lout[pos] = lo + j;
      ++pos;
    }
  }
  if (tid == 0) *count = k;
}

}  // namespace oasis
