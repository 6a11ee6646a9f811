// Delta selection and KV transfer into the HBM working set.
//
// Paper §4.2.3: the predicted set is intersected with the resident set (hits
// stay, no bytes move), non-selected residents are ranked by the step at which
// they were last selected and evicted least-recently-selected first, and each
// admitted miss is paired with one eviction target; at most fetch_cap pairs are
// admitted per KV head and step (§5.5.1: a fetch ratio of K), the highest-
// scoring misses first, and all other slots stay as they are. §4.3: a per-KV-head map
// records which logical block each GPU slot holds. §5.1: a gather kernel reads
// the selected block-head entries from pinned host memory over PCIe and
// writes them into the resident GPU pages.
//
// A small fixed grid of 256-thread workgroups walks the (request, KV head)
// pairs (workgroup w takes pairs w, w + grid, ...); for each pair it does:
//   plan   the slot map, stamps and selection sit in LDS; ranks come from
//          workgroup scans (free slots, misses) and from counting (stale
//          slots by (stamp, slot)); slot_map / slot_stamp are updated in place
//          and the (slot, page) pairs stay in LDS;
//   copy   the entries are streamed in batches of PF: the PCIe loads of a
//          whole batch (PF x 2 x B x d x 2 bytes) are issued before any is
//          stored, K goes to the pool token-major, V is transposed through LDS
//          into the d x B layout the attention kernel reads.
// Host reads wait microseconds in the memory system, and while they are
// outstanding they slow the HBM traffic of every concurrent kernel (measured
// on MI355X: 64 copying workgroups triple the duration of a concurrent block
// scan, 16 add about 20 %, and 16 x 8 KiB in flight already saturate the
// link). So the grid holds at most kCopyWorkgroups workgroups with about
// kCopyInflight entries in flight between them.
#include <climits>

#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kMaxK = 1024;
constexpr int kPer = kMaxK / kPlanThreads;  // items per thread in the scans
constexpr int kCopyWorkgroups = 32;
constexpr int kCopyInflight = 32;  // block-head entries (K and V) in flight over the whole grid

// Monotone map of a float onto uint32 (larger float, larger key; -0 and +0 equal).
__device__ inline unsigned order_key(float f) {
  unsigned u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ int wg_exclusive_scan(int v, int* s_wave) {
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
  int base = 0;
  for (int w = 0; w < wave; ++w) base += s_wave[w];
  int total = 0;
  for (int w = 0; w < kPlanThreads / 64; ++w) total += s_wave[w];
  __syncthreads();
  if (threadIdx.x == 0) s_wave[4] = total;
  __syncthreads();
  return base + x - v;
}

// Plan of one (request, KV head); returns the number of entries in s_slot/s_page.
__device__ int plan_entries(const StageArgs& a, int rh, int r, int* s_slot, int* s_page, int* s_wave) {
  const int tid = threadIdx.x;
  const int k = a.k;
  __shared__ int s_sel[kMaxK], s_map[kMaxK], s_stamp[kMaxK], s_hit[kMaxK], s_keep[kMaxK], s_vict[kMaxK];
  __shared__ unsigned s_key[kMaxK];

  const long long base = (long long)rh * k;
  int m = a.sel_count[rh];
  m = m < 0 ? 0 : (m > k ? k : m);
  for (int i = tid; i < k; i += kPlanThreads) {
    s_sel[i] = i < m ? a.sel[base + i] : INT_MAX;
    s_hit[i] = 0;
    s_map[i] = a.slot_map[base + i];
    s_stamp[i] = a.slot_stamp[base + i];
    s_vict[i] = -1;
  }
  __syncthreads();

  // resident hits: binary search of every resident block in the (ascending) selection
  for (int s = tid; s < k; s += kPlanThreads) {
    const int b = s_map[s];
    int keep = 0;
    if (b >= 0) {
      int lo = 0, hi = m;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (s_sel[mid] < b) lo = mid + 1; else hi = mid;
      }
      if (lo < m && s_sel[lo] == b) {
        s_hit[lo] = 1;
        keep = 1;
      }
    }
    s_keep[s] = keep;
  }
  __syncthreads();

  // items [tid*kPer, tid*kPer + kPer): misses (selection order) and free slots (slot order)
  const int i0 = tid * kPer;
  int n_miss_local = 0, n_free_local = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = i0 + j;
    if (i < m && !s_hit[i]) ++n_miss_local;
    if (i < k && s_map[i] < 0) ++n_free_local;
  }
  wg_exclusive_scan(n_miss_local, s_wave);
  const int n_miss = s_wave[4];
  const int free_base = wg_exclusive_scan(n_free_local, s_wave);
  const int n_free = s_wave[4];

  // admission: every miss, or under a binding cap the fetch_cap misses with the
  // highest score (ties: lowest block id, i.e. lowest selection index). Keys are
  // order-preserving integers, so the ranks are distinct even for NaN scores and
  // exactly fetch_cap misses are admitted.
  const bool capped = a.fetch_cap < n_miss;
  if (capped) {
    for (int i = tid; i < m; i += kPlanThreads) {
      const int b = s_sel[i];
      const float sc = (b >= 0 && b < a.NBmax) ? a.scores[(long long)rh * a.NBmax + b] : -__builtin_inff();
      s_key[i] = s_hit[i] ? 0u : order_key(sc);
    }
    __syncthreads();
  }
  unsigned adm_bits = 0;
  int n_adm_local = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = i0 + j;
    if (i >= m || s_hit[i]) continue;
    bool adm = true;
    if (capped) {
      const unsigned key = s_key[i];
      int rank = 0;
      for (int t = 0; t < m; ++t) {
        if (s_hit[t]) continue;
        const unsigned kt = s_key[t];
        rank += (kt > key) || (kt == key && t < i);
      }
      adm = rank < a.fetch_cap;
    }
    if (adm) {
      adm_bits |= 1u << j;
      ++n_adm_local;
    }
  }
  const int adm_base = wg_exclusive_scan(n_adm_local, s_wave);
  const int n_adm = s_wave[4];

  // victim order: free slots ascending, then stale residents by (stamp, slot)
  {
    int fr = free_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int s = i0 + j;
      if (s < k && s_map[s] < 0) s_vict[fr++] = s;
    }
  }
  for (int s = tid; s < k; s += kPlanThreads) {
    if (s_map[s] < 0 || s_keep[s]) continue;
    const int st = s_stamp[s];
    int rank = n_free;
    for (int t = 0; t < k; ++t) {
      if (s_map[t] < 0 || s_keep[t]) continue;
      const int su = s_stamp[t];
      rank += (su < st) || (su == st && t < s);
    }
    s_vict[rank] = s;
  }
  __syncthreads();

  // pair the i-th admitted miss (ascending block id) with the i-th victim
  int moved_local = 0;
  {
    int mr = adm_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = i0 + j;
      if (!(adm_bits >> j & 1u)) continue;
      // a slot map holding one block twice can leave fewer victims than misses
      const int v = mr < k ? s_vict[mr] : -1;
      const int blk = s_sel[i];
      int page = -1;
      if (v >= 0 && blk >= 0 && blk < a.NBmax) page = a.block_table[(long long)r * a.NBmax + blk];
      if (page < 0 || page >= a.num_pages) page = -1;
      s_slot[mr] = v;
      s_page[mr] = page;
      if (v >= 0) {
        s_map[v] = page >= 0 ? blk : -1;
        s_keep[v] = page >= 0;
      }
      moved_local += page >= 0;
      ++mr;
    }
  }
  wg_exclusive_scan(moved_local, s_wave);
  const int moved = s_wave[4];

  for (int s = tid; s < k; s += kPlanThreads) {
    a.slot_map[base + s] = s_map[s];
    if (s_keep[s]) a.slot_stamp[base + s] = a.step;
  }
  if (tid == 0 && a.moved) a.moved[rh] = moved;
  return n_adm;
}

template <int BS, int PF>
__global__ __launch_bounds__(kPlanThreads) void stage_kernel(StageArgs a) {
  const int tid = threadIdx.x;
  __shared__ int s_slot[kMaxK + 1], s_page[kMaxK + 1];
  __shared__ int s_wave[8];
  constexpr int kElems = BS * kHeadDim;          // one K (or V) block-head entry
  constexpr int kChunks = kElems / 8 / kPlanThreads;  // 16-byte chunks per thread
  __shared__ uint16_t tile[PF][kElems];

  for (int rh = blockIdx.x; rh < a.R * a.Hkv; rh += gridDim.x) {
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  int n = a.local_only ? 0 : plan_entries(a, rh, r, s_slot, s_page, s_wave);
  if (a.copy_local) {
    const Ctx c = ctx_blocks(a.ctx_len[r], BS, a.NBmax);
    if (c.nb > 0) {
      const int page = a.block_table[(long long)r * a.NBmax + c.nb - 1];
      if (tid == 0) {
        s_slot[n] = a.k;
        s_page[n] = (page >= 0 && page < a.num_pages) ? page : -1;
      }
      ++n;
    }
  }
  __syncthreads();

  for (int e0 = 0; e0 < n; e0 += PF) {
    u32x4 kr[PF][kChunks], vr[PF][kChunks];
    int slot[PF], page[PF];
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int e = e0 + p;
      slot[p] = e < n ? s_slot[e] : -1;
      page[p] = e < n ? s_page[e] : -1;
      const bool live = page[p] >= 0 && slot[p] >= 0 && slot[p] <= a.k;
      if (!live) page[p] = -1;
      const long long src = ((long long)(live ? page[p] : 0) * a.Hkv + h) * kElems;
#pragma unroll
      for (int q = 0; q < kChunks; ++q) {
        const int c = (q * kPlanThreads + tid) * 8;
        kr[p][q] = live ? ldg16(a.host_k + src + c) : u32x4{0, 0, 0, 0};
        vr[p][q] = live ? ldg16(a.host_v + src + c) : u32x4{0, 0, 0, 0};
      }
    }
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      if (page[p] < 0) continue;
      const long long dst = (((long long)r * (a.k + 1) + slot[p]) * a.Hkv + h) * kElems;
#pragma unroll
      for (int q = 0; q < kChunks; ++q) {
        const int c = (q * kPlanThreads + tid) * 8;
        *reinterpret_cast<u32x4*>(a.pool_k + dst + c) = kr[p][q];
        *reinterpret_cast<u32x4*>(&tile[p][c]) = vr[p][q];
      }
    }
    __syncthreads();
    // V: [BS][d] -> [d][BS]; thread -> (d, 8-token group)
    constexpr int kGroups = BS / 8;
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      if (page[p] < 0) continue;
      const long long dst = (((long long)r * (a.k + 1) + slot[p]) * a.Hkv + h) * kElems;
#pragma unroll
      for (int w = tid; w < kHeadDim * kGroups; w += kPlanThreads) {
        const int d = w / kGroups;
        const int t0 = (w % kGroups) * 8;
        u32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t lo = tile[p][(t0 + 2 * j) * kHeadDim + d];
          const uint32_t hi = tile[p][(t0 + 2 * j + 1) * kHeadDim + d];
          o[j] = lo | (hi << 16);
        }
        *reinterpret_cast<u32x4*>(a.pool_v + dst + (long long)d * BS + t0) = o;
      }
    }
    __syncthreads();
  }
  __syncthreads();  // LDS plan arrays are reused by the next pair
  }
}

}  // namespace

template <int BS>
hipError_t launch_bs(const StageArgs& a, hipStream_t s) {
  const int nrh = a.R * a.Hkv;
  const int grid = nrh < kCopyWorkgroups ? nrh : kCopyWorkgroups;
  const int pf = kCopyInflight / grid;  // entries per workgroup batch
  if (pf >= 8)
    hipLaunchKernelGGL((stage_kernel<BS, 8>), dim3(grid), dim3(kPlanThreads), 0, s, a);
  else if (pf >= 4)
    hipLaunchKernelGGL((stage_kernel<BS, 4>), dim3(grid), dim3(kPlanThreads), 0, s, a);
  else if (pf >= 2)
    hipLaunchKernelGGL((stage_kernel<BS, 2>), dim3(grid), dim3(kPlanThreads), 0, s, a);
  else
    hipLaunchKernelGGL((stage_kernel<BS, 1>), dim3(grid), dim3(kPlanThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s) {
  return a.B == 16 ? launch_bs<16>(a, s) : launch_bs<32>(a, s);
}

}  // namespace oasis
