// Delta selection and KV transfer into the HBM working set.
//
// Paper §4.2.3: the predicted set is intersected with the resident set (hits
// stay, no bytes move), non-selected residents are ranked by the step at which
// they were last selected and evicted least-recently-selected first, and each
// admitted miss is paired with one eviction target. §4.3: a per-KV-head map
// records which logical block each GPU slot holds. §5.1: a gather kernel reads
// the selected block-head entries from pinned host memory over PCIe and
// writes them into the resident GPU pages.
//
// plan kernel   one 256-thread workgroup per (request, KV head); the slot map,
//               stamps and selection sit in LDS; ranks come from block scans
//               (free slots, misses) and from counting (stale slots by
//               (stamp, slot)). It updates slot_map / slot_stamp in place and
//               writes (slot, page) pairs to the workspace.
// gather kernel one 256-thread workgroup per planned entry (plus one per head
//               for the local block): 16-byte loads from the host page (PCIe),
//               K stored token-major, V transposed through LDS to the d x B
//               layout the attention kernel consumes.
#include <climits>

#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kMaxK = 1024;
constexpr int kPer = kMaxK / kPlanThreads;  // items per thread in the scans

struct PlanEntry {
  int32_t slot;
  int32_t page;
};

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

__global__ __launch_bounds__(kPlanThreads) void stage_plan_kernel(StageArgs a) {
  const int rh = blockIdx.x;
  const int r = rh / a.Hkv;
  const int tid = threadIdx.x;
  const int k = a.k;
  __shared__ int s_sel[kMaxK], s_map[kMaxK], s_stamp[kMaxK], s_hit[kMaxK], s_keep[kMaxK], s_vict[kMaxK];
  __shared__ int s_wave[8];

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
  const int miss_base = wg_exclusive_scan(n_miss_local, s_wave);
  const int n_miss = s_wave[4];
  const int free_base = wg_exclusive_scan(n_free_local, s_wave);
  const int n_free = s_wave[4];

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

  // pair the i-th miss with the i-th victim
  PlanEntry* plan = reinterpret_cast<PlanEntry*>(a.plan) + base;
  int moved_local = 0;
  {
    int mr = miss_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = i0 + j;
      if (i >= m || s_hit[i]) continue;
      // a slot map holding one block twice can leave fewer victims than misses
      const int v = mr < k ? s_vict[mr] : -1;
      const int blk = s_sel[i];
      int page = -1;
      if (v >= 0 && blk >= 0 && blk < a.NBmax) page = a.block_table[(long long)r * a.NBmax + blk];
      if (page < 0 || page >= a.num_pages) page = -1;
      plan[mr] = PlanEntry{v, page};
      if (v >= 0) {
        s_map[v] = page >= 0 ? blk : -1;
        s_keep[v] = page >= 0;
      }
      moved_local += page >= 0;
      ++mr;
    }
  }
  // total copied entries (reuses the scan's total)
  wg_exclusive_scan(moved_local, s_wave);
  const int moved = s_wave[4];

  for (int s = tid; s < k; s += kPlanThreads) {
    a.slot_map[base + s] = s_map[s];
    if (s_keep[s]) a.slot_stamp[base + s] = a.step;
  }
  if (tid == 0) {
    a.plan_count[rh] = n_miss;
    if (a.moved) a.moved[rh] = moved;
  }
}

template <int BS>
__global__ __launch_bounds__(256) void stage_gather_kernel(StageArgs a) {
  const int rh = blockIdx.y;
  const int e = a.local_only ? a.k : (int)blockIdx.x;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const int tid = threadIdx.x;
  int slot, page;
  if (e < a.k) {
    if (e >= a.plan_count[rh]) return;
    const PlanEntry p = reinterpret_cast<const PlanEntry*>(a.plan)[(long long)rh * a.k + e];
    slot = p.slot;
    page = p.page;
    if (page < 0 || slot < 0 || slot >= a.k) return;
  } else {
    if (!a.copy_local) return;
    const Ctx c = ctx_blocks(a.ctx_len[r], BS, a.NBmax);
    if (c.nb == 0) return;
    page = a.block_table[(long long)r * a.NBmax + c.nb - 1];
    if (page < 0 || page >= a.num_pages) return;
    slot = a.k;
  }
  constexpr int kElems = BS * kHeadDim;
  const long long src = ((long long)page * a.Hkv + h) * kElems;
  const long long dst = (((long long)r * (a.k + 1) + slot) * a.Hkv + h) * kElems;
  __shared__ uint16_t tile[kElems];
#pragma unroll
  for (int c = tid; c < kElems / 8; c += 256) {
    const u32x4 kv = ldg16(a.host_k + src + c * 8);
    const u32x4 vv = ldg16(a.host_v + src + c * 8);
    *reinterpret_cast<u32x4*>(a.pool_k + dst + c * 8) = kv;
    *reinterpret_cast<u32x4*>(tile + c * 8) = vv;
  }
  __syncthreads();
  // V: [BS][d] -> [d][BS]; thread -> (d, 8-token group)
  constexpr int kGroups = BS / 8;
#pragma unroll
  for (int w = tid; w < kHeadDim * kGroups; w += 256) {
    const int d = w / kGroups;
    const int t0 = (w % kGroups) * 8;
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t lo = tile[(t0 + 2 * j) * kHeadDim + d];
      const uint32_t hi = tile[(t0 + 2 * j + 1) * kHeadDim + d];
      o[j] = lo | (hi << 16);
    }
    *reinterpret_cast<u32x4*>(a.pool_v + dst + (long long)d * BS + t0) = o;
  }
}

}  // namespace

size_t stage_workspace_bytes(int R, int Hkv, int k) {
  const size_t nrh = (size_t)R * Hkv;
  return nrh * (size_t)k * sizeof(PlanEntry) + nrh * sizeof(int32_t);
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s) {
  const unsigned nrh = (unsigned)(a.R * a.Hkv);
  if (!a.local_only) {
    hipLaunchKernelGGL(stage_plan_kernel, dim3(nrh), dim3(kPlanThreads), 0, s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const dim3 grid(a.local_only ? 1u : (unsigned)(a.k + 1), nrh);
  if (a.B == 16)
    hipLaunchKernelGGL(stage_gather_kernel<16>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(stage_gather_kernel<32>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace oasis
