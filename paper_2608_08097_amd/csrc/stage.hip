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
// A grid of 256-thread workgroups walks the (request, KV head) pairs
// (workgroup w takes pairs w, w + grid, ...); for each pair it does:
//   plan   the slot map, stamps and selection sit in LDS; misses and stale
//          slots are compacted by workgroup scans and ranked one item per
//          thread (misses by score under a cap, stale slots by (stamp, slot));
//          slot_map / slot_stamp are updated in place and the (slot, page)
//          pairs stay in LDS;
//   copy   the entries are streamed in batches of PF with two batches in
//          flight: the PCIe loads of the next batch are issued before the
//          current one is stored; K goes to the pool token-major, V is
//          transposed through LDS into the d x B layout the attention kernel
//          reads.
// Host reads take microseconds to return, so the plans run in parallel and
// each workgroup keeps a batch of entries in flight. Host reads beyond what
// saturates the link only queue inside the GPU, where they slow the HBM
// traffic of concurrent kernels (measured on MI355X: with 3 MB moved per step,
// 8 entries per workgroup in flight on 64 workgroups stretch a concurrent
// block scan from 57 to 98 us, 2 entries to 88 us). The grid is therefore one
// workgroup per two pairs, kept between kCopyWorkgroupsMin and
// kCopyWorkgroupsMax, with 2 entries in flight per workgroup (1 per batch;
// more on small grids, so that the link still fills). Keeping the second
// batch in flight while the first is stored raised the reasoning loop of
// 32 layers x 64 requests from 6,300 to 6,710 tokens/s (the transfer there
// paces the step) and changed 8 x 131,072 tokens by -1 %. Step rates measured
// before that change (steps/s) for
// 32 / 48 / 64 workgroups: 8 x 131,072 tokens (64 pairs) 10,490 / 9,790 /
// 9,290; 32 requests of 16K-32K tokens (256 pairs) 7,920 / 8,540 / 8,400;
// 16 x 65,536 tokens with B = 32 (128 pairs) 3,510 / 3,510 / 3,700. Fewer
// workgroups mean more plans in series per workgroup, which the last two
// cannot afford.
#include <climits>

#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kMaxK = 1024;
constexpr int kPer = kMaxK / kPlanThreads;  // items per thread in the scans
constexpr int kKeyPad = 4;
constexpr int kCopyWorkgroupsMin = 32;
constexpr int kCopyWorkgroupsMax = 64;
constexpr int kCopyInflightMin = 64;  // block-head entries (K and V) in flight over the whole grid, at least
constexpr int kLocalWorkgroups = 256;  // grid of a local-block-only call

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
//
// Misses and stale slots are first compacted (in ascending selection index and
// ascending slot, which is ascending block id and slot order); each thread then
// ranks one compacted item against all others, reading the keys four at a time
// from LDS, so no thread walks a long chain of dependent reads.
__device__ int plan_entries(const StageArgs& a, int rh, int r, int* s_slot, int* s_page, int* s_wave) {
  const int tid = threadIdx.x;
  const int k = a.k;
  // by selection index: s_sel, s_hit; by slot: s_map, s_stamp, s_keep; victims in order: s_vict;
  // compacted misses: key, selection index, admitted; compacted stale slots: stamp, slot
  __shared__ int s_sel[kMaxK], s_hit[kMaxK], s_map[kMaxK], s_stamp[kMaxK], s_keep[kMaxK], s_vict[kMaxK];
  __shared__ __align__(16) unsigned s_mkey[kMaxK + kKeyPad];
  __shared__ __align__(16) int s_skey[kMaxK + kKeyPad];
  __shared__ int s_midx[kMaxK], s_madm[kMaxK], s_sslot[kMaxK];
  // by selection index: the page of the block and its score key (under a possible cap)
  __shared__ int s_selpage[kMaxK];
  __shared__ unsigned s_selkey[kMaxK];

  const long long base = (long long)rh * k;
  int m = a.sel_count[rh];
  m = m < 0 ? 0 : (m > k ? k : m);
  // The page of every selected block (and, when a cap may bind, its score) is
  // fetched as soon as the block id arrives, so that these dependent loads
  // overlap the search below instead of stalling the pairing later.
  const bool may_cap = a.fetch_cap < m;
  int pg[kPer];
  unsigned ky[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kPlanThreads;
    pg[j] = -1;
    ky[j] = 0u;
    if (i < k) {
      const int sv = a.sel[base + i];  // in the row (k entries); loaded without waiting for the count
      const int b = i < m ? sv : INT_MAX;
      s_sel[i] = b;
      s_hit[i] = 0;
      s_map[i] = a.slot_map[base + i];
      s_stamp[i] = a.slot_stamp[base + i];
      if (i < m) {
        const bool in_row = b >= 0 && b < a.NBmax;
        if (in_row) pg[j] = a.block_table[(long long)r * a.NBmax + b];
        if (may_cap) ky[j] = order_key(in_row ? a.scores[(long long)rh * a.NBmax + b] : -__builtin_inff());
      }
    }
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
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kPlanThreads;
    if (i < k) {
      s_selpage[i] = pg[j];
      s_selkey[i] = ky[j];
    }
  }
  __syncthreads();

  // items [i0, i0 + kPer): selection entries (misses) and slots (free, stale)
  const int i0 = tid * kPer;
  int nm = 0, nf = 0, ns = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = i0 + j;
    if (i < m && !s_hit[i]) ++nm;
    if (i < k) {
      if (s_map[i] < 0) ++nf;
      else if (!s_keep[i]) ++ns;
    }
  }
  const int mf_base = wg_exclusive_scan(nm | (nf << 16), s_wave);  // two 16-bit counts (<= 1024 each)
  const int mf_tot = s_wave[4];
  const int st_base = wg_exclusive_scan(ns, s_wave);
  const int n_stale = s_wave[4];
  const int n_miss = mf_tot & 0xFFFF;
  const int n_free = mf_tot >> 16;

  // admission: every miss, or under a binding cap the fetch_cap misses with the
  // highest score (ties: lowest block id). Keys are order-preserving integers, so
  // the ranks are distinct even for NaN scores and exactly fetch_cap misses are
  // admitted.
  const bool capped = a.fetch_cap < n_miss;
  {
    int mr = mf_base & 0xFFFF, fr = mf_base >> 16, sr = st_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = i0 + j;
      if (i < m && !s_hit[i]) {
        s_mkey[mr] = capped ? s_selkey[i] : 0u;
        s_midx[mr] = i;
        ++mr;
      }
      if (i < k) {
        if (s_map[i] < 0) {
          s_vict[fr++] = i;
        } else if (!s_keep[i]) {
          s_skey[sr] = s_stamp[i];
          s_sslot[sr] = i;
          ++sr;
        }
      }
    }
    // pads read by the 4-wide loops below; they never rank ahead of a real item
    if (tid < kKeyPad) {
      s_mkey[n_miss + tid] = 0u;
      s_skey[n_stale + tid] = INT_MAX;
    }
  }
  __syncthreads();

  for (int c = tid; c < n_miss; c += kPlanThreads) {
    int adm = 1;
    if (capped) {
      const unsigned key = s_mkey[c];
      int rank = 0;
#pragma unroll 4
      for (int t = 0; t < n_miss; t += 4) {
        const u32x4 kt = *reinterpret_cast<const u32x4*>(&s_mkey[t]);
#pragma unroll
        for (int e = 0; e < 4; ++e) rank += (kt[e] > key) || (kt[e] == key && t + e < c);
      }
      adm = rank < a.fetch_cap;
    }
    s_madm[c] = adm;
  }
  // victim order: free slots ascending (already in s_vict), then stale slots by (stamp, slot)
  for (int c = tid; c < n_stale; c += kPlanThreads) {
    const int st = s_skey[c];
    int rank = 0;
#pragma unroll 4
    for (int t = 0; t < n_stale; t += 4) {
      const int4 kt = *reinterpret_cast<const int4*>(&s_skey[t]);
      rank += (kt.x < st) || (kt.x == st && t < c);
      rank += (kt.y < st) || (kt.y == st && t + 1 < c);
      rank += (kt.z < st) || (kt.z == st && t + 2 < c);
      rank += (kt.w < st) || (kt.w == st && t + 3 < c);
    }
    s_vict[n_free + rank] = s_sslot[c];
  }
  __syncthreads();

  // the i-th admitted miss (ascending block id) goes to the i-th victim
  int na = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = i0 + j;
    if (c < n_miss && s_madm[c]) ++na;
  }
  const int adm_base = wg_exclusive_scan(na, s_wave);
  const int n_adm = s_wave[4];
  const int n_vict = n_free + n_stale;
  int moved_local = 0;
  {
    int ar = adm_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int c = i0 + j;
      if (c >= n_miss || !s_madm[c]) continue;
      // a slot map holding one block twice can leave fewer victims than misses
      const int v = ar < n_vict ? s_vict[ar] : -1;
      const int blk = s_sel[s_midx[c]];
      int page = v >= 0 ? s_selpage[s_midx[c]] : -1;
      if (page < 0 || page >= a.num_pages) page = -1;
      s_slot[ar] = v;
      s_page[ar] = page;
      if (v >= 0) {
        s_map[v] = page >= 0 ? blk : -1;
        s_keep[v] = page >= 0;
      }
      moved_local += page >= 0;
      ++ar;
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

// One batch of PF block-head entries held in registers (K and V, 16-byte
// chunks of each entry spread over the workgroup).
template <int BS, int PF>
struct CopyBatch {
  static constexpr int kChunks = BS * kHeadDim / 8 / kPlanThreads;
  u32x4 k[PF][kChunks], v[PF][kChunks];
  int slot[PF], page[PF];
};

template <int BS, int PF>
__device__ __forceinline__ void fetch_batch(const StageArgs& a, CopyBatch<BS, PF>& b, int e0, int n, int r, int h,
                                            const int* s_slot, const int* s_page) {
  constexpr int kElems = BS * kHeadDim;
  const int tid = threadIdx.x;
  // placeholder source: slot 0 of this (r, h) in the pool
  const long long hold = (((long long)r * (a.k + 1)) * a.Hkv + h) * kElems;
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    const int e = e0 + p;
    b.slot[p] = e < n ? s_slot[e] : -1;
    b.page[p] = e < n ? s_page[e] : -1;
    const bool live = b.page[p] >= 0 && b.slot[p] >= 0 && b.slot[p] <= a.k;
    if (!live) b.page[p] = -1;
    const long long src = ((long long)(live ? b.page[p] : 0) * a.Hkv + h) * kElems;
    const uint16_t* ks = live ? a.host_k + src : a.pool_k + hold;
    const uint16_t* vs = live ? a.host_v + src : a.pool_k + hold;
#pragma unroll
    for (int q = 0; q < CopyBatch<BS, PF>::kChunks; ++q) {
      const int c = (q * kPlanThreads + tid) * 8;
      b.k[p][q] = ldg16(ks + c);
      b.v[p][q] = ldg16(vs + c);
    }
  }
}

// Store a fetched batch: K token-major into the pool, V transposed through LDS
// into the d x B layout the attention kernel reads.
template <int BS, int PF>
__device__ __forceinline__ void put_batch(const StageArgs& a, const CopyBatch<BS, PF>& b, int r, int h,
                                          uint16_t (*tile)[BS * kHeadDim]) {
  constexpr int kElems = BS * kHeadDim;
  const int tid = threadIdx.x;
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    if (b.page[p] < 0) continue;
    const long long dst = (((long long)r * (a.k + 1) + b.slot[p]) * a.Hkv + h) * kElems;
#pragma unroll
    for (int q = 0; q < CopyBatch<BS, PF>::kChunks; ++q) {
      const int c = (q * kPlanThreads + tid) * 8;
      *reinterpret_cast<u32x4*>(a.pool_k + dst + c) = b.k[p][q];
      *reinterpret_cast<u32x4*>(&tile[p][c]) = b.v[p][q];
    }
  }
  __syncthreads();
  // V: [BS][d] -> [d][BS]; thread -> (d, 8-token group)
  constexpr int kGroups = BS / 8;
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    if (b.page[p] < 0) continue;
    const long long dst = (((long long)r * (a.k + 1) + b.slot[p]) * a.Hkv + h) * kElems;
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

template <int BS, int PF>
__global__ __launch_bounds__(kPlanThreads) void stage_kernel(StageArgs a) {
  const int tid = threadIdx.x;
  __shared__ int s_slot[kMaxK + 1], s_page[kMaxK + 1];
  __shared__ int s_wave[8];
  constexpr int kElems = BS * kHeadDim;          // one K (or V) block-head entry
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

  // Batches of PF entries, two in flight: the host reads of the next batch are
  // issued before the current one is stored, so the link does not idle while
  // a batch is written and V is transposed. Every load is issued; an entry
  // past the end (or without a page) reads slot 0 of this (r, h) in the pool
  // instead (device memory, discarded), so the wait counts stay exact.
  CopyBatch<BS, PF> x, y;
  fetch_batch<BS, PF>(a, x, 0, n, r, h, s_slot, s_page);
  for (int e0 = 0; e0 < n; e0 += 2 * PF) {
    fetch_batch<BS, PF>(a, y, e0 + PF, n, r, h, s_slot, s_page);
    put_batch<BS, PF>(a, x, r, h, tile);
    if (e0 + PF >= n) break;
    fetch_batch<BS, PF>(a, x, e0 + 2 * PF, n, r, h, s_slot, s_page);
    put_batch<BS, PF>(a, y, r, h, tile);
  }
  __syncthreads();  // LDS plan arrays are reused by the next pair
  }
}

}  // namespace

template <int BS>
hipError_t launch_bs(const StageArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int nrh = a.R * a.Hkv;
  if (nrh <= 0) return hipSuccess;
  int grid = nrh / 2;
  grid = grid < kCopyWorkgroupsMin ? kCopyWorkgroupsMin : (grid > kCopyWorkgroupsMax ? kCopyWorkgroupsMax : grid);
  // the local block alone (no plan, one entry per pair, on the caller's critical path): spread wide
  if (a.local_only) grid = nrh < kLocalWorkgroups ? nrh : kLocalWorkgroups;
  if (grid > nrh) grid = nrh;
  // entries per batch; two batches are in flight per workgroup
  const int pf = grid * 2 >= kCopyInflightMin ? 1 : kCopyInflightMin / (2 * grid);
  if (pf >= 8)
    launch_kernel(stage_kernel<BS, 8>, dim3(grid), dim3(kPlanThreads), s, t, a);
  else if (pf >= 4)
    launch_kernel(stage_kernel<BS, 4>, dim3(grid), dim3(kPlanThreads), s, t, a);
  else if (pf >= 2)
    launch_kernel(stage_kernel<BS, 2>, dim3(grid), dim3(kPlanThreads), s, t, a);
  else
    launch_kernel(stage_kernel<BS, 1>, dim3(grid), dim3(kPlanThreads), s, t, a);
  return hipGetLastError();
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s, const LaunchTiming& t) {
  return a.B == 16 ? launch_bs<16>(a, s, t) : launch_bs<32>(a, s, t);
}

}  // namespace oasis
