// Delta selection and KV transfer into the HBM working set.
//
// Paper §4.2.3: the predicted set is intersected with the resident set (hits
// stay, no bytes move), non-selected residents are ranked by the step at which
// they were last selected and evicted least-recently-selected first, and each
// admitted miss is paired with one eviction target; at most fetch_cap pairs are
// admitted per KV head and step (§5.5.1: a fetch ratio of K), the highest-
// scoring misses first, and all other slots stay as they are. §4.3: a per-KV-head map
// records which logical block each GPU slot holds. §5.1: the copy is done by a
// kernel on the GPU that pulls each admitted (block, KV head) entry out of
// pinned host memory across PCIe and stores it straight into its pool slot.
//
// A grid of 256-thread workgroups walks the (request, KV head) pairs
// (workgroup w takes pairs w, w + grid, ...), as many pairs per pass as the
// LDS plan arrays hold (kMaxK / k, at most kMaxPairs); each pass does:
//   plan   the slot maps, stamps and selections of the pass's pairs sit in
//          LDS side by side. With k >= 64 one wave plans a pair alone
//          (plan_pair_wave): ballots and lane prefix counts compact misses and
//          stale slots, and under a cap of at most kPlanRounds the admitted
//          misses and the victims they need are picked in wave rounds, with
//          no workgroup barrier until every pair is done (measured on
//          MI355X, 8 x 131,072 tokens, 2 pairs per workgroup: staging alone
//          72.0 -> 69.5 us, plan phase 13 -> 10 us). With smaller k, where
//          a pair does not fill a wave, the whole workgroup plans the pass:
//          workgroup scans compact the items, which are ranked one item per
//          thread within their pair (misses by score under a cap, stale
//          slots by (stamp, slot)). Either way slot_map / slot_stamp are
//          updated in place and the (slot, page, pair) entries stay in LDS;
//   copy   the entries of all the pass's pairs are streamed in batches of PF
//          with two batches in flight: the PCIe loads of the next batch are
//          issued before the current one is stored; K goes to the pool
//          token-major, V is transposed through LDS into the d x B layout the
//          attention kernel reads.
// Host reads take microseconds to return, so the plans run in parallel and
// each workgroup keeps a batch of entries in flight. A plan costs a few
// dependent global reads and a dozen barriers, so the pairs of a workgroup
// are planned in one pass rather than one after another (measured on MI355X,
// 8 x 131,072 tokens, 2 pairs per workgroup: the plans alone take 25 us of
// an 80 us capped step when made in series; planned together, the step rate
// rose from 10,350 to 10,660 steps/s).
//
// Host reads beyond what saturates the link only queue inside the GPU, where
// they slow the HBM traffic of concurrent kernels (measured on MI355X: with
// 3 MB moved per step, 8 entries per workgroup in flight on 64 workgroups
// stretch a concurrent block scan from 57 to 98 us, 2 entries to 88 us). The
// grid is therefore small, with 2 entries in flight per workgroup (1 per
// batch; more on small grids, so that the link still fills): 32 workgroups at
// B = 16; at B = 32, whose 16 KiB entries take twice the stores and
// transposes, one per two pairs within 32 to 64. Step rates measured with
// batched plans, 32 against 64 workgroups: 32 requests of 16K-32K tokens
// (256 pairs) 9,020 against 8,220 steps/s; the reasoning loop of 32 layers x
// 64 requests (512 pairs) 3,360 against 3,180 layer-steps/s; 16 x 65,536
// tokens with B = 32 (128 pairs, paced by the transfer) 3,570 against 3,770.
// Fewer than 32 (16, 8) were slower at 8 x 131,072 tokens. Keeping the second
// batch in flight while the first is stored raised the reasoning loop from
// 6,300 to 6,710 tokens/s and changed 8 x 131,072 tokens by -1 %.
#include <climits>

#include "oasis_internal.h"
#include "score_core.h"
#include "select.h"

namespace oasis {

namespace {

constexpr int kPlanThreads = 256;
constexpr int kMaxK = 1024;
constexpr int kPer = kMaxK / kPlanThreads;  // items per thread of the staging kernel's passes
constexpr int kMaxPairs = 64;  // (request, KV head) pairs planned in one pass, at most
constexpr int kCopyWorkgroups = 32;
constexpr int kCopyInflightMin = 64;  // block-head entries (K and V) in flight over the whole grid, at least
constexpr int kLocalWorkgroups = 256;  // grid of a local-block-only call

// Monotone map of a float onto uint32 (larger float, larger key; -0 and +0 equal).
__device__ inline unsigned order_key(float f) {
  unsigned u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Wave-wide minimum of uint32 values, returned to every lane (the DPP steps of
// wave_min_max in select.h, one value).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  int a = (int)v;
#define OASIS_DPP_MIN(CTRL, ROWS) \
  a = (int)min((uint32_t)a, (uint32_t)__builtin_amdgcn_update_dpp((int)0xFFFFFFFF, a, CTRL, ROWS, 0xF, false));
  OASIS_DPP_MIN(0x111, 0xF)
  OASIS_DPP_MIN(0x112, 0xF)
  OASIS_DPP_MIN(0x114, 0xF)
  OASIS_DPP_MIN(0x118, 0xF)
  OASIS_DPP_MIN(0x142, 0xA)
  OASIS_DPP_MIN(0x143, 0xC)
#undef OASIS_DPP_MIN
  return (uint32_t)__builtin_amdgcn_readlane(a, 63);
}

// Up to this many admitted misses (or victims) of a pair are picked one at a
// time by a wave (wave_min_u32 rounds); beyond it every item is ranked against
// all others of its pair.
constexpr int kPlanRounds = 16;
static_assert(kMaxK / 64 <= 32, "a lane's items of a pair fit one 32-bit mask");

// Exclusive scan over an NTHR-thread workgroup; the total is left in
// s_wave[NTHR / 64] (s_wave holds NTHR / 64 + 1 ints).
template <int NTHR>
__device__ int wg_exclusive_scan(int v, int* s_wave) {
  constexpr int kWaves = NTHR / 64;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int x = wave_incl_sum(v);
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  int base = 0;
  for (int w = 0; w < wave; ++w) base += s_wave[w];
  int total = 0;
  for (int w = 0; w < kWaves; ++w) total += s_wave[w];
  __syncthreads();
  if (threadIdx.x == 0) s_wave[kWaves] = total;
  __syncthreads();
  return base + x - v;
}

// Orders the LDS accesses of one wave's lanes (a wave's LDS operations execute
// in program order; this keeps the compiler from moving them across).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Lanes below this one whose bit is set in `mask`.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// Shared-memory arrays of a plan pass (kMaxK items, kMaxPairs pairs).
struct PlanLds {
  int *sel, *hit, *map, *stamp, *keep, *selpage;
  unsigned *selkey, *mkey;
  int *midx, *madm, *skey, *sslot, *vstale, *free_;
};

// The plan of one (request, KV head) pair by one wave (k >= 64, so the pair
// fills the wave), with the semantics of the workgroup plan below: selection
// items [i0, i0 + k) and slot items [i0, i0 + k) of the pass arrays are this
// pair's, and only its wave touches them, so no workgroup barrier is needed
// until every pair is done. Compactions are ballots and lane prefix counts;
// admission and victim order are wave rounds (or ranking past kPlanRounds).
// Leaves the pair's entries (slot, page) at L.madm / L.hit [i0, i0 + nadm)
// and returns nadm.
__device__ int plan_pair_wave(const StageArgs& a, int rh, int i0, int m, const int* lsel, const PlanLds& L,
                              int* moved_out) {
  const int lane = threadIdx.x & 63;
  const int k = a.k;
  const long long row = (long long)rh * k;
  const int r = rh / a.Hkv;
  const bool capped = a.fetch_cap < m;
  // selection, slot map and stamps: all loads of a batch of four 64-item groups
  // are issued before any is stored
  for (int g0 = 0; g0 < k; g0 += 256) {
    int sv[4], mp[4], st[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int li = g0 + 64 * u + lane;
      if (li < k) {
        sv[u] = lsel ? lsel[li] : a.sel[row + li];
        mp[u] = a.slot_map[row + li];
        st[u] = a.slot_stamp[row + li];
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int li = g0 + 64 * u + lane;
      if (li < k) {
        L.sel[i0 + li] = li < m ? sv[u] : INT_MAX;
        L.hit[i0 + li] = 0;
        L.map[i0 + li] = mp[u];
        L.stamp[i0 + li] = st[u];
      }
    }
  }
  wave_lds_sync();
  // the page (and under a binding cap the score) of every selected block
  for (int g0 = 0; g0 < k; g0 += 256) {
    int pg[4];
    unsigned ky[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int li = g0 + 64 * u + lane;
      pg[u] = -1;
      ky[u] = 0u;
      if (li < m) {
        const int b = L.sel[i0 + li];
        const bool in_row = b >= 0 && b < a.NBmax;
        if (in_row) pg[u] = a.block_table[(long long)r * a.NBmax + b];
        if (capped) ky[u] = order_key(in_row ? a.scores[(long long)rh * a.NBmax + b] : -__builtin_inff());
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int li = g0 + 64 * u + lane;
      if (li < k) {
        L.selpage[i0 + li] = pg[u];
        L.selkey[i0 + li] = ky[u];
      }
    }
  }
  // resident hits: binary search of every resident block in the (ascending) selection
  for (int li = lane; li < k; li += 64) {
    const int b = L.map[i0 + li];
    int keep = 0;
    if (b >= 0) {
      int lo = 0, hi = m;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (L.sel[i0 + mid] < b) lo = mid + 1; else hi = mid;
      }
      if (lo < m && L.sel[i0 + lo] == b) {
        L.hit[i0 + lo] = 1;
        keep = 1;
      }
    }
    L.keep[i0 + li] = keep;
  }
  wave_lds_sync();
  // misses (selection side), free and stale slots, each compacted in ascending order
  int nm = 0, nf = 0, ns = 0;
  for (int g0 = 0; g0 < k; g0 += 64) {
    const int li = g0 + lane;
    const bool in = li < k;
    const int mp = in ? L.map[i0 + li] : -1;
    const bool miss = in && li < m && !L.hit[i0 + li];
    const bool fre = in && mp < 0;
    const bool stale = in && mp >= 0 && !L.keep[i0 + li];
    const uint64_t bm = __ballot(miss), bf = __ballot(fre), bs = __ballot(stale);
    if (miss) {
      const int at = i0 + nm + lanes_below(bm);
      L.mkey[at] = L.selkey[i0 + li];
      L.midx[at] = li;
    }
    if (fre) L.free_[i0 + nf + lanes_below(bf)] = li;
    if (stale) {
      const int at = i0 + ns + lanes_below(bs);
      L.skey[at] = L.stamp[i0 + li];
      L.sslot[at] = li;
    }
    nm += __popcll(bm);
    nf += __popcll(bf);
    ns += __popcll(bs);
  }
  wave_lds_sync();
  // admission: bit j of `adm` is miss lane + 64 j
  const int cap = a.fetch_cap;
  uint32_t adm = 0;
  int nadm = nm;
  if (cap >= nm) {
    for (int j = 0; lane + 64 * j < nm; ++j) adm |= 1u << j;
  } else if (cap <= kPlanRounds) {
    nadm = cap < 0 ? 0 : cap;
    for (int rd = 0; rd < cap; ++rd) {
      uint32_t bk = 0xFFFFFFFFu, bi = 0xFFFFFFFFu;  // complemented key: lowest = highest score
      for (int j = 0, c = lane; c < nm; ++j, c += 64) {
        const uint32_t kc = ~L.mkey[i0 + c];
        if (!((adm >> j) & 1u) && (kc < bk || bi == 0xFFFFFFFFu)) {  // ascending c: ties keep the lower
          bk = kc;
          bi = (uint32_t)c;
        }
      }
      const uint32_t wk = wave_min_u32(bi == 0xFFFFFFFFu ? 0xFFFFFFFFu : bk);
      const uint32_t wi = wave_min_u32(bi != 0xFFFFFFFFu && bk == wk ? bi : 0xFFFFFFFFu);
      if ((int)(wi & 63) == lane) adm |= 1u << (wi >> 6);
    }
  } else {
    nadm = cap;
    for (int j = 0, c = lane; c < nm; ++j, c += 64) {
      const unsigned key = L.mkey[i0 + c];
      int rank = 0;
#pragma unroll 4
      for (int t = 0; t < nm; ++t) {
        const unsigned kt = L.mkey[i0 + t];
        rank += (kt > key) || (kt == key && t < c);
      }
      if (rank < cap) adm |= 1u << j;
    }
  }
  // victims: free slots ascending, then stale slots by (stamp, slot); the first
  // (admitted - free) stale ones go to L.vstale
  int need = nadm - nf;
  need = need < 0 ? 0 : (need > ns ? ns : need);
  if (need <= kPlanRounds) {
    uint32_t taken = 0;
    for (int rd = 0; rd < need; ++rd) {
      uint32_t bs = 0xFFFFFFFFu, bi = 0xFFFFFFFFu;
      for (int j = 0, t = lane; t < ns; ++j, t += 64) {
        const uint32_t sk = (uint32_t)L.skey[i0 + t] ^ 0x80000000u;  // signed order
        if (!((taken >> j) & 1u) && (sk < bs || bi == 0xFFFFFFFFu)) {
          bs = sk;
          bi = (uint32_t)t;
        }
      }
      const uint32_t ws = wave_min_u32(bi == 0xFFFFFFFFu ? 0xFFFFFFFFu : bs);
      const uint32_t wi = wave_min_u32(bi != 0xFFFFFFFFu && bs == ws ? bi : 0xFFFFFFFFu);
      if ((int)(wi & 63) == lane) taken |= 1u << (wi >> 6);
      if (lane == 0) L.vstale[i0 + rd] = L.sslot[i0 + wi];
    }
  } else {
    for (int c = lane; c < ns; c += 64) {
      const int sk = L.skey[i0 + c];
      int rank = 0;
#pragma unroll 4
      for (int t = 0; t < ns; ++t) {
        const int kt = L.skey[i0 + t];
        rank += (kt < sk) || (kt == sk && t < c);
      }
      L.vstale[i0 + rank] = L.sslot[i0 + c];
    }
  }
  wave_lds_sync();
  // the a-th admitted miss (ascending block id) goes to the a-th victim
  int ar = 0, moved = 0;
  for (int j = 0; 64 * j < nm; ++j) {
    const int c = lane + 64 * j;
    const bool isadm = c < nm && ((adm >> j) & 1u);
    const uint64_t ba = __ballot(isadm);
    int page = -1;
    if (isadm) {
      const int e = ar + lanes_below(ba);
      const int v = e < nf ? L.free_[i0 + e] : (e < nf + ns ? L.vstale[i0 + e - nf] : -1);
      const int li = L.midx[i0 + c];
      const int blk = L.sel[i0 + li];
      page = v >= 0 ? L.selpage[i0 + li] : -1;
      if (page < 0 || page >= a.num_pages) page = -1;
      L.madm[i0 + e] = v;    // entry: slot of the pair (-1: none)
      L.hit[i0 + e] = page;  // entry: host page (-1: none)
      if (v >= 0) {
        L.map[i0 + v] = page >= 0 ? blk : -1;
        L.keep[i0 + v] = page >= 0;
      }
    }
    moved += __popcll(__ballot(isadm && page >= 0));
    ar += __popcll(ba);
  }
  wave_lds_sync();
  if (a.mode == kStagePlanOnly) {
    const long long nrhk = (long long)a.R * a.Hkv * k;
    int32_t* ws_map = a.ws;
    int32_t* ws_stamp = a.ws + nrhk;
    int2* ws_ent = reinterpret_cast<int2*>(a.ws + 2 * nrhk);
    int32_t* ws_cnt = a.ws + 4 * nrhk;
    for (int li = lane; li < k; li += 64) {
      ws_map[row + li] = L.map[i0 + li];
      ws_stamp[row + li] = L.keep[i0 + li] ? a.step : L.stamp[i0 + li];
    }
    for (int e = lane; e < nadm; e += 64) ws_ent[row + e] = make_int2(L.madm[i0 + e], L.hit[i0 + e]);
    if (lane == 0) ws_cnt[rh] = nadm;
  } else {
    for (int li = lane; li < k; li += 64) {
      a.slot_map[row + li] = L.map[i0 + li];
      if (L.keep[i0 + li]) a.slot_stamp[row + li] = a.step;
    }
  }
  *moved_out = moved;
  return nadm;
}

// Plans of np (request, KV head) pairs, pair0 + p * stride for p < np, made
// together (np * k <= kMaxK): item i of the pass is selection index and slot
// i % k of pair p = i / k. Returns the number of entries written to
// s_slot / s_page / s_epair (slot within the pair, host page, pair of the pass,
// in ascending block id per pair); s_prh[p] receives the pair index of p.
//
// With k >= 64 each pair is planned by one wave (plan_pair_wave), the waves
// taking the pass's pairs in turn, and the pairs' entries are then gathered in
// pair order. With smaller k the workgroup plans the pass together: misses,
// free slots and stale slots are compacted over the whole pass by workgroup
// scans (in item order, so each pair's items form one contiguous run in
// ascending block id or slot order); each thread then ranks one compacted item
// against the others of its pair (misses by score under a cap, stale slots by
// (stamp, slot)), and under a cap of at most kPlanRounds a wave per pair picks
// them in rounds instead. Planning the pairs of a workgroup in one pass pays
// the dependent global reads and the barriers once, not once per pair.
//
// With lsel (one pair, np = 1) the selection is taken from LDS (lsel[0, lsel_m)
// ascending) instead of a.sel / a.sel_count. NTHR threads call it (256 in the
// staging kernel, 1024 in the fused top-K and plan kernel).
template <int NTHR>
__device__ int plan_pass(const StageArgs& a, int pair0, int np, int stride, int* s_slot, int* s_page, int* s_epair,
                         int* s_prh, int* s_wave, const int* lsel = nullptr, int lsel_m = 0) {
  constexpr int kPer = kMaxK / NTHR;  // items per thread in the scans
  constexpr int kTot = NTHR / 64;     // where wg_exclusive_scan leaves its total
  const int tid = threadIdx.x;
  const int k = a.k;
  const int N = np * k;
  // by item: s_sel, s_hit (selection side), s_map, s_stamp, s_keep (slot side), s_selpage, s_selkey;
  // compacted misses: key, item, admitted; compacted stale slots: stamp, item; ranked stale items; free items
  __shared__ int s_sel[kMaxK], s_hit[kMaxK], s_map[kMaxK], s_stamp[kMaxK], s_keep[kMaxK];
  __shared__ int s_selpage[kMaxK];
  __shared__ unsigned s_selkey[kMaxK], s_mkey[kMaxK];
  __shared__ int s_midx[kMaxK], s_madm[kMaxK], s_skey[kMaxK], s_sslot[kMaxK], s_vstale[kMaxK], s_free[kMaxK];
  // per pair: selected count, run starts of misses / free / stale items (np + 1 entries), admitted start, moved
  __shared__ int s_pm[kMaxPairs], s_mstart[kMaxPairs + 1], s_fstart[kMaxPairs + 1], s_sstart[kMaxPairs + 1];
  __shared__ int s_astart[kMaxPairs], s_moved[kMaxPairs], s_nadm[kMaxPairs];

  if (k >= 64) {
    // a wave per pair (plan_pair_wave), then the pass's entries in pair order
    const PlanLds L{s_sel, s_hit, s_map, s_stamp, s_keep, s_selpage, s_selkey, s_mkey,
                    s_midx, s_madm, s_skey, s_sslot, s_vstale, s_free};
    for (int p = tid >> 6; p < np; p += NTHR / 64) {
      const int rh = pair0 + p * stride;
      int m = lsel ? lsel_m : a.sel_count[rh];
      m = m < 0 ? 0 : (m > k ? k : m);
      int moved = 0;
      const int nadm = plan_pair_wave(a, rh, p * k, m, lsel, L, &moved);
      if ((tid & 63) == 0) {
        s_nadm[p] = nadm;
        s_prh[p] = rh;
        if (a.moved) a.moved[rh] = moved;
      }
    }
    __syncthreads();
    if (tid == 0) {
      int o = 0;
      for (int p = 0; p < np; ++p) {
        s_astart[p] = o;
        o += s_nadm[p];
      }
      s_mstart[np] = o;
    }
    __syncthreads();
    const int n_adm = s_mstart[np];
    for (int p = 0; p < np; ++p) {
      const int na = s_nadm[p], at0 = s_astart[p];
      for (int e = tid; e < na; e += NTHR) {
        s_slot[at0 + e] = s_madm[p * k + e];
        s_page[at0 + e] = s_hit[p * k + e];
        s_epair[at0 + e] = p;
      }
    }
    __syncthreads();
    return n_adm;
  }

  // The page of every selected block (and, when a cap may bind, its score) is
  // fetched as soon as the block id arrives, so that these dependent loads
  // overlap the search below instead of stalling the pairing later.
  int pg[kPer];
  unsigned ky[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * NTHR;
    pg[j] = -1;
    ky[j] = 0u;
    if (i < N) {
      const int p = i / k;
      const int li = i - p * k;
      const int rh = pair0 + p * stride;
      const long long row = (long long)rh * k;
      const int sv = lsel ? lsel[li] : a.sel[row + li];  // in the row (k entries); loaded without waiting for the count
      int m = lsel ? lsel_m : a.sel_count[rh];
      m = m < 0 ? 0 : (m > k ? k : m);
      const int b = li < m ? sv : INT_MAX;
      s_sel[i] = b;
      s_hit[i] = 0;
      s_map[i] = a.slot_map[row + li];
      s_stamp[i] = a.slot_stamp[row + li];
      if (li == 0) {
        s_pm[p] = m;
        s_prh[p] = rh;
        s_moved[p] = 0;
        s_nadm[p] = 0;
      }
      if (li < m) {
        const int r = rh / a.Hkv;
        const bool in_row = b >= 0 && b < a.NBmax;
        if (in_row) pg[j] = a.block_table[(long long)r * a.NBmax + b];
        if (a.fetch_cap < m) ky[j] = order_key(in_row ? a.scores[(long long)rh * a.NBmax + b] : -__builtin_inff());
      }
    }
  }
  __syncthreads();

  // resident hits: binary search of every resident block in its pair's (ascending) selection
  for (int s = tid; s < N; s += NTHR) {
    const int p = s / k;
    const int off = p * k;
    const int m = s_pm[p];
    const int b = s_map[s];
    int keep = 0;
    if (b >= 0) {
      int lo = 0, hi = m;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (s_sel[off + mid] < b) lo = mid + 1; else hi = mid;
      }
      if (lo < m && s_sel[off + lo] == b) {
        s_hit[off + lo] = 1;
        keep = 1;
      }
    }
    s_keep[s] = keep;
  }
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * NTHR;
    if (i < N) {
      s_selpage[i] = pg[j];
      s_selkey[i] = ky[j];
    }
  }
  __syncthreads();

  // items [i0, i0 + kPer): misses (selection side), free and stale slots (slot side)
  const int i0 = tid * kPer;
  int nm = 0, nf = 0, ns = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = i0 + j;
    if (i < N) {
      const int p = i / k;
      if (i - p * k < s_pm[p] && !s_hit[i]) ++nm;
      if (s_map[i] < 0) ++nf;
      else if (!s_keep[i]) ++ns;
    }
  }
  const int mf_base = wg_exclusive_scan<NTHR>(nm | (nf << 16), s_wave);  // two 16-bit counts (<= 1024 each)
  const int mf_tot = s_wave[kTot];
  const int st_base = wg_exclusive_scan<NTHR>(ns, s_wave);
  const int n_stale = s_wave[kTot];
  const int n_miss = mf_tot & 0xFFFF;
  const int n_free = mf_tot >> 16;
  {
    int mr = mf_base & 0xFFFF, fr = mf_base >> 16, sr = st_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int i = i0 + j;
      if (i < N) {
        const int p = i / k;
        const int li = i - p * k;
        if (li == 0) {  // the pair's runs start here
          s_mstart[p] = mr;
          s_fstart[p] = fr;
          s_sstart[p] = sr;
        }
        if (li < s_pm[p] && !s_hit[i]) {
          s_mkey[mr] = s_selkey[i];
          s_midx[mr] = i;
          ++mr;
        }
        if (s_map[i] < 0) {
          s_free[fr++] = i;
        } else if (!s_keep[i]) {
          s_skey[sr] = s_stamp[i];
          s_sslot[sr] = i;
          ++sr;
        }
      }
    }
    if (tid == 0) {
      s_mstart[np] = n_miss;
      s_fstart[np] = n_free;
      s_sstart[np] = n_stale;
    }
  }
  __syncthreads();

  // admission: every miss of a pair, or under a binding cap its fetch_cap misses
  // with the highest score (ties: lowest block id). Keys are order-preserving
  // integers, so exactly fetch_cap misses are admitted even with NaN scores.
  // Victim order: free slots ascending (s_free), then stale slots by (stamp,
  // slot); only the first (admitted - free) stale slots are ever used. One wave
  // per pair: under a cap of at most kPlanRounds it picks the admitted misses,
  // and then the victims it needs, one round at a time (the best untaken item of
  // every lane, then wave minima: no barrier, no O(n^2) ranking); larger counts
  // rank every item of the pair against the others.
  {
    const int lane = tid & 63;
    for (int p = tid >> 6; p < np; p += NTHR / 64) {
      const int ms = s_mstart[p], me = s_mstart[p + 1];
      const int ss = s_sstart[p], se = s_sstart[p + 1];
      const int cap = a.fetch_cap;
      int nadm = me - ms;
      if (cap >= me - ms) {
        for (int c = ms + lane; c < me; c += 64) s_madm[c] = 1;
      } else if (cap <= kPlanRounds) {
        nadm = cap;
        uint32_t taken = 0;  // bit j: miss ms + lane + 64 j is admitted
        for (int rd = 0; rd < cap; ++rd) {
          uint32_t bk = 0xFFFFFFFFu;  // complemented key: the lowest is the highest score
          uint32_t bi = 0xFFFFFFFFu;
          for (int j = 0, c = ms + lane; c < me; ++j, c += 64) {
            const uint32_t kc = ~s_mkey[c];
            // ascending c: ties keep the lower one
            if (!((taken >> j) & 1u) && (kc < bk || bi == 0xFFFFFFFFu)) {
              bk = kc;
              bi = (uint32_t)c;
            }
          }
          // untaken misses remain (cap < misses), so some lane holds one
          const uint32_t wk = wave_min_u32(bi == 0xFFFFFFFFu ? 0xFFFFFFFFu : bk);
          const uint32_t wi = wave_min_u32(bi != 0xFFFFFFFFu && bk == wk ? bi : 0xFFFFFFFFu);
          if ((((int)wi - ms) & 63) == lane) taken |= 1u << (((int)wi - ms) >> 6);
        }
        for (int j = 0, c = ms + lane; c < me; ++j, c += 64) s_madm[c] = (taken >> j) & 1u;
      } else {
        nadm = cap;
        for (int c = ms + lane; c < me; c += 64) {
          const unsigned key = s_mkey[c];
          int rank = 0;
#pragma unroll 4
          for (int t = ms; t < me; ++t) {
            const unsigned kt = s_mkey[t];
            rank += (kt > key) || (kt == key && t < c);
          }
          s_madm[c] = rank < cap;
        }
      }
      int need = nadm - (s_fstart[p + 1] - s_fstart[p]);
      need = need < 0 ? 0 : (need > se - ss ? se - ss : need);
      if (need <= kPlanRounds) {
        uint32_t taken = 0;  // bit j: stale slot ss + lane + 64 j is a victim
        for (int rd = 0; rd < need; ++rd) {
          uint32_t bs = 0xFFFFFFFFu, bi = 0xFFFFFFFFu;
          for (int j = 0, t = ss + lane; t < se; ++j, t += 64) {
            const uint32_t st = (uint32_t)s_skey[t] ^ 0x80000000u;  // signed order
            if (!((taken >> j) & 1u) && (st < bs || bi == 0xFFFFFFFFu)) {
              bs = st;
              bi = (uint32_t)t;
            }
          }
          const uint32_t ws = wave_min_u32(bi == 0xFFFFFFFFu ? 0xFFFFFFFFu : bs);
          const uint32_t wi = wave_min_u32(bi != 0xFFFFFFFFu && bs == ws ? bi : 0xFFFFFFFFu);
          if ((((int)wi - ss) & 63) == lane) taken |= 1u << (((int)wi - ss) >> 6);
          if (lane == 0) s_vstale[ss + rd] = s_sslot[wi];
        }
      } else {
        for (int c = ss + lane; c < se; c += 64) {
          const int st = s_skey[c];
          int rank = 0;
#pragma unroll 4
          for (int t = ss; t < se; ++t) {
            const int kt = s_skey[t];
            rank += (kt < st) || (kt == st && t < c);
          }
          s_vstale[ss + rank] = s_sslot[c];
        }
      }
    }
  }
  __syncthreads();

  // the a-th admitted miss of a pair (ascending block id) goes to its a-th victim
  int na = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = i0 + j;
    if (c < n_miss && s_madm[c]) ++na;
  }
  const int adm_base = wg_exclusive_scan<NTHR>(na, s_wave);
  const int n_adm = s_wave[kTot];
  {
    int ar = adm_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int c = i0 + j;
      if (c < n_miss) {
        const int p = s_midx[c] / k;
        if (c == s_mstart[p]) s_astart[p] = ar;  // admitted misses of the pairs before p
        ar += s_madm[c];
      }
    }
  }
  __syncthreads();
  {
    int ar = adm_base;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int c = i0 + j;
      if (c >= n_miss || !s_madm[c]) continue;
      const int i = s_midx[c];
      const int p = i / k;
      const int rank = ar - s_astart[p];
      const int f0 = s_fstart[p], nfp = s_fstart[p + 1] - f0;
      const int s0 = s_sstart[p], nsp = s_sstart[p + 1] - s0;
      // a slot map holding one block twice can leave fewer victims than misses
      const int v = rank < nfp ? s_free[f0 + rank] : (rank < nfp + nsp ? s_vstale[s0 + rank - nfp] : -1);
      const int blk = s_sel[i];
      int page = v >= 0 ? s_selpage[i] : -1;
      if (page < 0 || page >= a.num_pages) page = -1;
      s_slot[ar] = v >= 0 ? v - p * k : -1;
      s_page[ar] = page;
      s_epair[ar] = p;
      if (v >= 0) {
        s_map[v] = page >= 0 ? blk : -1;
        s_keep[v] = page >= 0;
      }
      if (page >= 0) atomicAdd(&s_moved[p], 1);
      atomicAdd(&s_nadm[p], 1);
      ++ar;
    }
  }
  __syncthreads();

  if (a.mode == kStagePlanOnly) {
    // the new rows, the admitted entries and their counts go to the workspace
    const long long nrhk = (long long)a.R * a.Hkv * k;
    int32_t* ws_map = a.ws;
    int32_t* ws_stamp = a.ws + nrhk;
    int2* ws_ent = reinterpret_cast<int2*>(a.ws + 2 * nrhk);
    int32_t* ws_cnt = a.ws + 4 * nrhk;
    for (int s = tid; s < N; s += NTHR) {
      const int p = s / k;
      const long long at = (long long)s_prh[p] * k + (s - p * k);
      ws_map[at] = s_map[s];
      ws_stamp[at] = s_keep[s] ? a.step : s_stamp[s];
    }
    for (int e = tid; e < n_adm; e += NTHR) {
      const int p = s_epair[e];
      ws_ent[(long long)s_prh[p] * k + (e - s_astart[p])] = make_int2(s_slot[e], s_page[e]);
    }
    for (int p = tid; p < np; p += NTHR) ws_cnt[s_prh[p]] = s_nadm[p];
  } else {
    for (int s = tid; s < N; s += NTHR) {
      const int p = s / k;
      const long long at = (long long)s_prh[p] * k + (s - p * k);
      a.slot_map[at] = s_map[s];
      if (s_keep[s]) a.slot_stamp[at] = a.step;
    }
  }
  if (a.moved)
    for (int p = tid; p < np; p += NTHR) a.moved[s_prh[p]] = s_moved[p];
  return n_adm;
}

// Entries of a pass planned earlier (kStagePlanOnly): per pair its admitted
// (slot, page) entries from the workspace, compacted over the pass's pairs in
// LDS; the counts and all k entries of every pair are loaded together.
__device__ int load_planned(const StageArgs& a, int pair0, int np, int stride, int* s_slot, int* s_page,
                            int* s_epair, int* s_prh) {
  const int tid = threadIdx.x;
  const int k = a.k;
  const int N = np * k;
  const long long nrhk = (long long)a.R * a.Hkv * k;
  const int2* ws_ent = reinterpret_cast<const int2*>(a.ws + 2 * nrhk);
  const int32_t* ws_cnt = a.ws + 4 * nrhk;
  __shared__ int s_cnt[kMaxPairs], s_off[kMaxPairs + 1];
  int2 ent[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kPlanThreads;
    ent[j] = make_int2(-1, -1);
    if (i < N) {
      const int p = i / k;
      ent[j] = ws_ent[(long long)(pair0 + p * stride) * k + (i - p * k)];
    }
  }
  for (int p = tid; p < np; p += kPlanThreads) {
    const int rh = pair0 + p * stride;
    const int c = ws_cnt[rh];
    s_cnt[p] = c < 0 ? 0 : (c > k ? k : c);
    s_prh[p] = rh;
  }
  __syncthreads();
  if (tid == 0) {
    int o = 0;
    for (int p = 0; p < np; ++p) {
      s_off[p] = o;
      o += s_cnt[p];
    }
    s_off[np] = o;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = tid + j * kPlanThreads;
    if (i < N) {
      const int p = i / k;
      const int li = i - p * k;
      if (li < s_cnt[p]) {
        const int e = s_off[p] + li;
        int page = ent[j].y;
        if (page < 0 || page >= a.num_pages) page = -1;
        s_slot[e] = ent[j].x;
        s_page[e] = page;
        s_epair[e] = p;
      }
    }
  }
  return s_off[np];
}

// Commit the workspace rows of a pass's pairs to slot_map / slot_stamp.
__device__ void commit_planned(const StageArgs& a, int np, const int* s_prh) {
  const int k = a.k;
  const long long nrhk = (long long)a.R * a.Hkv * k;
  const int32_t* ws_map = a.ws;
  const int32_t* ws_stamp = a.ws + nrhk;
  for (int s = threadIdx.x; s < np * k; s += kPlanThreads) {
    const int p = s / k;
    const long long at = (long long)s_prh[p] * k + (s - p * k);
    a.slot_map[at] = ws_map[at];
    a.slot_stamp[at] = ws_stamp[at];
  }
}

// One batch of PF block-head entries held in registers (K and V, 16-byte
// chunks of each entry spread over the workgroup).
template <int BS, int PF>
struct CopyBatch {
  static constexpr int kChunks = BS * kHeadDim / 8 / kPlanThreads;
  u32x4 k[PF][kChunks], v[PF][kChunks];
  int rh[PF], slot[PF], page[PF];
};

template <int BS, int PF>
__device__ __forceinline__ void fetch_batch(const StageArgs& a, CopyBatch<BS, PF>& b, int e0, int n,
                                            const int* s_slot, const int* s_page, const int* s_epair,
                                            const int* s_prh) {
  constexpr int kElems = BS * kHeadDim;
  const int tid = threadIdx.x;
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    const int e = e0 + p;
    b.slot[p] = e < n ? s_slot[e] : -1;
    b.page[p] = e < n ? s_page[e] : -1;
    b.rh[p] = e < n ? s_prh[s_epair[e]] : 0;
    const bool live = b.page[p] >= 0 && b.slot[p] >= 0 && b.slot[p] <= a.k;
    if (!live) b.page[p] = -1;
    const int h = b.rh[p] % a.Hkv;
    const long long src = ((long long)(live ? b.page[p] : 0) * a.Hkv + h) * kElems;
    // placeholder source (no entry): the start of the pool (device memory, discarded)
    const uint16_t* ks = live ? a.host_k + src : a.pool_k;
    const uint16_t* vs = live ? a.host_v + src : a.pool_k;
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
__device__ __forceinline__ void put_batch(const StageArgs& a, const CopyBatch<BS, PF>& b,
                                          uint16_t (*tile)[BS * kHeadDim]) {
  constexpr int kElems = BS * kHeadDim;
  const int tid = threadIdx.x;
  long long dst[PF];
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    const int r = b.rh[p] / a.Hkv;
    const int h = b.rh[p] - r * a.Hkv;
    dst[p] = (((long long)r * (a.k + 1) + b.slot[p]) * a.Hkv + h) * kElems;
  }
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    if (b.page[p] < 0) continue;
#pragma unroll
    for (int q = 0; q < CopyBatch<BS, PF>::kChunks; ++q) {
      const int c = (q * kPlanThreads + tid) * 8;
      *reinterpret_cast<u32x4*>(a.pool_k + dst[p] + c) = b.k[p][q];
      *reinterpret_cast<u32x4*>(&tile[p][c]) = b.v[p][q];
    }
  }
  __syncthreads();
  // V: [BS][d] -> [d][BS]; thread -> (d, 8-token group)
  constexpr int kGroups = BS / 8;
#pragma unroll
  for (int p = 0; p < PF; ++p) {
    if (b.page[p] < 0) continue;
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
      *reinterpret_cast<u32x4*>(a.pool_v + dst[p] + (long long)d * BS + t0) = o;
    }
  }
  __syncthreads();
}

template <int BS, int PF, int TP>
__device__ __forceinline__ void copy_entries(const StageArgs& a, int n, const int* s_slot, const int* s_page,
                                             const int* s_epair, const int* s_prh, uint16_t (*tile)[TP]) {
  CopyBatch<BS, PF> x, y;
  fetch_batch<BS, PF>(a, x, 0, n, s_slot, s_page, s_epair, s_prh);
  for (int e0 = 0; e0 < n; e0 += 2 * PF) {
    fetch_batch<BS, PF>(a, y, e0 + PF, n, s_slot, s_page, s_epair, s_prh);
    put_batch<BS, PF>(a, x, tile);
    if (e0 + PF >= n) break;
    fetch_batch<BS, PF>(a, x, e0 + 2 * PF, n, s_slot, s_page, s_epair, s_prh);
    put_batch<BS, PF>(a, y, tile);
  }
}

// The in-kernel form of stream waits on counters (StageArgs::wait_flag): it
// saves the transfer stream a dispatch per counter and step. Thread 0 polls with relaxed
// agent-scope loads; the barrier holds the other waves; the acquire fence then
// orders every later read after the producer's writes, which its kernel's end
// released before the counter was raised. The poll is bounded (wait_polls, a
// few seconds by default): a counter that is never raised costs that time and
// a fault mark, not a hang.
__device__ __forceinline__ void stage_wait(const StageArgs& a) {
  if (!a.wait_flag[0] && !a.wait_flag[1]) return;
  if (threadIdx.x == 0) {
    uint32_t n = 0;
    for (int i = 0; i < 2; ++i) {
      if (!a.wait_flag[i]) continue;
      while (__hip_atomic_load(a.wait_flag[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < a.wait_value[i]) {
        if (++n >= a.wait_polls) {
          __hip_atomic_store(a.wait_fault, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

template <int BS, int PF>
__global__ __launch_bounds__(kPlanThreads) void stage_kernel(StageArgs a) {
  stage_wait(a);
  const int tid = threadIdx.x;
  __shared__ int s_slot[kMaxK + kMaxPairs], s_page[kMaxK + kMaxPairs], s_epair[kMaxK + kMaxPairs];
  __shared__ int s_prh[kMaxPairs];
  __shared__ int s_wave[8];
  constexpr int kElems = BS * kHeadDim;  // one K (or V) block-head entry
  __shared__ uint16_t tile[PF][kElems];

  // this workgroup's pairs: blockIdx.x, blockIdx.x + gridDim.x, ...; up to
  // kMaxK / k of them (kMaxPairs at most) are planned and copied per pass
  const int nrh = a.R * a.Hkv;
  const int stride = gridDim.x;
  const int mine = (int)blockIdx.x < nrh ? (nrh - 1 - (int)blockIdx.x) / stride + 1 : 0;
  int per_pass = a.local_only ? kMaxPairs : kMaxK / a.k;
  per_pass = per_pass < 1 ? 1 : (per_pass > kMaxPairs ? kMaxPairs : per_pass);
  for (int j0 = 0; j0 < mine; j0 += per_pass) {
    const int np = mine - j0 < per_pass ? mine - j0 : per_pass;
    const int pair0 = (int)blockIdx.x + j0 * stride;
    int n = 0;
    if (a.local_only) {
      for (int p = tid; p < np; p += kPlanThreads) s_prh[p] = pair0 + p * stride;
    } else if (a.mode == kStageCopyOnly) {
      n = load_planned(a, pair0, np, stride, s_slot, s_page, s_epair, s_prh);
    } else {
      n = plan_pass<kPlanThreads>(a, pair0, np, stride, s_slot, s_page, s_epair, s_prh, s_wave);
    }
    if (a.copy_local) {  // the local block of every pair of the pass, into slot k
      for (int p = tid; p < np; p += kPlanThreads) {
        const int rh = pair0 + p * stride;
        const int r = rh / a.Hkv;
        const Ctx c = ctx_blocks(a.ctx_len[r], BS, a.NBmax);
        int page = c.nb > 0 ? a.block_table[(long long)r * a.NBmax + c.nb - 1] : -1;
        if (page < 0 || page >= a.num_pages) page = -1;
        s_slot[n + p] = a.k;
        s_page[n + p] = page;
        s_epair[n + p] = p;
      }
      n += np;
    }
    __syncthreads();

    // Batches of PF entries, two in flight: the host reads of the next batch
    // are issued before the current one is stored, so the link does not idle
    // while a batch is written and V is transposed. Every load is issued; an
    // entry past the end (or without a page) reads the start of the pool
    // instead (device memory, discarded), so the wait counts stay exact.
    copy_entries<BS, PF>(a, n, s_slot, s_page, s_epair, s_prh, tile);
    if (a.mode == kStageCopyOnly && !a.local_only) commit_planned(a, np, s_prh);
    __syncthreads();  // LDS plan arrays are reused by the next pass
  }
}

// Top-K and plan in one kernel (the layer pipeline's prediction stream): a
// 1024-thread workgroup per (request, KV head) selects as the top-K kernel
// does, keeps the selection in LDS and plans the pair's transfer from it into
// the workspace (kStagePlanOnly), so the plan costs neither a launch nor a
// re-read of the selection, and the transfer stream only copies.
constexpr int kSelThreads = 1024;

template <int KPT>
__global__ __launch_bounds__(kSelThreads) void topk_plan_kernel(TopkArgs t, StageArgs a) {
  __shared__ SelectShared<kSelThreads, KPT> sh;
  __shared__ int s_lsel[kMaxK];
  __shared__ int s_slot[kMaxK + kMaxPairs], s_page[kMaxK + kMaxPairs], s_epair[kMaxK + kMaxPairs];
  __shared__ int s_prh[kMaxPairs];
  __shared__ int s_wave[kSelThreads / 64 + 1];
  const int rh = blockIdx.x;
  const int r = rh / t.Hkv;
  const Ctx c = ctx_blocks(t.ctx_len[r], t.B, t.NBmax);
  select_row<kSelThreads, KPT>(t.scores + (long long)rh * t.NBmax, c.n_cand, t.k, t.sel + (long long)rh * t.k,
                               t.sel_count + rh, sh, s_lsel);
  __syncthreads();
  const int m = c.n_cand < t.k ? (c.n_cand > 0 ? c.n_cand : 0) : t.k;
  plan_pass<kSelThreads>(a, rh, 1, 1, s_slot, s_page, s_epair, s_prh, s_wave, s_lsel, m);
}

// Scoring, top-K and, with PLAN, the transfer plan of one (request, KV head) in
// one workgroup of kScoreSelThreads threads (paper §4.2.1: the draft rows rank
// every block of the head; §4.2.2: top-K prediction; §4.2.3: delta selection).
// The workgroup scores its row's candidate tiles with the scorer's MFMA pieces
// (score_core.h, so the scores are bit-identical to the scoring kernel's),
// writes the row of scores, and selects from it after a workgroup barrier, so
// no other workgroup is waited for. The query operands sit in the selection's
// key staging area until the selection starts. Each wave scores kScoreSelTiles
// tiles at a time, all their loads issued before the first MFMA. Small
// workgroups let several rows share a CU, so that one row's selection overlaps
// another's loads. Worth trying where the rows are many and short, so that one
// workgroup per row fills the chip; with few long rows the two kernels spread
// a row over many workgroups.
constexpr int kScoreSelThreads = 256;
constexpr int kScoreSelTiles = 4;

template <int NRT, int KPT, bool PLAN>
__global__ __launch_bounds__(kScoreSelThreads) void score_select_kernel(ScoreArgs sa, TopkArgs t, StageArgs a) {
  constexpr int NTHR = kScoreSelThreads;
  constexpr int TPW = kScoreSelTiles;
  __shared__ __align__(16) SelectShared<NTHR, KPT> sh;
  __shared__ int s_lsel[PLAN ? kMaxK : 1];
  __shared__ int s_slot[PLAN ? kMaxK + kMaxPairs : 1], s_page[PLAN ? kMaxK + kMaxPairs : 1];
  __shared__ int s_epair[PLAN ? kMaxK + kMaxPairs : 1];
  __shared__ int s_prh[PLAN ? kMaxPairs : 1];
  __shared__ int s_wave[NTHR / 64 + 1];
  static_assert(sizeof(ScoreQOperands<NRT>) <= sizeof(sh.keys), "query operands must fit the key staging area");
  const int rh = blockIdx.x;
  const int r = rh / sa.Hkv;
  const int h = rh - r * sa.Hkv;
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int n = lane & 15;
  const Ctx c = ctx_blocks(sa.ctx_len[r], sa.B, sa.NBmax);
  ScoreQOperands<NRT>& s_q = *reinterpret_cast<ScoreQOperands<NRT>*>(sh.keys);
  for (int e = threadIdx.x; e < NRT * 256; e += NTHR) score_q_store<NRT>(s_q, e, score_q_raw(sa, r, h, e));

  const long long sum_base = (long long)rh * sa.NBmax * kHeadDim;
  const uint16_t* kmx = sa.kmax + sum_base;
  const uint16_t* kmn = sa.kmin + sum_base;
  float* srow = sa.scores + (long long)rh * sa.NBmax;
  const int ntile_c = (c.n_cand + 15) >> 4;
  __syncthreads();  // query operands are in
  for (int tile0 = wave * TPW; tile0 < ntile_c; tile0 += (NTHR / 64) * TPW) {
    u32x4 vmax[TPW][4], vmin[TPW][4];
#pragma unroll
    for (int u = 0; u < TPW; ++u) score_tile_load(kmx, kmn, tile0 + u, c.n_cand, g, n, vmax[u], vmin[u]);
    float best[TPW];
#pragma unroll
    for (int u = 0; u < TPW; ++u) best[u] = -INFINITY;
#pragma unroll
    for (int v = 0; v < NRT; ++v) {
      bf16x8 ap[4], an[4];
      score_q_tile<NRT>(s_q, v, lane, ap, an);
#pragma unroll
      for (int u = 0; u < TPW; ++u) best[u] = score_tile_fold(ap, an, vmax[u], vmin[u], best[u]);
    }
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      const float b = score_lane_reduce(best[u]);
      const int blk = (tile0 + u) * 16 + n;
      if (g == 0 && blk < c.n_cand) srow[blk] = b;
    }
  }
  for (int b = c.n_cand + threadIdx.x; b < sa.NBmax; b += NTHR) srow[b] = -INFINITY;
  __syncthreads();  // the score row is complete, and the query operands are no longer read
  select_row<NTHR, KPT>(srow, c.n_cand, t.k, t.sel + (long long)rh * t.k, t.sel_count + rh, sh,
                        PLAN ? s_lsel : nullptr);
  if (PLAN) {
    __syncthreads();
    const int m = c.n_cand < t.k ? (c.n_cand > 0 ? c.n_cand : 0) : t.k;
    plan_pass<NTHR>(a, rh, 1, 1, s_slot, s_page, s_epair, s_prh, s_wave, s_lsel, m);
  }
}

template <int NRT, int KPT>
hipError_t launch_score_select_t(const ScoreArgs& sa, const TopkArgs& t, const StageArgs* plan, hipStream_t s,
                                 const LaunchTiming& lt) {
  const dim3 grid((unsigned)(sa.R * sa.Hkv));
  if (plan)
    launch_kernel(score_select_kernel<NRT, KPT, true>, grid, dim3(kScoreSelThreads), s, lt, sa, t, *plan);
  else
    launch_kernel(score_select_kernel<NRT, KPT, false>, grid, dim3(kScoreSelThreads), s, lt, sa, t, StageArgs{});
  return hipGetLastError();
}

template <int NRT>
hipError_t launch_score_select_nrt(const ScoreArgs& sa, const TopkArgs& t, const StageArgs* plan, hipStream_t s,
                                   const LaunchTiming& lt) {
  // keys per thread; the staged keys also hold the query operands (8 KiB per row tile)
  const int per = (sa.NBmax + kScoreSelThreads - 1) / kScoreSelThreads;
  if constexpr (NRT == 1) {
    if (per <= 8) return launch_score_select_t<NRT, 8>(sa, t, plan, s, lt);
  }
  if (per <= 16) return launch_score_select_t<NRT, 16>(sa, t, plan, s, lt);
  if (per <= 32) return launch_score_select_t<NRT, 32>(sa, t, plan, s, lt);
  return launch_score_select_t<NRT, 64>(sa, t, plan, s, lt);
}

}  // namespace

bool score_select_supported(const ScoreArgs& sa) {
  const int rows = sa.num_draft * sa.G;
  return rows > kScoreValuMaxRows && rows <= kScoreSelectMaxRows && sa.NBmax <= kScoreSelectMaxBlocks;
}

hipError_t launch_score_select(const ScoreArgs& sa, const TopkArgs& t, const StageArgs* plan, hipStream_t s,
                               const LaunchTiming& lt) {
  if (!score_select_supported(sa)) return hipErrorInvalidValue;
  if (plan && (plan->mode != kStagePlanOnly || !plan->ws || plan->local_only)) return hipErrorInvalidValue;
  return (sa.num_draft * sa.G + 15) / 16 == 1 ? launch_score_select_nrt<1>(sa, t, plan, s, lt)
                                               : launch_score_select_nrt<2>(sa, t, plan, s, lt);
}

template <int BS>
hipError_t launch_bs(const StageArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int nrh = a.R * a.Hkv;
  if (nrh <= 0) return hipSuccess;
  // B = 16: kCopyWorkgroups; B = 32 (16 KiB entries, twice the stores and
  // transposes per entry): one workgroup per two pairs, up to twice as many
  int grid = BS == 16 ? kCopyWorkgroups : nrh / 2;
  grid = grid < kCopyWorkgroups ? kCopyWorkgroups : (grid > 2 * kCopyWorkgroups ? 2 * kCopyWorkgroups : grid);
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

hipError_t launch_topk_plan(const TopkArgs& t, const StageArgs& a, hipStream_t s, const LaunchTiming& lt) {
  if (a.mode != kStagePlanOnly || !a.ws || a.local_only) return hipErrorInvalidValue;
  // the candidate count of every request is at most NBmax - 1; beyond 16 keys
  // per thread they are re-read from memory (the staged row would not fit LDS
  // next to the plan)
  const int per = (t.NBmax + kSelThreads - 1) / kSelThreads;
  const dim3 grid((unsigned)(t.R * t.Hkv));
  if (per <= 8)
    launch_kernel(topk_plan_kernel<8>, grid, dim3(kSelThreads), s, lt, t, a);
  else if (per <= 16)
    launch_kernel(topk_plan_kernel<16>, grid, dim3(kSelThreads), s, lt, t, a);
  else
    launch_kernel(topk_plan_kernel<0>, grid, dim3(kSelThreads), s, lt, t, a);
  return hipGetLastError();
}

hipError_t launch_stage(const StageArgs& a, hipStream_t s, const LaunchTiming& t) {
  return a.B == 16 ? launch_bs<16>(a, s, t) : launch_bs<32>(a, s, t);
}

}  // namespace oasis
