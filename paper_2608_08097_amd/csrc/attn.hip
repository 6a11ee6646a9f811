// Block-sparse GQA decode attention over the HBM working set (paper §4.2.1:
// the normal and draft queries are stacked and attend one resident KV set in
// one call; §5.2: the K selected blocks plus the active local block).
//
// Work decomposition. The rows of one KV head are its G query heads times the
// T stacked query tokens (20 at G = 4, T = 5). The attended tokens of a
// (request, KV head) are cut into units of 32 tokens (two slots at B = 16,
// one at B = 32); a workgroup of 4 waves handles a contiguous range of units
// (a split) and every wave a strided subset of them, with its own online
// softmax. The waves are merged through LDS; with one split the workgroup
// writes the bf16 outputs and the log-sum-exp itself, otherwise each split
// writes one partial (unnormalised output, running max, running sum) per row
// and a second kernel merges the splits. (A merge by the last-arriving
// workgroup of a head inside the same kernel needs an agent-scope release
// per workgroup, which on MI355X writes back the XCD's L2; measured on a
// 256-workgroup stand-in, that cost 14.8 us per call against 2.6 us for the
// second launch.)
//
// One 32-token unit for one 16-row tile:
//   S^T (tokens x rows) = K (tokens x d) . Q^T (d x rows): 2 token tiles x
//       4 k-steps of v_mfma_f32_16x16x32_bf16. Token tile tau assigns MFMA row
//       i to unit token 8*(i/4) + 4*tau + i%4, so after both tiles lane (g, n)
//       holds query row n against unit tokens 8g .. 8g+7.
//   P (bf16) is then directly the B operand of
//   O^T (d x rows) += V^T (d x tokens) . P^T (tokens x rows): 8 d-tiles, one
//       MFMA each; lane (g, i) of the A operand needs V[8g .. 8g+7][d = i],
//       which is one 16-byte load because the pool keeps V transposed per
//       slot and head (d x B).
// So K and V go straight from HBM into MFMA registers with 16-byte loads and
// no LDS round trip; every lane owns one query row, so the running max and sum
// need only two cross-lane exchanges per unit.
//
// With more than two row tiles (G * T > 32 rows) the registers of one wave no
// longer hold every tile's accumulators next to two units of K and V; there a
// workgroup has one wave per row tile and the unit's K and V cross HBM once,
// into LDS, for all of them (attn_split_rows_kernel).
#include <mutex>
#include <utility>

#include "oasis_internal.h"

namespace oasis {
namespace {

constexpr int kW = 4;  // waves per workgroup
// Workgroups of one attention call: one per CU (the register-prefetching
// kernel of up to two row tiles holds one wave per SIMD; the many-row kernel
// one workgroup of up to five waves per CU).
constexpr int kTargetWorkgroups = 256;
constexpr int kMaxSplits = 16;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// XCD-aware placement: workgroup ids are dealt round-robin over the 8 XCDs, so
// the splits of one (request, KV head) are given ids that share id % 8 and
// therefore one L2 (the query rows they all read stay local).
__device__ __forceinline__ bool map_workgroup(int wg, int nrh, int nsplit, int& rh, int& split) {
  const int xcd = wg & 7;
  const int local = wg >> 3;
  const int rh_local = local / nsplit;
  split = local - rh_local * nsplit;
  rh = rh_local * 8 + xcd;
  return rh < nrh;
}

// K and V registers of one 32-token unit (the operands of its MFMAs).
struct UnitRegs {
  u32x4 k[2][4];
  u32x4 v[8];
};

// Unit u (wave-uniform) covers slots s0 = 2u, s1 = 2u + 1 at B = 16 or slot u
// at B = 32. Every load is unconditional: a slot index past the pool is
// clamped onto the local slot (always inside the pool) and only the token
// counts n0 / n1 decide which tokens count. Free slots may hold anything,
// even NaN; their K only yields masked scores and their V is cleared below.
//
// u < 0 is a placeholder unit: the loads are issued anyway (on the local slot,
// which is cache-resident after its first read) and count nothing. Issuing
// the same number of loads on every path keeps the compiler's wait counts
// exact, so waiting for the current unit never drains the prefetched one.
template <int BS>
__device__ __forceinline__ void load_unit(UnitRegs& ur, int u, int ks, const uint16_t* pk, const uint16_t* pv,
                                          long long slot_elems, int g, int i) {
  const bool real = u >= 0;
  const int s0 = real ? (BS == 16 ? 2 * u : u) : ks;
  const int s1raw = real ? (BS == 16 ? 2 * u + 1 : ks + 1) : ks + 1;
  const int s1 = s1raw <= ks ? s1raw : ks;
  const uint16_t* k0 = pk + (long long)s0 * slot_elems;
  const uint16_t* k1 = pk + (long long)s1 * slot_elems;
  const uint16_t* v0 = pv + (long long)s0 * slot_elems;
  const uint16_t* v1 = pv + (long long)s1 * slot_elems;
  // K: lane (g, i), token tile tau -> unit token 8*(i/4) + 4*tau + i%4
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    const int tok = 8 * (i >> 2) + 4 * tau + (i & 3);
    const uint16_t* src = BS == 16 ? ((tok < 16 ? k0 : k1) + (tok & 15) * kHeadDim + g * 8)
                                   : (k0 + tok * kHeadDim + g * 8);
#pragma unroll
    for (int st = 0; st < 4; ++st) ur.k[tau][st] = ldg16(src + st * 32);
  }
  // V^T: lane (g, i), d-tile dt -> V[tokens 8g .. 8g+7][d = dt*16 + i]
  const uint16_t* vsrc = BS == 16 ? ((g < 2 ? v0 : v1) + (g & 1) * 8) : (v0 + 8 * g);
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) ur.v[dt] = ldg16(vsrc + (long long)(dt * 16 + i) * BS);
}

// Attended tokens of the two slots of unit u (u < 0: none): a slot below k_slots
// counts B tokens when bit `bit` (first slot) / `bit + 1` (second slot, B = 16)
// of the validity mask is set; slot k_slots is the local block.
template <int BS>
__device__ __forceinline__ void unit_counts(int u, int ks, int local_len, uint64_t vmask, int bit, int& n0,
                                            int& n1) {
  const int s0 = BS == 16 ? 2 * u : u;
  const int s1 = s0 + 1;
  n0 = u < 0 ? 0 : (s0 < ks ? (((vmask >> bit) & 1) ? BS : 0) : (s0 == ks ? local_len : 0));
  n1 = (BS == 16 && u >= 0) ? (s1 < ks ? (((vmask >> (bit + 1)) & 1) ? BS : 0) : (s1 == ks ? local_len : 0)) : 0;
}

// Tokens of the unit that lane (g, i) scores: 8g .. 8g+7 of the unit (slot 0 holds
// unit tokens 0 .. B-1). The first `keep` of them are attended (0 .. 8).
template <int BS>
__device__ __forceinline__ int lane_keep(int n0, int n1, int g) {
  const int cnt = BS == 16 ? (g < 2 ? n0 : n1) : n0;
  const int k = cnt - (BS == 16 ? (g & 1) * 8 : 8 * g);
  return k < 0 ? 0 : (k > 8 ? 8 : k);
}

// Zero the V values of tokens that are not attended (their probability is 0,
// but 0 * NaN would poison the accumulator). Lane (g, i) holds V^T of the same
// 8 tokens it scores; only lanes with keep < 8 change anything.
__device__ __forceinline__ void mask_unit_v(UnitRegs& ur, int keep) {
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t lo = (2 * w) < keep ? 0x0000FFFFu : 0u;
      const uint32_t hi = (2 * w + 1) < keep ? 0xFFFF0000u : 0u;
      ur.v[dt][w] &= (lo | hi);
    }
}

// Online-softmax update of one wave with one 32-token unit (all row tiles).
//
// Lazy rescaling: every row keeps a reference maximum m_ref (the same in the
// four lanes of the row) and each lane a partial sum over its own tokens.
// Probabilities are exp2(x - m_ref); only when some score of the wave exceeds
// its row reference by more than kLazyTh (a wave-uniform branch, rare once the
// first unit has been seen) are the row maxima exchanged across lanes and the
// accumulators rescaled. Probabilities stay below 2^kLazyTh, far inside the
// fp32 range, and the result is the same softmax.
//
// `partial` (wave-uniform) is set when some lane has keep < 8: only then are
// unattended scores set to -inf; a fully attended unit skips that work.
constexpr float kLazyTh = 8.f;

template <int NT, int BS>
__device__ __forceinline__ void process_unit(const UnitRegs& cur, int keep, bool partial, const bf16x8 (&qb)[NT][4],
                                             float (&m_ref)[NT], float (&l_part)[NT], f32x4 (&acc)[NT][8],
                                             float scale_log2) {
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    f32x4 sc[2];
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 4; ++st)
        s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[tau][st]), qb[v][st], s4, 0, 0, 0);
      sc[tau] = s4;
    }
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = sc[e >> 2][e & 3] * scale_log2;
    if (partial) {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[e] = e < keep ? x[e] : -INFINITY;
    }
    const float lmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
    if (__builtin_amdgcn_ballot_w64(lmax > m_ref[v] + kLazyTh)) {
      float rmax = fmaxf(lmax, __shfl_xor(lmax, 16));
      rmax = fmaxf(rmax, __shfl_xor(rmax, 32));
      const float m_new = fmaxf(m_ref[v], rmax);
      const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_ref[v] - m_new);
      l_part[v] *= alpha;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) acc[v][dt] *= alpha;
      m_ref[v] = m_new;
    }
    const float m_use = m_ref[v] == -INFINITY ? 0.f : m_ref[v];
    bf16x8 pb;
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pe = fast_exp2(x[e] - m_use);
      psum += pe;
      pb[e] = (__bf16)pe;
    }
    l_part[v] += psum;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      acc[v][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.v[dt]), pb, acc[v][dt], 0, 0, 0);
  }
}

// Normalised bf16 output of 4 dimensions of one row, and its log-sum-exp.
__device__ __forceinline__ void write_output(const AttnArgs& a, int r, int h, int row, int c4, f32x4 o, float M,
                                             float L) {
  const int t = row / a.G;
  const int qh = h * a.G + (row - t * a.G);
  const long long orow = ((long long)r * a.T + t) * a.Hq + qh;
  const float inv = L > 0.f ? 1.f / L : 0.f;
  const uint32_t w0 = f32_to_bf16_bits(o[0] * inv) | (f32_to_bf16_bits(o[1] * inv) << 16);
  const uint32_t w1 = f32_to_bf16_bits(o[2] * inv) | (f32_to_bf16_bits(o[3] * inv) << 16);
  *reinterpret_cast<uint2*>(a.out + orow * kHeadDim + c4 * 4) = make_uint2(w0, w1);
  if (c4 == 0 && a.lse) a.lse[orow] = L > 0.f ? (M + __log2f(L)) * 0.69314718055994531f : -INFINITY;
}

// Slot-map validity of the wave's units t0 .. t0 + kChunk - 1 (unit t of the wave is
// u_first + t * kW): lane l reads the map entry of slot l % 2 of unit t0 + l / 2
// (B = 16) or of unit t0 + l (B = 32); ballot(slot < k_slots && entry >= 0) is then
// the mask unit_counts reads (bit 2j + e or j), so the unit loop loads no slot map.
// The load is split from the test: it is issued unconditionally (index clamped
// into the map; with k_slots = 0, where the map may be NULL, from `fallback`,
// any valid int, whose value the slot test then ignores), so that nothing waits
// for it until the mask is needed.
template <int BS>
__device__ __forceinline__ int unit_slot(int u_first, int t0, int lane) {
  const int j = BS == 16 ? lane >> 1 : lane;
  return BS == 16 ? 2 * (u_first + (t0 + j) * kW) + (lane & 1) : u_first + (t0 + j) * kW;
}
__device__ __forceinline__ const int32_t* map_addr(const int32_t* smap, int ks, int slot, const int32_t* fallback) {
  return ks > 0 ? smap + (slot < ks ? slot : ks - 1) : fallback;
}
__device__ __forceinline__ int map_load(const int32_t* smap, int ks, int slot, const int32_t* fallback) {
  return *map_addr(smap, ks, slot, fallback);
}
__device__ __forceinline__ uint64_t map_mask(int ks, int slot, int entry) {
  return __builtin_amdgcn_ballot_w64(slot < ks && entry >= 0);
}

// Split kernel for one or two row tiles (up to 32 rows): K and V straight
// into registers, every wave a strided subset of the split's units.
template <int NT, int BS>
__global__ __launch_bounds__(kW * 64) void attn_split_kernel(AttnArgs a) {
  static_assert(NT <= 2, "three or more row tiles take attn_split_rows_kernel");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int i = lane & 15;
  const int nrh = a.R * a.Hkv;
  int rh, split;
  if (!map_workgroup(blockIdx.x, nrh, a.nsplit, rh, split)) return;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const int ks = a.k_slots;
  const long long slot_elems = (long long)a.Hkv * BS * kHeadDim;
  const long long head_off = (long long)h * BS * kHeadDim;
  const uint16_t* pk = a.pool_k + (long long)r * (ks + 1) * slot_elems + head_off;
  const uint16_t* pv = a.pool_v + (long long)r * (ks + 1) * slot_elems + head_off;
  const int32_t* smap = a.slot_map + (long long)rh * ks;
  const int u_begin = split * a.units_per_split;
  const int u_end = min(a.n_units, u_begin + a.units_per_split);
  // unit t of this wave is u_first + t * kW, t < nt
  const int u_first = u_begin + wave;
  const int nt = u_first < u_end ? (u_end - u_first + kW - 1) / kW : 0;
  auto unit = [&](int t) { return t < nt ? u_first + t * kW : -1; };
  constexpr int kChunk = BS == 16 ? 32 : 64;  // units per validity mask
  auto bit_of = [&](int t) { return BS == 16 ? 2 * (t & (kChunk - 1)) : (t & (kChunk - 1)); };

  // The first unit's loads go out before anything else, so that no wave starts
  // by waiting for a scalar or query load; the queries, the slot map and the
  // context length follow.
  UnitRegs ua, ub;
  load_unit<BS>(ua, unit(0), ks, pk, pv, slot_elems, g, i);

  // Q^T operand: lane (g, i) holds row v*16 + i of tile v, dims st*32 + 8g .. +8.
  bf16x8 qb[NT][4];
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    const int row = v * 16 + i;
    if (row < a.rows) {
      const int tq = row / a.G;
      const int qh = h * a.G + (row - tq * a.G);
      const uint16_t* qrow = a.q + (((long long)r * a.T + tq) * a.Hq + qh) * kHeadDim;
#pragma unroll
      for (int st = 0; st < 4; ++st) qb[v][st] = as_bf16x8(ldg16(qrow + st * 32 + g * 8));
    } else {
#pragma unroll
      for (int st = 0; st < 4; ++st) qb[v][st] = as_bf16x8(u32x4{0, 0, 0, 0});
    }
  }
  const int map_slot = unit_slot<BS>(u_first, 0, lane);
  int map_entry = map_load(smap, ks, map_slot, a.ctx_len + r);
  // a vector load (relaxed atomic) whose value is pinned to a VGPR until the
  // next unit's loads are out, so that the wait for it comes after them
  int ctx_raw = __hip_atomic_load(a.ctx_len + r, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  __builtin_amdgcn_sched_barrier(0);

  float m_run[NT], l_run[NT];  // row reference maximum (log2 units) and this lane's partial sum
  f32x4 acc[NT][8];
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    m_run[v] = -INFINITY;
    l_run[v] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[v][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  int local_len = 0;
  // One unit: counts from the mask (reloaded at the first unit of every chunk
  // after the first), V of unattended tokens cleared, then the online softmax.
  uint64_t vmask = 0;
  auto run = [&](UnitRegs& cur, int t) {
    if (t > 0 && (t & (kChunk - 1)) == 0) {
      const int slot = unit_slot<BS>(u_first, t, lane);
      vmask = map_mask(ks, slot, map_load(smap, ks, slot, a.ctx_len + r));
    }
    int n0, n1;
    unit_counts<BS>(unit(t), ks, local_len, vmask, bit_of(t), n0, n1);
    const int keep = lane_keep<BS>(n0, n1, g);
    const bool partial = __builtin_amdgcn_ballot_w64(keep < 8) != 0;
    if (partial) mask_unit_v(cur, keep);
    process_unit<NT, BS>(cur, keep, partial, qb, m_run, l_run, acc, a.scale_log2);
  };

  // The next unit's K/V loads are issued before the current unit is computed
  // (one exposed memory latency per wave, not per unit). Loads past the wave's
  // last unit are placeholders on the local slot (cache-resident), so the
  // compiler's wait counts stay exact.
  auto settle = [&]() {  // the map entries and the context length are in
    asm volatile("" : "+v"(map_entry), "+v"(ctx_raw));
    vmask = map_mask(ks, map_slot, map_entry);
    local_len = ctx_blocks(ctx_raw, BS, a.NBmax).local_len;
  };
  load_unit<BS>(ub, unit(1), ks, pk, pv, slot_elems, g, i);
  __builtin_amdgcn_sched_barrier(0);  // both units' loads are issued before the first wait
  settle();
  for (int t = 0; t < nt;) {
    run(ua, t);
    if (++t >= nt) break;
    load_unit<BS>(ua, unit(t + 1), ks, pk, pv, slot_elems, g, i);
    run(ub, t);
    if (++t >= nt) break;
    load_unit<BS>(ub, unit(t + 1), ks, pk, pv, slot_elems, g, i);
  }
  // row sums: add the partial sums of the four lanes of every row
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    l_run[v] += __shfl_xor(l_run[v], 16);
    l_run[v] += __shfl_xor(l_run[v], 32);
  }

  // ---- merge the waves of this workgroup through LDS -----------------------
  // Each wave publishes its row maxima and sums; every lane then reads those of
  // all waves for its rows (all reads issued before any is used, no branch on
  // them), rescales its accumulators to the merged maximum and writes them to
  // its slice; finally every thread sums the slices of a few (row, 4-dimension)
  // positions, all their reads again issued at once.
  constexpr int kRows = NT * 16;
  constexpr int kPad = kHeadDim + 4;
  __shared__ float s_m[kW][kRows], s_l[kW][kRows], s_ml[2][kRows];
  __shared__ __align__(16) float s_o[kW][kRows][kPad];
  if (g == 0) {
#pragma unroll
    for (int v = 0; v < NT; ++v) {
      s_m[wave][v * 16 + i] = m_run[v];
      s_l[wave][v * 16 + i] = l_run[v];
    }
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    const int row = v * 16 + i;
    float mw[kW], lw[kW];
#pragma unroll
    for (int w = 0; w < kW; ++w) {
      mw[w] = s_m[w][row];
      lw[w] = s_l[w][row];
    }
    float M = mw[0];
#pragma unroll
    for (int w = 1; w < kW; ++w) M = fmaxf(M, mw[w]);
    float L = 0.f;
#pragma unroll
    for (int w = 0; w < kW; ++w) L += mw[w] == -INFINITY ? 0.f : lw[w] * fast_exp2(mw[w] - M);
    const float f = m_run[v] == -INFINITY ? 0.f : fast_exp2(m_run[v] - M);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[v][dt] *= f;
    if (wave == 0 && g == 0) {
      s_ml[0][row] = M;
      s_ml[1][row] = L;
    }
  }
#pragma unroll
  for (int v = 0; v < NT; ++v)
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
      *reinterpret_cast<f32x4*>(&s_o[wave][v * 16 + i][dt * 16 + 4 * g]) = acc[v][dt];
  __syncthreads();

  const int nsplit = a.nsplit;
  const long long pbase = ((long long)rh * nsplit + split) * a.rows;
  constexpr int kPer = (kRows * (kHeadDim / 4) + kW * 64 - 1) / (kW * 64);  // positions per thread
  const int npos = a.rows * (kHeadDim / 4);
  f32x4 o[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int pos = threadIdx.x + j * kW * 64;
    const int row = (pos < npos ? pos : 0) >> 5;
    const int c4 = pos & 31;
    o[j] = *reinterpret_cast<const f32x4*>(&s_o[0][row][c4 * 4]);
#pragma unroll
    for (int sl = 1; sl < kW; ++sl) o[j] += *reinterpret_cast<const f32x4*>(&s_o[sl][row][c4 * 4]);
  }
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int pos = threadIdx.x + j * kW * 64;
    if (pos >= npos) break;
    const int row = pos >> 5;
    const int c4 = pos & 31;
    const float M = s_ml[0][row], L = s_ml[1][row];
    if (nsplit == 1) {  // the only split: finish here
      write_output(a, r, h, row, c4, o[j], M, L);
    } else {
      *reinterpret_cast<f32x4*>(a.part_o + (pbase + row) * kHeadDim + c4 * 4) = o[j];
      if (c4 == 0) {
        a.part_ml[(pbase + row) * 2 + 0] = M;
        a.part_ml[(pbase + row) * 2 + 1] = L;
      }
    }
  }
}

// Split kernel for many row tiles (NT >= 3: G * T > 32 rows). A workgroup has
// one wave per row tile; every wave attends its 16 rows to every unit of the
// split, so the waves never merge softmax states and each writes its own rows.
// Each unit's K and V cross HBM once: its 16 chunks (8 of K, 8 of V, 16 bytes
// a lane, in the MFMA operand layout of load_unit) are loaded straight into
// LDS, dealt round-robin to the waves, and every wave reads all 16 back as
// conflict-free 16-byte LDS reads. A ring of kRowsStages units keeps
// kRowsStages - 1 units in flight; one barrier per unit publishes a unit to
// every wave and frees the stage of the one before.
//
// Measured on MI355X (16 requests x 8 KV heads x 72 rows, B = 32, 4,096
// tokens per head, 268 MB): 81.7 us for the register kernel (every wave loads
// the units of its own split range, five row tiles per wave), 63 to 66 us here
// with the merge and four stages; 1 to 2 us less with each unit's score
// products issued one step ahead of its softmax and PV products (below),
// about 1 us less again with the prologue's own loads on the DMA path
// (below), and 0.5 to 1.5 us less again with three stages instead of four
// (two: 80 us; six: no gain). Registers staged through VGPRs instead of
// direct-to-LDS loads, two units ahead: 67 to 70 us; two workgroups per CU: no
// gain; exact per-wave load counts instead of the surplus loads: 1 us slower.
constexpr int kRowsStages = 3;
typedef u32x4 UnitLds[17][64];  // [chunk][lane]; chunk 16 takes the surplus loads

template <int BS>
__device__ __forceinline__ const uint16_t* chunk_src(int u, int j, int ks, const uint16_t* pk, const uint16_t* pv,
                                                     long long slot_elems, int g, int i) {
  // lane (g, i)'s 16 bytes of chunk j of unit u: j < 8 is K token tile tau = j / 4 at
  // k-step st = j % 4, j >= 8 is V d-tile j - 8 (the addresses load_unit reads)
  const bool real = u >= 0;
  const int s0 = real ? (BS == 16 ? 2 * u : u) : ks;
  const int s1raw = real ? (BS == 16 ? 2 * u + 1 : ks + 1) : ks + 1;
  const int s1 = s1raw <= ks ? s1raw : ks;
  if (j < 8) {
    const int tau = j >> 2, st = j & 3;
    const int tok = 8 * (i >> 2) + 4 * tau + (i & 3);
    const uint16_t* k0 = pk + (long long)s0 * slot_elems;
    const uint16_t* k1 = pk + (long long)s1 * slot_elems;
    const uint16_t* src = BS == 16 ? ((tok < 16 ? k0 : k1) + (tok & 15) * kHeadDim + g * 8)
                                   : (k0 + tok * kHeadDim + g * 8);
    return src + st * 32;
  }
  const int dt = j - 8;
  const uint16_t* v0 = pv + (long long)s0 * slot_elems;
  const uint16_t* v1 = pv + (long long)s1 * slot_elems;
  const uint16_t* vsrc = BS == 16 ? ((g < 2 ? v0 : v1) + (g & 1) * 8) : (v0 + 8 * g);
  return vsrc + (long long)(dt * 16 + i) * BS;
}

// 16 bytes a lane from global memory straight into LDS (global_load_lds_dwordx4):
// lane L's bytes land at lds_row + 16 L, lds_row being the same in every lane.
// Written as inline assembly because the compiler, which cannot tell the ring's
// stages apart once they are reused, would otherwise wait for every earlier
// such load before each one (a full drain per unit); the waits are the
// explicit vmcnt counts of the kernel instead. The "memory" clobber keeps LDS
// reads and writes in program order around it, and M0 (the LDS base operand
// of the load) is restored after it.
__device__ __forceinline__ void lds_dma16(const void* gsrc, void* lds_row) {
  const uint32_t lds =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_row);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gsrc), "s"(lds)
      : "memory");
}

// 4 bytes a lane, as lds_dma16 (lane L's bytes land at lds_row + 4 L).
__device__ __forceinline__ void lds_dma4(const void* gsrc, void* lds_row) {
  const uint32_t lds =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds_row);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gsrc), "s"(lds)
      : "memory");
}

// s_waitcnt vmcnt(N) alone (expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// f(std::integral_constant<int, 0>{}), ..., f(std::integral_constant<int, N - 1>{})
template <typename F, int... S>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, S...>) {
  (f(std::integral_constant<int, S>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// One 32-token unit of one row tile in two halves, so that a wave can issue
// the next unit's score products before this unit's softmax and PV products
// (software pipelining across units): unit_scores gives S^T of the unit
// (lane (g, i): row i against unit tokens 8g .. 8g+7, as in process_unit);
// unit_softmax_pv is the rest of process_unit for one row tile.
__device__ __forceinline__ void unit_scores(const UnitRegs& cur, const bf16x8 (&qb)[4], f32x4 (&sc)[2]) {
#pragma unroll
  for (int tau = 0; tau < 2; ++tau) {
    f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 4; ++st)
      s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(cur.k[tau][st]), qb[st], s4, 0, 0, 0);
    sc[tau] = s4;
  }
}

__device__ __forceinline__ void unit_softmax_pv(const f32x4 (&sc)[2], const u32x4 (&vin)[8], int keep, bool partial,
                                                float& m_ref, float& l_part, f32x4 (&acc)[8], float scale_log2) {
  float x[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = sc[e >> 2][e & 3] * scale_log2;
  u32x4 v[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) v[dt] = vin[dt];
  if (partial) {
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = e < keep ? x[e] : -INFINITY;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t lo = (2 * w) < keep ? 0x0000FFFFu : 0u;
        const uint32_t hi = (2 * w + 1) < keep ? 0xFFFF0000u : 0u;
        v[dt][w] &= (lo | hi);
      }
  }
  const float lmax = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
  if (__builtin_amdgcn_ballot_w64(lmax > m_ref + kLazyTh)) {
    float rmax = fmaxf(lmax, __shfl_xor(lmax, 16));
    rmax = fmaxf(rmax, __shfl_xor(rmax, 32));
    const float m_new = fmaxf(m_ref, rmax);
    const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_ref - m_new);
    l_part *= alpha;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[dt] *= alpha;
    m_ref = m_new;
  }
  const float m_use = m_ref == -INFINITY ? 0.f : m_ref;
  bf16x8 pb;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float pe = fast_exp2(x[e] - m_use);
    psum += pe;
    pb[e] = (__bf16)pe;
  }
  l_part += psum;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt)
    acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(v[dt]), pb, acc[dt], 0, 0, 0);
}

template <int NT, int BS>
__global__ __launch_bounds__(NT * 64) void attn_split_rows_kernel(AttnArgs a) {
  static_assert(kRowsStages == 3, "one LDS variable per stage below");
  constexpr int kPer = (16 + NT - 1) / NT;  // chunk loads per wave and unit
  // One LDS variable per stage, always named with a compile-time stage, so the
  // compiler sees each read of a stage apart from the other stages' loads.
  // Every wave issues kPer loads a unit (the surplus ones re-read chunk 0 into
  // row 16), so that one vmcnt count fits every wave.
  __shared__ __align__(16) UnitLds s_st0;
  __shared__ __align__(16) UnitLds s_st1;
  __shared__ __align__(16) UnitLds s_st2;
  __shared__ __align__(16) u32x4 s_q[NT][4][64];  // each wave's query operand (4 k-steps)
  __shared__ int s_misc[NT][3][64];               // each wave's context length and two mask chunks
  auto stage_buf = [&](auto S) __attribute__((always_inline)) -> UnitLds& {
    constexpr int k = decltype(S)::value;
    if constexpr (k == 0) return s_st0;
    else if constexpr (k == 1) return s_st1;
    else return s_st2;
  };
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // this wave's row tile
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int i = lane & 15;
  const int nrh = a.R * a.Hkv;
  int rh, split;
  if (!map_workgroup(blockIdx.x, nrh, a.nsplit, rh, split)) return;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const int ks = a.k_slots;
  const long long slot_elems = (long long)a.Hkv * BS * kHeadDim;
  const long long head_off = (long long)h * BS * kHeadDim;
  const uint16_t* pk = a.pool_k + (long long)r * (ks + 1) * slot_elems + head_off;
  const uint16_t* pv = a.pool_v + (long long)r * (ks + 1) * slot_elems + head_off;
  const int32_t* smap = a.slot_map + (long long)rh * ks;
  const int u_begin = split * a.units_per_split;
  const int u_end = min(a.n_units, u_begin + a.units_per_split);
  const int nt = u_end > u_begin ? u_end - u_begin : 0;  // units of this workgroup, in order
  auto unit = [&](int t) __attribute__((always_inline)) { return t < nt ? u_begin + t : -1; };

  // this wave's chunk loads of unit t into stage S (past the last unit: the placeholder slot)
  auto issue = [&](int t, auto S) __attribute__((always_inline)) {
    UnitLds& buf = stage_buf(S);
    const int u = unit(t);
#pragma unroll
    for (int c = 0; c < kPer; ++c) {
      const int j = v + c * NT;
      lds_dma16(chunk_src<BS>(u, j < 16 ? j : 0, ks, pk, pv, slot_elems, g, i), &buf[j < 16 ? j : 16][0]);
    }
  };
  // validity mask of units t .. t + kChunkU - 1 (lane l: map entry of slot l % 2 of
  // unit t + l / 2 at B = 16, of unit t + l at B = 32)
  constexpr int kChunkU = BS == 16 ? 32 : 64;
  auto mask_slot = [&](int t) __attribute__((always_inline)) {
    const int jj = BS == 16 ? lane >> 1 : lane;
    return BS == 16 ? 2 * (u_begin + t + jj) + (lane & 1) : u_begin + t + jj;
  };
  // Everything else the unit loop reads (the context length, the slot-map
  // entries of the first two mask chunks, this wave's query operand) takes the
  // same LDS-DMA path, ahead of the ring's first units: the compiler cannot
  // count the DMA loads, so its wait for any load it issues after them would
  // drain the ring. Rows past the end load row 0's queries and are zeroed.
  const int row = v * 16 + i;
  {
    const int qr = row < a.rows ? row : 0;
    const int tq = qr / a.G;
    const int qh = h * a.G + (qr - tq * a.G);
    const uint16_t* qrow = a.q + (((long long)r * a.T + tq) * a.Hq + qh) * kHeadDim;
    lds_dma4(a.ctx_len + r, &s_misc[v][0][0]);
    lds_dma4(map_addr(smap, ks, mask_slot(0), a.ctx_len + r), &s_misc[v][1][0]);
    lds_dma4(map_addr(smap, ks, mask_slot(kChunkU), a.ctx_len + r), &s_misc[v][2][0]);
#pragma unroll
    for (int st = 0; st < 4; ++st) lds_dma16(qrow + st * 32 + g * 8, &s_q[v][st][0]);
  }
  static_for<kRowsStages - 1>([&](auto S) __attribute__((always_inline)) { issue(decltype(S)::value, S); });
  wait_vmcnt<kPer * (kRowsStages - 1)>();  // all but the ring's units are in

  // Q^T operand of row tile v
  bf16x8 qb[1][4];
#pragma unroll
  for (int st = 0; st < 4; ++st) qb[0][st] = as_bf16x8(row < a.rows ? s_q[v][st][lane] : u32x4{0, 0, 0, 0});
  const Ctx c = ctx_blocks(__builtin_amdgcn_readfirstlane(s_misc[v][0][lane]), BS, a.NBmax);
  const int local_len = c.local_len;

  float m_run[1] = {-INFINITY}, l_run[1] = {0.f};
  f32x4 acc[1][8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) acc[0][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint64_t vmask = map_mask(ks, mask_slot(0), s_misc[v][1][lane]);
  const bf16x8(&q1)[4] = qb[0];

  // The previous unit's scores, V operands and mask, finished one step late:
  // before the first unit they stand for an empty unit (no token attended).
  f32x4 sc_prev[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  u32x4 v_prev[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) v_prev[dt] = u32x4{0, 0, 0, 0};
  int keep_prev = 0;
  bool partial_prev = true;

  // unit t sits in stage t % kRowsStages
  auto step = [&](int t, auto S) __attribute__((always_inline)) {
    constexpr int k = decltype(S)::value;
    // this wave's loads of unit t are done (those of the kRowsStages - 2 later units may
    // still fly); the barrier publishes every wave's loads of unit t and tells that the
    // stage of unit t - 1 is no longer read
    wait_vmcnt<kPer * (kRowsStages - 2)>();
    __syncthreads();
    if (t > 0 && (t & (kChunkU - 1)) == 0) {
      // mask chunk t / kChunkU came in a chunk ago; the next one goes out now
      // (one more load ahead of the next unit's only makes later waits stricter)
      const int ch = t / kChunkU;
      vmask = map_mask(ks, mask_slot(t), s_misc[v][1 + (ch & 1)][lane]);
      lds_dma4(map_addr(smap, ks, mask_slot(t + kChunkU), a.ctx_len + r), &s_misc[v][1 + ((ch + 1) & 1)][0]);
    }
    issue(t + kRowsStages - 1, std::integral_constant<int, (k + kRowsStages - 1) % kRowsStages>{});
    const UnitLds& buf = stage_buf(S);
    UnitRegs cur;
#pragma unroll
    for (int tau = 0; tau < 2; ++tau)
#pragma unroll
      for (int st = 0; st < 4; ++st) cur.k[tau][st] = buf[tau * 4 + st][lane];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) cur.v[dt] = buf[8 + dt][lane];
    f32x4 sc[2];
    unit_scores(cur, q1, sc);
    // the previous unit's softmax and PV products run beside this unit's score products
    unit_softmax_pv(sc_prev, v_prev, keep_prev, partial_prev, m_run[0], l_run[0], acc[0], a.scale_log2);
    int n0, n1;
    const int bit = BS == 16 ? 2 * (t & (kChunkU - 1)) : (t & (kChunkU - 1));
    unit_counts<BS>(unit(t), ks, local_len, vmask, bit, n0, n1);
    keep_prev = lane_keep<BS>(n0, n1, g);
    partial_prev = __builtin_amdgcn_ballot_w64(keep_prev < 8) != 0;
    sc_prev[0] = sc[0];
    sc_prev[1] = sc[1];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) v_prev[dt] = cur.v[dt];
  };
  int t = 0;
  for (; t + kRowsStages <= nt; t += kRowsStages)
    static_for<kRowsStages>([&](auto S) __attribute__((always_inline)) { step(t + decltype(S)::value, S); });
  static_for<kRowsStages - 1>([&](auto S) __attribute__((always_inline)) {
    if (t + decltype(S)::value < nt) step(t + decltype(S)::value, S);
  });
  unit_softmax_pv(sc_prev, v_prev, keep_prev, partial_prev, m_run[0], l_run[0], acc[0], a.scale_log2);
  wait_vmcnt<0>();  // the placeholder loads past the last unit land before the workgroup ends
  float L = l_run[0] + __shfl_xor(l_run[0], 16);
  L += __shfl_xor(L, 32);
  const float M = m_run[0];
  if (row >= a.rows) return;
  if (a.nsplit == 1) {
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) write_output(a, r, h, row, dt * 4 + g, acc[0][dt], M, L);
    return;
  }
  const long long pr = ((long long)rh * a.nsplit + split) * a.rows + row;
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) *reinterpret_cast<f32x4*>(a.part_o + pr * kHeadDim + dt * 16 + 4 * g) = acc[0][dt];
  if (g == 0) *reinterpret_cast<float2*>(a.part_ml + pr * 2) = make_float2(M, L);
}

// Merge of the NS splits: a workgroup takes kMergeRows rows of one (request,
// KV head), 32 threads a row, each thread 4 dimensions; every thread issues its
// NS partial loads (16 bytes each) and the row's NS (max, sum) pairs at once.
// Workgroup ids are dealt so that the head's id % 8, which places its splits on
// one XCD, places its merge there too: the partials are read from the L2 that
// holds them.
constexpr int kMergeRows = 8;

template <int NS>
__global__ __launch_bounds__(kMergeRows * 32) void attn_merge_kernel(AttnArgs a) {
  const int nrh = a.R * a.Hkv;
  const int groups = (a.rows + kMergeRows - 1) / kMergeRows;
  const int wg = blockIdx.x;
  const int local = wg >> 3;
  const int rh_local = local / groups;
  const int grp = local - rh_local * groups;
  const int rh = rh_local * 8 + (wg & 7);
  const int row = grp * kMergeRows + (threadIdx.x >> 5);
  if (rh >= nrh || row >= a.rows) return;
  const int c4 = threadIdx.x & 31;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const long long base = (long long)rh * NS * a.rows + row;
  float2 ml[NS];
  f32x4 os[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const long long idx = base + (long long)s * a.rows;
    ml[s] = *reinterpret_cast<const float2*>(a.part_ml + idx * 2);
    os[s] = *reinterpret_cast<const f32x4*>(a.part_o + idx * kHeadDim + c4 * 4);
  }
  float M = ml[0].x;
#pragma unroll
  for (int s = 1; s < NS; ++s) M = fmaxf(M, ml[s].x);
  // a split with no attended token (max -inf) weighs 0; with none at all, L = 0
  float L = 0.f;
  f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const float f = ml[s].x == -INFINITY ? 0.f : fast_exp2(ml[s].x - M);
    L += ml[s].y * f;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] += os[s][e] * f;
  }
  float res[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) res[e] = L > 0.f ? o[e] / L : 0.f;
  const int t = row / a.G;
  const int qh = h * a.G + (row - t * a.G);
  const long long orow = ((long long)r * a.T + t) * a.Hq + qh;
  const uint32_t w0 = f32_to_bf16_bits(res[0]) | (f32_to_bf16_bits(res[1]) << 16);
  const uint32_t w1 = f32_to_bf16_bits(res[2]) | (f32_to_bf16_bits(res[3]) << 16);
  *reinterpret_cast<uint2*>(a.out + orow * kHeadDim + c4 * 4) = make_uint2(w0, w1);
  if (c4 == 0 && a.lse) a.lse[orow] = L > 0.f ? (M + __log2f(L)) * 0.69314718055994531f : -INFINITY;
}

template <int NS>
void launch_merge_ns(const AttnArgs& a, hipStream_t s, const LaunchTiming& t, int nrh8) {
  const int groups = (a.rows + kMergeRows - 1) / kMergeRows;
  launch_kernel(attn_merge_kernel<NS>, dim3((unsigned)(nrh8 * groups)), dim3(kMergeRows * 32), s, t, a);
}

void launch_merge(const AttnArgs& a, hipStream_t s, const LaunchTiming& t, int nrh8) {
  switch (a.nsplit) {
    case 2: return launch_merge_ns<2>(a, s, t, nrh8);
    case 3: return launch_merge_ns<3>(a, s, t, nrh8);
    case 4: return launch_merge_ns<4>(a, s, t, nrh8);
    case 5: return launch_merge_ns<5>(a, s, t, nrh8);
    case 6: return launch_merge_ns<6>(a, s, t, nrh8);
    case 7: return launch_merge_ns<7>(a, s, t, nrh8);
    case 8: return launch_merge_ns<8>(a, s, t, nrh8);
    case 9: return launch_merge_ns<9>(a, s, t, nrh8);
    case 10: return launch_merge_ns<10>(a, s, t, nrh8);
    case 11: return launch_merge_ns<11>(a, s, t, nrh8);
    case 12: return launch_merge_ns<12>(a, s, t, nrh8);
    case 13: return launch_merge_ns<13>(a, s, t, nrh8);
    case 14: return launch_merge_ns<14>(a, s, t, nrh8);
    case 15: return launch_merge_ns<15>(a, s, t, nrh8);
    default: return launch_merge_ns<kMaxSplits>(a, s, t, nrh8);
  }
}

template <int NT, int BS>
hipError_t launch_t(const AttnArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int nrh = a.R * a.Hkv;
  const int nrh8 = (nrh + 7) / 8 * 8;
  const bool merge = a.nsplit > 1;
  // timed as one span: from the split kernel's start to the merge kernel's end
  if constexpr (NT >= 3)
    launch_kernel(attn_split_rows_kernel<NT, BS>, dim3((unsigned)(nrh8 * a.nsplit)), dim3(NT * 64), s,
                  LaunchTiming{t.start, merge ? nullptr : t.stop}, a);
  else
    launch_kernel(attn_split_kernel<NT, BS>, dim3((unsigned)(nrh8 * a.nsplit)), dim3(kW * 64), s,
                  LaunchTiming{t.start, merge ? nullptr : t.stop}, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge) return e;
  launch_merge(a, s, LaunchTiming{nullptr, t.stop}, nrh8);
  return hipGetLastError();
}

template <int BS>
hipError_t launch_bs(const AttnArgs& a, hipStream_t s, const LaunchTiming& t) {
  switch ((a.rows + 15) / 16) {
    case 1: return launch_t<1, BS>(a, s, t);
    case 2: return launch_t<2, BS>(a, s, t);
    case 3: return launch_t<3, BS>(a, s, t);
    case 4: return launch_t<4, BS>(a, s, t);
    case 5: return launch_t<5, BS>(a, s, t);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

AttnPlan attn_plan(int R, int Hq, int Hkv, int T, int B, int k_slots) {
  AttnPlan p{};
  const int G = Hq / Hkv;
  p.rows = G * T;
  p.n_units = B == 16 ? (k_slots + 2) / 2 : k_slots + 1;
  const long long nrh = (long long)R * Hkv;
  long long want = (kTargetWorkgroups + nrh - 1) / (nrh > 0 ? nrh : 1);
  const long long most = (p.n_units + kW - 1) / kW;  // at least one unit per wave
  if (want > most) want = most;
  if (want > kMaxSplits) want = kMaxSplits;
  if (want < 1) want = 1;
  p.units_per_split = (int)((p.n_units + want - 1) / want);
  p.nsplit = (p.n_units + p.units_per_split - 1) / p.units_per_split;
  // partials exist only with several splits (one split writes the outputs itself)
  p.part_o_floats = p.nsplit > 1 ? (size_t)nrh * p.nsplit * p.rows * kHeadDim : 0;
  p.part_ml_floats = p.nsplit > 1 ? (size_t)nrh * p.nsplit * p.rows * 2 : 0;
  p.bytes = (p.part_o_floats + p.part_ml_floats) * sizeof(float);
  return p;
}

hipError_t launch_attn(const AttnArgs& a, hipStream_t s, const LaunchTiming& t) {
  return a.B == 16 ? launch_bs<16>(a, s, t) : launch_bs<32>(a, s, t);
}

// Scratch of the allocation-free attention entry point: the split partials, in
// a file-scope device array that every GPU the library runs on holds from
// module load until the process ends (kNoAllocScratchBytes each). Host code
// never passes the array's name to a kernel: that is a host-side stand-in, not
// a device address. Its address on each device comes from hipGetSymbolAddress,
// taken once per device with that device current, and only that address is
// handed to the kernels.
namespace {
__device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace oasis
