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
// and a second kernel merges the splits. (A last-arriving-workgroup merge in
// the same kernel measured slower on MI355X: its agent-scope release/acquire
// costs more than the second launch.)
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
#include "oasis_internal.h"

namespace oasis {

namespace {

constexpr int kW = 4;  // waves per workgroup
// Workgroups of one attention call: one per CU when the kernel prefetches
// (one wave per SIMD), two otherwise.
constexpr int kTargetWorkgroupsPrefetch = 256;
constexpr int kTargetWorkgroups = 512;
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

// K and V registers of one 32-token unit, plus the token counts of its two
// slots (0 = not attended).
struct UnitRegs {
  u32x4 k[2][4];
  u32x4 v[8];
  int n0, n1;
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
__device__ __forceinline__ void load_unit(UnitRegs& ur, int u, int ks, int local_len, const int32_t* smap,
                                          const uint16_t* pk, const uint16_t* pv, long long slot_elems, int g,
                                          int i) {
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
  // token counts of the two slots (0 = not attended)
  ur.n0 = !real ? 0 : (s0 < ks ? (smap[s0] >= 0 ? BS : 0) : (s0 == ks ? local_len : 0));
  ur.n1 = (BS == 16 && real) ? (s1raw < ks ? (smap[s1raw] >= 0 ? BS : 0) : (s1raw == ks ? local_len : 0)) : 0;
}

// Zero the V values of tokens that are not attended (their probability is 0,
// but 0 * NaN would poison the accumulator). Only lanes whose 8 tokens are not
// all attended (a free slot, the tail of the local block) do any work; in a
// full unit the whole wave skips it.
template <int BS>
__device__ __forceinline__ void mask_unit_v(UnitRegs& ur, int g) {
  const int cnt = BS == 16 ? (g < 2 ? ur.n0 : ur.n1) : ur.n0;
  const int t0 = BS == 16 ? (g & 1) * 8 : 8 * g;
  const int keep = cnt - t0;
  if (keep >= 8) return;
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
constexpr float kLazyTh = 8.f;

template <int NT, int BS>
__device__ __forceinline__ void process_unit(const UnitRegs& cur, const bf16x8 (&qb)[NT][4], float (&m_ref)[NT],
                                             float (&l_part)[NT], f32x4 (&acc)[NT][8], int g, float scale_log2) {
  // validity of the 8 unit tokens 8g + 4*tau + j this lane scores
  bool valid[2][4];
#pragma unroll
  for (int tau = 0; tau < 2; ++tau)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tok = 8 * g + 4 * tau + j;
      valid[tau][j] = BS == 16 ? (tok < 16 ? tok < cur.n0 : (tok - 16) < cur.n1) : tok < cur.n0;
    }
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
    float lmax = -INFINITY;
#pragma unroll
    for (int tau = 0; tau < 2; ++tau)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float z = valid[tau][j] ? sc[tau][j] * scale_log2 : -INFINITY;
        x[4 * tau + j] = z;
        lmax = fmaxf(lmax, z);
      }
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

template <int NT, int BS>
__global__ __launch_bounds__(kW * 64) void attn_split_kernel(AttnArgs a) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4;
  const int i = lane & 15;
  const int nrh = a.R * a.Hkv;
  int rh, split;
  if (!map_workgroup(blockIdx.x, nrh, a.nsplit, rh, split)) return;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const Ctx c = ctx_blocks(a.ctx_len[r], BS, a.NBmax);
  const int ks = a.k_slots;

  // Q^T operand: lane (g, i) holds row v*16 + i of tile v, dims st*32 + 8g .. +8.
  bf16x8 qb[NT][4];
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    const int row = v * 16 + i;
    if (row < a.rows) {
      const int t = row / a.G;
      const int qh = h * a.G + (row - t * a.G);
      const uint16_t* qrow = a.q + (((long long)r * a.T + t) * a.Hq + qh) * kHeadDim;
#pragma unroll
      for (int st = 0; st < 4; ++st) qb[v][st] = as_bf16x8(ldg16(qrow + st * 32 + g * 8));
    } else {
#pragma unroll
      for (int st = 0; st < 4; ++st) qb[v][st] = as_bf16x8(u32x4{0, 0, 0, 0});
    }
  }

  const long long slot_elems = (long long)a.Hkv * BS * kHeadDim;
  const long long head_off = (long long)h * BS * kHeadDim;
  const uint16_t* pk = a.pool_k + (long long)r * (ks + 1) * slot_elems + head_off;
  const uint16_t* pv = a.pool_v + (long long)r * (ks + 1) * slot_elems + head_off;
  const int32_t* smap = a.slot_map + (long long)rh * ks;

  float m_run[NT], l_run[NT];  // row reference maximum (log2 units) and this lane's partial sum
  f32x4 acc[NT][8];
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    m_run[v] = -INFINITY;
    l_run[v] = 0.f;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[v][dt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  const int u_begin = split * a.units_per_split;
  const int u_end = min(a.n_units, u_begin + a.units_per_split);

  // With few row tiles the next unit's K/V loads are issued before the current
  // unit is computed (one exposed memory latency per wave, not per unit); with
  // many row tiles the registers go to the accumulators instead.
  constexpr bool kPrefetch = NT <= 2;
  int u = u_begin + wave;
  if (kPrefetch) {
    // two register buffers used alternately (no copies between them)
    UnitRegs ua, ub;
    load_unit<BS>(ua, u < u_end ? u : -1, ks, c.local_len, smap, pk, pv, slot_elems, g, i);
    while (u < u_end) {
      load_unit<BS>(ub, u + kW < u_end ? u + kW : -1, ks, c.local_len, smap, pk, pv, slot_elems, g, i);
      mask_unit_v<BS>(ua, g);
      process_unit<NT, BS>(ua, qb, m_run, l_run, acc, g, a.scale_log2);
      u += kW;
      if (u >= u_end) break;
      load_unit<BS>(ua, u + kW < u_end ? u + kW : -1, ks, c.local_len, smap, pk, pv, slot_elems, g, i);
      mask_unit_v<BS>(ub, g);
      process_unit<NT, BS>(ub, qb, m_run, l_run, acc, g, a.scale_log2);
      u += kW;
    }
  } else {
    for (; u < u_end; u += kW) {
      UnitRegs cur;
      load_unit<BS>(cur, u, ks, c.local_len, smap, pk, pv, slot_elems, g, i);
      mask_unit_v<BS>(cur, g);
      process_unit<NT, BS>(cur, qb, m_run, l_run, acc, g, a.scale_log2);
    }
  }
  // row sums: add the partial sums of the four lanes of every row
#pragma unroll
  for (int v = 0; v < NT; ++v) {
    l_run[v] += __shfl_xor(l_run[v], 16);
    l_run[v] += __shfl_xor(l_run[v], 32);
  }

  // ---- merge the waves of this workgroup through LDS -----------------------
  // Row maxima first; every wave rescales its accumulators to them and writes
  // them to a slice (kSlices slices; with fewer slices than waves the other
  // waves add into them in a second round); then every thread sums the slices
  // of some (row, dimension) entries in a fixed order.
  constexpr int kRows = NT * 16;
  constexpr int kPad = kHeadDim + 4;
  constexpr int kSlices = NT <= 4 ? kW : 2;  // LDS: kSlices * kRows * kPad floats <= 160 KiB
  __shared__ float s_m[kW][kRows], s_l[kW][kRows];
  __shared__ float s_o[kSlices][kRows][kPad];
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
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kW; ++w) M = fmaxf(M, s_m[w][row]);
    const float f = M == -INFINITY ? 0.f : fast_exp2(m_run[v] - M);
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) acc[v][dt] *= f;
  }
#pragma unroll
  for (int round = 0; round < kW / kSlices; ++round) {
    if (wave / kSlices == round) {
      const int sl = wave % kSlices;
#pragma unroll
      for (int v = 0; v < NT; ++v)
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          float* dst = &s_o[sl][v * 16 + i][dt * 16 + 4 * g];
          f32x4 val = acc[v][dt];
          if (round > 0) {
            val[0] += dst[0];
            val[1] += dst[1];
            val[2] += dst[2];
            val[3] += dst[3];
          }
          dst[0] = val[0];
          dst[1] = val[1];
          dst[2] = val[2];
          dst[3] = val[3];
        }
    }
    __syncthreads();
  }

  const int nsplit = a.nsplit;
  const long long pbase = ((long long)rh * nsplit + split) * a.rows;
  // (row, 4-dimension group) entries of this split: max over waves, rescale, sum
  for (int idx = threadIdx.x; idx < a.rows * (kHeadDim / 4); idx += kW * 64) {
    const int row = idx / (kHeadDim / 4);
    const int c4 = idx - row * (kHeadDim / 4);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kW; ++w) M = fmaxf(M, s_m[w][row]);
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    float L = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kW; ++w) L += s_m[w][row] == -INFINITY ? 0.f : s_l[w][row] * fast_exp2(s_m[w][row] - M);
#pragma unroll
      for (int sl = 0; sl < kSlices; ++sl) {
        const float* src = &s_o[sl][row][c4 * 4];
        o[0] += src[0];
        o[1] += src[1];
        o[2] += src[2];
        o[3] += src[3];
      }
    }
    if (nsplit == 1) {  // the only split: finish here
      write_output(a, r, h, row, c4, o, M, L);
    } else {
      *reinterpret_cast<f32x4*>(a.part_o + (pbase + row) * kHeadDim + c4 * 4) = o;
      if (c4 == 0) {
        a.part_ml[(pbase + row) * 2 + 0] = M;
        a.part_ml[(pbase + row) * 2 + 1] = L;
      }
    }
  }
}

// Merge of the splits: one workgroup per (row, request x KV head), one thread
// per dimension; all partial loads of a thread are issued before any is used
// (nsplit <= kMaxSplits).
__global__ __launch_bounds__(kHeadDim) void attn_merge_kernel(AttnArgs a) {
  const int row = blockIdx.x;
  const int rh = blockIdx.y;
  const int d = threadIdx.x;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const long long base = (long long)rh * a.nsplit * a.rows + row;
  float ms[kMaxSplits], ls[kMaxSplits], os[kMaxSplits];
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) {
    const long long idx = base + (long long)s * a.rows;
    const bool live = s < a.nsplit;
    ms[s] = live ? a.part_ml[idx * 2] : -INFINITY;
    ls[s] = live ? a.part_ml[idx * 2 + 1] : 0.f;
    os[s] = live ? a.part_o[idx * kHeadDim + d] : 0.f;
  }
  float M = -INFINITY;
#pragma unroll
  for (int s = 0; s < kMaxSplits; ++s) M = fmaxf(M, ms[s]);
  float L = 0.f, o = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int s = 0; s < kMaxSplits; ++s) {
      const float f = ms[s] == -INFINITY ? 0.f : fast_exp2(ms[s] - M);
      L += ls[s] * f;
      o += os[s] * f;
    }
  }
  const float res = L > 0.f ? o / L : 0.f;
  const int t = row / a.G;
  const int qh = h * a.G + (row - t * a.G);
  const long long orow = ((long long)r * a.T + t) * a.Hq + qh;
  a.out[orow * kHeadDim + d] = (uint16_t)f32_to_bf16_bits(res);
  if (d == 0 && a.lse) a.lse[orow] = L > 0.f ? (M + __log2f(L)) * 0.69314718055994531f : -INFINITY;
}

template <int NT, int BS>
hipError_t launch_t(const AttnArgs& a, hipStream_t s, const LaunchTiming& t) {
  const int nrh = a.R * a.Hkv;
  const int nrh8 = (nrh + 7) / 8 * 8;
  const bool merge = a.nsplit > 1;
  // timed as one span: from the split kernel's start to the merge kernel's end
  launch_kernel(attn_split_kernel<NT, BS>, dim3((unsigned)(nrh8 * a.nsplit)), dim3(kW * 64), s,
                LaunchTiming{t.start, merge ? nullptr : t.stop}, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge) return e;
  launch_kernel(attn_merge_kernel, dim3((unsigned)a.rows, (unsigned)nrh), dim3(kHeadDim), s,
                LaunchTiming{nullptr, t.stop}, a);
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
  const int target = (p.rows + 15) / 16 <= 2 ? kTargetWorkgroupsPrefetch : kTargetWorkgroups;
  long long want = (target + nrh - 1) / (nrh > 0 ? nrh : 1);
  const long long most = (p.n_units + kW - 1) / kW;  // at least one unit per wave
  if (want > most) want = most;
  if (want > kMaxSplits) want = kMaxSplits;
  if (want < 1) want = 1;
  p.units_per_split = (int)((p.n_units + want - 1) / want);
  p.nsplit = (p.n_units + p.units_per_split - 1) / p.units_per_split;
  p.part_o_floats = (size_t)nrh * p.nsplit * p.rows * kHeadDim;
  p.part_ml_floats = (size_t)nrh * p.nsplit * p.rows * 2;
  p.bytes = (p.part_o_floats + p.part_ml_floats) * sizeof(float);
  return p;
}

hipError_t launch_attn(const AttnArgs& a, hipStream_t s, const LaunchTiming& t) {
  return a.B == 16 ? launch_bs<16>(a, s, t) : launch_bs<32>(a, s, t);
}

}  // namespace oasis
