// Block-sparse GQA decode attention over the HBM working set (paper §4.2.1:
// the normal and draft queries are stacked and attend one resident KV set in
// one call; §5.2: the K selected blocks plus the active local block).
//
// Work decomposition. The rows of one KV head are its G query heads times the
// T stacked query tokens (20 at G = 4, T = 5). The attended tokens of a
// (request, KV head) are cut into units of 32 tokens (two slots at B = 16,
// one at B = 32); a workgroup of 4 waves handles a contiguous range of units
// (a split) and every wave a strided subset of them, with its own online
// softmax. The waves are merged through LDS, each split writes one partial
// (unnormalised output, running max, running sum) per row, and a second kernel
// merges the splits and writes bf16 outputs and the log-sum-exp.
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

constexpr int kW = 4;                 // waves per workgroup
constexpr int kTargetWorkgroups = 512;

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

template <int NT, int BS>
__global__ __launch_bounds__(kW * 64) void attn_split_kernel(AttnArgs a) {
  const int wave = threadIdx.x >> 6;
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

  // Q^T operand: lane (g, i) holds row i of tile v, dims st*32 + 8g .. +8.
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

  float m_run[NT], l_run[NT];
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
  for (int u = u_begin + wave; u < u_end; u += kW) {
    // slots of this unit and their token counts (0 = not attended)
    int s0, s1, n0, n1;
    if (BS == 16) {
      s0 = 2 * u;
      s1 = 2 * u + 1;
    } else {
      s0 = u;
      s1 = -1;
    }
    n0 = s0 < ks ? (smap[s0] >= 0 ? BS : 0) : (s0 == ks ? c.local_len : 0);
    n1 = 0;
    if (BS == 16) n1 = s1 < ks ? (smap[s1] >= 0 ? BS : 0) : (s1 == ks ? c.local_len : 0);

    // K: lane (g, i), token tile tau -> unit token 8*(i/4) + 4*tau + i%4
    u32x4 kr[2][4];
#pragma unroll
    for (int tau = 0; tau < 2; ++tau) {
      const int tok = 8 * (i >> 2) + 4 * tau + (i & 3);
      int slot, row, cnt;
      if (BS == 16) {
        slot = tok < 16 ? s0 : s1;
        row = tok & 15;
        cnt = tok < 16 ? n0 : n1;
      } else {
        slot = s0;
        row = tok;
        cnt = n0;
      }
      const bool live = row < cnt;
      const uint16_t* src = pk + (long long)slot * slot_elems + row * kHeadDim + g * 8;
#pragma unroll
      for (int st = 0; st < 4; ++st) kr[tau][st] = live ? ldg16(src + st * 32) : u32x4{0, 0, 0, 0};
    }
    // V^T: lane (g, i), d-tile dt -> V[tokens 8g .. 8g+7][d = dt*16 + i]
    u32x4 vr[8];
    {
      int slot, t0, cnt;
      if (BS == 16) {
        slot = g < 2 ? s0 : s1;
        t0 = (g & 1) * 8;
        cnt = g < 2 ? n0 : n1;
      } else {
        slot = s0;
        t0 = 8 * g;
        cnt = n0;
      }
      const bool live = t0 < cnt;
      const uint16_t* src = pv + (long long)slot * slot_elems + t0;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) vr[dt] = live ? ldg16(src + (long long)(dt * 16 + i) * BS) : u32x4{0, 0, 0, 0};
      if (live && cnt - t0 < 8) {  // partial local block: clear the tokens past its end
        const int keep = cnt - t0;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t lo = (2 * w) < keep ? 0x0000FFFFu : 0u;
            const uint32_t hi = (2 * w + 1) < keep ? 0xFFFF0000u : 0u;
            vr[dt][w] &= (lo | hi);
          }
      }
    }

    // validity of the 8 unit tokens 8g + 4*tau + j this lane scores
    bool valid[2][4];
#pragma unroll
    for (int tau = 0; tau < 2; ++tau)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int tok = 8 * g + 4 * tau + j;
        valid[tau][j] = BS == 16 ? (tok < 16 ? tok < n0 : (tok - 16) < n1) : tok < n0;
      }

#pragma unroll
    for (int v = 0; v < NT; ++v) {
      f32x4 sc[2];
#pragma unroll
      for (int tau = 0; tau < 2; ++tau) {
        f32x4 s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < 4; ++st)
          s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kr[tau][st]), qb[v][st], s4, 0, 0, 0);
        sc[tau] = s4;
      }
      float x[8];
      float mx = -INFINITY;
#pragma unroll
      for (int tau = 0; tau < 2; ++tau)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float z = valid[tau][j] ? sc[tau][j] * a.scale_log2 : -INFINITY;
          x[4 * tau + j] = z;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[v], mx);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = fast_exp2(m_run[v] - m_use);
      float p[8];
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        p[e] = fast_exp2(x[e] - m_use);
        psum += p[e];
      }
      psum += __shfl_xor(psum, 16);
      psum += __shfl_xor(psum, 32);
      l_run[v] = l_run[v] * alpha + psum;
      m_run[v] = m_new;
      u32x4 pk4;
#pragma unroll
      for (int w = 0; w < 4; ++w) pk4[w] = f32_to_bf16_bits(p[2 * w]) | (f32_to_bf16_bits(p[2 * w + 1]) << 16);
      const bf16x8 pb = as_bf16x8(pk4);
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        acc[v][dt] *= alpha;
        acc[v][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vr[dt]), pb, acc[v][dt], 0, 0, 0);
      }
    }
  }

  // ---- merge the waves of this workgroup through LDS -----------------------
  constexpr int kRows = NT * 16;
  constexpr int kPad = kHeadDim + 4;
  __shared__ float s_m[kW][kRows], s_l[kW][kRows];
  __shared__ float s_M[kRows], s_L[kRows];
  __shared__ float s_o[kRows][kPad];
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
    if (wave == 0 && g == 0) {
      float L = 0.f;
#pragma unroll
      for (int w = 0; w < kW; ++w) L += M == -INFINITY ? 0.f : s_l[w][row] * fast_exp2(s_m[w][row] - M);
      s_M[row] = M;
      s_L[row] = L;
    }
  }
#pragma unroll
  for (int w = 0; w < kW; ++w) {
    if (wave == w) {
#pragma unroll
      for (int v = 0; v < NT; ++v)
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) {
          float* dst = &s_o[v * 16 + i][dt * 16 + 4 * g];
          f32x4 val = acc[v][dt];
          if (w > 0) {
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

  // ---- write this split's partial ------------------------------------------
  const long long pbase = ((long long)rh * a.nsplit + split) * a.rows;
  for (int idx = threadIdx.x; idx < a.rows * (kHeadDim / 4); idx += kW * 64) {
    const int row = idx / (kHeadDim / 4);
    const int c4 = idx - row * (kHeadDim / 4);
    const float* src = &s_o[row][c4 * 4];
    *reinterpret_cast<f32x4*>(a.part_o + (pbase + row) * kHeadDim + c4 * 4) = f32x4{src[0], src[1], src[2], src[3]};
  }
  for (int row = threadIdx.x; row < a.rows; row += kW * 64) {
    a.part_ml[(pbase + row) * 2 + 0] = s_M[row];
    a.part_ml[(pbase + row) * 2 + 1] = s_L[row];
  }
}

// One workgroup per (row, request x KV head); one thread per dimension.
__global__ __launch_bounds__(kHeadDim) void attn_merge_kernel(AttnArgs a) {
  const int row = blockIdx.x;
  const int rh = blockIdx.y;
  const int d = threadIdx.x;
  const int r = rh / a.Hkv;
  const int h = rh - r * a.Hkv;
  const long long base = (long long)rh * a.nsplit * a.rows + row;
  float M = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, a.part_ml[(base + (long long)s * a.rows) * 2]);
  float L = 0.f, o = 0.f;
  if (M != -INFINITY) {
    for (int s = 0; s < a.nsplit; ++s) {
      const long long idx = base + (long long)s * a.rows;
      const float ms = a.part_ml[idx * 2];
      if (ms == -INFINITY) continue;
      const float f = fast_exp2(ms - M);
      L += a.part_ml[idx * 2 + 1] * f;
      o += a.part_o[idx * kHeadDim + d] * f;
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
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
  const int nrh = a.R * a.Hkv;
  const int nrh8 = (nrh + 7) / 8 * 8;
  hipLaunchKernelGGL((attn_split_kernel<NT, BS>), dim3((unsigned)(nrh8 * a.nsplit)), dim3(kW * 64), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_merge_kernel, dim3((unsigned)a.rows, (unsigned)nrh), dim3(kHeadDim), 0, s, a);
  return hipGetLastError();
}

template <int BS>
hipError_t launch_bs(const AttnArgs& a, hipStream_t s) {
  switch ((a.rows + 15) / 16) {
    case 1: return launch_t<1, BS>(a, s);
    case 2: return launch_t<2, BS>(a, s);
    case 3: return launch_t<3, BS>(a, s);
    case 4: return launch_t<4, BS>(a, s);
    case 5: return launch_t<5, BS>(a, s);
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
  if (want < 1) want = 1;
  p.units_per_split = (int)((p.n_units + want - 1) / want);
  p.nsplit = (p.n_units + p.units_per_split - 1) / p.units_per_split;
  p.part_o_floats = (size_t)nrh * p.nsplit * p.rows * kHeadDim;
  p.part_ml_floats = (size_t)nrh * p.nsplit * p.rows * 2;
  p.bytes = (p.part_o_floats + p.part_ml_floats) * sizeof(float);
  return p;
}

hipError_t launch_attn(const AttnArgs& a, hipStream_t s) {
  return a.B == 16 ? launch_bs<16>(a, s) : launch_bs<32>(a, s);
}

}  // namespace oasis
