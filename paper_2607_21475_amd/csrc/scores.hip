// scores.hip -- importance scores from accumulated attention on gfx950 (App. "Experimental
// details", Harness: the sampler's scores are the attention that prefill queries, or a window
// of observation queries, pay to each cached key).
//
// score_i = sum_w softmax_w(scale q_w . k)_i over the rows query w sees, in two passes over K
// with one wave per (unit, split of its rows):
//   scores_stats  per split and query: the running max m and the sum z = sum 2^(l2 - m) of the
//                 base-2 logits l2 = scale log2e q.k over the split's rows the query sees
//   scores_accum  the unit's normalisers (M, Z) from its splits' (m, z), then for every row
//                 sum_w 2^(l2_w - M_w) / Z_w, written to (or added to) the scores
// q.k runs on MFMA 16x16x32 bf16 (exact products, fp32 sums): the K tile is the A operand
// (16 rows x 32 dims per k-block, loaded straight from HBM in operand layout) and each B
// operand block holds 16 queries.  Lane (g, c) of a block then holds rows 4g .. 4g+3 of
// query 16 b + c.  Tiles of 32 rows go through raw buffer loads bounded by the split, three in
// registers (two in flight while one is computed).
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

// Weights stay below 2^kLazy between moves of the running max (fp32 keeps their range).
constexpr float kLazyMax = 8.0f;

struct KTile {
  u32x4 k[8];  // subtile s (rows 32t + 16s + c): dims 32 kb + 8 g .. + 7 in k[4 s + kb]
  float old[2];  // accumulate mode: current score of row 32t + 16s + 4g + c (lanes c < 4)
};

template <bool ACC>
__device__ __forceinline__ void load_ktile(KTile &T, __amdgpu_buffer_rsrc_t rK,
                                           __amdgpu_buffer_rsrc_t rS, int t, int g, int c) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const uint32_t r = (uint32_t)(32 * t + 16 * s + c);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      T.k[4 * s + kb] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rK, r * 256u + (uint32_t)(64 * kb + 16 * g), 0, 0));
    if (ACC) {
      const uint32_t ro = (uint32_t)(32 * t + 16 * s + 4 * g + c);
      T.old[s] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(rS, c < 4 ? ro * 4u : 0xfffffff0u, 0, 0));
    }
  }
}

template <int NQB>
struct Queries {
  bf16x8 op[NQB][4];  // B operand blocks: column c of block b is query 16 b + c
  int lim[NQB];       // last unit row the query of this lane's column sees (-1: none)
};

template <int NQB>
__device__ __forceinline__ void load_queries(Queries<NQB> &Q, const ScoresLaunch &L, int u,
                                             int64_t n, int g, int c) {
#pragma unroll
  for (int b = 0; b < NQB; ++b) {
    const int w = 16 * b + c;
    const bool ok = w < L.W;
    const uint4 *qw =
        reinterpret_cast<const uint4 *>(L.q + ((int64_t)u * L.W + (ok ? w : 0)) * kHeadDim);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      Q.op[b][kb] = __builtin_bit_cast(bf16x8, ok ? qw[4 * kb + g] : make_uint4(0u, 0u, 0u, 0u));
    int lim = ok ? (int)(n - 1) : -1;
    if (ok && L.qpos) lim = min(lim, L.qpos[(int64_t)u * L.W + w]);
    Q.lim[b] = lim;
  }
}

// Base-2 logits of subtile s of a tile for every query block, -inf where the row is past the
// split or beyond what the query sees.  `rrel` is the split row of this lane's first row.
template <int NQB>
__device__ __forceinline__ void subtile_logits(const KTile &T, int s, const Queries<NQB> &Q,
                                               int rrel, int nrow, int row0, float sc2,
                                               float (&l)[NQB][4]) {
#pragma unroll
  for (int b = 0; b < NQB; ++b) {
    f32x4 acc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, T.k[4 * s + kb]),
                                                    Q.op[b][kb], acc, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool ok = (rrel + i < nrow) && (row0 + rrel + i <= Q.lim[b]);
      l[b][i] = ok ? acc[i] * sc2 : -INFINITY;
    }
  }
}

__device__ __forceinline__ float exp2_rel(float l, float m) {
  return l == -INFINITY ? 0.0f : fast_exp2(l - m);
}

}  // namespace

// Pass 1: per (unit, split) and query, the running max and exp-sum over the split's rows.
template <int NQB>
__global__ __launch_bounds__(64, 2) void scores_stats_kernel(ScoresLaunch L) {
  const int bid = blockIdx.x;
  const int sp = bid % L.nsplit, u = bid / L.nsplit;
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  const int64_t base = L.seq_off[u];
  // a unit longer than the launch was planned for is scored over its planned rows only
  const int64_t n = min(L.seq_off[u + 1] - base, (int64_t)L.nsplit * L.split_rows);
  const int row0 = sp * L.split_rows;
  if (row0 >= n) return;
  const int nrow = (int)min(n - row0, (int64_t)L.split_rows);

  Queries<NQB> Q;
  load_queries<NQB>(Q, L, u, n, g, c);
  float m[NQB], z[NQB];
#pragma unroll
  for (int b = 0; b < NQB; ++b) {
    m[b] = -INFINITY;
    z[b] = 0.0f;
  }
  const float sc2 = L.scale * kLog2e;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(L.K + (base + row0) * kHeadDim, (uint32_t)nrow * 256u);
  const int ntile = (nrow + 31) / 32;

  auto step = [&](const KTile &T, int t) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      float l[NQB][4];
      subtile_logits<NQB>(T, s, Q, 32 * t + 16 * s + 4 * g, nrow, row0, sc2, l);
#pragma unroll
      for (int b = 0; b < NQB; ++b) {
        const float lmax = fmaxf(fmaxf(l[b][0], l[b][1]), fmaxf(l[b][2], l[b][3]));
        if (__any(lmax > m[b] + kLazyMax)) {
          const float mnew = fmaxf(m[b], lmax);
          z[b] *= exp2_rel(m[b], mnew);
          m[b] = mnew;
        }
        const float ms = m[b] == -INFINITY ? 0.0f : m[b];  // no finite logit seen yet: l = -inf
        z[b] += exp2_rel(l[b][0], ms) + exp2_rel(l[b][1], ms) + exp2_rel(l[b][2], ms) +
                exp2_rel(l[b][3], ms);
      }
    }
  };
  KTile T0, T1, T2;
  const __amdgpu_buffer_rsrc_t rNone = rK;  // no score reads in this pass
  load_ktile<false>(T0, rK, rNone, 0, g, c);
  load_ktile<false>(T1, rK, rNone, 1, g, c);
  int t = 0;
  for (; t + 3 <= ntile; t += 3) {
    load_ktile<false>(T2, rK, rNone, t + 2, g, c);
    step(T0, t);
    load_ktile<false>(T0, rK, rNone, t + 3, g, c);
    step(T1, t + 1);
    load_ktile<false>(T1, rK, rNone, t + 4, g, c);
    step(T2, t + 2);
  }
  if (t < ntile) step(T0, t);
  if (t + 1 < ntile) step(T1, t + 1);

  // merge the four row groups of each query column
#pragma unroll
  for (int b = 0; b < NQB; ++b) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float mo = __shfl_xor(m[b], o), zo = __shfl_xor(z[b], o);
      const float mn = fmaxf(m[b], mo);
      z[b] = z[b] * exp2_rel(m[b], mn) + zo * exp2_rel(mo, mn);
      m[b] = mn;
    }
    const int w = 16 * b + c;
    if (g == 0 && w < L.W)
      L.stats[((int64_t)u * L.nsplit + sp) * L.W + w] = make_float2(m[b], z[b]);
  }
}

// Pass 2: the unit's normalisers, then every row's score.
template <int NQB, bool ACC>
__global__ __launch_bounds__(64, 2) void scores_accum_kernel(ScoresLaunch L) {
  const int bid = blockIdx.x;
  const int sp = bid % L.nsplit, u = bid / L.nsplit;
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  const int64_t base = L.seq_off[u];
  // a unit longer than the launch was planned for is scored over its planned rows only
  const int64_t n = min(L.seq_off[u + 1] - base, (int64_t)L.nsplit * L.split_rows);
  const int row0 = sp * L.split_rows;
  if (row0 >= n) return;
  const int nrow = (int)min(n - row0, (int64_t)L.split_rows);
  const int nsp = (int)((n + L.split_rows - 1) / L.split_rows);

  Queries<NQB> Q;
  load_queries<NQB>(Q, L, u, n, g, c);
  float M[NQB], iZ[NQB];
#pragma unroll
  for (int b = 0; b < NQB; ++b) {
    const int w = 16 * b + c;
    float mm = -INFINITY, zz = 0.0f;
    if (w < L.W) {
      const float2 *st = L.stats + (int64_t)u * L.nsplit * L.W + w;
      for (int s = 0; s < nsp; ++s) {
        const float2 v = st[(int64_t)s * L.W];
        const float mn = fmaxf(mm, v.x);
        zz = zz * exp2_rel(mm, mn) + v.y * exp2_rel(v.x, mn);
        mm = mn;
      }
    }
    M[b] = mm == -INFINITY ? 0.0f : mm;
    iZ[b] = zz > 0.0f ? 1.0f / zz : 0.0f;
  }
  const float sc2 = L.scale * kLog2e;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(L.K + (base + row0) * kHeadDim, (uint32_t)nrow * 256u);
  const __amdgpu_buffer_rsrc_t rS = make_rsrc(L.scores + base + row0, (uint32_t)nrow * 4u);
  const int ntile = (nrow + 31) / 32;

  auto step = [&](const KTile &T, int t) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int rrel = 32 * t + 16 * s + 4 * g;
      float l[NQB][4];
      subtile_logits<NQB>(T, s, Q, rrel, nrow, row0, sc2, l);
      float p[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int b = 0; b < NQB; ++b) {
#pragma unroll
        for (int i = 0; i < 4; ++i) p[i] += exp2_rel(l[b][i], M[b]) * iZ[b];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) p[i] = row16_sum(p[i]);  // over the 16 queries of the row group
      // lane (g, c < 4) stores row rrel + c; the other lanes' stores fall outside the range
      float v = c == 0 ? p[0] : (c == 1 ? p[1] : (c == 2 ? p[2] : p[3]));
      if (ACC) v += T.old[s];
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rS,
                                            c < 4 ? (uint32_t)(rrel + c) * 4u : 0xfffffff0u, 0, 0);
    }
  };
  KTile T0, T1, T2;
  load_ktile<ACC>(T0, rK, rS, 0, g, c);
  load_ktile<ACC>(T1, rK, rS, 1, g, c);
  int t = 0;
  for (; t + 3 <= ntile; t += 3) {
    load_ktile<ACC>(T2, rK, rS, t + 2, g, c);
    step(T0, t);
    load_ktile<ACC>(T0, rK, rS, t + 3, g, c);
    step(T1, t + 1);
    load_ktile<ACC>(T1, rK, rS, t + 4, g, c);
    step(T2, t + 2);
  }
  if (t < ntile) step(T0, t);
  if (t + 1 < ntile) step(T1, t + 1);
}

size_t scores_workspace_bytes(int32_t U, int32_t nsplit, int32_t W) {
  return ((size_t)U * (size_t)nsplit * (size_t)W * sizeof(float2) + 255) / 256 * 256;
}

hipError_t launch_scores_stats(const ScoresLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)L.U * L.nsplit)), block(64);
  switch ((L.W + 15) / 16) {
    case 1: hipLaunchKernelGGL(scores_stats_kernel<1>, grid, block, 0, s, L); break;
    case 2: hipLaunchKernelGGL(scores_stats_kernel<2>, grid, block, 0, s, L); break;
    case 3: hipLaunchKernelGGL(scores_stats_kernel<3>, grid, block, 0, s, L); break;
    default: hipLaunchKernelGGL(scores_stats_kernel<4>, grid, block, 0, s, L); break;
  }
  return hipGetLastError();
}

hipError_t launch_scores_accum(const ScoresLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)L.U * L.nsplit)), block(64);
  const bool acc = (L.flags & EBD_SCORES_ACCUMULATE) != 0;
  switch ((L.W + 15) / 16) {
    case 1:
      if (acc) hipLaunchKernelGGL((scores_accum_kernel<1, true>), grid, block, 0, s, L);
      else hipLaunchKernelGGL((scores_accum_kernel<1, false>), grid, block, 0, s, L);
      break;
    case 2:
      if (acc) hipLaunchKernelGGL((scores_accum_kernel<2, true>), grid, block, 0, s, L);
      else hipLaunchKernelGGL((scores_accum_kernel<2, false>), grid, block, 0, s, L);
      break;
    case 3:
      if (acc) hipLaunchKernelGGL((scores_accum_kernel<3, true>), grid, block, 0, s, L);
      else hipLaunchKernelGGL((scores_accum_kernel<3, false>), grid, block, 0, s, L);
      break;
    default:
      if (acc) hipLaunchKernelGGL((scores_accum_kernel<4, true>), grid, block, 0, s, L);
      else hipLaunchKernelGGL((scores_accum_kernel<4, false>), grid, block, 0, s, L);
      break;
  }
  return hipGetLastError();
}

}  // namespace ebd
