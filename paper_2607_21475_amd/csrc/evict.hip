// evict.hip -- the Poisson tail sampler on gfx950 (Sec. 3.3: eq. (2), certainty set, Poisson tail;
// Sec. 3.1: evicted rows are deleted, retained rows keep one stored pi each).
//
// Two launches per call:
//   evict_solve    one work-group per unit.  Reads the unit's scores once (kept in registers
//                  up to 16384 tokens), solves lambda with sum_T clip(lambda s, eps, 1) = m, then
//                  draws the mask once to count retained tokens per 2048-token chunk and writes
//                  the chunk offsets, count and status.
//   evict_compact  one work-group per (unit, chunk).  Recomputes pi and the Philox words of its
//                  2048 tokens (bit-identical to the solve pass), ranks the retained ones with a
//                  block scan and copies only the retained K/V rows (16 lanes x 16 B per row).
//                  Evicted rows are never read.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

__device__ __forceinline__ bool in_tail(int64_t i, int64_t n, int32_t n_sink, int32_t n_recent) {
  return i >= (int64_t)n_sink && i < n - (int64_t)n_recent;
}

// Non-finite and negative scores are read as 0 and flagged.
__device__ __forceinline__ float clean_score(float s, uint32_t &bad) {
  if (!(s >= 0.0f) || isinf(s)) {
    bad = 1u;
    return 0.0f;
  }
  return s;
}

// pi of one position; used identically by both launches so their masks agree bit for bit.
__device__ __forceinline__ float token_pi(bool tail, float s, float lam, float eps) {
  if (!tail) return 1.0f;
  if (isinf(lam)) return s > 0.0f ? 1.0f : eps;
  return fminf(fmaxf(lam * s, eps), 1.0f);
}

__device__ __forceinline__ uint64_t unit_seed(const EvictLaunch &L, int u) {
  return L.seed_per_unit ? L.seed_per_unit[u] : L.seed;
}

// Sum of three doubles over the 512-thread block; every thread gets the totals.
// `buf` alternates between calls so one barrier per call suffices.
__device__ __forceinline__ void block_sum3(double &a, double &b, double &c, double (*red)[8][3],
                                           int &buf) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  c = wave_sum(c);
  if (lane == 0) {
    red[buf][wv][0] = a;
    red[buf][wv][1] = b;
    red[buf][wv][2] = c;
  }
  __syncthreads();
  a = b = c = 0.0;
#pragma unroll
  for (int w = 0; w < kEvictThreads / 64; ++w) {
    a += red[buf][w][0];
    b += red[buf][w][1];
    c += red[buf][w][2];
  }
  buf ^= 1;
}

__device__ __forceinline__ void block_minmax(float &mx, float &mn, float (*red)[8][2], int &buf) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  mx = wave_max(mx);
  mn = wave_min(mn);
  if (lane == 0) {
    red[buf][wv][0] = mx;
    red[buf][wv][1] = mn;
  }
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kEvictThreads / 64; ++w) {
    mx = fmaxf(mx, red[buf][w][0]);
    mn = fminf(mn, red[buf][w][1]);
  }
  buf ^= 1;
}

// Scores of the thread's four-token groups: group k covers tokens 4 (t + 512 k) .. +3.
template <int RC>
struct ScoreRegs {
  float v[RC > 0 ? RC : 1][4];
};

template <int RC>
__device__ __forceinline__ void load_group(const float *sc, int64_t n, int64_t gi, float (&s)[4],
                                           uint32_t &bad) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t i = 4 * gi + j;
    s[j] = i < n ? clean_score(sc[i], bad) : 0.0f;
  }
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// evict_solve: lambda, per-chunk retained counts, count, status
// ---------------------------------------------------------------------------------------------
template <int RC>
__global__ __launch_bounds__(kEvictThreads) void evict_solve_kernel(EvictLaunch L) {
  __shared__ double red3[2][8][3];
  __shared__ float red2[2][8][2];
  int b3 = 0, b2 = 0;
  const int u = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t base = L.seq_off[u];
  const int64_t n = L.seq_off[u + 1] - base;
  const int64_t cap = L.cap_off[u + 1] - L.cap_off[u];
  const int64_t nprot = min(n, (int64_t)L.n_sink + (int64_t)L.n_recent);
  const double f = L.budget_per_unit ? (double)L.budget_per_unit[u] : (double)L.budget_frac;
  const double m = f * (double)n - (double)nprot;
  const float eps = L.pi_min;
  const float *sc = L.scores + base;
  const int64_t ngroups = (n + 3) / 4;
  if ((n + kEvictChunk - 1) / kEvictChunk > (int64_t)L.nchunk) {
    // longer than the launch was planned for: touch nothing of this unit
    if (t == 0) {
      L.count[u] = 0;
      L.status[u] = EBD_ST_BAD_LAYOUT;
      L.ws_lambda[u] = 0.0f;
      if (L.lambda_out) L.lambda_out[u] = 0.0f;
    }
    return;
  }

  ScoreRegs<RC> R;
  uint32_t bad = 0;
  if (RC > 0) {
#pragma unroll
    for (int k = 0; k < (RC > 0 ? RC : 1); ++k) load_group<RC>(sc, n, t + (int64_t)kEvictThreads * k, R.v[k], bad);
  }

  // Visit every token of the thread: f(i, s).
  auto for_tokens = [&](auto &&fn) {
    if (RC > 0) {
#pragma unroll
      for (int k = 0; k < (RC > 0 ? RC : 1); ++k) {
        const int64_t gi = t + (int64_t)kEvictThreads * k;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int64_t i = 4 * gi + j;
          if (i < n) fn(i, R.v[k][j]);
        }
      }
    } else {
      uint32_t dummy = 0;
      for (int64_t gi = t; gi < ngroups; gi += kEvictThreads) {
        float s[4];
        load_group<RC>(sc, n, gi, s, dummy);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int64_t i = 4 * gi + j;
          if (i < n) fn(i, s[j]);
        }
      }
    }
  };

  // Tail statistics: |T|, #positive, sum_T s, max s, min positive s; bad-score flag.
  double n_tail = 0.0, n_pos = 0.0, s_sum = 0.0;
  float s_max = 0.0f, s_minp = INFINITY;
  for_tokens([&](int64_t i, float s) {
    if (in_tail(i, n, L.n_sink, L.n_recent)) {
      n_tail += 1.0;
      s_sum += (double)s;
      if (s > 0.0f) {
        n_pos += 1.0;
        s_minp = fminf(s_minp, s);
      }
      s_max = fmaxf(s_max, s);
    }
  });
  if (RC == 0) {
    // streamed path: the flag is raised while reading raw scores
    for (int64_t i = t; i < n; i += kEvictThreads) {
      const float s = sc[i];
      if (!(s >= 0.0f) || isinf(s)) bad = 1u;
    }
  }
  double badd = (double)bad;
  block_sum3(n_tail, n_pos, s_sum, red3, b3);
  block_minmax(s_max, s_minp, red2, b2);
  {
    double z0 = badd, z1 = 0.0, z2 = 0.0;
    block_sum3(z0, z1, z2, red3, b3);
    badd = z0;
  }

  uint32_t st = badd > 0.0 ? EBD_ST_BAD_SCORE : 0u;
  const double n_zero = n_tail - n_pos;
  double lam = 0.0;
  if (n_tail == 0.0) {
    lam = 0.0;
  } else if (L.pi_mode == 1) {
    lam = (s_sum > 0.0 && m > 0.0) ? m / s_sum : 0.0;
    if (m <= (double)eps * n_tail) st |= EBD_ST_BUDGET_FLOOR;
  } else if (m <= (double)eps * n_tail) {
    lam = 0.0;
    st |= EBD_ST_BUDGET_FLOOR;
  } else if (m >= n_pos + (double)eps * n_zero) {
    lam = INFINITY;
    st |= EBD_ST_NO_EVICTION;
  } else {
    // g(lam) = H + eps L + lam S_mid is piecewise linear and nondecreasing.  Newton steps on the
    // current piece (exact once the piece is right), safeguarded by a bracket [lo, hi] with
    // g(lo) < m <= g(hi).
    double lo = (double)eps / (double)s_max;
    double hi = 1.0 / (double)s_minp;
    double cur = fmin(fmax(m / s_sum, lo), hi);
    double pH = -1.0, pL = -1.0, pS = -1.0;
    bool from_newton = false;
    for (int it = 0; it < 96; ++it) {
      const float lf = (float)cur;
      double H = 0.0, Lo = 0.0, S = 0.0;
      for_tokens([&](int64_t i, float s) {
        if (in_tail(i, n, L.n_sink, L.n_recent)) {
          const float p = lf * s;
          if (p >= 1.0f) H += 1.0;
          else if (p <= eps) Lo += 1.0;
          else S += (double)s;
        }
      });
      block_sum3(H, Lo, S, red3, b3);
      if (from_newton && H == pH && Lo == pL && S == pS) break;  // same piece: cur is exact
      const double g = H + (double)eps * Lo + (double)lf * S;
      if (g < m) lo = (double)lf;
      else hi = (double)lf;
      if (g == m) break;
      double nxt = S > 0.0 ? (m - H - (double)eps * Lo) / S : -1.0;
      from_newton = (nxt > lo && nxt < hi);
      if (!from_newton) nxt = 0.5 * (lo + hi);
      if ((float)nxt == lf || hi - lo <= 1e-9 * hi) {
        cur = from_newton ? nxt : cur;
        break;
      }
      pH = H;
      pL = Lo;
      pS = S;
      cur = nxt;
    }
    lam = cur;
  }
  const float lamf = (float)lam;

  // Retained count per chunk with the final pi: the same arithmetic evict_compact repeats.
  const uint64_t sd = unit_seed(L, u);
  const int64_t nch = (n + kEvictChunk - 1) / kEvictChunk;
  double total = 0.0;
  for (int64_t c = 0; c < nch; ++c) {
    const int64_t gi = c * kEvictThreads + t;
    double kept = 0.0;
    if (4 * gi < n) {
      float s[4];
      uint32_t dummy = 0;
      if (RC > 0) {
#pragma unroll
        for (int k = 0; k < (RC > 0 ? RC : 1); ++k)
          if (k == c) {
#pragma unroll
            for (int j = 0; j < 4; ++j) s[j] = R.v[k][j];
          }
      } else {
        load_group<RC>(sc, n, gi, s, dummy);
      }
      const uint4 x = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)u, L.epoch, kPhiloxTag),
                                    (uint32_t)sd, (uint32_t)(sd >> 32));
      const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t i = 4 * gi + j;
        if (i < n) {
          const float p = token_pi(in_tail(i, n, L.n_sink, L.n_recent), s[j], lamf, eps);
          kept += keep_token(xw[j], p) ? 1.0 : 0.0;
        }
      }
    }
    double z1 = 0.0, z2 = 0.0;
    block_sum3(kept, z1, z2, red3, b3);
    if (t == 0) L.ws_chunk_off[(int64_t)u * L.nchunk + c] = (int32_t)total;
    total += kept;
  }
  if (t == 0) {
    if ((int64_t)total > cap) st |= EBD_ST_CAP_OVERFLOW;
    L.count[u] = (int32_t)total;
    L.status[u] = st;
    L.ws_lambda[u] = lamf;
    if (L.lambda_out) L.lambda_out[u] = lamf;
  }
}

// ---------------------------------------------------------------------------------------------
// evict_compact: mask, rank, stable copy of retained rows
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kEvictThreads) void evict_compact_kernel(EvictLaunch L) {
  __shared__ int wave_tot[kEvictThreads / 64];
  __shared__ uint16_t list[kEvictChunk];
  const int64_t bid = blockIdx.x;
  const int c = (int)(bid % L.nchunk);
  const int u = (int)(bid / L.nchunk);
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t base = L.seq_off[u];
  const int64_t n = L.seq_off[u + 1] - base;
  if ((int64_t)c * kEvictChunk >= n) return;
  if ((n + kEvictChunk - 1) / kEvictChunk > (int64_t)L.nchunk) return;  // flagged by evict_solve
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const float lamf = L.ws_lambda[u];
  const float eps = L.pi_min;
  const uint64_t sd = unit_seed(L, u);

  const int64_t gi = (int64_t)c * kEvictThreads + t;
  float p[4] = {1.0f, 1.0f, 1.0f, 1.0f};
  uint32_t keep = 0;
  if (4 * gi < n) {
    uint32_t dummy = 0;
    float s[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i = 4 * gi + j;
      s[j] = i < n ? clean_score(L.scores[base + i], dummy) : 0.0f;
    }
    const uint4 x = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)u, L.epoch, kPhiloxTag),
                                  (uint32_t)sd, (uint32_t)(sd >> 32));
    const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i = 4 * gi + j;
      if (i < n) {
        p[j] = token_pi(in_tail(i, n, L.n_sink, L.n_recent), s[j], lamf, eps);
        if (keep_token(xw[j], p[j])) keep |= 1u << j;
        if (L.pi_full) L.pi_full[base + i] = p[j];
      }
    }
  }
  // Block exclusive scan of the per-thread retained counts.
  const int cnt = __popc(keep);
  int incl = cnt;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int y = __shfl_up(incl, d);
    if (lane >= d) incl += y;
  }
  if (lane == 63) wave_tot[wv] = incl;
  __syncthreads();
  int wpre = 0, nret = 0;
#pragma unroll
  for (int w = 0; w < kEvictThreads / 64; ++w) {
    const int v = wave_tot[w];
    wpre += w < wv ? v : 0;
    nret += v;
  }
  const int64_t chunk_off = L.ws_chunk_off[(int64_t)u * L.nchunk + c];
  int r = wpre + incl - cnt;  // rank within the chunk
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (keep & (1u << j)) {
      const int64_t g = chunk_off + r;
      if (g < cap) {
        L.pic[cbase + g] = p[j];
        L.idxc[cbase + g] = (int32_t)(4 * gi + j);
      }
      list[r] = (uint16_t)(4 * t + j);
      ++r;
    }
  }
  __syncthreads();

  // Copy the retained rows: 16 lanes per 256-byte row, 32 rows per pass, 4 passes in flight.
  const int sub = t & 15;
  const int row0 = t >> 4;
  const int64_t cbeg = (int64_t)c * kEvictChunk;
  const int64_t room = cap - chunk_off;  // rows of this chunk that still fit
  const int nrow = (int)min((int64_t)nret, max(room, (int64_t)0));
  const uint4 *K4 = reinterpret_cast<const uint4 *>(L.K);
  const uint4 *V4 = reinterpret_cast<const uint4 *>(L.V);
  uint4 *Kc4 = reinterpret_cast<uint4 *>(L.Kc);
  uint4 *Vc4 = reinterpret_cast<uint4 *>(L.Vc);
  constexpr int kRowsPerPass = kEvictThreads / 16;
  for (int rr = row0; rr < nrow; rr += 4 * kRowsPerPass) {
    uint4 kv[4], vv[4];
    int64_t dst[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int ro = rr + q * kRowsPerPass;
      dst[q] = -1;
      if (ro < nrow) {
        const int64_t src = (base + cbeg + list[ro]) * (kHeadDim / 8) + sub;
        kv[q] = K4[src];
        vv[q] = V4[src];
        dst[q] = (cbase + chunk_off + ro) * (kHeadDim / 8) + sub;
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (dst[q] >= 0) {
        Kc4[dst[q]] = kv[q];
        Vc4[dst[q]] = vv[q];
      }
    }
  }
}

size_t evict_workspace_bytes(int32_t U, int32_t nchunk) {
  const size_t a = ((size_t)U * sizeof(float) + 255) & ~(size_t)255;
  const size_t b = ((size_t)U * (size_t)nchunk * sizeof(int32_t) + 255) & ~(size_t)255;
  return a + b;
}

hipError_t launch_evict_solve(const EvictLaunch &L, hipStream_t s) {
  const dim3 grid(L.U), block(kEvictThreads);
  switch (L.reg_chunks) {
    case 1: hipLaunchKernelGGL(evict_solve_kernel<1>, grid, block, 0, s, L); break;
    case 2: hipLaunchKernelGGL(evict_solve_kernel<2>, grid, block, 0, s, L); break;
    case 4: hipLaunchKernelGGL(evict_solve_kernel<4>, grid, block, 0, s, L); break;
    case 8: hipLaunchKernelGGL(evict_solve_kernel<8>, grid, block, 0, s, L); break;
    default: hipLaunchKernelGGL(evict_solve_kernel<0>, grid, block, 0, s, L); break;
  }
  return hipGetLastError();
}

hipError_t launch_evict_compact(const EvictLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)L.U * L.nchunk)), block(kEvictThreads);
  hipLaunchKernelGGL(evict_compact_kernel, grid, block, 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
