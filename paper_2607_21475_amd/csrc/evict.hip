// evict.hip -- the Poisson tail sampler on gfx950 (Sec. 3.3: eq. (2), certainty set, Poisson tail;
// Sec. 3.1: evicted rows are deleted, retained rows keep one stored pi each).
//
// Launches per call:
//   evict_select_reg (units of at most 6144 tokens with a capacity of at least a sixth of their
//                 length) one work-group of 2 waves per unit, the scores in registers, so that
//                 every unit of a large batch is resident at once; the same steps as evict_select
//                 below with one barrier per reduction or prefix; then evict_copy gathers the rows.
//   evict_select  (every other launch) one work-group of 8 waves per unit, two per CU.  Stages the
//                 unit's scores in LDS (up to 16384 tokens, protected positions marked by a
//                 negative sentinel; longer units are re-read from memory), solves lambda with
//                 sum_T clip(lambda s, eps, 1) = m by safeguarded Newton steps on the piecewise
//                 linear g(lambda) (exact once the piece is found), then walks the unit in blocks
//                 of 4 tokens per thread: Philox words and the exact retention test (Poisson), or
//                 a block scan of the integer weights ceil(pi 2^32) against one start per unit
//                 (fixed-size systematic design), or the score threshold of a radix select (top-k
//                 comparison design); ballot ranks plus a cross-wave prefix give the order in
//                 which the stored pi and original position of every retained row are written,
//                 plus the count and status bits.  The same work-group then gathers its unit's
//                 retained K and V rows (the gathers of some units overlap the selection of
//                 others; no second launch).
//   evict_copy    one work-group per (unit, block of retained rows): gathers the retained K and
//                 V rows named by the index list (16 lanes x 16 B per 256-byte row, all loads of
//                 a thread in flight together, non-temporal loads and stores: every byte is
//                 touched once).  Evicted rows are never read.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

// Non-finite and negative scores are read as 0 and flagged.
__device__ __forceinline__ float clean_score(float s, uint32_t &bad) {
  if (!(s >= 0.0f) || isinf(s)) {
    bad = 1u;
    return 0.0f;
  }
  return s == 0.0f ? 0.0f : s;  // -0 becomes +0 (the top-k keys are the score bits)
}

// pi of a position: 1 outside the tail, clip(lambda s, eps, 1) in it.  With lambda = +inf (no
// eviction), lambda s is +inf for s > 0 (pi = 1) and NaN for s = 0, which fmaxf drops (pi = eps).
__device__ __forceinline__ float token_pi(bool tail, float s, float lam, float eps) {
  return tail ? fminf(fmaxf(lam * s, eps), 1.0f) : 1.0f;
}

// Block-wide reductions over the NW waves of evict_select.  `buf` alternates between calls so
// that one barrier per call suffices.
template <int NW>
struct BlockRed {
  double v[2][NW][4];
};



// Sums a, b, c (each exact in double for counts) over the block; all threads get the totals.
template <int NW>
__device__ __forceinline__ void block_sum3(double &a, double &b, double &c, BlockRed<NW> &R,
                                           int &buf) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  a = wave_sum(a);
  b = wave_sum(b);
  c = wave_sum(c);
  if (lane == 0) {
    R.v[buf][wv][0] = a;
    R.v[buf][wv][1] = b;
    R.v[buf][wv][2] = c;
  }
  __syncthreads();
  a = b = c = 0.0;
  for (int w = 0; w < NW; ++w) {
    a += R.v[buf][w][0];
    b += R.v[buf][w][1];
    c += R.v[buf][w][2];
  }
  buf ^= 1;
}

// As block_sum3 for a and b that are already wave totals (the same in every lane).
template <int NW>
__device__ __forceinline__ void block_sum_wave2(double &a, double &b, double &c, BlockRed<NW> &R,
                                                int &buf) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  c = wave_sum(c);
  if (lane == 0) {
    R.v[buf][wv][0] = a;
    R.v[buf][wv][1] = b;
    R.v[buf][wv][2] = c;
  }
  __syncthreads();
  a = b = c = 0.0;
  for (int w = 0; w < NW; ++w) {
    a += R.v[buf][w][0];
    b += R.v[buf][w][1];
    c += R.v[buf][w][2];
  }
  buf ^= 1;
}

template <int NW>
__device__ __forceinline__ void block_minmax(float &mx, float &mn, BlockRed<NW> &R, int &buf) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  mx = wave_max(mx);
  mn = wave_min(mn);
  if (lane == 0) {
    R.v[buf][wv][0] = (double)mx;
    R.v[buf][wv][1] = (double)mn;
  }
  __syncthreads();
  for (int w = 0; w < NW; ++w) {
    mx = fmaxf(mx, (float)R.v[buf][w][0]);
    mn = fminf(mn, (float)R.v[buf][w][1]);
  }
  buf ^= 1;
}

// Inclusive prefix sum over the wave (64-bit).
__device__ __forceinline__ uint64_t wave_scan_u64(uint64_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// Systematic design: points s + k 2^32 (k >= 0) strictly below C.
__device__ __forceinline__ uint64_t points_below(uint64_t C, uint32_t s) {
  return C > (uint64_t)s ? ((C - (uint64_t)s - 1u) >> 32) + 1u : 0u;
}

// Integer weight of a stored pi: ceil(pi 2^32), the Poisson test's exact threshold (pi 2^32 is
// exact in fp32; below 2^32 its ceiling fits 32 bits).
__device__ __forceinline__ uint64_t pi_weight(float pi) {
  const float t = pi * 4294967296.0f;
  return t >= 4294967296.0f ? (1ull << 32) : (uint64_t)(uint32_t)ceilf(t);
}

// Tail statistics of a unit: |T|, positive scores, their sum, the largest score and the smallest
// positive one.
struct TailStats {
  double n_tail, n_pos, s_sum;
  float s_max, s_minp;
};

// lambda of eq. (2) with sum_T clip(lambda s, eps, 1) = m, plus the status bits of the boundary
// cases.  `pass(lf, H, L, S, edges)` gives the unit's totals at lambda = lf: tail positions with
// lf s >= 1 (H), with lf s <= eps (L), and the sum of the scores in between (S).
// g(lambda) = H + eps L + lambda S is piecewise linear and nondecreasing: a Newton step on the
// current piece is exact once the piece is right, and the bracket [lo, hi] with
// g(lo) < m <= g(hi) guards every step (bisection when a step leaves it).
//
// The boundary cases (no tail, the literal lambda = m / sum s, the floor, no eviction): sets
// lambda and the status bits and returns true; false when lambda is interior and needs the
// iteration.
__device__ inline bool lambda_boundary(const TailStats &T, double m, float eps, int pi_mode,
                                       uint32_t &st, double &lam) {
  if (T.n_tail == 0.0) {
    lam = 0.0;
    return true;
  }
  if (pi_mode == 1) {
    if (m <= (double)eps * T.n_tail) st |= EBD_ST_BUDGET_FLOOR;
    lam = (T.s_sum > 0.0 && m > 0.0) ? m / T.s_sum : 0.0;
    return true;
  }
  if (m <= (double)eps * T.n_tail) {
    st |= EBD_ST_BUDGET_FLOOR;
    lam = 0.0;
    return true;
  }
  if (m >= T.n_pos + (double)eps * (T.n_tail - T.n_pos)) {
    st |= EBD_ST_NO_EVICTION;
    lam = INFINITY;
    return true;
  }
  return false;
}

// Where the scores of the evaluated piece lie: the smallest score of H, the largest and smallest
// of the middle, the largest tail score of L.  A lambda whose fp32 products keep every token on
// its side (monotone in s) gives a pass with exactly the same counts and sum.
struct PieceEdges {
  bool valid;  // false: not tracked by this pass
  float h_min, m_max, m_min, l_max;
  __device__ bool keeps(float lf, float eps) const {
    return valid && lf * h_min >= 1.0f && lf * m_max < 1.0f && lf * m_min > eps &&
           lf * l_max <= eps;
  }
};

// Streamed units (scores re-read from memory on every pass) start the iteration from a lambda
// solved on a histogram of their positive tail scores, gathered in the statistics pass: the bins
// are the fp32 bit patterns shifted right by kHistShift (the exponent and five mantissa bits, 32
// bins per octave over every positive float; 64 KB of LDS, which these units do not use for
// scores), each bin's scores taken at the bin's midpoint.  Started there, the iteration needs
// fewer passes over the scores than from the literal m / sum s (a CPU replay on Pareto scores:
// 2.0 instead of 3.6); the lambda it ends on is the same exact solve of the piece it finds.
// (Staged units gain nothing from it: their passes read LDS.)
constexpr int kHistShift = 18;
constexpr int kHistBins = 1 << (31 - kHistShift);

// The iteration for an interior lambda within the bracket [lo, hi] (g(lo) < m <= g(hi)),
// starting at cur.  pass(lf, H, L, S, edges) evaluates the piece at lf.  A Newton step that
// stays on the evaluated piece is final: the next pass would find the same piece and stop there,
// so a pass that reports the piece's edges saves that confirming pass.
template <class Pass>
__device__ double newton_lambda(double m, float eps, double lo, double hi, double cur,
                                Pass &&pass) {
  double pH = -1.0, pL = -1.0, pS = -1.0;
  bool from_newton = false;
  for (int it = 0; it < 96; ++it) {
    const float lf = (float)cur;
    double dH, dL, dS;
    PieceEdges e;
    pass(lf, dH, dL, dS, e);
    if (from_newton && dH == pH && dL == pL && dS == pS) break;  // same piece: cur is exact
    const double g = dH + (double)eps * dL + (double)lf * dS;
    if (g < m) lo = (double)lf;
    else hi = (double)lf;
    if (g == m) break;
    double nxt = dS > 0.0 ? (m - dH - (double)eps * dL) / dS : -1.0;
    from_newton = (nxt > lo && nxt < hi);
    if (!from_newton) nxt = 0.5 * (lo + hi);
    if ((float)nxt == lf || hi - lo <= 1e-9 * hi) {
      cur = from_newton ? nxt : cur;
      break;
    }
    if (from_newton && e.keeps((float)nxt, eps)) {
      cur = nxt;
      break;
    }
    pH = dH;
    pL = dL;
    pS = dS;
    cur = nxt;
  }
  return cur;
}

template <class Pass>
__device__ double solve_lambda(const TailStats &T, double m, float eps, int pi_mode, uint32_t &st,
                               Pass &&pass) {
  double lam;
  if (lambda_boundary(T, m, eps, pi_mode, st, lam)) return lam;
  const double lo = (double)eps / (double)T.s_max;
  const double hi = 1.0 / (double)T.s_minp;
  return newton_lambda(m, eps, lo, hi, fmin(fmax(m / T.s_sum, lo), hi), pass);
}

// Top-k threshold: the k-th largest key among the tail keys (score bits, which order like the
// non-negative cleaned scores), by radix select 8 bits per pass from the top over a histogram in
// LDS.  `count(prefix, pmask, shift)` adds to hist every tail key whose bits under pmask equal
// prefix, at digit (key >> shift) & 255.  Returns the key; `left` gets how many tail positions
// equal to it belong to the k largest.  Every thread of the NT-thread block calls it.
template <int NT, class Count>
__device__ uint32_t radix_kth(int k, int *hist, int *sel, int (*wtot)[NT / 64], int &left,
                              Count &&count) {
  // digits per thread, descending with the thread index (threads past digit 0 hold none)
  constexpr int DPT = NT >= 256 ? 1 : 256 / NT;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  uint32_t prefix = 0, pmask = 0;
  int krem = k, buf = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int d = t; d < 256; d += NT) hist[d] = 0;
    __syncthreads();
    count(prefix, pmask, shift);
    __syncthreads();
    int c[DPT], mine = 0;
#pragma unroll
    for (int e = 0; e < DPT; ++e) {
      c[e] = DPT * t + e < 256 ? hist[255 - DPT * t - e] : 0;
      mine += c[e];
    }
    int incl = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane == 63) wtot[buf][wv] = incl;
    __syncthreads();
    for (int w = 0; w < wv; ++w) incl += wtot[buf][w];
    buf ^= 1;
    int before = incl - mine;
#pragma unroll
    for (int e = 0; e < DPT; ++e) {
      if (c[e] > 0 && before < krem && krem <= before + c[e]) {  // the digit holding the krem-th largest key
        sel[0] = 255 - DPT * t - e;
        sel[1] = krem - before;
      }
      before += c[e];
    }
    __syncthreads();
    prefix |= (uint32_t)sel[0] << shift;
    pmask |= 255u << shift;
    krem = sel[1];
    __syncthreads();
  }
  left = krem;
  return prefix;
}

// Top-k size and threshold from the tail count: k = floor(m + 1/2) clipped to [0, |T|].  With
// 0 < k < |T| the radix select gives the threshold key and how many positions equal to it to
// keep; k = |T| keeps every tail key (threshold +0.0, no limit); k = 0 keeps none.
template <int NT, class Count>
__device__ uint32_t topk_threshold(double m, double n_tail, int *hist, int *sel,
                                   int (*wtot)[NT / 64], int &tleft, uint32_t &st, Count &&count) {
  int64_t k = (int64_t)floor(m + 0.5);
  if (k < 0) k = 0;
  if (k >= (int64_t)n_tail) {
    k = (int64_t)n_tail;
    if (n_tail > 0.0) st |= EBD_ST_NO_EVICTION;
  }
  if (k > 0 && k < (int64_t)n_tail) return radix_kth<NT>((int)k, hist, sel, wtot, tleft, count);
  if (k > 0) {
    tleft = INT32_MAX;
    return 0u;
  }
  tleft = 0;
  return 0xffffffffu;
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// evict_select: lambda, mask, stored pi and index of every retained row, count, status
// ---------------------------------------------------------------------------------------------
// The retained K and V rows of one unit, gathered in order by the NT threads of its work-group
// from the index list (idxc) the work-group wrote: 16 lanes per 256-byte row, 8 rows per thread
// with all their loads in flight, the next rows' indices loaded ahead.  Rows past the end
// re-load the unit's first retained row and skip the store.
template <int NT>
__device__ __forceinline__ void gather_rows(const EvictLaunch &L, int64_t base, int64_t cbase,
                                            int64_t nkeep) {
  constexpr int kGRows = NT / 16, kGIt = 8;  // rows per pass, passes per round
  const int t = threadIdx.x, sub = t & 15, grow = t >> 4;
  const u32x4 *K4 = reinterpret_cast<const u32x4 *>(L.K);
  const u32x4 *V4 = reinterpret_cast<const u32x4 *>(L.V);
  u32x4 *Kc4 = reinterpret_cast<u32x4 *>(L.Kc);
  u32x4 *Vc4 = reinterpret_cast<u32x4 *>(L.Vc);
  auto load_idx = [&](int64_t r0, int32_t (&src)[kGIt]) {
#pragma unroll
    for (int k = 0; k < kGIt; ++k) {
      const int64_t r = r0 + grow + k * kGRows;
      src[k] = L.idxc[cbase + (r < nkeep ? r : 0)];
    }
  };
  int32_t src[kGIt];
  if (nkeep > 0) load_idx(0, src);
  for (int64_t r0 = 0; r0 < nkeep; r0 += kGRows * kGIt) {
    u32x4 kv[kGIt], vv[kGIt];
#pragma unroll
    for (int k = 0; k < kGIt; ++k) {
      const int64_t sr = (base + src[k]) * (kHeadDim / 8) + sub;
      kv[k] = __builtin_nontemporal_load(&K4[sr]);  // streamed once: no cache retention
      vv[k] = __builtin_nontemporal_load(&V4[sr]);
    }
    if (r0 + kGRows * kGIt < nkeep) load_idx(r0 + kGRows * kGIt, src);
#pragma unroll
    for (int k = 0; k < kGIt; ++k) {
      const int64_t r = r0 + grow + k * kGRows;
      if (r < nkeep) {
        const int64_t d = (cbase + r) * (kHeadDim / 8) + sub;
        __builtin_nontemporal_store(kv[k], &Kc4[d]);
        __builtin_nontemporal_store(vv[k], &Vc4[d]);
      }
    }
  }
}

// The start of a streamed unit's lambda iteration from its score histogram (every thread of the
// NT-thread work-group calls it; the histogram's counts are complete in hc).  hc becomes the
// counts' exclusive prefix and hm that of count x bin midpoint.  With the scores of every bin at
// its midpoint, g(lambda) = H + eps L + lambda S is evaluated at each bin's breakpoint 1 / mid
// (the bin and those above it clip at 1; the bins at or below eps / lambda, and the zero scores,
// clip at eps); g falls as the bin rises, and the piece just below the highest bin whose
// breakpoint still has g >= m is solved for lambda.  Returns `fallback` when no bin qualifies.
template <int NT>
__device__ __forceinline__ double hist_start(int *hc, float *hm, int *s_wc, float *s_ww, int &s_bin,
                                             double m, float eps, double n_zero, double fallback) {
  constexpr int NW = NT / 64;
  constexpr int PER = kHistBins / NT;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  auto mid = [](int b) { return __uint_as_float(((uint32_t)b << kHistShift) | (1u << (kHistShift - 1))); };
  __syncthreads();  // the counts are complete
  int ct = 0;
  float wt = 0.0f;  // the start is approximate: fp32 sums of count x midpoint suffice
  for (int i = 0; i < PER; ++i) {
    const int c = hc[PER * t + i];
    ct += c;
    wt = fmaf((float)c, mid(PER * t + i), wt);
  }
  // exclusive prefix of (ct, wt) over the threads: within the wave, then over the waves
  int ic = ct;
  float iw = wt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int xc = __shfl_up(ic, o);
    const float xw = __shfl_up(iw, o);
    if (lane >= o) {
      ic += xc;
      iw += xw;
    }
  }
  if (lane == 63) {
    s_wc[wv] = ic;
    s_ww[wv] = iw;
  }
  __syncthreads();
  int pc = 0, nc = 0;
  float pw = 0.0f;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    if (w < wv) {
      pc += s_wc[w];
      pw += s_ww[w];
    }
    nc += s_wc[w];
  }
  pc += ic - ct;
  pw += iw - wt;
  if (t == 0) s_bin = -1;
  for (int i = 0; i < PER; ++i) {  // in place: this thread's bins only
    const int b = PER * t + i, c = hc[b];
    hc[b] = pc;
    hm[b] = pw;
    pc += c;
    pw = fmaf((float)c, mid(b), pw);
  }
  __syncthreads();  // the prefixes of every bin are in place
  const double N = (double)nc;
  auto count = [&](int b) { return (b + 1 < kHistBins ? hc[b + 1] : nc) - hc[b]; };
  // g at the breakpoint of bin b (lambda_b = 1 / mid_b): H = bins >= b, L = bins below the bin
  // of eps mid_b (and the zero scores), S = the bins between
  auto piece = [&](int b, double &H, double &Lo, double &S) {
    const int be = (int)(__float_as_uint(eps * mid(b)) >> kHistShift);
    H = N - (double)hc[b];
    Lo = (double)hc[be] + n_zero;
    S = (double)hm[b] - (double)hm[be];
  };
  int best = -1;
  for (int i = 0; i < PER; ++i) {
    const int b = PER * t + i;
    if (count(b) == 0) continue;
    double H, Lo, S;
    piece(b, H, Lo, S);
    if (H + (double)eps * Lo + S / (double)mid(b) >= m) best = b;  // bins ascend: the last that qualifies
  }
  if (best >= 0) atomicMax(&s_bin, best);
  __syncthreads();
  const int b = s_bin;
  if (b < 0) return fallback;
  // just below the breakpoint the bin itself leaves H for the middle
  double H, Lo, S;
  piece(b, H, Lo, S);
  const int cb = count(b);
  H -= (double)cb;
  S += (double)cb * (double)mid(b);
  const double top = 1.0 / (double)mid(b);
  const double lam = S > 0.0 ? (m - H - (double)eps * Lo) / S : top;
  return (lam > 0.0 && lam <= top) ? lam : top;
}

template <int NT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4)))
void evict_select_kernel(EvictLaunch L) {
  extern __shared__ float s_sc[];
  __shared__ BlockRed<NT / 64> R;
  __shared__ float4 s_edge[2][NT / 64];  // per wave: the edges of a streamed Newton pass
  __shared__ int s_tot[2][NT / 64];
  __shared__ int s_hist[256];
  __shared__ int s_sel[2];
  __shared__ int s_hc[NT / 64];     // streamed units: per-wave histogram totals (counts, ...
  __shared__ float s_hw[NT / 64];   // ... and count x midpoint) for the histogram's prefix
  __shared__ int s_hb;              // the histogram bin where g crosses m
  int rbuf = 0;
  const int u = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t base = L.seq_off[u];
  const int64_t n = L.seq_off[u + 1] - base;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  if (n > L.max_rows || cap > (int64_t)L.copy_blocks * kCopyRows) {
    // larger than the launch was planned for: touch nothing of this unit
    if (t == 0) {
      L.count[u] = 0;
      L.status[u] = EBD_ST_BAD_LAYOUT;
      if (L.lambda_out) L.lambda_out[u] = 0.0f;
    }
    return;
  }
  const int64_t nprot = min(n, (int64_t)L.n_sink + (int64_t)L.n_recent);
  const double f = L.budget_per_unit ? (double)L.budget_per_unit[u] : (double)L.budget_frac;
  const double m = f * (double)n - (double)nprot;
  const float eps = L.pi_min;
  const float *sc = L.scores + base;
  const int64_t ngroups = (n + 3) / 4;
  const int64_t tail_lo = L.n_sink, tail_hi = n - (int64_t)L.n_recent;  // T = [tail_lo, tail_hi)
  const bool staged = L.stage_rows > 0;
  const bool uniform = L.design == EBD_DESIGN_UNIFORM;  // tail scores taken as 1, not read
  const bool vec = ((base & 3) == 0);  // 16-byte aligned score groups

  // Raw scores of group gi (0 past the end).
  auto load_raw = [&](int64_t gi) -> float4 {
    const int64_t i = 4 * gi;
    if (uniform) return make_float4(1.0f, 1.0f, 1.0f, 1.0f);
    if (vec && i + 3 < n) return reinterpret_cast<const float4 *>(sc)[gi];
    float4 r;
    r.x = i < n ? sc[i] : 0.0f;
    r.y = i + 1 < n ? sc[i + 1] : 0.0f;
    r.z = i + 2 < n ? sc[i + 2] : 0.0f;
    r.w = i + 3 < n ? sc[i + 3] : 0.0f;
    return r;
  };
  // Cleaned tail scores of group gi; positions outside T (protected or past the end) read -1.
  auto tail4 = [&](int64_t gi, float4 raw, uint32_t &bad) -> float4 {
    float v[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t i = 4 * gi + j;
      const float c = clean_score(v[j], bad);
      v[j] = (i < n && i >= tail_lo && i < tail_hi) ? c : -1.0f;
    }
    return make_float4(v[0], v[1], v[2], v[3]);
  };
  auto group = [&](int64_t gi) -> float4 {
    if (staged) return reinterpret_cast<const float4 *>(s_sc)[gi];
    uint32_t dummy = 0;
    return tail4(gi, load_raw(gi), dummy);
  };

  // Streamed units: LDS holds the histogram of the positive tail scores (counts, later their
  // exclusive prefix) and the prefix of count x bin midpoint.
  const bool hist = !staged && L.design != EBD_DESIGN_TOPK;
  int *s_hcnt = reinterpret_cast<int *>(s_sc);
  float *s_hmid = s_sc + kHistBins;
  if (hist) {
    for (int b = t; b < kHistBins; b += NT) s_hcnt[b] = 0;
    __syncthreads();
  }

  // Pass 0: read (and stage) the scores; tail statistics; bad-score flag.  Four groups per
  // thread are loaded before any is used so their latencies overlap.
  uint32_t bad = 0;
  int c_tail = 0, c_pos = 0;
  double s_sum = 0.0;
  float s_max = 0.0f, s_minp = INFINITY;
  for (int64_t g0 = 0; g0 < ngroups; g0 += NT * 4) {
    float4 raw[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) raw[q] = load_raw(g0 + NT * q + t);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t gi = g0 + NT * q + t;
      if (gi >= ngroups) break;
      // every position is checked for bad values, protected ones included (positions past the
      // end read 0, which is not bad)
      const float4 tv = tail4(gi, raw[q], bad);
      const float v[4] = {tv.x, tv.y, tv.z, tv.w};
      float gsum = 0.0f;  // at most 4 terms in fp32, then the running sum in fp64
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool tail = v[j] >= 0.0f, pos = v[j] > 0.0f;
        c_tail += tail ? 1 : 0;
        c_pos += pos ? 1 : 0;
        gsum += tail ? v[j] : 0.0f;
        s_minp = fminf(s_minp, pos ? v[j] : INFINITY);
        s_max = fmaxf(s_max, v[j]);
        if (hist && pos) atomicAdd(&s_hcnt[__float_as_uint(v[j]) >> kHistShift], 1);
      }
      s_sum += (double)gsum;
      if (staged) reinterpret_cast<float4 *>(s_sc)[gi] = tv;
    }
  }
  double n_tail = (double)c_tail, n_pos = (double)c_pos;
  block_sum3(n_tail, n_pos, s_sum, R, rbuf);
  block_minmax(s_max, s_minp, R, rbuf);
  {
    double b0 = (double)bad, z1 = 0.0, z2 = 0.0;
    block_sum3(b0, z1, z2, R, rbuf);
    bad = b0 > 0.0 ? 1u : 0u;
  }
  uint32_t st = bad ? EBD_ST_BAD_SCORE : 0u;

  const bool topk = L.design == EBD_DESIGN_TOPK;
  // Top-k: tkey is the k-th largest tail key and tleft how many positions equal to it to keep.
  uint32_t tkey = 0xffffffffu;
  int tleft = 0;
  if (topk) {
    tkey = topk_threshold<NT>(
        m, n_tail, s_hist, s_sel, s_tot, tleft, st, [&](uint32_t prefix, uint32_t pmask, int shift) {
          for (int64_t gi = t; gi < ngroups; gi += NT) {
            const float4 s4 = group(gi);
            const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const uint32_t key = __float_as_uint(sv[j]);
              if (sv[j] >= 0.0f && (key & pmask) == prefix)
                atomicAdd(&s_hist[(key >> shift) & 255u], 1);
            }
          }
        });
  }
  const TailStats ts{n_tail, n_pos, s_sum, s_max, s_minp};
  // One evaluation of g's pieces at lambda = lf over the unit (LDS when staged; streamed scores
  // with four groups per thread in flight).  The loops are uniform over the work-group, so the
  // counts are wave ballots; slots past the unit read -1 like every slot outside the tail.  A
  // streamed pass, whose cost is the re-read of the scores, also reports the piece's edges so
  // that the solve can skip its confirming pass.
  auto newton_pass = [&](float lf, double &dH, double &dL, double &dS, PieceEdges &edges) {
    int H = 0, Lo = 0;  // wave totals
    float Sm = 0.0f;
    float h_min = INFINITY, m_max = 0.0f, m_min = INFINITY, l_max = 0.0f;
    auto add = [&](float4 s4, bool track) {
      const float sv[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p = lf * sv[j];
        const bool hb = p >= 1.0f, lb = p <= eps;
        H += __popcll(__ballot(hb));
        Lo += __popcll(__ballot(lb));
        const float mid = (hb || lb) ? 0.0f : sv[j];
        Sm += mid;
        if (track) {
          h_min = fminf(h_min, hb ? sv[j] : INFINITY);
          m_max = fmaxf(m_max, mid);
          m_min = fminf(m_min, (hb || lb) ? INFINITY : sv[j]);
          l_max = fmaxf(l_max, lb ? sv[j] : 0.0f);
        }
      }
      asm volatile("" : "+s"(H), "+s"(Lo));  // counted now: no lane masks held across groups
    };
    const float4 none = make_float4(-1.0f, -1.0f, -1.0f, -1.0f);
    int64_t slots = 0;  // slots visited by the work-group
    if (staged) {
      for (int64_t g0 = 0; g0 < ngroups; g0 += NT) {
        add(g0 + t < ngroups ? group(g0 + t) : none, false);
        slots += 4 * NT;
      }
    } else {
      for (int64_t g0 = 0; g0 < ngroups; g0 += NT * 4) {
        float4 raw[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) raw[q] = load_raw(g0 + NT * q + t);  // 0 past the end
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t dummy = 0;
          add(tail4(g0 + NT * q + t, raw[q], dummy), true);  // -1 past the end
        }
        slots += 16 * NT;
      }
    }
    edges.valid = !staged;
    if (!staged) {  // the edges over the work-group, published by the barrier of the sums below
      h_min = wave_min(h_min);
      m_max = wave_max(m_max);
      m_min = wave_min(m_min);
      l_max = wave_max(l_max);
      if (lane == 0) s_edge[rbuf][wv] = make_float4(h_min, m_max, m_min, l_max);
    }
    const int eb = rbuf;
    dH = (double)H;
    dL = (double)Lo;
    dS = Sm;
    block_sum_wave2(dH, dL, dS, R, rbuf);
    dL -= (double)slots - n_tail;  // every visited slot is either in the tail or not
    if (!staged) {
      edges.h_min = edges.m_min = INFINITY;
      edges.m_max = edges.l_max = 0.0f;
#pragma unroll
      for (int w = 0; w < NT / 64; ++w) {
        const float4 e4 = s_edge[eb][w];
        edges.h_min = fminf(edges.h_min, e4.x);
        edges.m_max = fmaxf(edges.m_max, e4.y);
        edges.m_min = fminf(edges.m_min, e4.z);
        edges.l_max = fmaxf(edges.l_max, e4.w);
      }
    }
  };
  double lam = 0.0;
  if (!topk && !lambda_boundary(ts, m, eps, L.pi_mode, st, lam)) {
    const double lo0 = (double)eps / (double)s_max, hi0 = 1.0 / (double)s_minp;
    double start = m / s_sum;
    if (hist) start = hist_start<NT>(s_hcnt, s_hmid, s_hc, s_hw, s_hb, m, eps, n_tail - n_pos, start);
    lam = newton_lambda(m, eps, lo0, hi0, fmin(fmax(start, lo0), hi0), newton_pass);
  }
  const float lamf = (float)lam;

  // Mask and in-order write of the retained rows' pi and positions, Q groups of 4 tokens per
  // thread at a time (a superblock of 4 Q NT tokens; group gi = g0 + NT q + t, so positions
  // ascend with (q, wave, lane, j)): ranks from per-(q, j) ballots plus one exchange of the
  // per-(q, wave) counts; the systematic design's weight prefix and the top-k design's ranks of
  // the threshold key take one exchange more.  Streamed scores: the next superblock's groups
  // load while this one is masked.
  constexpr int Q = 2;
  constexpr int NW = NT / 64;
  __shared__ int s_rk[2][Q][NW];
  __shared__ int s_eqx[2][Q][NW];
  __shared__ unsigned long long s_sys[2][Q][NW];
  const uint64_t sd = L.seed_per_unit ? L.seed_per_unit[u] : L.seed;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int design = L.design;
  // systematic design: one start per unit and the cumulative integer weight so far
  const uint32_t sys_start =
      philox4x32_10(make_uint4(0u, (uint32_t)u, L.epoch, kSystematicTag), (uint32_t)sd,
                    (uint32_t)(sd >> 32)).x;
  uint64_t csum = 0;
  int64_t eq_seen = 0;  // top-k: tail positions equal to the threshold key so far
  int64_t rank0 = 0;
  float4 nxt[Q];
  if (!staged) {
#pragma unroll
    for (int q = 0; q < Q; ++q) nxt[q] = load_raw((int64_t)NT * q + t);
  }
  int par = 0;
  for (int64_t g0 = 0; g0 < ngroups; g0 += (int64_t)Q * NT, par ^= 1) {
    float sv[Q][4], p[Q][4];
    bool inr[Q][4], keep[Q][4];
    {
      float4 cur[Q];
      if (!staged) {
#pragma unroll
        for (int q = 0; q < Q; ++q) {
          cur[q] = nxt[q];
          nxt[q] = load_raw(g0 + (int64_t)NT * (Q + q) + t);  // zeros past the end
        }
      }
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int64_t gi = g0 + (int64_t)NT * q + t;
        uint32_t dummy = 0;
        const float4 s4 = gi >= ngroups ? make_float4(-1.0f, -1.0f, -1.0f, -1.0f)
                                         : (staged ? group(gi) : tail4(gi, cur[q], dummy));
        const float v[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sv[q][j] = v[j];
          inr[q][j] = 4 * gi + j < n;
          p[q][j] = (inr[q][j] && !topk) ? token_pi(v[j] >= 0.0f, v[j], lamf, eps) : 1.0f;
          keep[q][j] = false;
        }
      }
    }
    if (design == EBD_DESIGN_SYSTEMATIC) {
      uint64_t a[Q][4], pre[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        uint64_t tsum = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          a[q][j] = inr[q][j] ? pi_weight(p[q][j]) : 0u;
          tsum += a[q][j];
        }
        const uint64_t incl = wave_scan_u64(tsum);
        pre[q] = incl - tsum;
        if (lane == 63) s_sys[par][q][wv] = incl;
      }
      __syncthreads();
      uint64_t acc = csum;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        uint64_t C = acc + pre[q];
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const uint64_t c = s_sys[par][q][w];
          C += w < wv ? c : 0u;
          acc += c;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint64_t Cn = C + a[q][j];
          keep[q][j] = inr[q][j] && points_below(Cn, sys_start) != points_below(C, sys_start);
          C = Cn;
        }
      }
      csum = acc;
    } else if (topk) {
      // tail positions at the threshold key are kept in position order while tleft lasts
      int eb[Q];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        int ebefore = 0, etot = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint64_t bal = __ballot(inr[q][j] && sv[q][j] >= 0.0f &&
                                        __float_as_uint(sv[q][j]) == tkey);
          ebefore += __popcll(bal & below);
          etot += __popcll(bal);
        }
        eb[q] = ebefore;
        if (lane == 0) s_eqx[par][q][wv] = etot;
      }
      __syncthreads();
      int64_t acc = eq_seen;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        // rank of this thread's first equal position among the unit's equal positions
        int64_t er = acc + eb[q];
#pragma unroll
        for (int w = 0; w < NW; ++w) {
          const int c = s_eqx[par][q][w];
          er += w < wv ? c : 0;
          acc += c;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool tail = sv[q][j] >= 0.0f;
          bool sel = false;
          if (inr[q][j] && tail) {
            const uint32_t key = __float_as_uint(sv[q][j]);
            if (key > tkey) sel = true;
            else if (key == tkey) sel = er++ < (int64_t)tleft;
          }
          p[q][j] = (!inr[q][j] || !tail) ? 1.0f : (sel ? 1.0f : 0.0f);
          keep[q][j] = inr[q][j] && (!tail || sel);
        }
      }
      eq_seen = acc;
    } else {
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int64_t gi = g0 + (int64_t)NT * q + t;
        if (gi >= ngroups) continue;
        const uint4 x = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)u, L.epoch, kPhiloxTag),
                                      (uint32_t)sd, (uint32_t)(sd >> 32));
        const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) keep[q][j] = inr[q][j] && keep_token(xw[j], p[q][j]);
      }
    }
    if (L.pi_full) {
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int64_t gi = g0 + (int64_t)NT * q + t;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (inr[q][j]) L.pi_full[base + 4 * gi + j] = p[q][j];
      }
    }
    int before[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      int b = 0, wtot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint64_t bal = __ballot(keep[q][j]);
        b += __popcll(bal & below);
        wtot += __popcll(bal);
      }
      before[q] = b;
      if (lane == 0) s_rk[par][q][wv] = wtot;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int64_t gi = g0 + (int64_t)NT * q + t;
      int64_t r = rank0 + before[q];
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int c = s_rk[par][q][w];
        r += w < wv ? c : 0;
        rank0 += c;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (keep[q][j]) {
          if (r < cap) {
            L.pic[cbase + r] = p[q][j];
            L.idxc[cbase + r] = (int32_t)(4 * gi + j);
          }
          ++r;
        }
      }
    }
  }
  if (t == 0) {
    if (rank0 > cap) st |= EBD_ST_CAP_OVERFLOW;
    L.count[u] = (int32_t)rank0;
    L.status[u] = st;
    if (L.lambda_out) L.lambda_out[u] = lamf;
  }

  // The unit's retained K and V rows, gathered by the same work-group from the index list it
  // has just written (visible to it after the barrier).  Units of this kernel run in many
  // generations, so one unit's gather overlaps other units' selection.
  __syncthreads();
  gather_rows<NT>(L, base, cbase, min(rank0, cap));
}

// ---------------------------------------------------------------------------------------------
// evict_select_reg: the same selection for units of at most 512 G4 tokens (G4 <= 12, so up to
// 6144 tokens; longer units take evict_select), two waves per unit
// with the scores in registers (G4 groups of 4 tokens per thread; group gi = 128 q + thread, so
// loads are coalesced and positions ascend with (q, wave, lane, j)).  Without LDS staging every
// unit of a large batch is resident at once.  Each reduction or prefix costs one barrier: the
// mask bits of the whole unit are drawn first, then one exchange of the per-(q, wave) counts
// gives every retained row its output slot.
// ---------------------------------------------------------------------------------------------
template <int G4>
__global__ __launch_bounds__(kSelectRegThreads) __attribute__((amdgpu_waves_per_eu(4)))
void evict_select_reg_kernel(EvictLaunch L) {
  constexpr int NT = kSelectRegThreads, NW = NT / 64;
  __shared__ double s_d[2][NW][3];
  __shared__ float s_f[NW][2];
  __shared__ int s_i[NW][3];
  __shared__ int s_cnt[G4][NW];
  __shared__ unsigned long long s_c64[G4][NW];
  __shared__ int s_hist[256];
  __shared__ int s_sel[2];
  __shared__ int s_wtot[2][NW];
  const int u = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int64_t base = L.seq_off[u];
  const int64_t n64 = L.seq_off[u + 1] - base;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  if (n64 > L.max_rows || n64 > 512 * G4 || cap > (int64_t)L.copy_blocks * kCopyRows) {
    if (t == 0) {
      L.count[u] = 0;
      L.status[u] = EBD_ST_BAD_LAYOUT;
      if (L.lambda_out) L.lambda_out[u] = 0.0f;
    }
    return;
  }
  const int n = (int)n64;
  const int64_t nprot = min(n64, (int64_t)L.n_sink + (int64_t)L.n_recent);
  const double f = L.budget_per_unit ? (double)L.budget_per_unit[u] : (double)L.budget_frac;
  const double m = f * (double)n - (double)nprot;
  const float eps = L.pi_min;
  // T = [tail_lo, tail_hi), as 32-bit positions (the unit has at most 512 G4 tokens)
  const int tail_lo = (int)min((int64_t)L.n_sink, n64);
  const int tail_hi = (int)max(n64 - (int64_t)L.n_recent, (int64_t)0);
  const int design = L.design;
  const bool uniform = design == EBD_DESIGN_UNIFORM;  // tail scores taken as 1, not read
  const bool topk = design == EBD_DESIGN_TOPK;
  const bool vec = ((base & 3) == 0);
  const float *sc = L.scores + base;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int rb = 0;

  // Unit totals of two wave-uniform counts and a per-lane fp32 partial (summed in fp64); all
  // threads get them.
  auto bsum = [&](int a, int b, float c, double &A, double &B, double &C) {
    const double cw = wave_sum((double)c);
    if (lane == 0) {
      s_d[rb][wv][0] = (double)a;
      s_d[rb][wv][1] = (double)b;
      s_d[rb][wv][2] = cw;
    }
    __syncthreads();
    A = B = C = 0.0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      A += s_d[rb][w][0];
      B += s_d[rb][w][1];
      C += s_d[rb][w][2];
    }
    rb ^= 1;
  };

  // Scores: cleaned tail scores, -1 outside the tail (protected or past the end); every position
  // is checked for bad values, protected ones included.
  float sv[G4][4];
  int n_tail = 0, n_pos = 0, n_bad = 0;  // wave totals (ballots)
  float s_sum = 0.0f, s_max = 0.0f, s_minp = INFINITY;
  {
    // raw buffer loads bounded by the unit: positions past its end read 0
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(sc, (uint32_t)(4 * n));
    float4 raw[G4];
    if (uniform) {
#pragma unroll
      for (int q = 0; q < G4; ++q) raw[q] = make_float4(1.0f, 1.0f, 1.0f, 1.0f);
    } else if (vec) {
#pragma unroll
      for (int q = 0; q < G4; ++q)
        raw[q] = __builtin_bit_cast(
            float4, __builtin_amdgcn_raw_buffer_load_b128(rs, 16u * (uint32_t)(q * NT + t), 0, 0));
    } else {
#pragma unroll
      for (int q = 0; q < G4; ++q) {
        const uint32_t off = 16u * (uint32_t)(q * NT + t);
        raw[q].x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
        raw[q].y = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + 4, 0, 0));
        raw[q].z = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + 8, 0, 0));
        raw[q].w = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + 12, 0, 0));
      }
    }
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      const float rv[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = 4 * (q * NT + t) + j;
        uint32_t b = 0;
        const float c = clean_score(rv[j], b);
        const bool tail = i < n && i >= tail_lo && i < tail_hi;
        sv[q][j] = tail ? c : -1.0f;
        n_bad += __popcll(__ballot(i < n && b));
        n_tail += __popcll(__ballot(tail));
        n_pos += __popcll(__ballot(tail && c > 0.0f));
        s_sum += tail ? c : 0.0f;
        s_max = fmaxf(s_max, tail ? c : 0.0f);
        s_minp = fminf(s_minp, (tail && c > 0.0f) ? c : INFINITY);
      }
      asm volatile("" : "+s"(n_bad), "+s"(n_tail), "+s"(n_pos));  // counted now, masks dropped
      __builtin_amdgcn_sched_barrier(0);  // one group at a time: bounded register pressure
    }
  }
  // From here on a slot's class is read from its value alone: hiding how it was formed keeps
  // the compiler from carrying 48 per-slot lane masks through every phase instead.
#pragma unroll
  for (int q = 0; q < G4; ++q)
#pragma unroll
    for (int j = 0; j < 4; ++j) asm volatile("" : "+v"(sv[q][j]));
  double d_tail, d_pos, d_sum;
  {
    s_max = wave_max(s_max);
    s_minp = wave_min(s_minp);
    if (lane == 0) {
      s_i[wv][0] = n_bad;
      s_f[wv][0] = s_max;
      s_f[wv][1] = s_minp;
    }
    bsum(n_tail, n_pos, s_sum, d_tail, d_pos, d_sum);  // its barrier also publishes s_i, s_f
    n_bad = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      n_bad += s_i[w][0];
      s_max = fmaxf(s_max, s_f[w][0]);
      s_minp = fminf(s_minp, s_f[w][1]);
    }
    n_tail = (int)d_tail;
  }
  const uint32_t bad = n_bad > 0 ? 1u : 0u;
  uint32_t st = bad ? EBD_ST_BAD_SCORE : 0u;

  uint32_t tkey = 0xffffffffu;
  int tleft = 0;
  if (topk) {
    tkey = topk_threshold<NT>(m, (double)n_tail, s_hist, s_sel, s_wtot, tleft, st,
                              [&](uint32_t prefix, uint32_t pmask, int shift) {
#pragma unroll
                                for (int q = 0; q < G4; ++q)
#pragma unroll
                                  for (int j = 0; j < 4; ++j) {
                                    const uint32_t key = __float_as_uint(sv[q][j]);
                                    if (sv[q][j] >= 0.0f && (key & pmask) == prefix)
                                      atomicAdd(&s_hist[(key >> shift) & 255u], 1);
                                  }
                              });
  }
  // Slots outside the tail hold -1: lf (-1) <= eps counts them in L, so L is corrected by their
  // number (every slot of the unit's G4 x 4 x NT is one or the other).
  const double n_out = (double)(4 * G4 * NT) - (double)n_tail;
  const TailStats ts{d_tail, d_pos, d_sum, s_max, s_minp};
  const double lam =
      topk ? 0.0
           : solve_lambda(ts, m, eps, L.pi_mode, st, [&](float lf, double &dH, double &dL, double &dS,
                                                          PieceEdges &edges) {
               edges.valid = false;
               int H = 0, Lo = 0;  // wave totals (ballots)
               float Sm = 0.0f;
#pragma unroll
               for (int q = 0; q < G4; ++q) {
#pragma unroll
                 for (int j = 0; j < 4; ++j) {
                   const float p = lf * sv[q][j];
                   const bool hb = p >= 1.0f, lb = p <= eps;
                   H += __popcll(__ballot(hb));
                   Lo += __popcll(__ballot(lb));
                   Sm += (hb || lb) ? 0.0f : sv[q][j];
                 }
                 // counted per group: the compiler would otherwise keep 2 x 4 G4 lane masks until
                 // the one lane that publishes the totals
                 asm volatile("" : "+s"(H), "+s"(Lo));
               }
               bsum(H, Lo, Sm, dH, dL, dS);
               dL -= n_out;
             });
  float lamf = (float)lam;

  // pi of slot (q, j): 1 outside the tail; the clipped lambda s in the tail (top-k: 1 or 0 by
  // the keep bit).
  auto slot_pi = [&](int q, int j, bool keep) -> float {
    if (!(sv[q][j] >= 0.0f)) return 1.0f;
    if (topk) return keep ? 1.0f : 0.0f;
    return token_pi(true, sv[q][j], lamf, eps);
  };
  // The per-slot range tests are taken again in each phase: kept as lane masks across the
  // phases they would crowd the scalar registers.
  int nn = n, tb = 4 * t;  // this thread's first position, as an opaque value
  asm volatile("" : "+s"(nn), "+v"(tb));
  uint64_t keep = 0;  // bit 4 q + j
  const uint64_t sd = L.seed_per_unit ? L.seed_per_unit[u] : L.seed;
  if (design == EBD_DESIGN_SYSTEMATIC) {
    // integer weights ceil(pi 2^32) in position order against one start per unit; the wave
    // scans are taken twice (totals, then prefixes) rather than kept across the exchange
    const uint32_t start =
        philox4x32_10(make_uint4(0u, (uint32_t)u, L.epoch, kSystematicTag), (uint32_t)sd,
                      (uint32_t)(sd >> 32)).x;
    auto weights = [&](int q, uint64_t (&a)[4]) {
      uint64_t tsum = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a[j] = tb + 4 * NT * q + j < nn ? pi_weight(slot_pi(q, j, false)) : 0u;
        tsum += a[j];
      }
      return tsum;
    };
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      uint64_t a[4];
      const uint64_t incl = wave_scan_u64(weights(q, a));
      if (lane == 63) s_c64[q][wv] = incl;
    }
    __syncthreads();
    asm volatile("" : "+v"(lamf));  // recompute pi here rather than keep every slot's value live
    uint64_t acc = 0;
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      uint64_t a[4];
      const uint64_t tsum = weights(q, a);
      uint64_t C = acc + wave_scan_u64(tsum) - tsum;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const uint64_t c = s_c64[q][w];
        C += w < wv ? c : 0u;
        acc += c;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint64_t Cn = C + a[j];
        if (a[j] != 0u && points_below(Cn, start) != points_below(C, start))
          keep |= 1ull << (4 * q + j);
        C = Cn;
      }
    }
  } else if (topk) {
    // tail positions at the threshold key are kept in position order while tleft lasts; the
    // ballots are taken twice (totals, then ranks) rather than kept across the exchange
    auto eq_ballot = [&](int q, int j) {
      return __ballot(sv[q][j] >= 0.0f && __float_as_uint(sv[q][j]) == tkey);
    };
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      int etot = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) etot += __popcll(eq_ballot(q, j));
      if (lane == 0) s_cnt[q][wv] = etot;
    }
    __syncthreads();
    int acc = 0;
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      int er = acc;
#pragma unroll
      for (int j = 0; j < 4; ++j) er += __popcll(eq_ballot(q, j) & below);
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const int c = s_cnt[q][w];
        er += w < wv ? c : 0;
        acc += c;
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (!(sv[q][j] >= 0.0f)) {
          if (tb + 4 * NT * q + j < nn) keep |= 1ull << (4 * q + j);  // protected
          continue;
        }
        const uint32_t key = __float_as_uint(sv[q][j]);
        bool sel = key > tkey;
        if (key == tkey) sel = er++ < tleft;
        if (sel) keep |= 1ull << (4 * q + j);
      }
    }
    __syncthreads();  // s_cnt is reused for the output ranks
  } else {
#pragma unroll
    for (int q = 0; q < G4; ++q) {
      const int gi = (tb >> 2) + NT * q;  // group index: positions 4 gi .. 4 gi + 3
      if (4 * gi >= nn) continue;
      const uint4 x = philox4x32_10(make_uint4((uint32_t)gi, (uint32_t)u, L.epoch, kPhiloxTag),
                                    (uint32_t)sd, (uint32_t)(sd >> 32));
      const uint32_t xw[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (4 * gi + j < nn && keep_token(xw[j], slot_pi(q, j, false)))
          keep |= 1ull << (4 * q + j);
    }
  }

  // Output slots: per-(q, wave) retained counts, one exchange, then every retained row writes its
  // pi and position; the unit's full pi vector on request.
#pragma unroll
  for (int q = 0; q < G4; ++q) {
    int wtot = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) wtot += __popcll(__ballot((keep >> (4 * q + j)) & 1ull));
    if (lane == 0) s_cnt[q][wv] = wtot;
  }
  __syncthreads();
  asm volatile("" : "+v"(lamf), "+v"(tb));  // as above: recomputed per slot for the output
  // buffer stores: a slot at or past the capacity (or a dropped row, sent past it) writes nothing
  const uint32_t capw = (uint32_t)min(cap, (int64_t)INT32_MAX / 4);
  const __amdgpu_buffer_rsrc_t rpi = make_rsrc(L.pic + cbase, 4u * capw);
  const __amdgpu_buffer_rsrc_t rix = make_rsrc(L.idxc + cbase, 4u * capw);
  const __amdgpu_buffer_rsrc_t rfull = make_rsrc(L.pi_full ? L.pi_full + base : nullptr,
                                                 L.pi_full ? 4u * (uint32_t)n : 0u);
  int total = 0;  // running count of the rows before block q, then the unit's count
#pragma unroll
  for (int q = 0; q < G4; ++q) {
    int r = total;
#pragma unroll
    for (int j = 0; j < 4; ++j) r += __popcll(__ballot((keep >> (4 * q + j)) & 1ull) & below);
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int c = s_cnt[q][w];
      r += w < wv ? c : 0;
      total += c;
    }
    float pv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool kj = (keep >> (4 * q + j)) & 1ull;
      pv[j] = slot_pi(q, j, kj);
      const uint32_t off = kj ? 4u * (uint32_t)r : 0xfffffff0u;
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, pv[j]), rpi, off, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32((uint32_t)(tb + 4 * NT * q + j), rix, off, 0, 0);
      r += kj ? 1 : 0;
    }
    if (L.pi_full) {
      if (vec) {
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(u32x4, make_float4(pv[0], pv[1], pv[2], pv[3])), rfull,
            4u * (uint32_t)(tb + 4 * NT * q), 0, 0);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, pv[j]), rfull,
                                                4u * (uint32_t)(tb + 4 * NT * q + j), 0, 0);
      }
    }
  }
  if (t == 0) {
    if (total > cap) st |= EBD_ST_CAP_OVERFLOW;
    L.count[u] = total;
    L.status[u] = st;
    if (L.lambda_out) L.lambda_out[u] = lamf;
  }
}

// ---------------------------------------------------------------------------------------------
// evict_copy: gather the retained K and V rows in order
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kCopyThreads) void evict_copy_kernel(EvictLaunch L) {
  const int64_t bid = blockIdx.x;
  const int blk = (int)(bid % L.copy_blocks);
  const int u = (int)(bid / L.copy_blocks);
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int64_t nkeep = min((int64_t)L.count[u], cap);
  const int64_t r0 = (int64_t)blk * kCopyRows;
  if (r0 >= nkeep || (L.seq_off[u + 1] - L.seq_off[u]) > L.max_rows) return;
  const int64_t base = L.seq_off[u];
  const int sub = threadIdx.x & 15;
  const int row = threadIdx.x >> 4;
  constexpr int kPass = kCopyThreads / 16;  // rows per pass
  constexpr int kIter = kCopyRows / kPass;  // passes per block
  const u32x4 *K4 = reinterpret_cast<const u32x4 *>(L.K);
  const u32x4 *V4 = reinterpret_cast<const u32x4 *>(L.V);
  u32x4 *Kc4 = reinterpret_cast<u32x4 *>(L.Kc);
  u32x4 *Vc4 = reinterpret_cast<u32x4 *>(L.Vc);
  // Rows past the end load a valid row (the block's first) and skip the store, so every load
  // is unconditional and all of a thread's loads are in flight together.
  int32_t src[kIter];
  bool ok[kIter];
#pragma unroll
  for (int k = 0; k < kIter; ++k) {
    const int64_t r = r0 + row + k * kPass;
    ok[k] = r < nkeep;
    src[k] = L.idxc[cbase + (ok[k] ? r : r0)];
  }
  u32x4 kv[kIter], vv[kIter];
#pragma unroll
  for (int k = 0; k < kIter; ++k) {
    const int64_t s = (base + src[k]) * (kHeadDim / 8) + sub;
    kv[k] = __builtin_nontemporal_load(&K4[s]);  // streamed once: no cache retention
    vv[k] = __builtin_nontemporal_load(&V4[s]);
  }
#pragma unroll
  for (int k = 0; k < kIter; ++k) {
    if (ok[k]) {
      const int64_t d = (cbase + r0 + row + k * kPass) * (kHeadDim / 8) + sub;
      __builtin_nontemporal_store(kv[k], &Kc4[d]);
      __builtin_nontemporal_store(vv[k], &Vc4[d]);
    }
  }
}

// The eight-wave evict_select (which also gathers the rows) takes units longer than the register
// kernel holds, and units whose capacity is under a sixth of their length: with few rows to
// gather, its selection overlapping other units' gathers wins over the register kernel plus a
// copy launch (measured on 6144-token units: 240 against 261 us at a 10% budget, 571 against
// 561 us at 25%).
bool evict_select_gathers(const EvictLaunch &L) {
  return (L.max_rows + 511) / 512 > 12 || (int64_t)L.copy_blocks * kCopyRows * 6 < L.max_rows;
}

hipError_t launch_evict_select(const EvictLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)L.U), reg(kSelectRegThreads);
  const int64_t g4 = (L.max_rows + 511) / 512;  // groups of 4 tokens per thread (two waves)
  if (evict_select_gathers(L)) {
    // eight waves per unit, two units per CU: scores staged in LDS (up to 64 KB per unit) or,
    // for longer units, streamed from memory on every pass
    const size_t lds = L.stage_rows > 0 ? (size_t)((L.stage_rows + 3) / 4) * 16
                                         : (size_t)kHistBins * (sizeof(int) + sizeof(float));
    hipLaunchKernelGGL(evict_select_kernel<kSelectThreads>, grid, dim3(kSelectThreads), lds, s, L);
  } else if (g4 <= 2) hipLaunchKernelGGL(evict_select_reg_kernel<2>, grid, reg, 0, s, L);
  else if (g4 <= 4) hipLaunchKernelGGL(evict_select_reg_kernel<4>, grid, reg, 0, s, L);
  else if (g4 <= 8) hipLaunchKernelGGL(evict_select_reg_kernel<8>, grid, reg, 0, s, L);
  else hipLaunchKernelGGL(evict_select_reg_kernel<12>, grid, reg, 0, s, L);
  return hipGetLastError();
}

hipError_t launch_evict_copy(const EvictLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)L.U * L.copy_blocks)), block(kCopyThreads);
  hipLaunchKernelGGL(evict_copy_kernel, grid, block, 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
