// attend.hip -- certified decode attention over the retained rows on gfx950.
//
// Per (unit, query head h), over the retained set S (Sec. 3.3 eq. (3), Theorem 2; Sec. 3.4 eq. (4)),
// in base-2 logits (l2 = l log2 e):
//   l2_j = scale log2e q_h.k_j - log2 pi_j           (Hajek weight a_j / pi_j as a logit offset)
//   w_j = 2^(l2_j - m),  m = running max              (online softmax)
//   yhat = sum w v / sum w,   ln Nhat = m ln 2 + ln sum w
//   c_j = (1 - pi_j) w_j^2 = (1 - pi)/pi^2 a^2 2^{-2m}: Vhat = sum c |v - yhat|^2 / (sum w)^2,
//     accumulated in one pass as C2 - 2 yhat.Cv + |yhat|^2 C0 with C0 = sum c, Cv = sum c v,
//     C2 = sum c |v|^2 (the 2^{-2m} factors cancel against (sum w)^2)
//   b = max_j sqrt(1 - pi_j) w_j |v_j - yhat| / sum w  (exact: candidates + bound check)
//
// attend_split (one work-group of four waves per (unit, split of the retained rows)):
//   Each wave walks 16-row tiles with the next tile's loads in flight while the current one is
//   computed.  q.k runs on MFMA (16x16x32 bf16, exact products, fp32 sums): A = K tile (16 rows x
//   32 dims per k-block, loaded straight from HBM in operand layout), B = [q_0 .. q_{GB-1},
//   q_0 .. q_{GB-1}, 0 ..] (16 columns).  Each lane then holds 4 rows x 1 column of logits;
//   columns < GB become weights w, columns GB..2GB-1 (same logits) become variance weights c.
//   f32 16x16x4 MFMAs then form o = sum w v (rows < GB) and Cv = sum c v (rows GB..2GB-1)
//   together, with V in its natural row-major layout (no transpose, exact fp32 products).
//   Range-term candidates: every weight lane keeps its four largest g^2 |v|^2 (g^2 = (1 - pi) w^2)
//   among its rows, plus the maxima of g^2 |v|^2 and of g^2 over what it dropped; the
//   work-group stores the 32 largest per head, their largest |v| and the non-candidate maxima.
//   The running max m moves lazily (only by jumps of more than 2^8 in weight).
// attend_finalize (one wave per (unit, query head)): log-sum-exp combine of the split records,
//   yhat, Vhat, ln Nhat, the exact range term b (only candidates whose bound can still win are
//   re-read; a split is rescanned only if its non-candidate bound cannot exclude a larger term)
//   and the radius r.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float fast_sqrt(float x) { return __builtin_amdgcn_sqrtf(x); }

__device__ __forceinline__ float scale_of(float mw, float M) {
  return (mw == -INFINITY) ? 0.0f : fast_exp2(mw - M);
}

struct Tile {
  uint4 k[4];  // K rows rb + c, dims 32 kb + 8 g .. + 7 (A operand of q.k)
  uint4 v[4];  // V rows rb + 4 g + j, dims 8 c .. 8 c + 7 (B operand of the weighted sums)
  float p[4];  // pi of rows rb + 4 g + j
};

// Row offsets are unsigned 32-bit (a unit's region is < 2^31 rows), so the loads use a uniform
// base plus a 32-bit lane offset.
__device__ __forceinline__ void load_tile(Tile &T, const uint4 *Kb, const uint4 *Vb,
                                          const float *Pb, int rb, int rlast, int g, int c) {
  const uint32_t rk = (uint32_t)min(rb + c, rlast);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) T.k[kb] = Kb[rk * (kHeadDim / 8) + (uint32_t)(4 * kb + g)];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t r = (uint32_t)min(rb + 4 * g + j, rlast);
    T.v[j] = Vb[r * (kHeadDim / 8) + (uint32_t)c];
    T.p[j] = Pb[r];
  }
}

struct SplitState {
  f32x4 acc[8];
  float mrun, s0, s1;
  float ck[4], cg[4], dk, dg;  // candidate lists (descending g^2 |v|^2, with g^2) and dropped maxima
  int cr[4];
  int rowbase;                 // row of this lane's first logit in the current tile
};

// The running max moves only when a logit exceeds it by more than kLazy (log2 units): weights then
// stay below 2^kLazy, which fp32 accumulates without loss of range, and the common tile needs no
// cross-lane max.
constexpr float kLazy = 8.0f;

__device__ __forceinline__ void split_tile(SplitState &S, const Tile &T, const bf16x8 (&qop)[4],
                                           int nvalid, int g, bool isC, float scale2) {
  f32x4 sacc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, T.k[kb]), qop[kb],
                                                   sacc, 0, 0, 0);
  // log2 pi of the 4 rows of this row group: quad lane i computes row i, the quad shares it.
  const int qi = __lane_id() & 3;
  const float pq = qi == 0 ? T.p[0] : (qi == 1 ? T.p[1] : (qi == 2 ? T.p[2] : T.p[3]));
  const float lq = fast_log2(pq);
  float lp[4];
  lp[0] = dpp_f<0x00>(lq);  // quad_perm [0,0,0,0]
  lp[1] = dpp_f<0x55>(lq);  // quad_perm [1,1,1,1]
  lp[2] = dpp_f<0xAA>(lq);  // quad_perm [2,2,2,2]
  lp[3] = dpp_f<0xFF>(lq);  // quad_perm [3,3,3,3]
  // lane (g, c): base-2 logits of rows rb + 4g + i for head slot c (nvalid <= 0 masks all)
  float lg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) lg[i] = i < nvalid ? fmaf(sacc[i], scale2, -lp[i]) : -INFINITY;
  const float lmax = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
  if (__any(lmax > S.mrun + kLazy)) {
    float tmax = fmaxf(lmax, __shfl_xor(lmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(S.mrun, tmax);
    const float alpha = (mnew > S.mrun) ? fast_exp2(S.mrun - mnew) : 1.0f;
    const float as = isC ? alpha * alpha : alpha;  // variance terms carry 2^{-2m}
    const float a2 = alpha * alpha;               // candidate keys are squares
    S.s0 *= as;
    S.s1 *= as;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      S.ck[e] *= a2;
      S.cg[e] *= a2;
    }
    S.dk *= a2;
    S.dg *= a2;
    float ai[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ai[i] = __shfl(as, 4 * (__lane_id() >> 4) + i);  // row 4g + i
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int i = 0; i < 4; ++i) S.acc[db][i] *= ai[i];
    }
    S.mrun = mnew;
  }

  float vf[4][8], nv2[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t w4[4] = {T.v[j].x, T.v[j].y, T.v[j].z, T.v[j].w};
    float sq = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      vf[j][2 * k] = bf16_lo(w4[k]);
      vf[j][2 * k + 1] = bf16_hi(w4[k]);
      sq = fmaf(vf[j][2 * k], vf[j][2 * k], sq);
      sq = fmaf(vf[j][2 * k + 1], vf[j][2 * k + 1], sq);
    }
    nv2[j] = row16_sum(sq);
  }

  // Weights (w for weight columns, c for variance columns), one MFMA operand per row group.
  // Candidate keys: kappa^2 = g^2 |v|^2 with g^2 = c.
  float val[4], kap[4], gsq[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float w = fast_exp2(lg[i] - S.mrun);  // 0 for masked rows (lg = -inf)
    const float cc = (1.0f - T.p[i]) * w * w;
    val[i] = isC ? cc : w;
    S.s0 += val[i];
    S.s1 = fmaf(cc, nv2[i], S.s1);
    gsq[i] = cc;
    kap[i] = cc * nv2[i];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int db = 0; db < 8; ++db)
      S.acc[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(val[j], vf[j][db], S.acc[db], 0, 0, 0);
  }

  // Range-term candidates: every row of the tile is offered to the lane's sorted top-4; whatever
  // falls off the end only raises the dropped maxima.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float nk = kap[i], ng = gsq[i];
    int nr = S.rowbase + i;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool sw = nk > S.ck[e];
      const float tk = sw ? S.ck[e] : nk, tg = sw ? S.cg[e] : ng;
      const int tr = sw ? S.cr[e] : nr;
      S.ck[e] = sw ? nk : S.ck[e];
      S.cg[e] = sw ? ng : S.cg[e];
      S.cr[e] = sw ? nr : S.cr[e];
      nk = tk;
      ng = tg;
      nr = tr;
    }
    S.dk = fmaxf(S.dk, nk);
    S.dg = fmaxf(S.dg, ng);
  }
}

}  // namespace

template <int GB>
__global__ __launch_bounds__(kAttendThreads, 2) void attend_split_kernel(AttendLaunch L, int h0) {
  __shared__ float s_acc[4][16][kHeadDim];
  __shared__ float s_m[4][16], s_s0[4][16], s_s1[4][16];
  __shared__ float s_ck[GB][64], s_cg[GB][64];
  __shared__ int s_cr[GB][64];
  __shared__ float s_dk[GB][16], s_dg[GB][16];
  __shared__ __align__(16) float s_key[4][64];

  const int bid = blockIdx.x;
  const int sp = bid % L.nsplit;
  const int u = bid / L.nsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  if (bid == 0 && tid == 0 && h0 == 0) L.diag[0] = 0u;

  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int cnt = (int)min(min((int64_t)L.count[u], cap), (int64_t)L.nsplit * L.split_rows);
  const int row0 = sp * L.split_rows;
  if (row0 >= cnt) return;  // empty split: the finalize pass skips it
  const int row1 = min(cnt, row0 + L.split_rows);

  const bool isW = c < GB;
  const bool isC = (c >= GB) && (c < 2 * GB);
  const bool active = isW || isC;
  const int hs = isW ? c : (isC ? c - GB : 0);

  // B operand of the q.k MFMA: column c holds q_{hs}; lane (g, c) supplies dims 32kb + 8g .. +7.
  bf16x8 qop[4];
  {
    const uint4 *qh = reinterpret_cast<const uint4 *>(L.q + ((int64_t)u * L.G + h0 + hs) * kHeadDim);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const uint4 w = active ? qh[4 * kb + g] : make_uint4(0u, 0u, 0u, 0u);
      qop[kb] = __builtin_bit_cast(bf16x8, w);
    }
  }

  SplitState S;
#pragma unroll
  for (int db = 0; db < 8; ++db) S.acc[db] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  S.mrun = active ? -INFINITY : 0.0f;
  S.s0 = S.s1 = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    S.ck[e] = S.cg[e] = 0.0f;
    S.cr[e] = -1;
  }
  S.dk = S.dg = 0.0f;

  const uint4 *Kb = reinterpret_cast<const uint4 *>(L.Kc + cbase * kHeadDim);
  const uint4 *Vb = reinterpret_cast<const uint4 *>(L.Vc + cbase * kHeadDim);
  const float *Pb = L.pic + cbase;
  const float scale2 = L.scale * kLog2e;
  const int ntile = (row1 - row0 + 15) / 16;
  const int rlast = row1 - 1;

  // Two tiles in registers: the next one loads while the current one is computed.  The
  // prefetch is unconditional (clamped to the last tile) so the compiler can wait for exactly
  // the current tile's loads.
  Tile TA, TB;
  const int tlast = ntile - 1;
  const int gmask = active ? 0 : (1 << 30);  // inactive columns see no valid rows
  int tt = wave;
  if (tt < ntile) load_tile(TA, Kb, Vb, Pb, row0 + 16 * tt, rlast, g, c);
  while (tt < ntile) {
    load_tile(TB, Kb, Vb, Pb, row0 + 16 * min(tt + 4, tlast), rlast, g, c);
    S.rowbase = row0 + 16 * tt + 4 * g;
    split_tile(S, TA, qop, row1 - S.rowbase - gmask, g, isC, scale2);
    tt += 4;
    if (tt >= ntile) break;
    load_tile(TA, Kb, Vb, Pb, row0 + 16 * min(tt + 4, tlast), rlast, g, c);
    S.rowbase = row0 + 16 * tt + 4 * g;
    split_tile(S, TB, qop, row1 - S.rowbase - gmask, g, isC, scale2);
    tt += 4;
  }

  // ---- wave results to LDS -------------------------------------------------------------------
  float s0 = S.s0, s1 = S.s1;
  s0 += __shfl_xor(s0, 16);
  s0 += __shfl_xor(s0, 32);
  s1 += __shfl_xor(s1, 16);
  s1 += __shfl_xor(s1, 32);
  if (g == 0) {
    s_m[wave][c] = S.mrun;
    s_s0[wave][c] = s0;
    s_s1[wave][c] = s1;
  }
#pragma unroll
  for (int db = 0; db < 8; ++db) {
#pragma unroll
    for (int i = 0; i < 4; ++i) s_acc[wave][4 * g + i][8 * c + db] = S.acc[db][i];
  }
  if (isW) {
    const int e = wave * 16 + g * 4;  // 64 entries per head: (wave, g, rank)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      s_ck[c][e + q] = S.ck[q];
      s_cg[c][e + q] = S.cg[q];
      s_cr[c][e + q] = S.cr[q];
    }
    s_dk[c][wave * 4 + g] = S.dk;
    s_dg[c][wave * 4 + g] = S.dg;
  }
  __syncthreads();

  // ---- merge the four waves and write one record per head ------------------------------------
  float *rec_base = L.part + (((int64_t)u * L.nsplit + sp) * L.G + h0) * kRec;
  for (int e = tid; e < 2 * GB * kHeadDim; e += kAttendThreads) {
    const int slot = e / kHeadDim, d = e % kHeadDim;
    const int hh = slot < GB ? slot : slot - GB;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][hh]);
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      float f = scale_of(s_m[w][hh], M);
      if (slot >= GB) f *= f;
      sum += f * s_acc[w][slot][d];
    }
    rec_base[(int64_t)hh * kRec + (slot < GB ? kRecO : kRecCv) + d] = sum;
  }
  // candidates: wave w merges heads w and w + 4 (64 entries -> the kCand largest by rank)
  for (int hh = wave; hh < GB; hh += 4) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][hh]);
    // keys are squares: scale by f^2, compare, and take square roots only for what is stored
    float f = scale_of(s_m[lane >> 4][hh], M);
    f *= f;
    const int row = s_cr[hh][lane];
    const float k = row >= 0 ? f * s_ck[hh][lane] : 0.0f;
    const float gv = row >= 0 ? f * s_cg[hh][lane] : 0.0f;
    s_key[wave][lane] = k;  // written and read by this wave only
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the keys are in LDS
    int rank = 0;
    const float4 *kk = reinterpret_cast<const float4 *>(s_key[wave]);
#pragma unroll 4
    for (int e4 = 0; e4 < 16; ++e4) {
      const float4 q = kk[e4];
      const float qe[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int e = 4 * e4 + t;
        rank += (qe[t] > k || (qe[t] == k && e < lane)) ? 1 : 0;
      }
    }
    const bool chosen = row >= 0 && k > 0.0f && rank < kCand;
    float dA = chosen ? 0.0f : k, dB = chosen ? 0.0f : gv;
    if (lane < 16) {
      float fw = scale_of(s_m[lane >> 2][hh], M);
      fw *= fw;
      dA = fmaxf(dA, fw * s_dk[hh][lane]);
      dB = fmaxf(dB, fw * s_dg[hh][lane]);
    }
    dA = sqrtf(wave_max(dA));
    dB = sqrtf(wave_max(dB));
    const float vmax = sqrtf(wave_max(chosen && gv > 0.0f ? k / gv : 0.0f));
    // chosen ranks are distinct and < kCand; unfilled candidate slots get row -1
    const int nchosen = __popcll(__ballot(chosen));
    float *rec = rec_base + (int64_t)hh * kRec;
    if (chosen) {
      rec[kRecCandG + rank] = sqrtf(gv);
      rec[kRecCandI + rank] = __int_as_float(row);
    }
    if (lane == 0) rec[kRecVmax] = vmax;
    if (lane >= nchosen && lane < kCand) {
      rec[kRecCandG + lane] = 0.0f;
      rec[kRecCandI + lane] = __int_as_float(-1);
    }
    if (lane == 0) {
      float lsum = 0.0f, c0 = 0.0f, c2 = 0.0f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float fw = scale_of(s_m[w][hh], M);
        lsum += fw * s_s0[w][hh];
        c0 += fw * fw * s_s0[w][GB + hh];
        c2 += fw * fw * s_s1[w][GB + hh];
      }
      rec[kRecM] = M;
      rec[kRecL] = lsum;
      rec[kRecC0] = c0;
      rec[kRecC2] = c2;
      rec[kRecA] = dA;
      rec[kRecB] = dB;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// attend_finalize: one wave per (unit, query head)
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(64) void attend_finalize_kernel(AttendLaunch L) {
  __shared__ float s_y[kHeadDim];
  __shared__ float s_q[kHeadDim];
  const int64_t bid = blockIdx.x;
  const int u = (int)(bid / L.G), h = (int)(bid % L.G);
  const int lane = threadIdx.x;
  const int64_t uh = bid;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int cnt = (int)min(min((int64_t)L.count[u], cap), (int64_t)L.nsplit * L.split_rows);
  float2 *yout = reinterpret_cast<float2 *>(L.y + uh * kHeadDim);
  if (cnt == 0) {
    yout[lane] = make_float2(0.0f, 0.0f);
    if (lane == 0) {
      L.vhat[uh] = 0.0f;
      L.lse[uh] = -INFINITY;
      if (L.brange) L.brange[uh] = 0.0f;
      if (L.radius) L.radius[uh] = 0.0f;
    }
    return;
  }
  const int nsp = (cnt + L.split_rows - 1) / L.split_rows;
  const float *rec0 = L.part + ((int64_t)u * L.nsplit * L.G + h) * kRec;
  const int64_t rstride = (int64_t)L.G * kRec;

  float M = -INFINITY;
  for (int s = lane; s < nsp; s += 64) M = fmaxf(M, rec0[s * rstride + kRecM]);
  M = wave_max(M);
  float l = 0.0f, C0 = 0.0f, C2 = 0.0f;
  for (int s = lane; s < nsp; s += 64) {
    const float *r = rec0 + s * rstride;
    const float f = scale_of(r[kRecM], M);
    l += f * r[kRecL];
    C0 += f * f * r[kRecC0];
    C2 += f * f * r[kRecC2];
  }
  l = wave_sum(l);
  C0 = wave_sum(C0);
  C2 = wave_sum(C2);

  float2 o = make_float2(0.0f, 0.0f), cv = make_float2(0.0f, 0.0f);
  for (int s = 0; s < nsp; ++s) {
    const float *r = rec0 + s * rstride;
    const float f = scale_of(r[kRecM], M);
    const float2 a = reinterpret_cast<const float2 *>(r + kRecO)[lane];
    const float2 b = reinterpret_cast<const float2 *>(r + kRecCv)[lane];
    o.x += f * a.x;
    o.y += f * a.y;
    cv.x += f * f * b.x;
    cv.y += f * f * b.y;
  }
  const float y0 = o.x / l, y1 = o.y / l;
  s_y[2 * lane] = y0;
  s_y[2 * lane + 1] = y1;
  {
    const uint32_t qw = reinterpret_cast<const uint32_t *>(L.q + uh * kHeadDim)[lane];
    s_q[2 * lane] = bf16_lo(qw);
    s_q[2 * lane + 1] = bf16_hi(qw);
  }
  const float ynorm2 = wave_sum(y0 * y0 + y1 * y1);
  const float ycv = wave_sum(y0 * cv.x + y1 * cv.y);
  const float V = fmaxf(C2 - 2.0f * ycv + ynorm2 * C0, 0.0f) / (l * l);
  const float ynorm = sqrtf(ynorm2);
  __syncthreads();

  // Range term, exact at the candidate rows.  A candidate's value f g |v - yhat| / l is at most
  // f g (Vmax + |yhat|) / l; the most promising candidate is evaluated first (whole wave), then
  // only the candidates whose bound still exceeds the best value so far (one per lane).
  const uint16_t *Vrows = L.Vc + cbase * kHeadDim;
  const int ncand = nsp * kCand;
  auto cand_bound = [&](int e, int &row, float &fg) -> float {
    const float *r = rec0 + (e / kCand) * rstride;
    row = __float_as_int(r[kRecCandI + (e % kCand)]);
    fg = scale_of(r[kRecM], M) * r[kRecCandG + (e % kCand)] / l;
    return row >= 0 ? fg * (r[kRecVmax] + ynorm) : 0.0f;
  };
  // the candidate with the largest bound, by the whole wave
  float best_ub = 0.0f;
  int best_e = -1;
  for (int e = lane; e < ncand; e += 64) {
    int row;
    float fg;
    const float ub = cand_bound(e, row, fg);
    if (ub > best_ub) {
      best_ub = ub;
      best_e = e;
    }
  }
  {
    const float m = wave_max(best_ub);
    const uint64_t who = __ballot(best_ub == m && best_e >= 0);
    best_e = who ? __shfl(best_e, (int)__ffsll((unsigned long long)who) - 1) : -1;
  }
  float lb = 0.0f;
  if (best_e >= 0) {
    int row;
    float fg;
    cand_bound(best_e, row, fg);
    const uint32_t w = reinterpret_cast<const uint32_t *>(Vrows + (int64_t)row * kHeadDim)[lane];
    const float d0 = bf16_lo(w) - y0, d1 = bf16_hi(w) - y1;
    lb = fg * sqrtf(wave_sum(d0 * d0 + d1 * d1));
  }
  for (int e = lane; e < ncand; e += 64) {
    int row;
    float fg;
    const float ub = cand_bound(e, row, fg);
    if (!(ub > lb) || e == best_e) continue;
    // keep yhat in LDS (re-read per candidate) instead of 128 registers
    asm volatile("" ::: "memory");
    const uint4 *vr = reinterpret_cast<const uint4 *>(Vrows + (int64_t)row * kHeadDim);
    uint4 vv[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) vv[k] = vr[k];
    float d2 = 0.0f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const uint32_t w4[4] = {vv[k].x, vv[k].y, vv[k].z, vv[k].w};
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float a = bf16_lo(w4[t]) - s_y[8 * k + 2 * t];
        const float b = bf16_hi(w4[t]) - s_y[8 * k + 2 * t + 1];
        d2 = fmaf(a, a, d2);
        d2 = fmaf(b, b, d2);
      }
    }
    lb = fmaxf(lb, fg * sqrtf(d2));
  }
  lb = wave_max(lb);
  // ... and a rescan of any split whose bound max(g|v|) + max(g)|yhat| could exceed it.
  const float scale2 = L.scale * kLog2e;
  for (int s = 0; s < nsp; ++s) {
    const float *r = rec0 + s * rstride;
    const float f = scale_of(r[kRecM], M);
    const float ub = f * (r[kRecA] + r[kRecB] * ynorm) / l;
    if (!(ub > lb)) continue;
    if (lane == 0) atomicAdd(L.diag, 1u);
    const int ra = s * L.split_rows, rz = min(cnt, ra + L.split_rows);
    const float ms = r[kRecM];
    float best = 0.0f;
    for (int j = ra + lane; j < rz; j += 64) {
      const uint4 *kr = reinterpret_cast<const uint4 *>(L.Kc + (cbase + j) * kHeadDim);
      const uint4 *vr = reinterpret_cast<const uint4 *>(Vrows + (int64_t)j * kHeadDim);
      const float pj = L.pic[cbase + j];
      float dot = 0.0f, d2 = 0.0f;
      for (int half = 0; half < 2; ++half) {  // half a row per step keeps the registers down
        asm volatile("" ::: "memory");  // q and yhat stay in LDS
        uint4 kq[8], vq[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          kq[k] = kr[8 * half + k];
          vq[k] = vr[8 * half + k];
        }
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const uint32_t kw[4] = {kq[k].x, kq[k].y, kq[k].z, kq[k].w};
          const uint32_t vw[4] = {vq[k].x, vq[k].y, vq[k].z, vq[k].w};
          const int d0 = 64 * half + 8 * k;
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            dot = fmaf(s_q[d0 + 2 * t], bf16_lo(kw[t]), dot);
            dot = fmaf(s_q[d0 + 2 * t + 1], bf16_hi(kw[t]), dot);
            const float a = bf16_lo(vw[t]) - s_y[d0 + 2 * t];
            const float b = bf16_hi(vw[t]) - s_y[d0 + 2 * t + 1];
            d2 = fmaf(a, a, d2);
            d2 = fmaf(b, b, d2);
          }
        }
      }
      const float w = fast_exp2(dot * scale2 - fast_log2(pj) - ms);
      best = fmaxf(best, sqrtf(1.0f - pj) * w * sqrtf(d2));
    }
    lb = fmaxf(lb, wave_max(f * best / l));
  }
  const float Ld = logf(1.0f / L.delta);
  yout[lane] = make_float2(y0, y1);
  if (lane == 0) {
    L.vhat[uh] = V;
    L.lse[uh] = M * kLn2 + logf(l);
    if (L.brange) L.brange[uh] = lb;
    if (L.radius) L.radius[uh] = (sqrtf(2.0f * V * Ld) + lb * Ld) / (ynorm + L.eps0);
  }
}

size_t attend_workspace_bytes(int32_t U, int32_t nsplit, int32_t G) {
  return 256 + (size_t)U * (size_t)nsplit * (size_t)G * kRec * sizeof(float);
}

hipError_t launch_attend_split(const AttendLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)((int64_t)L.U * L.nsplit)), block(kAttendThreads);
  for (int h0 = 0; h0 < L.G; h0 += kHeadBlock) {
    const int gb = min(kHeadBlock, L.G - h0);
    switch (gb) {
      case 1: hipLaunchKernelGGL(attend_split_kernel<1>, grid, block, 0, s, L, h0); break;
      case 2: hipLaunchKernelGGL(attend_split_kernel<2>, grid, block, 0, s, L, h0); break;
      case 3: hipLaunchKernelGGL(attend_split_kernel<3>, grid, block, 0, s, L, h0); break;
      case 4: hipLaunchKernelGGL(attend_split_kernel<4>, grid, block, 0, s, L, h0); break;
      case 5: hipLaunchKernelGGL(attend_split_kernel<5>, grid, block, 0, s, L, h0); break;
      case 6: hipLaunchKernelGGL(attend_split_kernel<6>, grid, block, 0, s, L, h0); break;
      case 7: hipLaunchKernelGGL(attend_split_kernel<7>, grid, block, 0, s, L, h0); break;
      default: hipLaunchKernelGGL(attend_split_kernel<8>, grid, block, 0, s, L, h0); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attend_finalize(const AttendLaunch &L, hipStream_t s) {
  hipLaunchKernelGGL(attend_finalize_kernel, dim3((unsigned)((int64_t)L.U * L.G)), dim3(64), 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
