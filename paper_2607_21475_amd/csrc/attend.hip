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
// attend_split (one wave per (unit, split of the retained rows, block of <= 8 query heads)):
//   The wave walks its split in 16-row tiles with two tiles' loads in flight while a third is
//   computed (raw buffer loads bounded by the split, so tail rows read as zero).  q.k runs on
//   MFMA (16x16x32 bf16, exact products, fp32 sums): A = K tile (16 rows x 32 dims per k-block,
//   loaded straight from HBM in operand layout), B = [q_0 .. q_{GB-1}, q_0 .. q_{GB-1}, 0 ..]
//   (16 columns).  Each lane then holds 4 rows x 1 column of logits; columns < GB become weights
//   w, columns GB..2GB-1 (same logits) become variance weights c.  bf16 16x16x32 MFMAs then form
//   o = sum w v (rows < GB) and Cv = sum c v (rows GB..2GB-1) together, with V in its natural
//   row-major layout (no transpose): each fp32 weight enters as an exact three-term bf16 sum,
//   so every product is exact and only the fp32 sums round.
//   Range-term candidates, per 512-row chunk: in every tile the weight lane of a head takes
//   rows 0 and 1 of its 4-row group and the variance lane (same logits) rows 2 and 3; each lane
//   keeps its four largest
//   g^2 |v|^2 (g^2 = (1 - pi) w^2) plus the maxima of g |v| and of g over what it dropped, so
//   a chunk holds 32 candidates per head with bounds for the rest.
//   The running max m moves lazily (only by jumps of more than 2^8 in weight).
//   A unit cut into 2..4 splits (when their LDS fits one work-group) runs them as the waves
//   of one work-group instead of as separate work-groups.
// Finalize (yhat, Vhat, ln Nhat, the exact range term b and the radius r): a unit that is one
//   split is finalized by the same wave from LDS; a unit whose splits share a work-group by the
//   wave that arrives last (an LDS counter, work-group fences); any other unit cut into splits
//   by attend_finalize (one wave per (unit, head block)).  The split records are combined by
//   log-sum-exp.  Candidates are bounded a chunk block at a time; only those whose bound can
//   still win are re-read, and a chunk is rescanned only if its non-candidate bound cannot
//   exclude a larger term.  Where C2 - 2 yhat.Cv + |yhat|^2 C0 has cancelled (one tail row
//   dominates both yhat and the variance, so yhat ~ v of that row), Vhat of that head is summed
//   again directly, sum (1 - pi) w^2 |v - yhat|^2 over the unit's retained rows.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

__device__ __forceinline__ float scale_of(float mw, float M) {
  return (mw == -INFINITY) ? 0.0f : fast_exp2(mw - M);
}

// Upper bound of a finite x >= 0 in bf16 (round toward +inf), as the high 16 bits.
__device__ __forceinline__ uint32_t bf16_up(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b >> 16) + ((b & 0xffffu) ? 1u : 0u);
}

struct Tile {
  u32x4 k[4];  // K rows 16t + c, dims 32 kb + 8 g .. + 7 (A operand of q.k)
  u32x4 v[4];  // V rows 16t + 4 g + j, dims 8 c .. 8 c + 7 (B operand of the weighted sums)
  float p[4];  // pi of rows 16t + 4 g + j
};

// Tile t of a split (rows 16t .. 16t + 15 counted from the split's first row).  Every byte of the
// retained rows is read once per step, so the loads are non-temporal (kLoadNT): streamed without
// being kept in the caches, which on this GPU reads markedly faster than the default policy.
__device__ __forceinline__ void load_tile(Tile &T, __amdgpu_buffer_rsrc_t rK, __amdgpu_buffer_rsrc_t rV,
                                          __amdgpu_buffer_rsrc_t rP, int t, int g, int c) {
  const uint32_t rk = (uint32_t)(16 * t + c);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    T.k[kb] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            rK, rk * 256u + (uint32_t)(64 * kb + 16 * g), 0, kLoadNT));
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t r = (uint32_t)(16 * t + 4 * g + j);
    T.v[j] = __builtin_bit_cast(u32x4,
                                __builtin_amdgcn_raw_buffer_load_b128(rV, r * 256u + 16u * c, 0, kLoadNT));
  }
  // pi of the row group's 4 consecutive rows in one 16-byte load (the range check is per dword:
  // rows past the split read as zero, those before it are loaded)
  const u32x4 pw = __builtin_bit_cast(
      u32x4, __builtin_amdgcn_raw_buffer_load_b128(rP, (uint32_t)(16 * t + 4 * g) * 4u, 0, kLoadNT));
  T.p[0] = __uint_as_float(pw.x);
  T.p[1] = __uint_as_float(pw.y);
  T.p[2] = __uint_as_float(pw.z);
  T.p[3] = __uint_as_float(pw.w);
}

struct SplitState {
  f32x4 acc[8];
  float mrun, s0, s1;
  float pl;  // logit of this lane's head's current pivot (-inf: none yet)
  float ck[4], cg[4], dk, dg;  // candidate lists (descending g^2 |v|^2, with g^2) and dropped maxima
  int cr[4];
};

// The running max moves only when a logit exceeds it by more than kLazy (log2 units): weights then
// stay below 2^kLazy, which fp32 accumulates without loss of range, and the common tile needs no
// cross-lane max.
constexpr float kLazy = 8.0f;

// Pivot rows.  One row that outweighs the rest of a head makes yhat ~ its v, and then the one-pass
// C2 - 2 yhat.Cv + |yhat|^2 C0 cancels (a row drawn near a small floor carries 1/pi up to 1e6).
// So each head keeps its largest-weight row out of every sum: a row becomes the head's pivot when
// its logit exceeds the current pivot's by more than kPivGap (a factor 8 in weight), is recorded
// in the head's list (row, logit, pi) and gets weight 0 in the sums and the candidate lists.  A
// row that outweighs every other row by more than 8x is then the last pivot, whatever the order;
// the finalize adds the earlier pivots back exactly and treats the last one in closed form.  With
// the gap, a head takes a new pivot a few times per split at most (the first tile always).
constexpr float kPivGap = 3.0f;

// One 16-row tile: rows 16t + 4g + i of the split for this lane's head slot; `nvalid` rows of the
// lane's row group are real (<= 0 masks them all), `rowbase` is the unit row of its first one.
// kPivLogit: the slot of a pivot list that holds the head's current pivot logit when it is kept in
// LDS rather than in a register (the eight-head kernel, whose registers are otherwise exhausted).
constexpr int kPivLogit = 25;

template <bool PL_LDS>
__device__ __forceinline__ void split_tile(SplitState &S, const Tile &T, const bf16x8 (&qop)[4],
                                           int nvalid, int rowbase, bool isC, bool plain,
                                           float scale2, float *s_piv, int hslot, bool isW) {
  f32x4 sacc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
    sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, T.k[kb]), qop[kb],
                                                   sacc, 0, 0, 0);
  // log2 pi of the 4 rows of this row group: quad lane i computes row i, the quad shares it.
  const int qi = __lane_id() & 3;
  const float p01 = (qi & 1) ? T.p[1] : T.p[0], p23 = (qi & 1) ? T.p[3] : T.p[2];
  const float pq = (qi & 2) ? p23 : p01;  // selects, not an indexed (scratch) array
  const float lq = plain ? 0.0f : fast_log2(pq);  // the uncorrected pass drops the offset
  float lp[4];
  lp[0] = dpp_f<0x00>(lq);  // quad_perm [0,0,0,0]
  lp[1] = dpp_f<0x55>(lq);  // quad_perm [1,1,1,1]
  lp[2] = dpp_f<0xAA>(lq);  // quad_perm [2,2,2,2]
  lp[3] = dpp_f<0xFF>(lq);  // quad_perm [3,3,3,3]
  float lg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) lg[i] = i < nvalid ? fmaf(sacc[i], scale2, -lp[i]) : -INFINITY;
  float lmax = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
  const float pl = PL_LDS ? s_piv[hslot * kPivFloats + kPivLogit] : S.pl;
  if (__any(lmax > pl + kPivGap)) {
    // a new pivot for some head: the tile's largest logit of each column and its row (the lowest
    // of equal ones); both columns of a head see the same logits and decide alike
    const int g = __lane_id() >> 4;
    float tm = fmaxf(lmax, __shfl_xor(lmax, 16));
    tm = fmaxf(tm, __shfl_xor(tm, 32));
    int r = 16;
#pragma unroll
    for (int i = 3; i >= 0; --i) r = (lg[i] == tm) ? 4 * g + i : r;
    r = min(r, __shfl_xor(r, 16));
    r = min(r, __shfl_xor(r, 32));
    const int rr = r & 15;
    const int pn = __float_as_int(s_piv[hslot * kPivFloats]);  // the list's count
    if (tm > pl + kPivGap && pn < kPivMax) {
      if (isW && g == (rr >> 2)) {  // the weight lane holding the row records it
        float *e = s_piv + hslot * kPivFloats;
        const float pa = (rr & 1) ? T.p[1] : T.p[0], pb = (rr & 1) ? T.p[3] : T.p[2];
        e[1 + 3 * pn] = __int_as_float(rowbase - 4 * g + rr);
        e[2 + 3 * pn] = tm;
        e[3 + 3 * pn] = (rr & 2) ? pb : pa;
        e[0] = __int_as_float(pn + 1);
        if (PL_LDS) e[kPivLogit] = tm;
      }
      if (!PL_LDS) S.pl = tm;
#pragma unroll
      for (int i = 0; i < 4; ++i) lg[i] = (g == (rr >> 2) && i == (rr & 3)) ? -INFINITY : lg[i];
      lmax = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
    }
  }
  if (__any(lmax > S.mrun + kLazy)) {
    float tmax = fmaxf(lmax, __shfl_xor(lmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(S.mrun, tmax);
    const float alpha = (mnew > S.mrun) ? fast_exp2(S.mrun - mnew) : 1.0f;
    const float as = isC ? alpha * alpha : alpha;  // variance terms carry 2^{-2m}
    const float a2 = alpha * alpha;               // candidate keys and C2 are squares
    S.s0 *= as;
    S.s1 *= a2;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      S.ck[e] *= a2;
      S.cg[e] *= a2;
    }
    S.dk *= a2;
    S.dg *= a2;
    float ai[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ai[i] = __shfl(as, 4 * (__lane_id() >> 4) + i);  // slot 4g + i
#pragma unroll
    for (int db = 0; db < 8; ++db) {
#pragma unroll
      for (int i = 0; i < 4; ++i) S.acc[db][i] *= ai[i];
    }
    S.mrun = mnew;
  }

  // |v|^2 of the lane's 4 rows (exact fp32 products; the bf16 pair dot instruction is not
  // accurate enough here: the variance moved by 2.5% with it)
  float nv2[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float sq = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float a = bf16_lo(T.v[j][k]), b = bf16_hi(T.v[j][k]);
      sq = fmaf(a, a, sq);
      sq = fmaf(b, b, sq);
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
  // o and Cv on bf16 MFMAs (16x16x32), exactly: every fp32 weight is split into three bf16
  // terms hi + mid + lo (successive 8-bit pieces of its significand, each difference exact), and
  // V (bf16) times each term is an exact product, so only the fp32 summation rounds.  The
  // contraction runs over this row group's 4 rows x {hi, mid} in one MFMA (A = [hi_0 .. hi_3,
  // mid_0 .. mid_3]) and 4 rows x {lo, 0} in a second (A = [lo_0 .. lo_3, 0 x 4]), against
  // B = [v_0, v_1, v_2, v_3, v_0, v_1, v_2, v_3] at one dim.  Lane (g, c) holds rows 4g + j at
  // dims 8c .. 8c + 7 of V, which is the B operand for dims 8c + e, e = 0..7.
  uint32_t hb[4], mb[4], lb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    hb[i] = __float_as_uint(val[i]) & 0xffff0000u;
    const float r = val[i] - __uint_as_float(hb[i]);  // exact: the low 16 significand bits
    mb[i] = __float_as_uint(r) & 0xffff0000u;
    lb[i] = __float_as_uint(r - __uint_as_float(mb[i]));  // exact, and exact in bf16
  }
  // the high halves of two words, the first one's in the low half
  auto hh = [](uint32_t x, uint32_t y) { return __builtin_amdgcn_perm(y, x, 0x07060302u); };
  const u32x4 whm = {hh(hb[0], hb[1]), hh(hb[2], hb[3]), hh(mb[0], mb[1]), hh(mb[2], mb[3])};
  const u32x4 wlo = {hh(lb[0], lb[1]), hh(lb[2], lb[3]), 0u, 0u};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    // element e of rows (0, 1) and of rows (2, 3), each pair in one word
    const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
    const uint32_t p01 = __builtin_amdgcn_perm(T.v[1][e >> 1], T.v[0][e >> 1], sel);
    const uint32_t p23 = __builtin_amdgcn_perm(T.v[3][e >> 1], T.v[2][e >> 1], sel);
    const u32x4 bop = {p01, p23, p01, p23};
    S.acc[e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, whm),
                                                      __builtin_bit_cast(bf16x8, bop), S.acc[e], 0,
                                                      0, 0);
    S.acc[e] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wlo),
                                                      __builtin_bit_cast(bf16x8, bop), S.acc[e], 0,
                                                      0, 0);
  }

  // Range-term candidates: the weight lane of a head takes rows 0 and 1 of its row group, the
  // variance lane (same logits, so the same keys) rows 2 and 3.  Each such row is offered to the
  // lane's sorted top-4; whatever falls off the end only raises the dropped maxima.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float nk = isC ? kap[i + 2] : kap[i], ng = isC ? gsq[i + 2] : gsq[i];
    int nr = rowbase + (isC ? i + 2 : i);
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

// End of a chunk: the lane lists of head h (weight lanes (g, h), variance lanes (g, GB + h))
// become the chunk's 32 candidates in LDS, with the chunk's dropped maxima and the running max
// they are scaled by; the lists restart empty for the next chunk.  `c0` is the chunk's first
// unit row.
template <int GB>
__device__ __forceinline__ void flush_chunk(SplitState &S, float *s_chunk, int k, int g, int c,
                                            int c0) {
  float dk = S.dk, dg = S.dg, vm = 0.0f;
#pragma unroll
  for (int e = 0; e < 4; ++e) vm = fmaxf(vm, S.cg[e] > 0.0f ? S.ck[e] / S.cg[e] : 0.0f);
  const float al = fast_sqrt(dk);              // this lane's own dropped maximum of g |v|
  const float ao = __shfl_xor(al, 16);         // ... and that of row group g ^ 1
  dk = fmaxf(dk, __shfl_xor(dk, 16));
  dk = fmaxf(dk, __shfl_xor(dk, 32));
  dg = fmaxf(dg, __shfl_xor(dg, 16));
  dg = fmaxf(dg, __shfl_xor(dg, 32));
  vm = fmaxf(vm, __shfl_xor(vm, 16));
  vm = fmaxf(vm, __shfl_xor(vm, 32));
  const int lane = __lane_id();
  const int partner = (lane + GB) & 63;  // the variance lane of the same head and row group
  dk = fmaxf(dk, __shfl(dk, partner));
  dg = fmaxf(dg, __shfl(dg, partner));
  vm = fmaxf(vm, __shfl(vm, partner));
  if (c < 2 * GB) {
    const int h = c < GB ? c : c - GB;
    const int j0 = (c < GB ? 0 : 16) + 4 * g;
    float *blk = s_chunk + (k * GB + h) * kChunkFloats;
    uint32_t off[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool real = S.cr[e] >= 0 && S.ck[e] > 0.0f;
      blk[kChG + j0 + e] = real ? fast_sqrt(S.cg[e]) : 0.0f;
      off[e] = real ? (uint32_t)(S.cr[e] - c0) : 0u;
    }
    blk[kChI + j0 / 2] = __uint_as_float(off[0] | (off[1] << 16));
    blk[kChI + j0 / 2 + 1] = __uint_as_float(off[2] | (off[3] << 16));
    if ((g & 1) == 0)  // lanes 4w + g and 4w + g + 1 (w = 0 weight, 1 variance lanes)
      blk[kChAL + g / 2 + (c < GB ? 0 : 2)] = __uint_as_float(bf16_up(al) | (bf16_up(ao) << 16));
    if (c < GB && g == 0) {
      blk[kChA] = fast_sqrt(dk);
      blk[kChB] = fast_sqrt(dg);
      blk[kChVmax] = fast_sqrt(vm);
      blk[kChM] = S.mrun;
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    S.ck[e] = S.cg[e] = 0.0f;
    S.cr[e] = -1;
  }
  S.dk = S.dg = 0.0f;
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// Finalize of a block of GB heads of one unit: yhat, Vhat, ln Nhat, the exact range term b and
// the radius r, from the combined sums in LDS and the candidate blocks of every chunk.
// ---------------------------------------------------------------------------------------------
constexpr int kListCap = 256;  // candidates evaluated per batch
// per-head table: M, l, C0, C2, |yhat|, lb, Vhat, redo, then the pivot: logit (-inf: none), pi,
// row, key (split * kPivMax + entry)
constexpr int kHs = 12;
constexpr int kHsM = 0, kHsL = 1, kHsC0 = 2, kHsC2 = 3, kHsYn = 4, kHsLb = 5, kHsV = 6, kHsRedo = 7;
constexpr int kHsPl = 8, kHsPp = 9, kHsPr = 10, kHsPk = 11;
// The one-pass form C2 - 2 yhat.Cv + |yhat|^2 C0 of sum c |v - yhat|^2 carries a rounding error of
// a few ulps of (sqrt(C2) + |yhat| sqrt(C0))^2 (each sum is of exact products, rounded in fp32);
// below this fraction of that scale the head's Vhat is summed again directly.
constexpr float kCancelFrac = 1.0f / 1024.0f;

// Per (unit, head block) diagnostic words at the start of the workspace: the 512-row chunks
// rescanned for the range term, and the heads whose Vhat was summed directly.
__device__ __forceinline__ uint32_t *diag_of(const AttendLaunch &L, int u, int h0) {
  return L.diag + 2 * ((int64_t)u * L.nhb + h0 / kHeadBlock);
}

// LDS of the finalize, carved from one dynamic buffer.
template <int GB>
struct FinLds {
  float *o;                  // [2 GB][128]: o, later yhat (slots < GB); Cv, later q (the rest)
  float *hs;                 // [GB][kHs]
  unsigned long long *best;  // [GB]: (bound bits << 32) | candidate index of the largest bound
  int *list;                 // [kListCap]
  __device__ explicit FinLds(float *base) {
    o = base;
    hs = o + 2 * GB * kHeadDim;
    best = reinterpret_cast<unsigned long long *>(hs + GB * kHs);
    list = reinterpret_cast<int *>(best + GB);
  }
  static constexpr size_t bytes() {
    return (2 * GB * kHeadDim + GB * kHs) * sizeof(float) + GB * sizeof(unsigned long long) +
           kListCap * sizeof(int);
  }
};

// Where the candidate block of (split s, chunk k, head h) lives: LDS for a fused split, the
// split records in the workspace otherwise.
struct CandSrc {
  const float *base;
  int64_t sstride;
  int kstride, hstride;
};

// Where the pivot list of (split s, head h) lives: LDS for a fused split, the records otherwise.
struct PivSrc {
  const float *base;
  int64_t sstride;
  int hstride;
  __device__ const float *at(int s, int h) const { return base + s * sstride + h * hstride; }
};

// Calls f(row, logit, pi, key) for every pivot entry of head h over the splits, in a fixed order
// (split, entry); key = split * kPivMax + entry.  All lanes of a head run the same iterations.
template <class Fn>
__device__ __forceinline__ void for_each_pivot(const PivSrc &P, int nsp, int h, bool act, Fn &&f) {
  for (int s = 0; s < nsp; ++s) {
    const float *pl = P.at(s, h);
    const int n = act ? __float_as_int(pl[0]) : 0;
#pragma unroll
    for (int e = 0; e < kPivMax; ++e)
      if (e < n) f(__float_as_int(pl[1 + 3 * e]), pl[2 + 3 * e], pl[3 + 3 * e], s * kPivMax + e);
  }
}

// Before the finalize: per head, the entry with the largest logit over all splits becomes the
// pivot (kept in the head's table), the running max is raised to its logit if needed (the sums
// rescaled), and every other entry is added back into l, o, C0, Cv, C2 exactly.  8 lanes per
// head, 16 dims per lane.
template <int GB>
__device__ __forceinline__ void pivot_prepare(const AttendLaunch &L, int64_t cbase, int nsp, const PivSrc &P,
                              const FinLds<GB> &F) {
  const int lane = threadIdx.x & 63;
  const int h = lane >> 3, j = lane & 7;
  const bool act = h < GB;
  const int hh = act ? h : 0;
  wave_sync();  // the sums are in LDS
  // the pivot: lanes of a head look at every eighth split, then compare
  float bl = -INFINITY;
  int bk = 0x7fffffff;
  for (int s = j; s < nsp; s += 8) {
    const float *pl = P.at(s, hh);
    const int n = act ? __float_as_int(pl[0]) : 0;
#pragma unroll
    for (int e = 0; e < kPivMax; ++e) {
      if (e < n && pl[2 + 3 * e] > bl) {
        bl = pl[2 + 3 * e];
        bk = s * kPivMax + e;
      }
    }
  }
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) {
    const float ol = __shfl_xor(bl, o);
    const int ok = __shfl_xor(bk, o);
    if (ol > bl || (ol == bl && ok < bk)) {
      bl = ol;
      bk = ok;
    }
  }
  float *hs = F.hs + hh * kHs;
  const float M0 = hs[kHsM], M1 = fmaxf(M0, bl);
  const float f = scale_of(M0, M1), f2 = f * f;
  float o16[16], c16[16];
  {
    const float4 *op = reinterpret_cast<const float4 *>(F.o + hh * kHeadDim + 16 * j);
    const float4 *cp = reinterpret_cast<const float4 *>(F.o + (GB + hh) * kHeadDim + 16 * j);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 a = op[q], b = cp[q];
      o16[4 * q] = a.x * f, o16[4 * q + 1] = a.y * f, o16[4 * q + 2] = a.z * f, o16[4 * q + 3] = a.w * f;
      c16[4 * q] = b.x * f2, c16[4 * q + 1] = b.y * f2, c16[4 * q + 2] = b.z * f2, c16[4 * q + 3] = b.w * f2;
    }
  }
  float la = 0.0f, c0a = 0.0f, c2a = 0.0f;
  for_each_pivot(P, nsp, hh, act, [&](int row, float lgt, float p, int key) {
    if (key == bk) return;
    const float w = fast_exp2(lgt - M1), cc = (1.0f - p) * w * w;
    const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + row) * kHeadDim + 16 * j);
    const uint4 va = vr[0], vb = vr[1];
    const uint32_t vw[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
    float nv = 0.0f;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float x0 = bf16_lo(vw[t]), x1 = bf16_hi(vw[t]);
      o16[2 * t] = fmaf(w, x0, o16[2 * t]);
      o16[2 * t + 1] = fmaf(w, x1, o16[2 * t + 1]);
      c16[2 * t] = fmaf(cc, x0, c16[2 * t]);
      c16[2 * t + 1] = fmaf(cc, x1, c16[2 * t + 1]);
      nv = fmaf(x0, x0, nv);
      nv = fmaf(x1, x1, nv);
    }
    nv += __shfl_xor(nv, 1);
    nv += __shfl_xor(nv, 2);
    nv += __shfl_xor(nv, 4);
    la += w;
    c0a += cc;
    c2a = fmaf(cc, nv, c2a);
  });
  wave_sync();  // every lane has read the sums it rescales
  if (act) {
    float4 *op = reinterpret_cast<float4 *>(F.o + hh * kHeadDim + 16 * j);
    float4 *cp = reinterpret_cast<float4 *>(F.o + (GB + hh) * kHeadDim + 16 * j);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      op[q] = make_float4(o16[4 * q], o16[4 * q + 1], o16[4 * q + 2], o16[4 * q + 3]);
      cp[q] = make_float4(c16[4 * q], c16[4 * q + 1], c16[4 * q + 2], c16[4 * q + 3]);
    }
    if (j == 0) {
      hs[kHsL] = fmaf(hs[kHsL], f, la);
      hs[kHsC0] = fmaf(hs[kHsC0], f2, c0a);
      hs[kHsC2] = fmaf(hs[kHsC2], f2, c2a);
      hs[kHsM] = M1;
      hs[kHsPl] = bl;
      hs[kHsPk] = __int_as_float(bk);
      if (bl > -INFINITY) {
        const float *pe = P.at(bk / kPivMax, hh) + 1 + 3 * (bk % kPivMax);
        hs[kHsPr] = pe[0];
        hs[kHsPp] = pe[2];
      }
    }
  }
  wave_sync();
}

template <int GB>
__device__ __forceinline__ void finalize_block(const AttendLaunch &L, int u, int h0, int cnt, int64_t cbase,
                               int nsp, const CandSrc &C, const PivSrc &P, const FinLds<GB> &F) {
  const int lane = threadIdx.x & 63;
  const int64_t uh0 = (int64_t)u * L.G + h0;

  // (1) yhat, Vhat, ln Nhat: 8 lanes per head, 16 dims per lane.  With a pivot p (weight w_p,
  //     value v_p) outside the rest sums l_r, o_r, C0, Cv, C2:
  //       l = l_r + w_p,  yhat = (o_r + w_p v_p) / l,  d = yhat - v_p = (o_r - l_r v_p) / l,
  //       Vhat l^2 = [C2 - 2 yhat.Cv + |yhat|^2 C0] + c_p |d|^2,   c_p = (1 - pi_p) w_p^2,
  //     where neither the bracket (rest rows only) nor d cancels when the pivot dominates.
  {
    const int h = lane >> 3, j = lane & 7;
    float yy = 0.0f, ycv = 0.0f, dd = 0.0f;
    if (h < GB) {
      const float *hs = F.hs + h * kHs;
      const float lr = hs[kHsL];
      const bool piv = hs[kHsPl] > -INFINITY;
      float wp = 0.0f, vp[16];
#pragma unroll
      for (int t = 0; t < 16; ++t) vp[t] = 0.0f;
      if (piv) {
        wp = fast_exp2(hs[kHsPl] - hs[kHsM]);
        const uint4 *vr = reinterpret_cast<const uint4 *>(
            L.Vc + (cbase + __float_as_int(hs[kHsPr])) * kHeadDim + 16 * j);
        const uint4 va = vr[0], vb = vr[1];
        const uint32_t vw[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          vp[2 * t] = bf16_lo(vw[t]);
          vp[2 * t + 1] = bf16_hi(vw[t]);
        }
      }
      const float il = 1.0f / (lr + wp);
      float4 *oh = reinterpret_cast<float4 *>(F.o + h * kHeadDim + 16 * j);
      const float4 *cv = reinterpret_cast<const float4 *>(F.o + (GB + h) * kHeadDim + 16 * j);
      float4 *yo = reinterpret_cast<float4 *>(L.y + (uh0 + h) * kHeadDim + 16 * j);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 a = oh[q], b = cv[q];
        const float ov[4] = {a.x, a.y, a.z, a.w}, cvv[4] = {b.x, b.y, b.z, b.w};
        float yv[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          yv[t] = fmaf(wp, vp[4 * q + t], ov[t]) * il;
          const float dv = fmaf(-lr, vp[4 * q + t], ov[t]) * il;
          yy = fmaf(yv[t], yv[t], yy);
          ycv = fmaf(yv[t], cvv[t], ycv);
          dd = fmaf(dv, dv, dd);
        }
        oh[q] = make_float4(yv[0], yv[1], yv[2], yv[3]);
        yo[q] = oh[q];
      }
    }
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) {
      yy += __shfl_xor(yy, o);
      ycv += __shfl_xor(ycv, o);
      dd += __shfl_xor(dd, o);
    }
    if (h < GB && j == 0) {
      float *hs = F.hs + h * kHs;
      const bool piv = hs[kHsPl] > -INFINITY;
      const float wp = piv ? fast_exp2(hs[kHsPl] - hs[kHsM]) : 0.0f;
      const float pp = piv ? hs[kHsPp] : 1.0f;
      const float l = hs[kHsL] + wp;
      const float num = hs[kHsC2] - 2.0f * ycv + yy * hs[kHsC0] + (1.0f - pp) * wp * wp * dd;
      const float sc = sqrtf(hs[kHsC2]) + sqrtf(yy * hs[kHsC0]);
      const bool redo = num < kCancelFrac * sc * sc;  // never when the rest has no tail row
      const float V = fmaxf(num, 0.0f) / (l * l);
      if (!L.plain && !redo) L.vhat[uh0 + h] = V;
      L.lse[uh0 + h] = hs[kHsM] * kLn2 + logf(l);
      hs[kHsL] = l;
      hs[kHsYn] = sqrtf(yy);
      hs[kHsLb] = piv ? sqrtf(1.0f - pp) * wp * sqrtf(dd) / l : 0.0f;  // the pivot's range term
      hs[kHsV] = V;
      hs[kHsRedo] = redo ? 1.0f : 0.0f;
      F.best[h] = 0ull;
    }
  }
  wave_sync();
  if (L.plain) return;  // the uncorrected pass only replaces y and ln N

  // (1c) The range terms of the pivot list entries added back in pivot_prepare (they are in no
  //      candidate list): sqrt(1 - pi) w |v - yhat| / l, exactly.
  {
    const int h = lane >> 3, j = lane & 7;
    const bool act = h < GB;
    const int hh = act ? h : 0;
    const float *hs = F.hs + hh * kHs;
    const int pk = __float_as_int(hs[kHsPk]);
    const float M = hs[kHsM], il = 1.0f / hs[kHsL];
    const float *yh = F.o + hh * kHeadDim + 16 * j;
    float bmax = 0.0f;
    for_each_pivot(P, nsp, hh, act, [&](int row, float lgt, float p, int key) {
      if (key == pk) return;
      const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + row) * kHeadDim + 16 * j);
      const uint4 va = vr[0], vb = vr[1];
      const uint32_t vw[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
      float d2 = 0.0f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float a = bf16_lo(vw[t]) - yh[2 * t], b = bf16_hi(vw[t]) - yh[2 * t + 1];
        d2 = fmaf(a, a, d2);
        d2 = fmaf(b, b, d2);
      }
      d2 += __shfl_xor(d2, 1);
      d2 += __shfl_xor(d2, 2);
      d2 += __shfl_xor(d2, 4);
      bmax = fmaxf(bmax, sqrtf(1.0f - p) * fast_exp2(lgt - M) * sqrtf(d2) * il);
    });
    if (act && j == 0) F.hs[h * kHs + kHsLb] = fmaxf(F.hs[h * kHs + kHsLb], bmax);
    wave_sync();
  }

  // q of every head into the Cv slots, once Cv is no longer needed (the direct variance sums and
  // the range-term rescans recompute logits).
  bool qloaded = false;
  auto load_q = [&]() {
    if (qloaded) return;
    for (int e = lane; e < GB * kHeadDim / 2; e += 64) {
      const int h = e / (kHeadDim / 2), d2 = e % (kHeadDim / 2);
      const uint32_t qw = reinterpret_cast<const uint32_t *>(L.q + (uh0 + h) * kHeadDim)[d2];
      F.o[(GB + h) * kHeadDim + 2 * d2] = bf16_lo(qw);
      F.o[(GB + h) * kHeadDim + 2 * d2 + 1] = bf16_hi(qw);
    }
    wave_sync();
    qloaded = true;
  };

  uint32_t redo = 0u;
#pragma unroll
  for (int h = 0; h < GB; ++h) redo |= (F.hs[h * kHs + kHsRedo] != 0.0f ? 1u : 0u) << h;

  // (2) Candidate bounds: a candidate's value f g |v - yhat| / l is at most f g (Vmax + |yhat|)/l.
  //     Candidate e = ((s nchunk + k) GB + h) kCand + j.
  const int R = L.split_rows;
  auto decode = [&](int e, int &h, int &row, float &fg, float &ub) -> bool {
    const int j = e % kCand;
    int r = e / kCand;
    h = r % GB;
    r /= GB;
    const int k = r % L.nchunk, s = r / L.nchunk;
    if (k * kChunkRows >= min(cnt - s * R, R)) return false;  // no such chunk
    const float *blk = C.base + s * C.sstride + k * C.kstride + h * C.hstride;
    const float gj = blk[kChG + j];
    if (!(gj > 0.0f)) return false;
    row = s * R + k * kChunkRows + (int)((__float_as_uint(blk[kChI + j / 2]) >> (16 * (j & 1))) & 0xffffu);
    const float *hs = F.hs + h * kHs;
    fg = scale_of(blk[kChM], hs[kHsM]) * gj / hs[kHsL];
    ub = fg * (blk[kChVmax] + hs[kHsYn]);
    return true;
  };
  // Chunk block x = (s nchunk + k) GB + h (16-byte aligned), or null for a chunk that is absent.
  const int nx = nsp * L.nchunk * GB;
  auto block_at = [&](int x, int &h) -> const float * {
    h = x % GB;
    const int sk = x / GB, s = sk / L.nchunk, k = sk - s * L.nchunk;
    if (x >= nx || k * kChunkRows >= min(cnt - s * R, R)) return nullptr;
    return C.base + s * C.sstride + k * C.kstride + h * C.hstride;
  };
  // One lane per block: candidate j's bound is g_j F with F = f (Vmax + |yhat|) / l, so the
  // block's largest g decides; per head, the largest bound (and its candidate) goes to F.best.
  for (int x0 = 0; x0 < nx; x0 += 64) {
    int h;
    const float *blk = block_at(x0 + lane, h);
    if (blk) {
      const float4 *g4 = reinterpret_cast<const float4 *>(blk + kChG);
      float gmax = 0.0f;
      int jmax = 0;
#pragma unroll
      for (int q = 0; q < kCand / 4; ++q) {
        const float4 v = g4[q];
        const float gq[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (gq[t] > gmax) {
            gmax = gq[t];
            jmax = 4 * q + t;
          }
        }
      }
      const float *hs = F.hs + h * kHs;
      const float ub = scale_of(blk[kChM], hs[kHsM]) * gmax / hs[kHsL] * (blk[kChVmax] + hs[kHsYn]);
      if (ub > 0.0f)
        atomicMax(&F.best[h], ((unsigned long long)__float_as_uint(ub) << 32) |
                                  (unsigned)((x0 + lane) * kCand + jmax));
    }
  }
  wave_sync();

  // (3) The most promising candidate of every head, 8 lanes per head.
  {
    const int h = lane >> 3, j = lane & 7;
    float d2 = 0.0f, fg = 0.0f;
    bool have = false;
    if (h < GB && F.best[h] != 0ull) {
      int hh, row;
      float ub;
      have = decode((int)(F.best[h] & 0xffffffffull), hh, row, fg, ub);
      if (have) {
        const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + row) * kHeadDim) + 2 * j;
        const float *yh = F.o + h * kHeadDim + 16 * j;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const uint4 w = vr[q];
          const uint32_t w4[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const float a = bf16_lo(w4[t]) - yh[8 * q + 2 * t];
            const float b = bf16_hi(w4[t]) - yh[8 * q + 2 * t + 1];
            d2 = fmaf(a, a, d2);
            d2 = fmaf(b, b, d2);
          }
        }
      }
    }
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) d2 += __shfl_xor(d2, o);
    if (have && j == 0) F.hs[h * kHs + kHsLb] = fmaxf(F.hs[h * kHs + kHsLb], fg * sqrtf(d2));
  }
  wave_sync();

  // (4) Every other candidate whose bound exceeds its head's best value: listed, then evaluated
  //     sixteen at a time (four lanes per value row).
  auto eval_list = [&](int n) {
    wave_sync();  // the list is in LDS
    const int t4 = lane & 3;  // four lanes per candidate, 32 dims each
    for (int i0 = 0; i0 < n; i0 += 16) {
      const int i = i0 + (lane >> 2);
      int h = 0, row = 0;
      float fg = 0.0f, ub;
      const bool have = i < n && decode(F.list[i], h, row, fg, ub);
      float d2 = 0.0f;
      if (have) {
        const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + row) * kHeadDim) + 4 * t4;
        const float *yh = F.o + h * kHeadDim + 32 * t4;
        uint4 vv[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) vv[k] = vr[k];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t w4[4] = {vv[k].x, vv[k].y, vv[k].z, vv[k].w};
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const float a = bf16_lo(w4[t]) - yh[8 * k + 2 * t];
            const float b = bf16_hi(w4[t]) - yh[8 * k + 2 * t + 1];
            d2 = fmaf(a, a, d2);
            d2 = fmaf(b, b, d2);
          }
        }
      }
      d2 += __shfl_xor(d2, 1);
      d2 += __shfl_xor(d2, 2);
      if (have && t4 == 0)
        atomicMax(reinterpret_cast<unsigned *>(F.hs + h * kHs + kHsLb), __float_as_uint(fg * sqrtf(d2)));
    }
    wave_sync();
  };
  // One lane per block marks the candidates whose bound, with a relative margin for rounding,
  // exceeds the head's best value; a wave scan of the counts places them in the list.
  int n = 0;
  for (int x0 = 0; x0 < nx; x0 += 64) {
    const int x = x0 + lane;
    int h;
    const float *blk = block_at(x, h);
    uint32_t bits = 0;
    if (blk) {
      const float *hs = F.hs + h * kHs;
      // candidate j is listed iff f g_j (Vmax + |yhat|) / l, with a margin, exceeds the best value
      const float thr = hs[kHsLb] / (scale_of(blk[kChM], hs[kHsM]) / hs[kHsL] *
                                     (blk[kChVmax] + hs[kHsYn]) * 1.0002f);
      const float4 *g4 = reinterpret_cast<const float4 *>(blk + kChG);
#pragma unroll
      for (int q = 0; q < kCand / 4; ++q) {
        const float4 v = g4[q];
        bits |= (v.x > thr ? 1u : 0u) << (4 * q);
        bits |= (v.y > thr ? 1u : 0u) << (4 * q + 1);
        bits |= (v.z > thr ? 1u : 0u) << (4 * q + 2);
        bits |= (v.w > thr ? 1u : 0u) << (4 * q + 3);
      }
      const unsigned long long bk = F.best[h];  // evaluated in step (3)
      const unsigned jb = (unsigned)(bk & 0xffffffffull) - (unsigned)(x * kCand);
      if (bk && jb < (unsigned)kCand) bits &= ~(1u << jb);
    }
    // exclusive prefix of the counts by bit planes (counts are at most kCand = 32)
    const int mine = __popc(bits);
    int excl = 0, total = 0;
#pragma unroll
    for (int b = 0; b < 6; ++b) {
      const uint64_t m = __ballot((mine >> b) & 1);
      excl += (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) << b;
      total += (int)__popcll(m) << b;
    }
    // entries p of this group (p = excl .. excl + mine - 1 for this lane) go out in list-sized
    // windows
    for (int done = 0; done < total;) {
      const int take = min(kListCap - n, total - done);
      int p = excl;
      for (uint32_t m = bits; m; m &= m - 1, ++p)
        if (p >= done && p < done + take) F.list[n + p - done] = x * kCand + __builtin_ctz(m);
      n += take;
      done += take;
      if (n == kListCap) {
        eval_list(n);
        n = 0;
      }
    }
  }
  if (n > 0) eval_list(n);

  // (5) A chunk whose non-candidate bound f (A + B |yhat|) / l still exceeds the best value is
  //     rescanned row by row.
  const float scale2 = L.scale * kLog2e;
  for (int x0 = 0; x0 < nx; x0 += 64) {
    const int x = x0 + lane;  // (s nchunk + k) GB + h
    bool need = false;
    if (x < nx) {
      const int h = x % GB, sk = x / GB, s = sk / L.nchunk, k = sk % L.nchunk;
      if (k * kChunkRows < min(cnt - s * R, R)) {
        const float *blk = C.base + s * C.sstride + k * C.kstride + h * C.hstride;
        const float *hs = F.hs + h * kHs;
        const float ub = scale_of(blk[kChM], hs[kHsM]) * (blk[kChA] + blk[kChB] * hs[kHsYn]) / hs[kHsL];
        need = ub > hs[kHsLb];
      }
    }
    uint64_t m = __ballot(need);
    if (m) load_q();
    while (m) {
      const int xx = x0 + (int)__builtin_ctzll(m);
      m &= m - 1;
      const int h = xx % GB, sk = xx / GB, s = sk / L.nchunk, k = sk % L.nchunk;
      const int ra = s * R + k * kChunkRows;
      const int rz = min(min(cnt, (s + 1) * R), ra + kChunkRows);
      const float *hs = F.hs + h * kHs;
      const float M = hs[kHsM];
      const float *qh = F.o + (GB + h) * kHeadDim;
      const float *yh = F.o + h * kHeadDim;
      const float *blk = C.base + s * C.sstride + k * C.kstride + h * C.hstride;
      const float fk = scale_of(blk[kChM], M) / hs[kHsL];
      const float bterm = blk[kChB] * hs[kHsYn];
      // only the rows of a candidate lane whose own bound still exceeds the best value: lane i
      // kept rows 2 (i / 4) and 2 (i / 4) + 1 of row group i % 4 in every tile of the chunk
      // (64 rows)
      const int i = lane >> 3;  // lane group i decides for candidate lane i
      const float ai = __uint_as_float(
          ((__float_as_uint(blk[kChAL + (i & 3) / 2 + 2 * (i >> 2)]) >> (16 * (i & 1))) & 0xffffu) << 16);
      const uint64_t lanes = __ballot((lane & 7) == 0 && fk * (ai + bterm) > hs[kHsLb]);
      // rows in the split's pivot list are in no sum here; their terms were taken in step (1c)
      const float *plist = P.at(s, h);
      const int pn = __float_as_int(plist[0]);
      float best = 0.0f;
      for (uint64_t lm = lanes; lm; lm &= lm - 1) {
        const int li = (int)__builtin_ctzll(lm) >> 3;
        if (lane == 0) atomicAdd(diag_of(L, u, h0), 1u);
        const int j = ra + 16 * (lane >> 1) + 4 * (li & 3) + 2 * (li >> 2) + (lane & 1);
        if (j >= rz) continue;
        bool listed = false;
#pragma unroll
        for (int e = 0; e < kPivMax; ++e) listed |= e < pn && __float_as_int(plist[1 + 3 * e]) == j;
        if (listed) continue;
        const uint4 *kr = reinterpret_cast<const uint4 *>(L.Kc + (cbase + j) * kHeadDim);
        const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + j) * kHeadDim);
        const float pj = L.pic[cbase + j];
        float dot = 0.0f, d2 = 0.0f;
        for (int half = 0; half < 2; ++half) {  // half a row per step keeps the registers down
          asm volatile("" ::: "memory");       // q and yhat stay in LDS
          uint4 kq[8], vq[8];
#pragma unroll
          for (int k2 = 0; k2 < 8; ++k2) {
            kq[k2] = kr[8 * half + k2];
            vq[k2] = vr[8 * half + k2];
          }
#pragma unroll
          for (int k2 = 0; k2 < 8; ++k2) {
            const uint32_t kw[4] = {kq[k2].x, kq[k2].y, kq[k2].z, kq[k2].w};
            const uint32_t vw[4] = {vq[k2].x, vq[k2].y, vq[k2].z, vq[k2].w};
            const int d0 = 64 * half + 8 * k2;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              dot = fmaf(qh[d0 + 2 * t], bf16_lo(kw[t]), dot);
              dot = fmaf(qh[d0 + 2 * t + 1], bf16_hi(kw[t]), dot);
              const float a = bf16_lo(vw[t]) - yh[d0 + 2 * t];
              const float b = bf16_hi(vw[t]) - yh[d0 + 2 * t + 1];
              d2 = fmaf(a, a, d2);
              d2 = fmaf(b, b, d2);
            }
          }
        }
        const float w = fast_exp2(dot * scale2 - fast_log2(pj) - M);
        best = fmaxf(best, sqrtf(1.0f - pj) * w * sqrtf(d2));
      }
      best = wave_max(best) / hs[kHsL];
      if (lane == 0) F.hs[h * kHs + kHsLb] = fmaxf(F.hs[h * kHs + kHsLb], best);
      wave_sync();
    }
  }

  // (5b) Heads whose one-pass variance cancelled (step (1)): Vhat and b again, directly over the
  //      unit's retained rows and about the reference point c0 = yhat (fp32) in LDS.  One row
  //      then dominates yhat, and yhat - c0 is of the order of c0's own rounding, so the pass
  //      accumulates l' = sum w, o' = sum w (v - c0), C0 = sum c, Cv' = sum c (v - c0) and
  //      S1 = sum c |v - c0|^2 (v - c0 is exact near the dominating row), then
  //        delta = o' / l',   Vhat l'^2 = S1 - 2 delta.Cv' + |delta|^2 C0
  //      (none of these terms cancels), and a second pass takes b exactly as
  //      max sqrt(1 - pi) w |(v - c0) - delta| / l'.  Heads go in groups of four; 16 lanes per
  //      row, 8 dims per lane, four rows per lane in flight.
  if (redo) {
    load_q();
    const int rq = lane >> 4, c = lane & 15;
    const float scale2d = L.scale * kLog2e;
    for (int hg = 0; hg < GB; hg += 4) {
      if (!((redo >> hg) & 0xfu)) continue;
      bool act[4];
      float q8[4][8], c8[4][8], Mh[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int h = hg + k;
        act[k] = h < GB && ((redo >> h) & 1u);
        const float *qs = F.o + (GB + (act[k] ? h : 0)) * kHeadDim + 8 * c;
        const float *cs = F.o + (act[k] ? h : 0) * kHeadDim + 8 * c;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          q8[k][e] = qs[e];
          c8[k][e] = cs[e];
        }
        Mh[k] = F.hs[(act[k] ? h : 0) * kHs + kHsM];
      }
      // Rows of a step: lane group rq takes rows j0 + 4 i + rq.  Rows past cnt get w = 0.
      constexpr int kIn = 4;
      auto load_rows = [&](int j0, uint4 (&kw)[kIn], uint4 (&vw)[kIn], float (&pj)[kIn],
                           bool (&ok)[kIn]) {
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
          const int j = j0 + 4 * i + rq;
          ok[i] = j < cnt;
          kw[i] = ok[i] ? reinterpret_cast<const uint4 *>(L.Kc + (cbase + j) * kHeadDim)[c]
                        : make_uint4(0u, 0u, 0u, 0u);
          vw[i] = ok[i] ? reinterpret_cast<const uint4 *>(L.Vc + (cbase + j) * kHeadDim)[c]
                        : make_uint4(0u, 0u, 0u, 0u);
          pj[i] = ok[i] ? L.pic[cbase + j] : 1.0f;
        }
      };
      // logit weight w of one row for head slot k (every lane of the row gets it)
      auto weight = [&](int k, const uint4 &kw, float p, bool ok) -> float {
        const uint32_t kk[4] = {kw.x, kw.y, kw.z, kw.w};
        float dot = 0.0f;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          dot = fmaf(q8[k][2 * t], bf16_lo(kk[t]), dot);
          dot = fmaf(q8[k][2 * t + 1], bf16_hi(kk[t]), dot);
        }
        dot = row16_sum(dot);
        return ok ? fast_exp2(fmaf(dot, scale2d, -fast_log2(p)) - Mh[k]) : 0.0f;
      };
      // pass 1: the sums about c0
      float op[4][8], cv[4][8], lp[4], c0s[4], s1[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        lp[k] = c0s[k] = s1[k] = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) op[k][e] = cv[k][e] = 0.0f;
      }
      for (int j0 = 0; j0 < cnt; j0 += 4 * kIn) {
        uint4 kw[kIn], vw[kIn];
        float pj[kIn];
        bool ok[kIn];
        load_rows(j0, kw, vw, pj, ok);
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
          const uint32_t vv[4] = {vw[i].x, vw[i].y, vw[i].z, vw[i].w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (!act[k]) continue;
            const float w = weight(k, kw[i], pj[i], ok[i]);
            const float cc = (1.0f - pj[i]) * w * w;
            float n2 = 0.0f;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const float d0 = bf16_lo(vv[t]) - c8[k][2 * t], d1 = bf16_hi(vv[t]) - c8[k][2 * t + 1];
              op[k][2 * t] = fmaf(w, d0, op[k][2 * t]);
              op[k][2 * t + 1] = fmaf(w, d1, op[k][2 * t + 1]);
              cv[k][2 * t] = fmaf(cc, d0, cv[k][2 * t]);
              cv[k][2 * t + 1] = fmaf(cc, d1, cv[k][2 * t + 1]);
              n2 = fmaf(d0, d0, n2);
              n2 = fmaf(d1, d1, n2);
            }
            n2 = row16_sum(n2);
            lp[k] += w;
            c0s[k] += cc;
            s1[k] = fmaf(cc, n2, s1[k]);
          }
        }
      }
      // combine the four row groups: vectors by lane exchange (every lane then holds the sums of
      // its 8 dims), scalars from one lane per row group
      float lt[4], vt[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!act[k]) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          op[k][e] += __shfl_xor(op[k][e], 16);
          op[k][e] += __shfl_xor(op[k][e], 32);
          cv[k][e] += __shfl_xor(cv[k][e], 16);
          cv[k][e] += __shfl_xor(cv[k][e], 32);
        }
        lt[k] = wave_sum(c == 0 ? lp[k] : 0.0f);
        const float c0t = wave_sum(c == 0 ? c0s[k] : 0.0f);
        const float s1t = wave_sum(c == 0 ? s1[k] : 0.0f);
        float dcv = 0.0f, dd = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          op[k][e] /= lt[k];  // delta, dims 8c .. 8c + 7
          dcv = fmaf(op[k][e], cv[k][e], dcv);
          dd = fmaf(op[k][e], op[k][e], dd);
        }
        dcv = row16_sum(dcv);  // every row group holds all 128 dims: one row's lanes suffice
        dd = row16_sum(dd);
        vt[k] = fmaxf(s1t - 2.0f * dcv + dd * c0t, 0.0f) / (lt[k] * lt[k]);
      }
      // pass 2: the range term with delta known
      float bm[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int j0 = 0; j0 < cnt; j0 += 4 * kIn) {
        uint4 kw[kIn], vw[kIn];
        float pj[kIn];
        bool ok[kIn];
        load_rows(j0, kw, vw, pj, ok);
#pragma unroll
        for (int i = 0; i < kIn; ++i) {
          const uint32_t vv[4] = {vw[i].x, vw[i].y, vw[i].z, vw[i].w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            if (!act[k]) continue;
            const float w = weight(k, kw[i], pj[i], ok[i]);
            float n2 = 0.0f;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const float d0 = (bf16_lo(vv[t]) - c8[k][2 * t]) - op[k][2 * t];
              const float d1 = (bf16_hi(vv[t]) - c8[k][2 * t + 1]) - op[k][2 * t + 1];
              n2 = fmaf(d0, d0, n2);
              n2 = fmaf(d1, d1, n2);
            }
            n2 = row16_sum(n2);
            bm[k] = fmaxf(bm[k], sqrtf(1.0f - pj[i]) * w * sqrtf(n2));
          }
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (!act[k]) continue;
        const float b = wave_max(bm[k]) / lt[k];
        if (lane == 0) {
          float *hs = F.hs + (hg + k) * kHs;
          hs[kHsV] = vt[k];
          hs[kHsLb] = b;
          L.vhat[uh0 + hg + k] = vt[k];
        }
      }
    }
    if (lane == 0) diag_of(L, u, h0)[1] = (uint32_t)__popc(redo);
    wave_sync();
  }

  // (6) b and the radius of eq. (4).
  if (lane < GB) {
    const float *hs = F.hs + lane * kHs;
    const float Ld = logf(1.0f / L.delta);
    const float b = hs[kHsLb];
    if (L.brange) L.brange[uh0 + lane] = b;
    if (L.radius) L.radius[uh0 + lane] = (sqrtf(2.0f * hs[kHsV] * Ld) + b * Ld) / (hs[kHsYn] + L.eps0);
  }
}

// Outputs of a unit with no retained rows.
template <int GB>
__device__ __forceinline__ void finalize_empty(const AttendLaunch &L, int u, int h0) {
  const int lane = threadIdx.x & 63;
  const int64_t uh0 = (int64_t)u * L.G + h0;
  for (int e = lane; e < GB * kHeadDim; e += 64) L.y[uh0 * kHeadDim + e] = 0.0f;
  if (lane < GB) {
    L.lse[uh0 + lane] = -INFINITY;
    if (!L.plain) {
      L.vhat[uh0 + lane] = 0.0f;
      if (L.brange) L.brange[uh0 + lane] = 0.0f;
      if (L.radius) L.radius[uh0 + lane] = 0.0f;
    }
  }
  if (lane == 0 && !L.plain) diag_of(L, u, h0)[0] = diag_of(L, u, h0)[1] = 0u;
}

template <int GB>
__device__ __forceinline__ void finalize_records(const AttendLaunch &L, int u, int h0, float *s_fin);

// One wave per (unit, split, head block).  Lane (g, c): MFMA column c is head slot c (weights for
// c < GB, variance weights for GB <= c < 2 GB, idle above); g selects the row group.
// Work-groups: one wave each (L.wpg = 1; units of several splits are then finalized by
// attend_finalize), or, when a unit is cut into L.wpg = L.nsplit splits, the unit's splits as the
// waves of one work-group: each writes its split record, counts itself in an LDS word, and the
// wave that arrives last finalizes the unit from the records (no second launch).  Waves of empty
// splits leave at once; the only work-group barrier is the one after the counter is cleared,
// which every wave reaches.
template <int GB, bool COOP>
__global__ __launch_bounds__(COOP ? 64 * kCoopMaxSplits : 64, 2) void attend_split_kernel(
    AttendLaunch L, int h0) {
  extern __shared__ float s_lds[];
  const int bid = blockIdx.x;
  const int wave = COOP ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
  constexpr bool coop = COOP;
  const int sp = coop ? wave : bid % L.nsplit;
  const int u = coop ? bid : bid / L.nsplit;
  const int lane = (int)__lane_id();  // recomputed where needed rather than kept live (registers)
  const int g = lane >> 4, c = lane & 15;
  // this wave's LDS: [nchunk][GB][kChunkFloats] chunk blocks, then [GB][kPivFloats] pivot lists
  float *s_chunk = s_lds + (coop ? (size_t)wave * (L.nchunk * kChunkFloats + kPivFloats) * GB : 0);
  int *s_arrived = reinterpret_cast<int *>(s_lds + L.coop_counter);
  if (coop) {
    if (threadIdx.x == 0) *s_arrived = 0;
    __syncthreads();  // before any wave can leave or arrive
  }
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int64_t held = min((int64_t)L.count[u], cap);
  const int cnt = (int)min(held, (int64_t)L.nsplit * L.split_rows);
  if (L.status && sp == 0 && h0 == 0 && lane == 0 && !L.plain)
    L.status[u] = ((int64_t)L.count[u] > cap ? EBD_ST_CAP_OVERFLOW : 0u) |
                  (held > (int64_t)cnt ? EBD_ST_BAD_LAYOUT : 0u);
  const int row0 = sp * L.split_rows;
  if (row0 >= cnt) {  // empty split: the finalize skips it; an empty unit gets empty outputs
    if (sp == 0 && (COOP || L.nsplit == 1)) finalize_empty<GB>(L, u, h0);
    return;
  }
  const int nrow = min(cnt - row0, L.split_rows);

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
  // A finite floor rather than -inf: a split whose only rows are pivots keeps no row in its sums,
  // and its weights exp2(-inf - floor) are then 0 (exp2(-inf + inf) would be NaN); scale factors
  // from that floor to any real maximum underflow to 0 as well.
  S.mrun = active ? -1e30f : 0.0f;
  S.s0 = S.s1 = 0.0f;
  S.pl = -INFINITY;
  float *s_piv = s_chunk + L.nchunk * GB * kChunkFloats;  // [GB][kPivFloats]
  if (isW && g == 0) {  // empty lists
    s_piv[c * kPivFloats] = __int_as_float(0);
    s_piv[c * kPivFloats + kPivLogit] = -INFINITY;
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    S.ck[e] = S.cg[e] = 0.0f;
    S.cr[e] = -1;
  }
  S.dk = S.dg = 0.0f;

  // The split's rows only: anything past them reads as zero.
  const int64_t r0 = cbase + row0;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(L.Kc + r0 * kHeadDim, (uint32_t)nrow * 256u);
  const __amdgpu_buffer_rsrc_t rV = make_rsrc(L.Vc + r0 * kHeadDim, (uint32_t)nrow * 256u);
  const __amdgpu_buffer_rsrc_t rP = make_rsrc(L.pic + r0, (uint32_t)nrow * 4u);
  const float scale2 = L.scale * kLog2e;
  const bool plain = L.plain != 0;
  const int ntile = (nrow + 15) / 16;
  const int nv0 = active ? nrow - 4 * g : -1;  // valid rows of this lane's row group in tile 0
  const int rb0 = row0 + 4 * g;

  // Three tiles in registers: two load while the third is computed.  The loop body is straight
  // line (whole triples), so the compiler waits for exactly the tile it is about to use.
  Tile T0, T1, T2;
  load_tile(T0, rK, rV, rP, 0, g, c);
  load_tile(T1, rK, rV, rP, 1, g, c);
  constexpr int kChunkTiles = kChunkRows / 16;
  // tile tt of the split, then the flush of its chunk if tt ends one
  auto step = [&](const Tile &T, int tt) {
    split_tile<(GB > 7)>(S, T, qop, nv0 - 16 * tt, rb0 + 16 * tt, isC, plain, scale2, s_piv, hs, isW);
    if ((tt + 1) % kChunkTiles == 0)
      flush_chunk<GB>(S, s_chunk, tt / kChunkTiles, g, c, row0 + (tt / kChunkTiles) * kChunkRows);
  };
  int t = 0;
  for (; t + 3 <= ntile; t += 3) {
    load_tile(T2, rK, rV, rP, t + 2, g, c);
    step(T0, t);
    load_tile(T0, rK, rV, rP, t + 3, g, c);
    step(T1, t + 1);
    load_tile(T1, rK, rV, rP, t + 4, g, c);
    step(T2, t + 2);
  }
  if (t < ntile) step(T0, t);
  if (t + 1 < ntile) step(T1, t + 1);
  // every chunk is flushed once: full ones where they end, a partial last one here
  const int nck = (ntile + kChunkTiles - 1) / kChunkTiles;
  if (ntile % kChunkTiles != 0)
    flush_chunk<GB>(S, s_chunk, nck - 1, g, c, row0 + (nck - 1) * kChunkRows);

  // ---- epilogue ------------------------------------------------------------------------------
  float s0 = S.s0, s1 = S.s1;
  s0 += __shfl_xor(s0, 16);
  s0 += __shfl_xor(s0, 32);
  s1 += __shfl_xor(s1, 16);
  s1 += __shfl_xor(s1, 32);
  if (!COOP && L.nsplit == 1) {
    // The unit is this one split: its sums go to LDS beside the chunk blocks and the wave
    // finalizes its heads itself (no record, no second launch).
    FinLds<GB> F(s_piv + GB * kPivFloats);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int slot = 4 * g + i;
      if (slot < 2 * GB) {
        float4 *dst = reinterpret_cast<float4 *>(F.o + slot * kHeadDim + 8 * c);
        dst[0] = make_float4(S.acc[0][i], S.acc[1][i], S.acc[2][i], S.acc[3][i]);
        dst[1] = make_float4(S.acc[4][i], S.acc[5][i], S.acc[6][i], S.acc[7][i]);
      }
    }
    if (g == 0 && isW) {
      F.hs[c * kHs + kHsM] = S.mrun;
      F.hs[c * kHs + kHsL] = s0;
    } else if (g == 0 && isC) {
      F.hs[(c - GB) * kHs + kHsC0] = s0;
      F.hs[(c - GB) * kHs + kHsC2] = s1;
    }
    if (lane == 0 && !L.plain) diag_of(L, u, h0)[0] = diag_of(L, u, h0)[1] = 0u;
    wave_sync();
    const CandSrc C{s_chunk, 0, GB * kChunkFloats, kChunkFloats};
    const PivSrc P{s_piv, 0, kPivFloats};
    pivot_prepare<GB>(L, cbase, 1, P, F);
    finalize_block<GB>(L, u, h0, cnt, cbase, 1, C, P, F);
    return;
  }
  // Several splits: this one's record (sums from registers, chunk blocks from LDS).
  float *rec_base = L.part + (((int64_t)u * L.nsplit + sp) * L.G + h0) * L.rec;
  // o (slots < GB) and Cv (slots GB .. 2GB-1): lane (g, c) holds slots 4g + i, dims 8c .. 8c + 7
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int slot = 4 * g + i;
    if (slot < 2 * GB) {
      const int hh = slot < GB ? slot : slot - GB;
      float4 *dst = reinterpret_cast<float4 *>(rec_base + (int64_t)hh * L.rec +
                                               (slot < GB ? kRecO : kRecCv) + 8 * c);
      dst[0] = make_float4(S.acc[0][i], S.acc[1][i], S.acc[2][i], S.acc[3][i]);
      dst[1] = make_float4(S.acc[4][i], S.acc[5][i], S.acc[6][i], S.acc[7][i]);
    }
  }
  if (g == 0 && isW) {
    float *rec = rec_base + (int64_t)c * L.rec;
    rec[kRecM] = S.mrun;
    rec[kRecL] = s0;
  } else if (g == 0 && isC) {
    float *rec = rec_base + (int64_t)(c - GB) * L.rec;
    rec[kRecC0] = s0;
    rec[kRecC2] = s1;
  }
  wave_sync();  // the chunk blocks and the pivot lists are in LDS
  for (int e = lane; e < GB * kPivFloats; e += 64)
    rec_base[(int64_t)(e / kPivFloats) * L.rec + kRecPiv + e % kPivFloats] = s_piv[e];
  const int nblk = nck * GB * kChunkFloats;
  for (int e = lane; e < nblk; e += 64) {
    const int k = e / (GB * kChunkFloats), r = e % (GB * kChunkFloats);
    const int hh = r / kChunkFloats, j = r % kChunkFloats;
    rec_base[(int64_t)hh * L.rec + kRecChunks + k * kChunkFloats + j] = s_chunk[e];
  }
  if (!COOP) return;
  // The record is complete (the release makes it visible to the work-group's other waves before
  // the count moves); the last of the unit's nsp waves to arrive finalizes.  Its FinLds reuses
  // the LDS of the splits, whose waves are all done with it by then.
  const int nsp = (cnt + L.split_rows - 1) / L.split_rows;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  int before = 0;
  if (lane == 0) before = __hip_atomic_fetch_add(s_arrived, 1, __ATOMIC_RELAXED,
                                                 __HIP_MEMORY_SCOPE_WORKGROUP);
  before = __builtin_amdgcn_readfirstlane(before);
  if (before != nsp - 1) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  finalize_records<GB>(L, u, h0, s_lds);
}

// attend_finalize: one wave per (unit, head block) when units are cut into several splits.  The
// split records are combined into LDS, then the unit is finalized like a fused split, reading
// the candidate blocks from the records (a lane per block, whole blocks as float4).  Every global
// read of the records is issued in batches, so the wave waits on a handful of round trips rather
// than one per split or candidate.
// Float offset of the split scale factors in the finalize's LDS (after FinLds).
template <int GB>
__host__ __device__ constexpr size_t fin_scale_off() {
  return FinLds<GB>::bytes() / sizeof(float);
}

// The finalize of unit u from its split records, by one wave (s_fin: FinLds, then the split
// scale factors).
template <int GB>
__device__ __forceinline__ void finalize_records(const AttendLaunch &L, int u, int h0, float *s_fin) {
  const int lane = threadIdx.x & 63;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int cnt = (int)min(min((int64_t)L.count[u], cap), (int64_t)L.nsplit * L.split_rows);
  if (cnt == 0) {
    finalize_empty<GB>(L, u, h0);
    return;
  }
  if (lane == 0 && !L.plain) diag_of(L, u, h0)[0] = diag_of(L, u, h0)[1] = 0u;
  wave_sync();  // the zeroed words are in place before the finalize's own updates
  const int nsp = (cnt + L.split_rows - 1) / L.split_rows;
  const float *rec0 = L.part + ((int64_t)u * L.nsplit * L.G + h0) * L.rec;  // (s, h) at s G rec + h rec
  const int64_t sstride = (int64_t)L.G * L.rec;
  FinLds<GB> F(s_fin);
  float *fsc = s_fin + fin_scale_off<GB>();  // [nsplit][GB]: scale of (s, h)

  // Scalars (M, l, C0, C2) of every (split, head): one float4 per lane and head, all in flight.
  for (int s0 = 0; s0 < nsp; s0 += 64) {
    const int sl = s0 + lane;
    float4 r[GB];
#pragma unroll
    for (int h = 0; h < GB; ++h)
      r[h] = sl < nsp ? *reinterpret_cast<const float4 *>(rec0 + sl * sstride + h * L.rec + kRecM)
                      : make_float4(-INFINITY, 0.0f, 0.0f, 0.0f);
#pragma unroll
    for (int h = 0; h < GB; ++h) {
      if (sl < nsp) fsc[sl * GB + h] = r[h].x;  // the split's running max, for now
      const float M = wave_max(r[h].x);
      const float mo = s0 == 0 ? -INFINITY : F.hs[h * kHs + kHsM];  // earlier batches
      const float Mn = fmaxf(M, mo);
      const float f = scale_of(r[h].x, Mn);
      float l = wave_sum(f * r[h].y), c0 = wave_sum(f * f * r[h].z), c2 = wave_sum(f * f * r[h].w);
      if (lane == 0) {
        const float fo = s0 == 0 ? 0.0f : scale_of(mo, Mn);
        F.hs[h * kHs + kHsM] = Mn;
        F.hs[h * kHs + kHsL] = l + (s0 == 0 ? 0.0f : fo * F.hs[h * kHs + kHsL]);
        F.hs[h * kHs + kHsC0] = c0 + (s0 == 0 ? 0.0f : fo * fo * F.hs[h * kHs + kHsC0]);
        F.hs[h * kHs + kHsC2] = c2 + (s0 == 0 ? 0.0f : fo * fo * F.hs[h * kHs + kHsC2]);
      }
      wave_sync();
    }
  }
  // the scale of every split to the combined max
  for (int e = lane; e < nsp * GB; e += 64) fsc[e] = scale_of(fsc[e], F.hs[(e % GB) * kHs + kHsM]);
  wave_sync();

  // o and Cv: two dims per lane, every slot of SP splits in flight at once.
  {
    constexpr int SP = GB <= 4 ? 4 : 2;
    float2 acc[2 * GB];
#pragma unroll
    for (int slot = 0; slot < 2 * GB; ++slot) acc[slot] = make_float2(0.0f, 0.0f);
    for (int sp = 0; sp < nsp; sp += SP) {
      float2 a[SP][2 * GB];
#pragma unroll
      for (int q = 0; q < SP; ++q)
#pragma unroll
        for (int slot = 0; slot < 2 * GB; ++slot) {
          const int h = slot < GB ? slot : slot - GB;
          const int off = slot < GB ? kRecO : kRecCv;
          a[q][slot] = sp + q < nsp ? reinterpret_cast<const float2 *>(
                                          rec0 + (sp + q) * sstride + h * L.rec + off)[lane]
                                    : make_float2(0.0f, 0.0f);
        }
#pragma unroll
      for (int q = 0; q < SP; ++q) {
        if (sp + q >= nsp) break;
#pragma unroll
        for (int slot = 0; slot < 2 * GB; ++slot) {
          const int h = slot < GB ? slot : slot - GB;
          float f = fsc[(sp + q) * GB + h];
          if (slot >= GB) f *= f;
          acc[slot].x = fmaf(f, a[q][slot].x, acc[slot].x);
          acc[slot].y = fmaf(f, a[q][slot].y, acc[slot].y);
        }
      }
    }
#pragma unroll
    for (int slot = 0; slot < 2 * GB; ++slot)
      reinterpret_cast<float2 *>(F.o + slot * kHeadDim)[lane] = acc[slot];
  }

  wave_sync();
  const CandSrc C{rec0 + kRecChunks, sstride, kChunkFloats, L.rec};
  const PivSrc P{rec0 + kRecPiv, sstride, L.rec};
  pivot_prepare<GB>(L, cbase, nsp, P, F);
  finalize_block<GB>(L, u, h0, cnt, cbase, nsp, C, P, F);
}

template <int GB>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(1, 2)))
void attend_finalize_kernel(AttendLaunch L, int h0) {
  extern __shared__ float s_fin[];
  finalize_records<GB>(L, blockIdx.x, h0, s_fin);
}

template <int GB>
size_t attend_finalize_lds(const AttendLaunch &L) {
  return (fin_scale_off<GB>() + (size_t)L.nsplit * GB) * sizeof(float);
}

size_t attend_workspace_bytes(int32_t U, int32_t nsplit, int32_t G, int32_t split_rows) {
  const size_t nhb = (size_t)((G + kHeadBlock - 1) / kHeadBlock);
  const size_t diag = ((size_t)U * nhb * 2 * sizeof(uint32_t) + 255) / 256 * 256;
  if (nsplit <= 1) return diag;  // fused: no split records
  return diag + (size_t)U * (size_t)nsplit * (size_t)G * (size_t)attend_record_floats(split_rows) *
                    sizeof(float);
}

size_t attend_finalize_lds_gb(const AttendLaunch &L, int gb) {
  switch (gb) {
    case 1: return attend_finalize_lds<1>(L);
    case 2: return attend_finalize_lds<2>(L);
    case 3: return attend_finalize_lds<3>(L);
    case 4: return attend_finalize_lds<4>(L);
    case 5: return attend_finalize_lds<5>(L);
    case 6: return attend_finalize_lds<6>(L);
    case 7: return attend_finalize_lds<7>(L);
    default: return attend_finalize_lds<8>(L);
  }
}

// Float offset of the arrival count of a work-group of a unit's splits: after the splits' own
// LDS and after the finalize's, which reuses the splits' space.
int32_t attend_coop_counter(const AttendLaunch &L, int gb) {
  const size_t part = ((size_t)L.nchunk * kChunkFloats + kPivFloats) * gb;
  const size_t fin = attend_finalize_lds_gb(L, gb) / sizeof(float);
  const size_t need = part * (size_t)L.wpg > fin ? part * (size_t)L.wpg : fin;
  return (int32_t)((need + 3) / 4 * 4);
}

size_t attend_split_lds(const AttendLaunch &L, int gb) {
  size_t b = ((size_t)L.nchunk * kChunkFloats + kPivFloats) * gb * sizeof(float);
  if (L.nsplit > 1 && L.wpg > 1) return ((size_t)attend_coop_counter(L, gb) + 4) * sizeof(float);
  if (L.nsplit == 1) {
    size_t f = 0;
    switch (gb) {
      case 1: f = FinLds<1>::bytes(); break;
      case 2: f = FinLds<2>::bytes(); break;
      case 3: f = FinLds<3>::bytes(); break;
      case 4: f = FinLds<4>::bytes(); break;
      case 5: f = FinLds<5>::bytes(); break;
      case 6: f = FinLds<6>::bytes(); break;
      case 7: f = FinLds<7>::bytes(); break;
      default: f = FinLds<8>::bytes(); break;
    }
    b += f;
  }
  return b;
}

size_t attend_fused_lds_bytes(int32_t split_rows, int gb) {
  AttendLaunch L{};
  L.nsplit = 1;
  L.wpg = 1;
  L.nchunk = attend_chunks(split_rows);
  return attend_split_lds(L, gb);
}

size_t attend_part_lds_bytes(int32_t split_rows, int gb) {
  AttendLaunch L{};
  L.nsplit = 2;
  L.wpg = 1;
  L.nchunk = attend_chunks(split_rows);
  return attend_split_lds(L, gb);
}

hipError_t launch_attend_split(const AttendLaunch &L0, hipStream_t s) {
  if (L0.wpg != 1 && (L0.wpg != L0.nsplit || L0.wpg > kCoopMaxSplits)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((int64_t)L0.U * (L0.wpg > 1 ? 1 : L0.nsplit))),
      block(kAttendThreads * L0.wpg);
  for (int h0 = 0; h0 < L0.G; h0 += kHeadBlock) {
    const int gb = min(kHeadBlock, L0.G - h0);
    AttendLaunch L = L0;
    L.coop_counter = L.wpg > 1 ? attend_coop_counter(L, gb) : 0;
    const size_t lds = attend_split_lds(L, gb);
    const bool coop = L.wpg > 1;
    switch (gb) {
#define EBD_SPLIT(N)                                                                              \
  case N:                                                                                         \
    if (coop)                                                                                     \
      hipLaunchKernelGGL((attend_split_kernel<N, true>), grid, block, lds, s, L, h0);             \
    else                                                                                          \
      hipLaunchKernelGGL((attend_split_kernel<N, false>), grid, block, lds, s, L, h0);            \
    break;
      EBD_SPLIT(1)
      EBD_SPLIT(2)
      EBD_SPLIT(3)
      EBD_SPLIT(4)
      EBD_SPLIT(5)
      EBD_SPLIT(6)
      EBD_SPLIT(7)
      default: EBD_SPLIT(8)
#undef EBD_SPLIT
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_attend_finalize(const AttendLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)L.U), block(64);
  for (int h0 = 0; h0 < L.G; h0 += kHeadBlock) {
    const int gb = min(kHeadBlock, L.G - h0);
    switch (gb) {
#define EBD_FIN(N)                                                                             \
  case N:                                                                                      \
    hipLaunchKernelGGL(attend_finalize_kernel<N>, grid, block, attend_finalize_lds<N>(L), s, L, \
                       h0);                                                                    \
    break;
      EBD_FIN(1)
      EBD_FIN(2)
      EBD_FIN(3)
      EBD_FIN(4)
      EBD_FIN(5)
      EBD_FIN(6)
      EBD_FIN(7)
      default: EBD_FIN(8)
#undef EBD_FIN
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace ebd
