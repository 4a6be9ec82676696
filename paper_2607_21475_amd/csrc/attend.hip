// attend.hip -- certified decode attention over the retained rows on gfx950.
//
// Per (unit, query head h), over the retained set S (Sec. 3.3 eq. (3), Theorem 2; Sec. 3.4 eq. (4)):
//   l_j = scale q_h.k_j - ln pi_j                 (Hajek weight a_j / pi_j as a logit offset)
//   w_j = exp(l_j - m),  m = running max          (online softmax)
//   yhat = sum w v / sum w,   ln Nhat = m + ln sum w
//   c_j = (1 - pi_j) w_j^2 = (1 - pi)/pi^2 a^2 e^{-2m}:  Vhat = sum c |v - yhat|^2 / (sum w)^2,
//     accumulated in one pass as C2 - 2 yhat.Cv + |yhat|^2 C0 with C0 = sum c, Cv = sum c v,
//     C2 = sum c |v|^2 (the e^{-2m} factors cancel against (sum w)^2)
//   b = max_j sqrt(1 - pi_j) w_j |v_j - yhat| / sum w  (exact: streaming candidates + bound check)
//
// attend_split (one work-group of four waves per (unit, split of the retained rows)):
//   A 16-row tile per wave step.  q.k runs on MFMA (16x16x32 bf16, exact products, fp32 sums):
//   A = K tile (16 rows x 32 dims per k-block, loaded straight from HBM in operand layout),
//   B = [q_0 .. q_{GB-1}, q_0 .. q_{GB-1}, 0 ..] (16 columns).  Each lane then holds 4 rows x 1
//   column of logits; columns < GB become weights w, columns GB..2GB-1 (same logits) become
//   variance weights c.  One f32 16x16x4 MFMA per (row group, 8-dim block) then forms
//   o = sum w v (rows < GB) and Cv = sum c v (rows GB..2GB-1) together, with V taken directly in
//   its natural row-major layout (no transpose, exact fp32 products).
// attend_finalize (one work-group per unit): log-sum-exp combine of the split records, yhat,
//   Vhat, ln Nhat, the exact range term b (candidate rows re-read; a split is rescanned only if
//   its bound cannot exclude a larger term) and the radius r.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

__device__ __forceinline__ void topc_insert(float kap, float gb, int row, float (&ck)[4],
                                            float (&cg)[4], int (&ci)[4], float &dk, float &dg) {
  if (kap > ck[3]) {
    dk = fmaxf(dk, ck[3]);
    dg = fmaxf(dg, cg[3]);
    if (kap > ck[1]) {
      ck[3] = ck[2]; cg[3] = cg[2]; ci[3] = ci[2];
      ck[2] = ck[1]; cg[2] = cg[1]; ci[2] = ci[1];
      if (kap > ck[0]) {
        ck[1] = ck[0]; cg[1] = cg[0]; ci[1] = ci[0];
        ck[0] = kap; cg[0] = gb; ci[0] = row;
      } else {
        ck[1] = kap; cg[1] = gb; ci[1] = row;
      }
    } else {
      if (kap > ck[2]) {
        ck[3] = ck[2]; cg[3] = cg[2]; ci[3] = ci[2];
        ck[2] = kap; cg[2] = gb; ci[2] = row;
      } else {
        ck[3] = kap; cg[3] = gb; ci[3] = row;
      }
    }
  } else {
    dk = fmaxf(dk, kap);
    dg = fmaxf(dg, gb);
  }
}

__device__ __forceinline__ float scale_of(float mw, float M) {
  return (mw == -INFINITY) ? 0.0f : __expf(mw - M);
}

}  // namespace

template <int GB>
__global__ __launch_bounds__(kAttendThreads) void attend_split_kernel(AttendLaunch L, int h0) {
  __shared__ float s_acc[4][16][kHeadDim];
  __shared__ float s_m[4][16], s_s0[4][16], s_s1[4][16];
  __shared__ float s_ck[4][GB][4][4], s_cg[4][GB][4][4];
  __shared__ int s_ci[4][GB][4][4];
  __shared__ float s_dk[4][GB][4], s_dg[4][GB][4];

  const int bid = blockIdx.x;
  const int sp = bid % L.nsplit;
  const int u = bid / L.nsplit;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, c = lane & 15;
  if (bid == 0 && tid == 0 && h0 == 0) L.diag[0] = 0u;

  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int64_t cnt = min(min((int64_t)L.count[u], cap), (int64_t)L.nsplit * L.split_rows);
  const int64_t row0 = (int64_t)sp * L.split_rows;
  if (row0 >= cnt) return;  // empty split: the finalize pass skips it
  const int64_t row1 = min(cnt, row0 + (int64_t)L.split_rows);

  const bool isW = c < GB;
  const bool isC = (c >= GB) && (c < 2 * GB);
  const int hs = isW ? c : (isC ? c - GB : 0);

  // B operand of the q.k MFMA: column c holds q_{hs}; lane (g, c) supplies dims 32kb + 8g .. +7.
  bf16x8 qop[4];
  {
    const uint4 *qh = reinterpret_cast<const uint4 *>(L.q + ((int64_t)u * L.G + h0 + hs) * kHeadDim);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      const uint4 w = (isW || isC) ? qh[4 * kb + g] : make_uint4(0u, 0u, 0u, 0u);
      qop[kb] = __builtin_bit_cast(bf16x8, w);
    }
  }

  f32x4 acc[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) acc[db] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float mrun = -INFINITY, s0 = 0.0f, s1 = 0.0f;
  float ck[4] = {0.0f, 0.0f, 0.0f, 0.0f}, cg[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  int ci[4] = {-1, -1, -1, -1};
  float dk = 0.0f, dg = 0.0f;

  const uint4 *Kb = reinterpret_cast<const uint4 *>(L.Kc + cbase * kHeadDim);
  const uint4 *Vb = reinterpret_cast<const uint4 *>(L.Vc + cbase * kHeadDim);
  const float *Pb = L.pic + cbase;
  const float scale = L.scale;
  const int ntile = (int)((row1 - row0 + 15) / 16);

  for (int tt = wave; tt < ntile; tt += 4) {
    const int64_t rb = row0 + 16 * (int64_t)tt;
    // K tile rows rb + c (A operand, row = c); invalid rows read row0 and are masked below.
    const int64_t rk = (rb + c < row1) ? rb + c : row0;
    uint4 kraw[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) kraw[kb] = Kb[rk * (kHeadDim / 8) + 4 * kb + g];
    // V rows rb + 4g + j, dims 8c .. 8c + 7 (B operand of the weighted sums).
    uint4 vraw[4];
    float p[4];
    bool tv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t r = rb + 4 * g + j;
      tv[j] = r < row1;
      const int64_t rv = tv[j] ? r : row0;
      vraw[j] = Vb[rv * (kHeadDim / 8) + c];
      p[j] = tv[j] ? Pb[r] : 1.0f;
    }

    f32x4 sacc = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kraw[kb]), qop[kb],
                                                     sacc, 0, 0, 0);
    // lane (g, c): logits of rows rb + 4g + i for head slot c
    float lg[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      lg[i] = (tv[i] && (isW || isC)) ? sacc[i] * scale - __logf(p[i]) : -INFINITY;

    float tmax = fmaxf(fmaxf(lg[0], lg[1]), fmaxf(lg[2], lg[3]));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(mrun, tmax);
    if (__any(mnew > mrun)) {
      const float alpha = (mnew > mrun) ? __expf(mrun - mnew) : 1.0f;
      const float as = isC ? alpha * alpha : alpha;  // variance terms carry e^{-2m}
      s0 *= as;
      s1 *= as;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        ck[e] *= alpha;
        cg[e] *= alpha;
      }
      dk *= alpha;
      dg *= alpha;
      float ai[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) ai[i] = __shfl(as, 4 * g + i);  // factor of accumulator row 4g + i
#pragma unroll
      for (int db = 0; db < 8; ++db) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[db][i] *= ai[i];
      }
      mrun = mnew;
    }

    float vf[4][8], nv2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w4[4] = {vraw[j].x, vraw[j].y, vraw[j].z, vraw[j].w};
      float sq = 0.0f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        vf[j][2 * k] = bf16_lo(w4[k]);
        vf[j][2 * k + 1] = bf16_hi(w4[k]);
        sq += vf[j][2 * k] * vf[j][2 * k] + vf[j][2 * k + 1] * vf[j][2 * k + 1];
      }
      nv2[j] = row16_sum(sq);
    }

    float val[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float w = (lg[i] == -INFINITY) ? 0.0f : __expf(lg[i] - mrun);
      const float omp = 1.0f - p[i];
      if (isW) {
        val[i] = w;
        s0 += w;
        const float gb = sqrtf(omp) * w;
        topc_insert(gb * sqrtf(nv2[i]), gb, (int)(rb + 4 * g + i), ck, cg, ci, dk, dg);
      } else if (isC) {
        const float cc = omp * w * w;
        val[i] = cc;
        s0 += cc;
        s1 += cc * nv2[i];
      } else {
        val[i] = 0.0f;
      }
    }

#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int db = 0; db < 8; ++db)
        acc[db] = __builtin_amdgcn_mfma_f32_16x16x4f32(val[j], vf[j][db], acc[db], 0, 0, 0);
    }
  }

  // ---- wave results to LDS -------------------------------------------------------------------
  s0 += __shfl_xor(s0, 16);
  s0 += __shfl_xor(s0, 32);
  s1 += __shfl_xor(s1, 16);
  s1 += __shfl_xor(s1, 32);
  if (g == 0) {
    s_m[wave][c] = mrun;
    s_s0[wave][c] = s0;
    s_s1[wave][c] = s1;
  }
#pragma unroll
  for (int db = 0; db < 8; ++db) {
#pragma unroll
    for (int i = 0; i < 4; ++i) s_acc[wave][4 * g + i][8 * c + db] = acc[db][i];
  }
  if (isW) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      s_ck[wave][c][g][e] = ck[e];
      s_cg[wave][c][g][e] = cg[e];
      s_ci[wave][c][g][e] = ci[e];
    }
    s_dk[wave][c][g] = dk;
    s_dg[wave][c][g] = dg;
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
  if (tid < GB) {
    const int hh = tid;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) M = fmaxf(M, s_m[w][hh]);
    float lsum = 0.0f, c0 = 0.0f, c2 = 0.0f, A = 0.0f, B = 0.0f;
    float tk[kCand], tg[kCand];
    int ti[kCand];
#pragma unroll
    for (int k = 0; k < kCand; ++k) {
      tk[k] = 0.0f;
      tg[k] = 0.0f;
      ti[k] = -1;
    }
    for (int w = 0; w < 4; ++w) {
      const float f = scale_of(s_m[w][hh], M);
      lsum += f * s_s0[w][hh];
      c0 += f * f * s_s0[w][GB + hh];
      c2 += f * f * s_s1[w][GB + hh];
      for (int gg = 0; gg < 4; ++gg) {
        A = fmaxf(A, f * s_dk[w][hh][gg]);
        B = fmaxf(B, f * s_dg[w][hh][gg]);
        for (int e = 0; e < 4; ++e) {
          float kap = f * s_ck[w][hh][gg][e];
          float gv = f * s_cg[w][hh][gg][e];
          int row = s_ci[w][hh][gg][e];
          if (row < 0) continue;
          if (kap > tk[kCand - 1]) {
            // insert into the sorted list; the displaced entry becomes a non-candidate
            A = fmaxf(A, tk[kCand - 1]);
            B = fmaxf(B, tg[kCand - 1]);
            int k = kCand - 1;
            while (k > 0 && tk[k - 1] < kap) {
              tk[k] = tk[k - 1];
              tg[k] = tg[k - 1];
              ti[k] = ti[k - 1];
              --k;
            }
            tk[k] = kap;
            tg[k] = gv;
            ti[k] = row;
          } else {
            A = fmaxf(A, kap);
            B = fmaxf(B, gv);
          }
        }
      }
    }
    float *rec = rec_base + (int64_t)hh * kRec;
    rec[kRecM] = M;
    rec[kRecL] = lsum;
    rec[kRecC0] = c0;
    rec[kRecC2] = c2;
    rec[kRecA] = A;
    rec[kRecB] = B;
    for (int k = 0; k < kCand; ++k) {
      rec[kRecCandG + k] = tg[k];
      rec[kRecCandI + k] = __int_as_float(ti[k]);
    }
  }
}

// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ float block_sum256(float v, float *red) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}
__device__ __forceinline__ float block_max256(float v, float *red) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[wv] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ __launch_bounds__(kAttendThreads) void attend_finalize_kernel(AttendLaunch L) {
  __shared__ float s_y[kHeadDim];
  __shared__ float red[4];
  const int u = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int64_t cnt = min(min((int64_t)L.count[u], cap), (int64_t)L.nsplit * L.split_rows);
  const int nsp = (int)((cnt + L.split_rows - 1) / L.split_rows);
  const float Ld = logf(1.0f / L.delta);

  for (int h = 0; h < L.G; ++h) {
    const int64_t uh = (int64_t)u * L.G + h;
    if (cnt == 0) {
      if (tid < kHeadDim) L.y[uh * kHeadDim + tid] = 0.0f;
      if (tid == 0) {
        L.vhat[uh] = 0.0f;
        L.lse[uh] = -INFINITY;
        if (L.brange) L.brange[uh] = 0.0f;
        if (L.radius) L.radius[uh] = 0.0f;
      }
      continue;
    }
    const float *rec0 = L.part + ((int64_t)u * L.nsplit * L.G + h) * kRec;
    const int64_t rstride = (int64_t)L.G * kRec;
    float M = -INFINITY;
    for (int s = 0; s < nsp; ++s) M = fmaxf(M, rec0[s * rstride + kRecM]);
    float l = 0.0f, C0 = 0.0f, C2 = 0.0f;
    for (int s = 0; s < nsp; ++s) {
      const float *r = rec0 + s * rstride;
      const float f = scale_of(r[kRecM], M);
      l += f * r[kRecL];
      C0 += f * f * r[kRecC0];
      C2 += f * f * r[kRecC2];
    }
    float yv = 0.0f, cv = 0.0f;
    if (tid < kHeadDim) {
      for (int s = 0; s < nsp; ++s) {
        const float *r = rec0 + s * rstride;
        yv += scale_of(r[kRecM], M) * r[kRecO + tid];
      }
      yv /= l;
      s_y[tid] = yv;
    } else {
      const int d = tid - kHeadDim;
      for (int s = 0; s < nsp; ++s) {
        const float *r = rec0 + s * rstride;
        const float f = scale_of(r[kRecM], M);
        cv += f * f * r[kRecCv + d];
      }
    }
    __syncthreads();
    const float ynorm2 = block_sum256(tid < kHeadDim ? yv * yv : 0.0f, red);
    const float ycv = block_sum256(tid >= kHeadDim ? s_y[tid - kHeadDim] * cv : 0.0f, red);
    const float V = fmaxf(C2 - 2.0f * ycv + ynorm2 * C0, 0.0f) / (l * l);
    const float ynorm = sqrtf(ynorm2);

    // Range term: exact value at the candidate rows ...
    const uint16_t *Vrows = L.Vc + cbase * kHeadDim;
    const float y0 = s_y[2 * lane], y1 = s_y[2 * lane + 1];
    float lb = 0.0f;
    for (int e = wv; e < nsp * kCand; e += 4) {
      const float *r = rec0 + (e / kCand) * rstride;
      const int row = __float_as_int(r[kRecCandI + (e % kCand)]);
      const float gv = r[kRecCandG + (e % kCand)];
      if (row < 0 || !(gv > 0.0f)) continue;
      const uint32_t w = reinterpret_cast<const uint32_t *>(Vrows + (int64_t)row * kHeadDim)[lane];
      const float d0 = bf16_lo(w) - y0, d1 = bf16_hi(w) - y1;
      const float dist = sqrtf(wave_sum(d0 * d0 + d1 * d1));
      lb = fmaxf(lb, scale_of(r[kRecM], M) * gv * dist / l);
    }
    lb = block_max256(lb, red);
    // ... and a rescan of any split whose bound max(g|v|) + max(g)|yhat| could exceed it.
    for (int s = 0; s < nsp; ++s) {
      const float *r = rec0 + s * rstride;
      const float f = scale_of(r[kRecM], M);
      const float ub = f * (r[kRecA] + r[kRecB] * ynorm) / l;
      if (!(ub > lb)) continue;
      if (tid == 0) atomicAdd(L.diag, 1u);
      const int64_t ra = (int64_t)s * L.split_rows, rz = min(cnt, ra + (int64_t)L.split_rows);
      const uint32_t qw = reinterpret_cast<const uint32_t *>(L.q + uh * kHeadDim)[lane];
      const float q0 = bf16_lo(qw), q1 = bf16_hi(qw);
      const float ms = r[kRecM];
      float best = 0.0f;
      for (int64_t j = ra + wv; j < rz; j += 4) {
        const uint32_t kw = reinterpret_cast<const uint32_t *>(L.Kc + (cbase + j) * kHeadDim)[lane];
        const uint32_t vw = reinterpret_cast<const uint32_t *>(Vrows + j * kHeadDim)[lane];
        const float dot = wave_sum(q0 * bf16_lo(kw) + q1 * bf16_hi(kw));
        const float d0 = bf16_lo(vw) - y0, d1 = bf16_hi(vw) - y1;
        const float dist = sqrtf(wave_sum(d0 * d0 + d1 * d1));
        const float pj = L.pic[cbase + j];
        const float w = __expf(dot * L.scale - __logf(pj) - ms);
        best = fmaxf(best, sqrtf(1.0f - pj) * w * dist);
      }
      lb = fmaxf(lb, block_max256(f * best / l, red));
    }
    const float b = lb;
    if (tid < kHeadDim) L.y[uh * kHeadDim + tid] = yv;
    if (tid == 0) {
      L.vhat[uh] = V;
      L.lse[uh] = M + logf(l);
      if (L.brange) L.brange[uh] = b;
      if (L.radius) L.radius[uh] = (sqrtf(2.0f * V * Ld) + b * Ld) / (ynorm + L.eps0);
    }
    __syncthreads();
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
  hipLaunchKernelGGL(attend_finalize_kernel, dim3(L.U), dim3(kAttendThreads), 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
