// finegrain.hip -- fine-grained attribution and the deployed certificate on gfx950 (Sec. 6
// "Finer grains"; App. "Experimental details": the fine-grained probe and the certificate
// averaged over sampled heads and maximized over decode steps).
//
// block_contrib  one wave per (unit, block of <= 8 query heads), one retained row per lane:
//                kappa_hj = (1 - pi_j) (a_hj / (pi_j Nhat_h))^2 |v_j - yhat_h|^2, the summand of
//                Theorem 2, with a/(pi Nhat) = exp(scale q.k - ln pi - ln Nhat) from the certified
//                attention's own outputs; summed over the heads and into the LDS bin of the
//                row's original position / block_rows, then written (first head block) or added
//                (later head blocks, launched in order) to the unit's blocks.
// cert_step      one work-group per sequence: the mean radius over the sampled (unit, query
//                head) pairs, folded into a running maximum.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

template <int GB>
__global__ __launch_bounds__(64) void block_contrib_kernel(BlocksLaunch L, int h0) {
  extern __shared__ float s_bin[];  // [nblocks], then q [GB][128], yhat [GB][128], lse [GB]
  float *s_q = s_bin + L.nblocks;
  float *s_y = s_q + GB * kHeadDim;
  float *s_l = s_y + GB * kHeadDim;
  const int u = blockIdx.x;
  const int lane = threadIdx.x;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int cnt = (int)min(min((int64_t)L.count[u], cap), L.max_rows);
  const int64_t uh0 = (int64_t)u * L.G + h0;

  for (int64_t b = lane; b < L.nblocks; b += 64) s_bin[b] = 0.0f;
  for (int e = lane; e < GB * kHeadDim / 2; e += 64) {
    const int h = e / (kHeadDim / 2), d2 = e % (kHeadDim / 2);
    const uint32_t qw = reinterpret_cast<const uint32_t *>(L.q + (uh0 + h) * kHeadDim)[d2];
    s_q[h * kHeadDim + 2 * d2] = bf16_lo(qw);
    s_q[h * kHeadDim + 2 * d2 + 1] = bf16_hi(qw);
    const float2 yv = reinterpret_cast<const float2 *>(L.y + (uh0 + h) * kHeadDim)[d2];
    s_y[h * kHeadDim + 2 * d2] = yv.x;
    s_y[h * kHeadDim + 2 * d2 + 1] = yv.y;
  }
  if (lane < GB) s_l[lane] = L.lse[uh0 + lane];
  __syncthreads();

  const float scale2 = L.scale * kLog2e;
  for (int j = lane; j < cnt; j += 64) {
    const float pj = L.pic[cbase + j];
    const int pos = L.idxc[cbase + j];
    // certainty rows (pi = 1) and rows without a position (appended) carry no term
    if (!(pj < 1.0f) || pos < 0) continue;
    const int64_t bin = pos / L.block_rows;
    if (bin >= L.nblocks) continue;
    const uint4 *kr = reinterpret_cast<const uint4 *>(L.Kc + (cbase + j) * kHeadDim);
    const uint4 *vr = reinterpret_cast<const uint4 *>(L.Vc + (cbase + j) * kHeadDim);
    float dot[GB], d2[GB];
#pragma unroll
    for (int h = 0; h < GB; ++h) dot[h] = d2[h] = 0.0f;
    for (int half = 0; half < 2; ++half) {  // half a row per step keeps the registers down
      asm volatile("" ::: "memory");       // q and yhat stay in LDS
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
          const float k0 = bf16_lo(kw[t]), k1 = bf16_hi(kw[t]);
          const float v0 = bf16_lo(vw[t]), v1 = bf16_hi(vw[t]);
#pragma unroll
          for (int h = 0; h < GB; ++h) {
            const float *qh = s_q + h * kHeadDim + d0 + 2 * t;
            const float *yh = s_y + h * kHeadDim + d0 + 2 * t;
            dot[h] = fmaf(qh[0], k0, dot[h]);
            dot[h] = fmaf(qh[1], k1, dot[h]);
            const float a = v0 - yh[0], b = v1 - yh[1];
            d2[h] = fmaf(a, a, d2[h]);
            d2[h] = fmaf(b, b, d2[h]);
          }
        }
      }
    }
    const float lp = fast_log2(pj);
    float kap = 0.0f;
#pragma unroll
    for (int h = 0; h < GB; ++h) {
      // a/(pi Nhat) in base 2: scale log2e q.k - log2 pi - log2e ln Nhat
      const float wn = fast_exp2(dot[h] * scale2 - lp - s_l[h] * kLog2e);
      kap = fmaf((1.0f - pj) * wn * wn, d2[h], kap);
    }
    atomicAdd(&s_bin[bin], kap);
  }
  __syncthreads();
  float *out = L.blocks + (int64_t)u * L.nblocks;
  for (int64_t b = lane; b < L.nblocks; b += 64) out[b] = (h0 == 0 ? 0.0f : out[b]) + s_bin[b];
}

__global__ __launch_bounds__(256) void cert_step_kernel(CertLaunch L) {
  __shared__ double s_sum[4];
  __shared__ int s_cnt[4];
  const int sq = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  double sum = 0.0;
  int cnt = 0;
  for (int u = t; u < L.U; u += 256) {
    if (L.unit_seq[u] != sq) continue;
    const int64_t h0 = L.unit_head0 ? L.unit_head0[u] : 0;
    for (int g = 0; g < L.G; ++g) {
      if ((h0 + g) % L.head_stride != 0) continue;
      sum += (double)L.radius[(int64_t)u * L.G + g];
      ++cnt;
    }
  }
  sum = wave_sum(sum);
  cnt = wave_sum(cnt);
  if (lane == 0) {
    s_sum[wv] = sum;
    s_cnt[wv] = cnt;
  }
  __syncthreads();
  if (t == 0) {
    const double total = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    const int n = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    const float mean = n > 0 ? (float)(total / (double)n) : 0.0f;
    if (L.mean_out) L.mean_out[sq] = mean;
    if (n > 0) L.cert[sq] = fmaxf(L.cert[sq], mean);
  }
}

size_t block_contrib_lds(int64_t nblocks, int gb) {
  return (size_t)(nblocks + 2 * gb * kHeadDim + gb) * sizeof(float);
}

hipError_t launch_block_contrib(const BlocksLaunch &L, hipStream_t s) {
  const dim3 grid((unsigned)L.U), block(64);
  for (int h0 = 0; h0 < L.G; h0 += kHeadBlock) {
    const int gb = min(kHeadBlock, L.G - h0);
    const size_t lds = block_contrib_lds(L.nblocks, gb);
    switch (gb) {
      case 1: hipLaunchKernelGGL(block_contrib_kernel<1>, grid, block, lds, s, L, h0); break;
      case 2: hipLaunchKernelGGL(block_contrib_kernel<2>, grid, block, lds, s, L, h0); break;
      case 3: hipLaunchKernelGGL(block_contrib_kernel<3>, grid, block, lds, s, L, h0); break;
      case 4: hipLaunchKernelGGL(block_contrib_kernel<4>, grid, block, lds, s, L, h0); break;
      case 5: hipLaunchKernelGGL(block_contrib_kernel<5>, grid, block, lds, s, L, h0); break;
      case 6: hipLaunchKernelGGL(block_contrib_kernel<6>, grid, block, lds, s, L, h0); break;
      case 7: hipLaunchKernelGGL(block_contrib_kernel<7>, grid, block, lds, s, L, h0); break;
      default: hipLaunchKernelGGL(block_contrib_kernel<8>, grid, block, lds, s, L, h0); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_cert_step(const CertLaunch &L, hipStream_t s) {
  hipLaunchKernelGGL(cert_step_kernel, dim3((unsigned)L.S), dim3(256), 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
