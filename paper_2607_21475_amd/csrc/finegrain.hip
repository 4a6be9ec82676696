// finegrain.hip -- fine-grained attribution and the deployed certificate on gfx950 (Sec. 6
// "Finer grains"; App. "Experimental details": the fine-grained probe and the certificate
// averaged over sampled heads and maximized over decode steps).
//
// block_contrib  one wave per (unit, block of <= 8 query heads), 16 retained rows per step on
//                MFMA: kappa_hj = (1 - pi_j) (a_hj / (pi_j Nhat_h))^2 |v_j - yhat_h|^2, the
//                summand of Theorem 2, with a/(pi Nhat) = exp(scale q.k - ln pi - ln Nhat) from
//                the certified attention's own outputs; summed over the heads and into the LDS
//                bin of the row's original position / block_rows, then written (first head
//                block) or added (later head blocks, launched in order) to the unit's blocks.
// cert_step      one work-group per sequence: the mean radius over the sampled (unit, query
//                head) pairs, folded into a running maximum.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

namespace {

// 16 retained rows of a unit: K and V in the B-operand layout of the 16x16x32 MFMA (lane (g, c):
// row 16t + c, dims 32 kb + 8 g .. + 7), and pi and the original position of row 16t + c.
struct BTile {
  u32x4 k[4], v[4];
  float p;
  int ix;
};

__device__ __forceinline__ void load_btile(BTile &T, __amdgpu_buffer_rsrc_t rK,
                                           __amdgpu_buffer_rsrc_t rV, __amdgpu_buffer_rsrc_t rP,
                                           __amdgpu_buffer_rsrc_t rI, int t, int g, int c) {
  const uint32_t r = (uint32_t)(16 * t + c);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const uint32_t off = r * 256u + (uint32_t)(64 * kb + 16 * g);
    T.k[kb] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rK, off, 0, 0));
    T.v[kb] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rV, off, 0, 0));
  }
  T.p = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rP, r * 4u, 0, 0));
  T.ix = (int)__builtin_amdgcn_raw_buffer_load_b32(rI, r * 4u, 0, 0);
}

// Top 16 bits of x as a bf16 (truncation: x - value is exact in fp32).
__device__ __forceinline__ uint32_t bf16_top(float x) { return __float_as_uint(x) >> 16; }

}  // namespace

// One wave per (unit, block of <= 8 query heads), 16 retained rows per step.  Two MFMA
// contractions give, for every (head, row) pair, q_h.k_j (A = the heads' queries) and
// yhat_h.v_j (A = yhat split exactly into three bf16 pieces, so that every product is exact and
// only the fp32 sums round); with |v_j|^2 from the lane's own V dims, |v - yhat|^2 =
// |v|^2 - 2 yhat.v + |yhat|^2.  Where that loses more than 8 bits to cancellation (v close to
// yhat), the tile recomputes the squared distance directly.  Lane (g, c) holds heads 4g .. 4g+3
// for row 16t + c; the heads' terms are summed over the four row groups and added to the LDS bin
// of the row's original position.
template <int GB>
__global__ __launch_bounds__(64, 2) void block_contrib_kernel(BlocksLaunch L, int h0) {
  extern __shared__ float s_bin[];  // [nblocks], then |yhat|^2 [8], ln Nhat [8], yhat [GB][128]
  float *s_yy = s_bin + L.nblocks;
  float *s_l = s_yy + 8;
  float *s_y = s_l + 8;
  const int u = blockIdx.x;
  const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int cnt = (int)min(min((int64_t)L.count[u], cap), L.max_rows);
  const int64_t uh0 = (int64_t)u * L.G + h0;

  for (int64_t b = lane; b < L.nblocks; b += 64) s_bin[b] = 0.0f;
  // A operands: row c is head c (zero above GB); lane (g, c) holds dims 32 kb + 8 g .. + 7
  bf16x8 qa[4], ya[3][4];
  float yy = 0.0f;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const int d0 = 32 * kb + 8 * g;
    uint4 qw = make_uint4(0u, 0u, 0u, 0u);
    float yv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) yv[e] = 0.0f;
    if (c < GB) {
      qw = *reinterpret_cast<const uint4 *>(L.q + (uh0 + c) * kHeadDim + d0);
      const float2 *yr = reinterpret_cast<const float2 *>(L.y + (uh0 + c) * kHeadDim + d0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float2 y2 = yr[e];
        yv[2 * e] = y2.x;
        yv[2 * e + 1] = y2.y;
      }
    }
    qa[kb] = __builtin_bit_cast(bf16x8, qw);
    uint32_t hw[4], mw[4], lw[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint32_t pk[3][2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const float x = yv[2 * e + h2];
        yy = fmaf(x, x, yy);
        const uint32_t hi = bf16_top(x);
        const float r = x - __uint_as_float(hi << 16);
        const uint32_t mid = bf16_top(r);
        const float lo = r - __uint_as_float(mid << 16);
        pk[0][h2] = hi;
        pk[1][h2] = mid;
        pk[2][h2] = bf16_top(lo);  // lo has at most 8 significant bits: exact in bf16
      }
      hw[e] = pk[0][0] | (pk[0][1] << 16);
      mw[e] = pk[1][0] | (pk[1][1] << 16);
      lw[e] = pk[2][0] | (pk[2][1] << 16);
    }
    ya[0][kb] = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
    ya[1][kb] = __builtin_bit_cast(bf16x8, make_uint4(mw[0], mw[1], mw[2], mw[3]));
    ya[2][kb] = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
  }
  yy += __shfl_xor(yy, 16);
  yy += __shfl_xor(yy, 32);
  if (g == 0 && c < 8) {
    s_yy[c] = c < GB ? yy : 0.0f;
    s_l[c] = c < GB ? L.lse[uh0 + c] : 0.0f;
  }
  for (int e = lane; e < GB * kHeadDim; e += 64) s_y[e] = L.y[uh0 * kHeadDim + e];
  __syncthreads();

  const float scale2 = L.scale * kLog2e;
  const __amdgpu_buffer_rsrc_t rK = make_rsrc(L.Kc + cbase * kHeadDim, (uint32_t)cnt * 256u);
  const __amdgpu_buffer_rsrc_t rV = make_rsrc(L.Vc + cbase * kHeadDim, (uint32_t)cnt * 256u);
  const __amdgpu_buffer_rsrc_t rP = make_rsrc(L.pic + cbase, (uint32_t)cnt * 4u);
  const __amdgpu_buffer_rsrc_t rI = make_rsrc(L.idxc + cbase, (uint32_t)cnt * 4u);
  const int ntile = (cnt + 15) / 16;

  auto step = [&](const BTile &T, int t) {
    f32x4 s = f32x4{0.0f, 0.0f, 0.0f, 0.0f}, d = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[kb], __builtin_bit_cast(bf16x8, T.k[kb]), s,
                                                  0, 0, 0);
#pragma unroll
    for (int pc = 0; pc < 3; ++pc)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ya[pc][kb], __builtin_bit_cast(bf16x8, T.v[kb]),
                                                    d, 0, 0, 0);
    // |v|^2 of row 16t + c: the lane's 32 dims, then the four row groups
    float nv = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float a = bf16_lo(T.v[kb][e]), b = bf16_hi(T.v[kb][e]);
        nv = fmaf(a, a, nv);
        nv = fmaf(b, b, nv);
      }
    nv += __shfl_xor(nv, 16);
    nv += __shfl_xor(nv, 32);
    const bool row_ok = 16 * t + c < cnt && T.p < 1.0f && T.ix >= 0 &&
                        (int64_t)T.ix / L.block_rows < L.nblocks;
    float d2[4];
    bool exact = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float yh = s_yy[(4 * g + i) & 7];
      d2[i] = nv - 2.0f * d[i] + yh;
      exact |= row_ok && 4 * g + i < GB && d2[i] < 0.00390625f * (nv + yh);
    }
    if (__any(exact)) {
      // direct sums over the lane's 32 dims, one head at a time, then over the row groups
#pragma unroll 1
      for (int h = 0; h < GB; ++h) {
        float dd = 0.0f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int dim = 32 * kb + 8 * g + 2 * e;
            const float ea = bf16_lo(T.v[kb][e]) - s_y[h * kHeadDim + dim];
            const float eb = bf16_hi(T.v[kb][e]) - s_y[h * kHeadDim + dim + 1];
            dd = fmaf(ea, ea, dd);
            dd = fmaf(eb, eb, dd);
          }
        dd += __shfl_xor(dd, 16);
        dd += __shfl_xor(dd, 32);
#pragma unroll
        for (int i = 0; i < 4; ++i) d2[i] = (h == 4 * g + i) ? dd : d2[i];
      }
    }
    float kap = 0.0f;
    if (row_ok) {
      const float lp = fast_log2(T.p);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int h = 4 * g + i;
        if (h < GB) {
          // a/(pi Nhat) in base 2: scale log2e q.k - log2 pi - log2e ln Nhat
          const float wn = fast_exp2(s[i] * scale2 - lp - s_l[h] * kLog2e);
          kap = fmaf((1.0f - T.p) * wn * wn, fmaxf(d2[i], 0.0f), kap);
        }
      }
    }
    kap += __shfl_xor(kap, 16);
    kap += __shfl_xor(kap, 32);
    if (g == 0 && row_ok) atomicAdd(&s_bin[T.ix / L.block_rows], kap);
  };
  BTile T0, T1, T2;
  load_btile(T0, rK, rV, rP, rI, 0, g, c);
  load_btile(T1, rK, rV, rP, rI, 1, g, c);
  int t = 0;
  for (; t + 3 <= ntile; t += 3) {
    load_btile(T2, rK, rV, rP, rI, t + 2, g, c);
    step(T0, t);
    load_btile(T0, rK, rV, rP, rI, t + 3, g, c);
    step(T1, t + 1);
    load_btile(T1, rK, rV, rP, rI, t + 4, g, c);
    step(T2, t + 2);
  }
  if (t < ntile) step(T0, t);
  if (t + 1 < ntile) step(T1, t + 1);
  __syncthreads();
  float *out = L.blocks + (int64_t)u * L.nblocks;
  for (int64_t b = lane; b < L.nblocks; b += 64) out[b] = (h0 == 0 ? 0.0f : out[b]) + s_bin[b];
}

constexpr int kCertThreads = 1024;

__global__ __launch_bounds__(kCertThreads) void cert_step_kernel(CertLaunch L) {
  constexpr int NW = kCertThreads / 64;
  __shared__ double s_sum[NW];
  __shared__ int s_cnt[NW];
  const int sq = blockIdx.x;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  double sum = 0.0;
  int cnt = 0;
  // (unit, head) pairs e = u G + g spread over the threads, up to eight per thread with all their
  // reads issued together (walked by unit, a sequence's units can all fall to a few threads);
  // 32-bit indices (the call checks U G < 2^31)
  const uint32_t total = (uint32_t)L.U * (uint32_t)L.G, G = (uint32_t)L.G;
  const uint32_t stride = (uint32_t)L.head_stride;
  constexpr int kB = 8;
  for (uint32_t e0 = (uint32_t)t; e0 < total; e0 += (uint32_t)kCertThreads * kB) {
    int seq[kB];
    uint32_t hg[kB];
    float rv[kB];
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      const uint32_t e = e0 + (uint32_t)kCertThreads * k;
      const bool in = e < total;
      const uint32_t u = in ? e / G : 0u;
      seq[k] = in ? L.unit_seq[u] : -1;
      const uint32_t h0 = (in && L.unit_head0) ? (uint32_t)L.unit_head0[u] : 0u;
      hg[k] = h0 + (e - u * G);  // the head's index in its layer
      rv[k] = in ? L.radius[e] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < kB; ++k) {
      if (seq[k] == sq && hg[k] % stride == 0u) {
        sum += (double)rv[k];
        ++cnt;
      }
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
    double tsum = 0.0;
    int n = 0;
    for (int w = 0; w < NW; ++w) {
      tsum += s_sum[w];
      n += s_cnt[w];
    }
    const float mean = n > 0 ? (float)(tsum / (double)n) : 0.0f;
    if (L.mean_out) L.mean_out[sq] = mean;
    if (n > 0) L.cert[sq] = fmaxf(L.cert[sq], mean);
  }
}

size_t block_contrib_lds(int64_t nblocks, int gb) {
  return (size_t)(nblocks + 16 + gb * kHeadDim) * sizeof(float);
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
  hipLaunchKernelGGL(cert_step_kernel, dim3((unsigned)L.S), dim3(kCertThreads), 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
