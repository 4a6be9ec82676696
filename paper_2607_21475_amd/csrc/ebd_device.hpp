// ebd_device.hpp -- device helpers shared by the gfx950 kernels of libebd.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ebd {

constexpr uint32_t kPhiloxTag = 0x45424431u;      // "EBD1": fourth counter word of the mask stream
constexpr uint32_t kSystematicTag = 0x45424453u;  // "EBDS": ... of the systematic start

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Hardware transcendental approximations (v_exp_f32, v_log_f32, v_sqrt_f32).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float fast_sqrt(float x) { return __builtin_amdgcn_sqrtf(x); }

// Buffer resources (gfx9 raw buffers: stride 0, range checked per access).  Loads at or beyond
// the range return zeros and stores there are dropped, without touching memory, so tail tiles
// and prefetches past a range need no clamping.
constexpr int kRsrcWord3 = 0x00020000;  // 32-bit data format, untyped access
// Cache-policy operand of the raw buffer loads: the non-temporal hint (nt), for data read once.
constexpr int kLoadNT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)nbytes,
                                           kRsrcWord3);
}

// Ordering of LDS and global memory between the lanes of one wave: what __syncthreads gives a
// one-wave work-group (every prior access of the wave complete, no compiler motion across it),
// without the work-group barrier.  Code that one wave of a larger work-group runs alone (the
// attention finalize) synchronises with this.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// bf16 halves of a 32-bit word -> fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Philox4x32-10 (Salmon et al., SC 2011).  Returns the four output words.  Each round's two
// 32x32 -> 64-bit products are taken whole (one v_mad_u64_u32 each rather than a low and a high
// multiply).
__device__ __forceinline__ uint4 philox4x32_10(uint4 ctr, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * ctr.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * ctr.z;
    ctr = make_uint4((uint32_t)(p1 >> 32) ^ ctr.y ^ k0, (uint32_t)p1,
                     (uint32_t)(p0 >> 32) ^ ctr.w ^ k1, (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return ctr;
}

// Exact retention test x < pi * 2^32 for a stored fp32 pi in [0, 1]: pi * 2^32 is exact in
// fp32, pi = 1 keeps every x, and below 2^32, for an integer x, x < t  <=>  x < ceil(t), which
// fits 32 bits.
__device__ __forceinline__ bool keep_token(uint32_t x, float pi) {
  const float t = pi * 4294967296.0f;
  return t >= 4294967296.0f || x < (uint32_t)ceilf(t);
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over each 16-lane row; every lane of the row receives the row total.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp_f<0x141>(x);  // row_half_mirror
  x += dpp_f<0x140>(x);  // row_mirror
  return x;
}

// Wave reductions: DPP within each 16-lane row (every lane of a row gets the row's result), then
// the four row results by lane reads, so the result is the same in every lane and the order of
// the operations is fixed.  Every lane of the wave must be active.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
  return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, false);
}
template <class T>
struct LaneBits;
template <>
struct LaneBits<float> {
  template <int CTRL>
  __device__ static float dpp(float x) { return __int_as_float(dpp_i<CTRL>(__float_as_int(x))); }
  __device__ static float read(float x, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
  }
};
template <>
struct LaneBits<int> {
  template <int CTRL>
  __device__ static int dpp(int x) { return dpp_i<CTRL>(x); }
  __device__ static int read(int x, int l) { return __builtin_amdgcn_readlane(x, l); }
};
template <>
struct LaneBits<double> {
  template <int CTRL>
  __device__ static double dpp(double x) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = (unsigned)dpp_i<CTRL>((int)(unsigned)b);
    const unsigned hi = (unsigned)dpp_i<CTRL>((int)(unsigned)(b >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
  }
  __device__ static double read(double x, int l) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)b, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
  }
};

template <class T, class Op>
__device__ __forceinline__ T wave_reduce(T x, Op op) {
  using B = LaneBits<T>;
  x = op(x, B::template dpp<0xB1>(x));   // quad_perm [1,0,3,2]
  x = op(x, B::template dpp<0x4E>(x));   // quad_perm [2,3,0,1]
  x = op(x, B::template dpp<0x141>(x));  // row_half_mirror
  x = op(x, B::template dpp<0x140>(x));  // row_mirror
  return op(op(B::read(x, 0), B::read(x, 16)), op(B::read(x, 32), B::read(x, 48)));
}

__device__ __forceinline__ float wave_sum(float x) {
  return wave_reduce(x, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ double wave_sum(double x) {
  return wave_reduce(x, [](double a, double b) { return a + b; });
}
__device__ __forceinline__ int wave_sum(int x) {
  return wave_reduce(x, [](int a, int b) { return a + b; });
}
__device__ __forceinline__ float wave_max(float x) {
  return wave_reduce(x, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ float wave_min(float x) {
  return wave_reduce(x, [](float a, float b) { return fminf(a, b); });
}

}  // namespace ebd
