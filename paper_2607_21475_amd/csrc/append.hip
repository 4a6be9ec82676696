// append.hip -- append one decode-step token per unit to its retained set with pi = 1.
// The sampled draw is reused across decode steps (App. A.2); tokens that arrive after eviction
// join the certainty set (recency), so they carry no offset and no variance term.
#include "ebd.h"
#include "ebd_device.hpp"
#include "ebd_internal.hpp"

namespace ebd {

__global__ __launch_bounds__(64) void append_certain_kernel(AppendLaunch L) {
  const int u = blockIdx.x;
  const int t = threadIdx.x;
  const int64_t cbase = L.cap_off[u];
  const int64_t cap = L.cap_off[u + 1] - cbase;
  const int32_t cnt = L.count[u];
  __syncthreads();  // every lane has read count[u] before lane 0 updates it
  if ((int64_t)cnt >= cap || cnt < 0) {
    if (t == 0 && L.status) L.status[u] |= EBD_ST_CAP_OVERFLOW;
    return;
  }
  const int64_t row = cbase + cnt;
  if (t < 16) {
    reinterpret_cast<uint4 *>(L.Kc + row * kHeadDim)[t] =
        reinterpret_cast<const uint4 *>(L.k_new + (int64_t)u * kHeadDim)[t];
  } else if (t < 32) {
    reinterpret_cast<uint4 *>(L.Vc + row * kHeadDim)[t - 16] =
        reinterpret_cast<const uint4 *>(L.v_new + (int64_t)u * kHeadDim)[t - 16];
  } else if (t == 32) {
    L.pic[row] = 1.0f;
    if (L.idxc) L.idxc[row] = L.pos_new ? L.pos_new[u] : -1;
  }
  __syncthreads();
  if (t == 0) L.count[u] = cnt + 1;
}

hipError_t launch_append_certain(const AppendLaunch &L, hipStream_t s) {
  hipLaunchKernelGGL(append_certain_kernel, dim3(L.U), dim3(64), 0, s, L);
  return hipGetLastError();
}

}  // namespace ebd
