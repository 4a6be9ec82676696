// ebd_internal.hpp -- launch descriptors shared by the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

namespace ebd {

constexpr int kHeadDim = 128;                // rows of K, V and q are 128 bf16
constexpr int kEvictThreads = 512;            // one work-group per (unit, chunk)
constexpr int kEvictChunk = 4 * kEvictThreads;  // tokens per chunk: four per thread (one Philox block)
constexpr int kEvictRegChunks = 8;            // scores held in registers up to 8 chunks (16384 tokens)

constexpr int kAttendThreads = 256;  // four waves per (unit, split, head block)
constexpr int kHeadBlock = 8;        // query heads handled together (MFMA rows: 8 weight + 8 variance)
constexpr int kCand = 8;             // range-term candidates kept per (split, head)
constexpr int kRec = 288;            // floats per (unit, split, head) partial record

// Partial record layout (floats):
//   [0] m  running logit max        [1] l  = sum w        (scale e^{-m})
//   [2] C0 = sum c                  [3] C2 = sum c |v|^2  (scale e^{-2m})
//   [4] A  max over non-candidates of g |v|   [5] B  max over non-candidates of g
//   [8..15] candidate g             [16..23] candidate row (int bits, -1 = none)
//   [24..151] o = sum w v           [152..279] Cv = sum c v
//   with w = exp(l - m), c = (1 - pi) w^2, g = sqrt(1 - pi) w.
constexpr int kRecM = 0, kRecL = 1, kRecC0 = 2, kRecC2 = 3, kRecA = 4, kRecB = 5;
constexpr int kRecCandG = 8, kRecCandI = 16, kRecO = 24, kRecCv = 152;

struct EvictLaunch {
  int32_t U;
  int32_t nchunk;  // chunks per unit in the compact grid = ceil(max_rows / kEvictChunk)
  int32_t reg_chunks;  // 1, 2, 4, 8: scores in registers; 0: streamed from memory
  const int64_t *seq_off;
  const int64_t *cap_off;
  int32_t n_sink, n_recent;
  float budget_frac;
  const float *budget_per_unit;
  float pi_min;
  int32_t pi_mode;
  uint64_t seed;
  const uint64_t *seed_per_unit;
  uint32_t epoch;
  const float *scores;
  const uint16_t *K, *V;
  uint16_t *Kc, *Vc;
  float *pic;
  int32_t *idxc;
  int32_t *count;
  float *lambda_out;
  float *pi_full;
  uint32_t *status;
  float *ws_lambda;        // [U]
  int32_t *ws_chunk_off;   // [U * nchunk]
};

struct AttendLaunch {
  int32_t U, G, nsplit, split_rows, nhb;
  const int64_t *cap_off;
  const int32_t *count;
  const uint16_t *q, *Kc, *Vc;
  const float *pic;
  float scale, delta, eps0;
  float *part;          // [U * nsplit * G * kRec]
  uint32_t *diag;       // [0]: number of split rescans taken for the range term
  float *y, *vhat, *lse, *brange, *radius;
};

struct AppendLaunch {
  int32_t U;
  const int64_t *cap_off;
  int32_t *count;
  const uint16_t *k_new, *v_new;
  const int32_t *pos_new;
  uint16_t *Kc, *Vc;
  float *pic;
  int32_t *idxc;
  uint32_t *status;
};

size_t evict_workspace_bytes(int32_t U, int32_t nchunk);
size_t attend_workspace_bytes(int32_t U, int32_t nsplit, int32_t G);

hipError_t launch_evict_solve(const EvictLaunch &L, hipStream_t s);
hipError_t launch_evict_compact(const EvictLaunch &L, hipStream_t s);
hipError_t launch_attend_split(const AttendLaunch &L, hipStream_t s);
hipError_t launch_attend_finalize(const AttendLaunch &L, hipStream_t s);
hipError_t launch_append_certain(const AppendLaunch &L, hipStream_t s);

}  // namespace ebd
