// ebd_internal.hpp -- launch descriptors shared by the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stddef.h>
#include <stdint.h>

#include "ebd.h"

namespace ebd {

constexpr int kHeadDim = 128;                // rows of K, V and q are 128 bf16
constexpr int kEvictStageMax = 16384;        // scores staged in LDS (64 KB) up to this length
constexpr int kSelectThreads = 512;          // evict_select (scores in LDS or streamed): eight waves per unit
constexpr int kSelectRegThreads = 128;       // evict_select_reg: two waves per unit, <= 6144 tokens
constexpr int kCopyThreads = 256;            // evict_copy: 16 lanes per 256-byte row
constexpr int kCopyRows = 128;               // retained rows per evict_copy work-group

constexpr int kAttendThreads = 64;   // one wave per (unit, split, head block); wpg waves per work-group
constexpr int kHeadBlock = 8;        // query heads handled together (MFMA rows: 8 weight + 8 variance)
constexpr int kSplitMaxRows = 4096;  // default split length cap (bounds the launch's tail)
constexpr int kSplitMinRows = 256;   // default split length floor
constexpr int kSplitWaves = 1536;    // default: cut units until the launch has this many waves
constexpr int kSplitRowsLimit = 8192;  // largest split a caller may ask for (LDS of one wave)
constexpr int kMaxSplits = 4096;       // splits per unit (the finalize keeps a scale per split and head in LDS)
constexpr int kCoopMaxSplits = 4;      // units of 2..4 splits run them as the waves of one work-group
constexpr size_t kCoopLdsMax = 61440;  // ... and their LDS stays within 60 KB per work-group
constexpr size_t kSplitLdsBudget = 20480;  // LDS of one split wave at two waves per SIMD (160 KB / 8)
constexpr int kResidentWaves = 2048;       // attention waves resident at once: two per SIMD, 256 CUs
constexpr int kScoresMaxQueries = 64;  // queries per ebd_scores call (four MFMA blocks)
constexpr int kChunkRows = 512;      // range-term candidates are kept per chunk of a split
constexpr int kCand = 32;            // candidates per (chunk, head)

// Partial record per (unit, split, head), floats, logits in base 2:
//   [0] m  final running max        [1] l  = sum w        (scale 2^{-m})
//   [2] C0 = sum c                  [3] C2 = sum c |v|^2  (scale 2^{-2m})
//   [8..135] o = sum w v            [136..263] Cv = sum c v
//   [264..291] the split's pivot list: [0] entry count (int bits), then per entry (row as int
//     bits, base-2 logit, pi); these rows are in none of the sums above nor in any candidate list
//   then one block of kChunkFloats per chunk of kChunkRows rows:
//     [0] A  max over the chunk's non-candidates of g |v|   [1] B  ... of g
//     [2] Vmax  max |v| over the candidates   [3] m_k  running max the block is scaled by
//     [4..35] candidate g (0 = no candidate)  [36..51] candidate rows, two 16-bit offsets from
//     the chunk's first row per word (candidate j in word j / 2, half j % 2)
//     [52..55] A of each of the 8 lanes that kept candidates (bf16 rounded up, two per word:
//     lane i in word i / 2, half i % 2; lane i owns row group i % 4 of the tiles of parity i / 4)
//   with w = 2^(l2 - m), c = (1 - pi) w^2, g = sqrt(1 - pi) w.
constexpr int kRecM = 0, kRecL = 1, kRecC0 = 2, kRecC2 = 3, kRecO = 8, kRecCv = 136;
constexpr int kPivMax = 8;      // pivot entries per (split, head)
constexpr int kPivFloats = 28;  // count, kPivMax x (row, logit, pi), padding to 16 bytes
constexpr int kRecPiv = 264;
constexpr int kRecChunks = kRecPiv + kPivFloats;
constexpr int kChunkFloats = 56;
constexpr int kChA = 0, kChB = 1, kChVmax = 2, kChM = 3, kChG = 4, kChI = 36, kChAL = 52;

inline int32_t attend_chunks(int32_t split_rows) { return (split_rows + kChunkRows - 1) / kChunkRows; }
inline int32_t attend_record_floats(int32_t split_rows) {
  return kRecChunks + kChunkFloats * attend_chunks(split_rows);
}

struct EvictLaunch {
  int32_t U;
  int64_t max_rows;     // longest unit the launch was planned for
  int64_t stage_rows;   // LDS staging length of evict_select (0: scores streamed from memory)
  int32_t copy_blocks;  // evict_copy work-groups per unit = ceil(max capacity / kCopyRows)
  const int64_t *seq_off;
  const int64_t *cap_off;
  int32_t n_sink, n_recent;
  float budget_frac;
  const float *budget_per_unit;
  float pi_min;
  int32_t pi_mode;
  int32_t design;  // EBD_DESIGN_*
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
};

struct AttendLaunch {
  int32_t U, G, nsplit, split_rows, nhb;
  int32_t wpg;           // waves per work-group: 1, or nsplit (a unit's splits in one work-group)
  int32_t coop_counter;  // float offset in LDS of the arrival count (wpg > 1; set per head block)
  int32_t nchunk, rec;  // chunks per split, floats per record
  int32_t plain;        // 1: the uncorrected pass (no offset; writes y and lse only)
  const int64_t *cap_off;
  const int32_t *count;
  const uint16_t *q, *Kc, *Vc;
  const float *pic;
  float scale, delta, eps0;
  float *part;          // [U * nsplit * G * rec]
  uint32_t *diag;       // [U * nhb * 2]: range-term chunk rescans, heads with Vhat summed directly
  float *y, *vhat, *lse, *brange, *radius;
  uint32_t *status;     // [U] or NULL: rows the step could not see (EBD_ST_*)
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

struct ScoresLaunch {
  int32_t U, W, nsplit, split_rows;
  const int64_t *seq_off;
  const int32_t *qpos;  // [U, W] last row each query sees, or NULL (every row)
  const uint16_t *q, *K;
  float scale;
  uint32_t flags;
  float *scores;
  float2 *stats;        // [U, nsplit, W] (max, exp-sum) per split and query
};

struct BlocksLaunch {
  int32_t U, G, block_rows;
  int64_t nblocks, max_rows;
  const int64_t *cap_off;
  const int32_t *count;
  const uint16_t *q, *Kc, *Vc;
  const float *pic;
  const int32_t *idxc;
  const float *y, *lse;
  float scale;
  float *blocks;  // [U, nblocks]
};

struct CertLaunch {
  int32_t U, G, S, head_stride;
  const int32_t *unit_seq, *unit_head0;
  const float *radius;
  float *cert, *mean_out;
};

constexpr int64_t kMaxBlocks = 8192;  // blocks per unit of ebd_block_contributions (LDS bins)

size_t attend_workspace_bytes(int32_t U, int32_t nsplit, int32_t G, int32_t split_rows);
size_t attend_fused_lds_bytes(int32_t split_rows, int gb);  // LDS of a split that also finalizes
size_t attend_part_lds_bytes(int32_t split_rows, int gb);   // LDS of one split of several
size_t scores_workspace_bytes(int32_t U, int32_t nsplit, int32_t W);

// The attention entry points' shared parts (ebd_api.cpp): argument checks (need = workspace
// bytes the launch uses), the device check, and the launches on a given workspace.
ebd_status attend_check(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                        const uint16_t *Vc, const float *pic, const int32_t *count, const float *y,
                        const float *vhat, const float *lse, size_t *need);
ebd_status device_ok();
ebd_status attend_launch(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                         const uint16_t *Vc, const float *pic, const int32_t *count, float *y,
                         float *vhat, float *lse, float *brange, float *radius, uint32_t *status,
                         void *workspace, void *stream, bool timing);

hipError_t launch_evict_select(const EvictLaunch &L, hipStream_t s);
hipError_t launch_evict_copy(const EvictLaunch &L, hipStream_t s);
bool evict_select_gathers(const EvictLaunch &L);  // evict_select also gathers the rows (no copy launch)
hipError_t launch_attend_split(const AttendLaunch &L, hipStream_t s);
hipError_t launch_attend_finalize(const AttendLaunch &L, hipStream_t s);
hipError_t launch_append_certain(const AppendLaunch &L, hipStream_t s);
hipError_t launch_scores_stats(const ScoresLaunch &L, hipStream_t s);
hipError_t launch_scores_accum(const ScoresLaunch &L, hipStream_t s);
hipError_t launch_block_contrib(const BlocksLaunch &L, hipStream_t s);
hipError_t launch_cert_step(const CertLaunch &L, hipStream_t s);

}  // namespace ebd
