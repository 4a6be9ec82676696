// ebd_api.cpp -- the C ABI of libebd: argument validation, workspace layout, launch planning and
// optional per-kernel timing.  Every step of the path runs in the HIP kernels; this file only
// checks arguments and launches them.
#include "ebd.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "ebd_internal.hpp"

namespace {

using namespace ebd;

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// The library runs on gfx950 only.  Checked once per device.
ebd_status check_device() {
  static std::mutex mu;
  static std::map<int, bool> ok;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return EBD_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(mu);
  auto it = ok.find(dev);
  if (it == ok.end()) {
    hipDeviceProp_t prop;
    bool good = false;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess)
      good = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
    it = ok.emplace(dev, good).first;
  }
  return it->second ? EBD_OK : EBD_ERR_UNSUPPORTED;
}

// ---- optional kernel timing ----------------------------------------------------------------
struct TimingRec {
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending;
  std::vector<hipEvent_t> pool;
  double ms = 0.0;
  int64_t launches = 0;
};
std::mutex g_tmu;
std::atomic<bool> g_timing{false};
std::map<std::string, TimingRec> g_trec;

hipEvent_t pooled_event(TimingRec &r) {
  if (!r.pool.empty()) {
    hipEvent_t e = r.pool.back();
    r.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
hipError_t timed(const char *name, hipStream_t s, F &&launch) {
  if (!g_timing.load(std::memory_order_acquire)) return launch();
  std::lock_guard<std::mutex> lk(g_tmu);
  TimingRec &r = g_trec[name];
  hipEvent_t a = pooled_event(r), b = pooled_event(r);
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, s);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, s);
  if (e != hipSuccess) return e;
  r.pending.emplace_back(a, b);
  return hipSuccess;
}

// The sampler keeps no state between its two launches except the index list it writes.
constexpr size_t kEvictWorkspace = 256;

// Rows per split (a multiple of 16).  Unless the caller fixes it: one split per unit when there
// are enough units for kSplitWaves waves, else units are cut into equal splits until there are;
// splits stay within [kSplitMinRows, kSplitMaxRows] rows.  When the units alone give enough
// waves, a whole unit of up to kSplitRowsLimit rows stays one split (which then also finalizes
// its unit, with no second launch) as long as that split's LDS still lets two waves share a SIMD.
// Splits may also run longer than kSplitMaxRows, up to the same LDS limit, when that makes the
// whole launch one generation of resident waves (kResidentWaves): a launch of two generations
// ends with the second one's stragglers (1024 units of about 14000 rows, G = 4: two splits per
// unit took 1150 us where four took 1190 us).
int32_t attend_split_rows(const ebd_attend_params *p) {
  if (p->split_rows > 0) return p->split_rows;
  const int64_t cap = p->max_rows > 0 ? p->max_rows : 1;
  const int64_t U = p->num_units > 0 ? p->num_units : 1;
  const int32_t G = p->group > 0 ? p->group : 1;
  const int64_t waves = U * ((G + kHeadBlock - 1) / kHeadBlock);
  if (waves >= kSplitWaves && cap <= kSplitRowsLimit &&
      attend_fused_lds_bytes((int32_t)cap, std::min(G, kHeadBlock)) <= kSplitLdsBudget)
    return (int32_t)((cap + 15) / 16 * 16);
  int64_t ns = (kSplitWaves + U - 1) / U;
  ns = std::max<int64_t>(ns, (cap + kSplitMaxRows - 1) / kSplitMaxRows);
  const int gb = std::min(G, kHeadBlock);
  const int64_t lds_rows =
      (int64_t)(kSplitLdsBudget / attend_part_lds_bytes(kChunkRows, gb)) * kChunkRows;
  const int64_t rmax = std::min<int64_t>(kSplitRowsLimit, lds_rows);
  const int64_t ns1 = std::max<int64_t>((kSplitWaves + U - 1) / U, (cap + rmax - 1) / rmax);
  if (ns1 < ns && U * ns1 <= kResidentWaves) ns = ns1;  // each head block is its own launch
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, cap / kSplitMinRows));
  const int64_t sr = ((cap + ns - 1) / ns + 15) / 16 * 16;
  return (int32_t)sr;
}

int32_t attend_nsplit(const ebd_attend_params *p, int32_t sr) {
  const int64_t ns = (p->max_rows + sr - 1) / sr;
  return (int32_t)(ns > 0 ? ns : 1);
}

// Rows per scores split: as for attention, one split per unit when the units give enough
// waves, else equal splits (at least 256 rows, at most 8192).
int32_t scores_split_rows(const ebd_scores_params *p) {
  if (p->split_rows > 0) return p->split_rows;
  const int64_t n = p->max_rows > 0 ? p->max_rows : 1;
  const int64_t U = p->num_units > 0 ? p->num_units : 1;
  int64_t ns = (kSplitWaves + U - 1) / U;
  ns = std::max<int64_t>(ns, (n + 8191) / 8192);
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, n / 256));
  return (int32_t)(((n + ns - 1) / ns + 15) / 16 * 16);
}

int32_t scores_nsplit(const ebd_scores_params *p, int32_t sr) {
  const int64_t ns = (p->max_rows + sr - 1) / sr;
  return (int32_t)(ns > 0 ? ns : 1);
}

bool valid_scores_params(const ebd_scores_params *p) {
  if (!p) return false;
  if (p->num_units < 0 || p->max_rows < 0 || p->max_rows > ((int64_t)1 << 31)) return false;
  if (p->num_queries < 1 || p->num_queries > kScoresMaxQueries) return false;
  if (p->num_units > 0 && !p->seq_off) return false;
  if (p->split_rows != 0 && (p->split_rows < 16 || p->split_rows > 65536 || p->split_rows % 16))
    return false;
  if ((p->flags & ~EBD_SCORES_ACCUMULATE) != 0u) return false;
  if (p->scale < 0.0f || !std::isfinite(p->scale)) return false;
  return true;
}

bool valid_evict_params(const ebd_evict_params *p) {
  if (!p) return false;
  if (p->num_units < 0 || p->max_rows < 0 || p->max_rows > ((int64_t)1 << 31)) return false;
  if (p->max_capacity < 0 || p->max_capacity > ((int64_t)1 << 31)) return false;
  if (p->num_units > 0 && (!p->seq_off || !p->cap_off)) return false;
  if (p->n_sink < 0 || p->n_recent < 0) return false;
  if (!(p->pi_min > 0.0f && p->pi_min <= 1.0f)) return false;
  if (p->pi_mode != 0 && p->pi_mode != 1) return false;
  if (p->design < EBD_DESIGN_POISSON || p->design > EBD_DESIGN_UNIFORM) return false;
  if (!p->budget_per_unit && !std::isfinite(p->budget_frac)) return false;
  return true;
}

bool valid_attend_params(const ebd_attend_params *p) {
  if (!p) return false;
  if (p->num_units < 0 || p->group < 1 || p->max_rows < 0 || p->max_rows > ((int64_t)1 << 31))
    return false;
  if (p->num_units > 0 && !p->cap_off) return false;
  if (p->split_rows != 0 &&
      (p->split_rows < 16 || p->split_rows > kSplitRowsLimit || p->split_rows % 16))
    return false;
  if ((p->flags & ~EBD_F_NO_OFFSET) != 0u) return false;
  if (p->scale < 0.0f || !std::isfinite(p->scale)) return false;
  if (p->delta < 0.0f || p->delta >= 1.0f) return false;
  if (p->eps0 < 0.0f || !std::isfinite(p->eps0)) return false;
  return true;
}

}  // namespace

namespace ebd {

ebd_status device_ok() { return check_device(); }

ebd_status attend_check(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                        const uint16_t *Vc, const float *pic, const int32_t *count, const float *y,
                        const float *vhat, const float *lse, size_t *need) {
  if (!valid_attend_params(p)) return EBD_ERR_INVALID_ARG;
  if (p->head_dim != kHeadDim) return EBD_ERR_UNSUPPORTED;
  *need = 0;
  if (p->num_units == 0) return EBD_OK;
  if (!q || !Kc || !Vc || !pic || !count || !y || !vhat || !lse) return EBD_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(Kc, 16) || !aligned(Vc, 16) || !aligned(pic, 4) ||
      !aligned(y, 16))
    return EBD_ERR_INVALID_ARG;
  const int32_t sr = attend_split_rows(p);
  if (attend_nsplit(p, sr) > kMaxSplits) return EBD_ERR_UNSUPPORTED;
  *need = attend_workspace_bytes(p->num_units, attend_nsplit(p, sr), p->group, sr);
  return EBD_OK;
}

ebd_status attend_launch(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                         const uint16_t *Vc, const float *pic, const int32_t *count, float *y,
                         float *vhat, float *lse, float *brange, float *radius, uint32_t *status,
                         void *workspace, void *stream, bool timing) {
  const int32_t sr = attend_split_rows(p);
  const int32_t nsplit = attend_nsplit(p, sr);
  AttendLaunch L;
  L.U = p->num_units;
  L.G = p->group;
  L.nsplit = nsplit;
  // a unit of 2..4 splits runs them as one work-group's waves, the last of which finalizes
  L.wpg = (nsplit > 1 && nsplit <= kCoopMaxSplits &&
           (size_t)nsplit * attend_part_lds_bytes(sr, std::min(p->group, kHeadBlock)) <= kCoopLdsMax)
              ? nsplit
              : 1;
  L.coop_counter = 0;
  L.split_rows = sr;
  L.nchunk = attend_chunks(sr);
  L.rec = attend_record_floats(sr);
  L.nhb = (p->group + kHeadBlock - 1) / kHeadBlock;
  L.cap_off = p->cap_off;
  L.count = count;
  L.q = q;
  L.Kc = Kc;
  L.Vc = Vc;
  L.pic = pic;
  L.scale = p->scale > 0.0f ? p->scale : 1.0f / std::sqrt((float)kHeadDim);
  L.delta = p->delta > 0.0f ? p->delta : 0.1f;
  L.eps0 = p->eps0 > 0.0f ? p->eps0 : 1e-9f;
  char *ws = static_cast<char *>(workspace);
  L.diag = reinterpret_cast<uint32_t *>(ws);
  L.part = reinterpret_cast<float *>(ws + attend_workspace_bytes(p->num_units, 1, p->group, sr));
  L.y = y;
  L.vhat = vhat;
  L.lse = lse;
  L.brange = brange;
  L.radius = radius;
  L.status = status;

  hipStream_t s = static_cast<hipStream_t>(stream);
  L.plain = 0;
  const int passes = (p->flags & EBD_F_NO_OFFSET) ? 2 : 1;
  for (int pass = 0; pass < passes; ++pass) {
    L.plain = pass;  // the second pass replaces y and ln N by the uncorrected softmax
    const hipError_t e1 = timing ? timed("attend_split", s, [&] { return launch_attend_split(L, s); })
                                 : launch_attend_split(L, s);
    if (e1 != hipSuccess) return EBD_ERR_HIP;
    if (L.nsplit > 1 && L.wpg == 1) {
      const hipError_t e2 =
          timing ? timed("attend_finalize", s, [&] { return launch_attend_finalize(L, s); })
                 : launch_attend_finalize(L, s);
      if (e2 != hipSuccess) return EBD_ERR_HIP;
    }
  }
  return EBD_OK;
}

}  // namespace ebd

extern "C" {

const char *ebd_version(void) { return "ebd-gfx950 0.1.0"; }

const char *ebd_status_string(ebd_status s) {
  switch (s) {
    case EBD_OK: return "ok";
    case EBD_ERR_INVALID_ARG: return "invalid argument";
    case EBD_ERR_UNSUPPORTED: return "unsupported (head_dim must be 128; device must be gfx950)";
    case EBD_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case EBD_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t ebd_workspace_size(int32_t which, const void *params) {
  if (which == EBD_WS_EVICT) {
    const ebd_evict_params *p = static_cast<const ebd_evict_params *>(params);
    if (!valid_evict_params(p)) return 0;
    return kEvictWorkspace;
  }
  if (which == EBD_WS_ATTEND) {
    const ebd_attend_params *p = static_cast<const ebd_attend_params *>(params);
    if (!valid_attend_params(p)) return 0;
    const int32_t sr = attend_split_rows(p);
    return attend_workspace_bytes(p->num_units, attend_nsplit(p, sr), p->group, sr);
  }
  if (which == EBD_WS_SCORES) {
    const ebd_scores_params *p = static_cast<const ebd_scores_params *>(params);
    if (!valid_scores_params(p)) return 0;
    const int32_t sr = scores_split_rows(p);
    return scores_workspace_bytes(p->num_units, scores_nsplit(p, sr), p->num_queries);
  }
  return 0;
}

ebd_status ebd_evict(const ebd_evict_params *p, const float *scores, const uint16_t *K,
                     const uint16_t *V, uint16_t *Kc, uint16_t *Vc, float *pic, int32_t *idxc,
                     int32_t *count, float *lambda_out, float *pi_full, uint32_t *status,
                     void *workspace, size_t ws_bytes, void *stream) {
  if (!valid_evict_params(p)) return EBD_ERR_INVALID_ARG;
  if (p->head_dim != kHeadDim) return EBD_ERR_UNSUPPORTED;
  if (p->num_units == 0) return EBD_OK;
  if (!scores || !K || !V || !Kc || !Vc || !pic || !idxc || !count || !status)
    return EBD_ERR_INVALID_ARG;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(Kc, 16) || !aligned(Vc, 16) ||
      !aligned(scores, 4) || !aligned(pic, 4) || !aligned(idxc, 4))
    return EBD_ERR_INVALID_ARG;
  if (!workspace || ws_bytes < kEvictWorkspace || !aligned(workspace, 256)) return EBD_ERR_WORKSPACE;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;

  EvictLaunch L;
  L.U = p->num_units;
  L.max_rows = p->max_rows;
  L.stage_rows = p->max_rows <= kEvictStageMax ? p->max_rows : 0;
  L.copy_blocks = (int32_t)((p->max_capacity + kCopyRows - 1) / kCopyRows);
  L.seq_off = p->seq_off;
  L.cap_off = p->cap_off;
  L.n_sink = p->n_sink;
  L.n_recent = p->n_recent;
  L.budget_frac = p->budget_frac;
  L.budget_per_unit = p->budget_per_unit;
  L.pi_min = p->pi_min;
  L.pi_mode = p->pi_mode;
  L.design = p->design;
  L.seed = p->seed;
  L.seed_per_unit = p->seed_per_unit;
  L.epoch = p->epoch;
  L.scores = scores;
  L.K = K;
  L.V = V;
  L.Kc = Kc;
  L.Vc = Vc;
  L.pic = pic;
  L.idxc = idxc;
  L.count = count;
  L.lambda_out = lambda_out;
  L.pi_full = pi_full;
  L.status = status;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (timed("evict_select", s, [&] { return launch_evict_select(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  if (L.copy_blocks > 0 && !evict_select_gathers(L) &&
      timed("evict_copy", s, [&] { return launch_evict_copy(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  return EBD_OK;
}

ebd_status ebd_attend_certify(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                              const uint16_t *Vc, const float *pic, const int32_t *count,
                              float *y, float *vhat, float *lse, float *brange, float *radius,
                              uint32_t *status, void *workspace, size_t ws_bytes, void *stream) {
  size_t need = 0;
  const ebd_status cs = ebd::attend_check(p, q, Kc, Vc, pic, count, y, vhat, lse, &need);
  if (cs != EBD_OK || p->num_units == 0) return cs;
  if (!workspace || ws_bytes < need || !aligned(workspace, 256)) return EBD_ERR_WORKSPACE;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;
  return ebd::attend_launch(p, q, Kc, Vc, pic, count, y, vhat, lse, brange, radius, status,
                            workspace, stream, true);
}

ebd_status ebd_scores(const ebd_scores_params *p, const uint16_t *q, const uint16_t *K,
                      float *scores, void *workspace, size_t ws_bytes, void *stream) {
  if (!valid_scores_params(p)) return EBD_ERR_INVALID_ARG;
  if (p->head_dim != kHeadDim) return EBD_ERR_UNSUPPORTED;
  if (p->num_units == 0) return EBD_OK;
  if (!q || !K || !scores) return EBD_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(K, 16) || !aligned(scores, 4)) return EBD_ERR_INVALID_ARG;
  const int32_t sr = scores_split_rows(p);
  const int32_t nsplit = scores_nsplit(p, sr);
  const size_t need = scores_workspace_bytes(p->num_units, nsplit, p->num_queries);
  if (!workspace || ws_bytes < need || !aligned(workspace, 256)) return EBD_ERR_WORKSPACE;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;

  ScoresLaunch L;
  L.U = p->num_units;
  L.W = p->num_queries;
  L.nsplit = nsplit;
  L.split_rows = sr;
  L.seq_off = p->seq_off;
  L.qpos = p->qpos;
  L.q = q;
  L.K = K;
  L.scale = p->scale > 0.0f ? p->scale : 1.0f / std::sqrt((float)kHeadDim);
  L.flags = p->flags;
  L.scores = scores;
  L.stats = static_cast<float2 *>(workspace);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (timed("scores_stats", s, [&] { return launch_scores_stats(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  if (timed("scores_accum", s, [&] { return launch_scores_accum(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  return EBD_OK;
}

ebd_status ebd_block_contributions(const ebd_blocks_params *p, const uint16_t *q,
                                   const uint16_t *Kc, const uint16_t *Vc, const float *pic,
                                   const int32_t *idxc, const int32_t *count, const float *y,
                                   const float *lse, float *blocks, void *stream) {
  if (!p) return EBD_ERR_INVALID_ARG;
  if (p->num_units < 0 || p->group < 1 || p->block_rows < 1 || p->nblocks < 1 ||
      p->nblocks > kMaxBlocks || p->max_rows < 0 || p->scale < 0.0f || !std::isfinite(p->scale))
    return EBD_ERR_INVALID_ARG;
  if (p->head_dim != kHeadDim) return EBD_ERR_UNSUPPORTED;
  // one wave reads a unit through 32-bit buffer ranges of 256-byte rows: 2^24 rows would wrap
  if (p->max_rows >= ((int64_t)1 << 24)) return EBD_ERR_UNSUPPORTED;
  if (p->num_units == 0) return EBD_OK;
  if (!p->cap_off || !q || !Kc || !Vc || !pic || !idxc || !count || !y || !lse || !blocks)
    return EBD_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(Kc, 16) || !aligned(Vc, 16) || !aligned(y, 8))
    return EBD_ERR_INVALID_ARG;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;
  BlocksLaunch L;
  L.U = p->num_units;
  L.G = p->group;
  L.block_rows = p->block_rows;
  L.nblocks = p->nblocks;
  L.max_rows = p->max_rows;
  L.cap_off = p->cap_off;
  L.count = count;
  L.q = q;
  L.Kc = Kc;
  L.Vc = Vc;
  L.pic = pic;
  L.idxc = idxc;
  L.y = y;
  L.lse = lse;
  L.scale = p->scale > 0.0f ? p->scale : 1.0f / std::sqrt((float)kHeadDim);
  L.blocks = blocks;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (timed("block_contrib", s, [&] { return launch_block_contrib(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  return EBD_OK;
}

ebd_status ebd_certificate_step(const ebd_cert_params *p, const float *radius, float *cert,
                                float *mean_out, void *stream) {
  if (!p || p->num_units < 0 || p->group < 1 || p->num_seqs < 0 || p->head_stride < 1 ||
      (int64_t)p->num_units * p->group >= ((int64_t)1 << 31))
    return EBD_ERR_INVALID_ARG;
  if (p->num_seqs == 0) return EBD_OK;
  if (!cert || (p->num_units > 0 && (!p->unit_seq || !radius))) return EBD_ERR_INVALID_ARG;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;
  CertLaunch L;
  L.U = p->num_units;
  L.G = p->group;
  L.S = p->num_seqs;
  L.head_stride = p->head_stride;
  L.unit_seq = p->unit_seq;
  L.unit_head0 = p->unit_head0;
  L.radius = radius;
  L.cert = cert;
  L.mean_out = mean_out;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (timed("cert_step", s, [&] { return launch_cert_step(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  return EBD_OK;
}

ebd_status ebd_append_certain(int32_t num_units, int32_t head_dim, const int64_t *cap_off,
                              int32_t *count, const uint16_t *k_new, const uint16_t *v_new,
                              const int32_t *pos_new, uint16_t *Kc, uint16_t *Vc, float *pic,
                              int32_t *idxc, uint32_t *status, void *stream) {
  if (num_units < 0) return EBD_ERR_INVALID_ARG;
  if (head_dim != kHeadDim) return EBD_ERR_UNSUPPORTED;
  if (num_units == 0) return EBD_OK;
  if (!cap_off || !count || !k_new || !v_new || !Kc || !Vc || !pic) return EBD_ERR_INVALID_ARG;
  if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(Kc, 16) || !aligned(Vc, 16))
    return EBD_ERR_INVALID_ARG;
  const ebd_status ds = check_device();
  if (ds != EBD_OK) return ds;
  AppendLaunch L;
  L.U = num_units;
  L.cap_off = cap_off;
  L.count = count;
  L.k_new = k_new;
  L.v_new = v_new;
  L.pos_new = pos_new;
  L.Kc = Kc;
  L.Vc = Vc;
  L.pic = pic;
  L.idxc = idxc;
  L.status = status;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (timed("append_certain", s, [&] { return launch_append_certain(L, s); }) != hipSuccess)
    return EBD_ERR_HIP;
  return EBD_OK;
}

ebd_status ebd_timing_enable(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing.store(enable != 0, std::memory_order_release);
  return EBD_OK;
}

ebd_status ebd_timing_read(const char *name, double *total_ms, int64_t *launches) {
  if (!name || !total_ms || !launches) return EBD_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_tmu);
  auto it = g_trec.find(name);
  *total_ms = 0.0;
  *launches = 0;
  if (it == g_trec.end()) return EBD_OK;
  TimingRec &r = it->second;
  ebd_status st = EBD_OK;
  for (auto &ev : r.pending) {
    float ms = 0.0f;
    if (hipEventSynchronize(ev.second) != hipSuccess ||
        hipEventElapsedTime(&ms, ev.first, ev.second) != hipSuccess) {
      st = EBD_ERR_HIP;
    } else {
      r.ms += ms;
      r.launches += 1;
    }
    r.pool.push_back(ev.first);
    r.pool.push_back(ev.second);
  }
  r.pending.clear();
  *total_ms = r.ms;
  *launches = r.launches;
  r.ms = 0.0;
  r.launches = 0;
  return st;
}

}  // extern "C"
