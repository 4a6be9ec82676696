/*
 * ebd.h -- C ABI of the MI355X (gfx950) eviction-by-design (EBD) library, libebd.so.
 *
 * Method: "Error Certificates for KV-Cache Eviction via Randomized Design".
 * A "unit" is one KV-head cache (one layer, one batch row, one KV head), the
 * object of Sec. 3.1.  Each unit is sampled independently: a certainty set
 * (protected positions plus tokens whose eq. (2) allocation clips at 1) is
 * always kept and the tail is Poisson-sampled at the stored probabilities pi.
 * Decode attention then runs over the retained rows with the Hajek weights of
 * eq. (3) and, in the same pass, produces the Theorem 2 variance estimate and
 * the eq. (4) radius for every query head.
 *
 * Conventions for every entry point:
 *   - All data pointers are DEVICE pointers owned by the caller.  The library
 *     allocates nothing and frees nothing; scratch space is the caller's
 *     `workspace` buffer, sized by ebd_workspace_size().
 *   - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 *   - Rows are head_dim contiguous elements; head_dim must be 128.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the default
 *     stream).  Host-detectable argument errors are returned synchronously and
 *     nothing is launched.  Data-dependent conditions are reported per unit
 *     in the `status` words (EBD_ST_*), written by the kernels.
 *   - Calls on different streams may run concurrently if they do not share
 *     output or workspace buffers.
 */
#ifndef EBD_H
#define EBD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum ebd_status {
    EBD_OK = 0,
    EBD_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, bad parameter */
    EBD_ERR_UNSUPPORTED = 2, /* head_dim != 128, no gfx950 device current, or a size beyond
                                a limit documented at the entry point */
    EBD_ERR_WORKSPACE = 3,   /* workspace NULL or smaller than ebd_workspace_size() */
    EBD_ERR_HIP = 4          /* a HIP runtime call failed (launch, event) */
} ebd_status;

/* Per-unit status bits written by ebd_evict (status[u]), ebd_append_certain and
   ebd_attend_certify. */
#define EBD_ST_CAP_OVERFLOW 1u /* retained count exceeds the unit's capacity: rows at or
                                  beyond the capacity are NOT written; count[u] holds the
                                  true count; re-run with a larger capacity */
#define EBD_ST_BUDGET_FLOOR 2u /* m <= pi_min * |T|: every tail pi equals pi_min, so the
                                  expected size exceeds the budget */
#define EBD_ST_NO_EVICTION 4u  /* the budget covers every positive-score tail token: all
                                  of them get pi = 1 (zero scores keep pi_min) */
#define EBD_ST_BAD_SCORE 8u    /* a NaN, infinite or negative score was seen; it is
                                  treated as 0 (pi = pi_min) */
#define EBD_ST_BAD_LAYOUT 16u  /* ebd_evict: the unit exceeds params.max_rows or
                                  params.max_capacity: nothing was sampled or written for it
                                  and count[u] = 0.  ebd_attend_certify: the unit holds more
                                  rows than params.max_rows; those past it were not seen */

/*
 * Sampler parameters (Sec. 3.3, eq. (2) and the certainty set).
 *   seq_off  [U+1] device int64: unit u owns full-cache rows seq_off[u] .. seq_off[u+1]-1
 *            of `scores`, `K`, `V` (non-decreasing; uniform caches: u * n).
 *   cap_off  [U+1] device int64: unit u owns compacted rows cap_off[u] .. cap_off[u+1]-1
 *            of Kc, Vc, pic, idxc (its capacity).
 *   max_rows host value >= max_u (seq_off[u+1] - seq_off[u]); units longer than this are
 *            flagged EBD_ST_BAD_LAYOUT and left untouched.
 *   max_capacity host value >= max_u (cap_off[u+1] - cap_off[u]); sizes the copy grid.
 *            Units outside either bound are flagged EBD_ST_BAD_LAYOUT (nothing written).
 *   n_sink, n_recent: protected positions i < n_sink and i >= n - n_recent (pi = 1).
 *   budget_frac f: expected resident tokens per unit = f * n, protected ones included,
 *            so the tail budget is m = f n - |P| (real valued).
 *   budget_per_unit [U] device float or NULL: per-unit f overriding budget_frac.
 *   pi_min   eps > 0, the floor of eq. (2).
 *   pi_mode  0: lambda solves sum_T clip(lambda s_i, eps, 1) = m (expected tail size = m);
 *            1: lambda = m / sum_T s_i, eq. (2) taken verbatim (then clipped).
 *   seed, seed_per_unit [U] (device or NULL), epoch: the Philox4x32-10 stream.  Token i of
 *            unit u is kept iff x < pi_i * 2^32, x = word (i mod 4) of
 *            Philox4x32-10(counter = (i/4, u, epoch, 0x45424431), key = (seed lo, seed hi)).
 *   design   EBD_DESIGN_POISSON (0, Sec. 3.3): independent retention as above.
 *            EBD_DESIGN_SYSTEMATIC (1, App. "Experimental details", fixed-size systematic
 *            sampling at the same pi): integer weights a_i = ceil(pi_i 2^32), cumulative sums
 *            C_i over the unit, one start s = word 0 of Philox4x32-10(counter = (0, u, epoch,
 *            0x45424453), key = seed); position i is kept iff a point s + k 2^32 (k >= 0) lies
 *            in [C_{i-1}, C_i).  The retained size is floor or ceil of sum_i a_i / 2^32.
 *            EBD_DESIGN_TOPK (2, the deterministic comparison arm): the protected positions
 *            and the k = floor(m + 1/2) largest tail scores (ties to the lower position), all
 *            with pi = 1; other positions get pi = 0; lambda_out is 0.
 *            EBD_DESIGN_UNIFORM (3, the uniform comparison arm): every tail score is taken
 *            as 1 (scores are not read), so pi = clip(m / |T|, eps, 1) on the tail.
 */
#define EBD_DESIGN_POISSON 0
#define EBD_DESIGN_SYSTEMATIC 1
#define EBD_DESIGN_TOPK 2
#define EBD_DESIGN_UNIFORM 3

typedef struct ebd_evict_params {
    int32_t num_units;
    int32_t head_dim;
    int64_t max_rows;
    int64_t max_capacity;
    const int64_t *seq_off;
    const int64_t *cap_off;
    int32_t n_sink;
    int32_t n_recent;
    float budget_frac;
    const float *budget_per_unit;
    float pi_min;
    int32_t pi_mode;
    uint64_t seed;
    const uint64_t *seed_per_unit;
    uint32_t epoch;
    int32_t design;
} ebd_evict_params;

/*
 * ebd_evict -- the tail sampler for U units (Sec. 3.3; Sec. 3.1 for deletion).
 *   scores [rows] fp32 importance (input of eq. (2)); K, V [rows, 128] bf16.
 *   Outputs (compacted, stable: ascending original position):
 *     Kc, Vc [cap rows, 128] bf16   retained rows
 *     pic    [cap rows] fp32        stored inclusion probability of each retained row
 *     idxc   [cap rows] int32       original position (within its unit) of each row
 *     count  [U] int32              retained rows per unit (true count, even on overflow)
 *     lambda_out [U] fp32 or NULL   the solved scale (+inf when nothing is evicted)
 *     pi_full [rows] fp32 or NULL   pi of every full-cache position
 *     status [U] uint32             EBD_ST_* bits
 *   workspace: at least ebd_workspace_size(EBD_WS_EVICT, p) bytes, 256-byte aligned
 *   (currently reserved: the sampler's launches share only the idxc list they write).
 *   Launches whose units are at most 6144 tokens long, with capacities of at least a sixth
 *   of that, take two kernels (selection, then the row gather "evict_copy"); other launches
 *   one ("evict_select" also gathers the rows).
 *   Rows of Kc/Vc/pic/idxc beyond count[u] are left untouched.
 */
ebd_status ebd_evict(const ebd_evict_params *p, const float *scores, const uint16_t *K,
                     const uint16_t *V, uint16_t *Kc, uint16_t *Vc, float *pic, int32_t *idxc,
                     int32_t *count, float *lambda_out, float *pi_full, uint32_t *status,
                     void *workspace, size_t ws_bytes, void *stream);

/*
 * Certified decode attention parameters (Sec. 3.3 eq. (3), Theorem 2; Sec. 3.4 eq. (4)).
 *   group G: query heads per KV head (q is [U, G, 128]); any G >= 1.
 *   cap_off [U+1] device int64: the compacted layout written by ebd_evict.
 *   max_rows host value >= the most rows any unit holds; sizes the split grid (rows of a unit
 *   beyond it are not seen, and flagged in the status words).
 *   scale: logit scale (0 means 1/sqrt(head_dim)); delta (0 means 0.1) and eps0
 *   (0 means 1e-9): the confidence level and normaliser of eq. (4).
 *   split_rows: retained rows per split, one wave each (0 = library choice; else a
 *   multiple of 16 in [16, 8192]).
 *   A unit spans at most 4096 splits: max_rows above 4096 split rows (with the library's
 *   choice, above 4096 x 4096 rows) returns EBD_ERR_UNSUPPORTED.
 *   flags: 0, or EBD_F_NO_OFFSET: y and ln N are those of the uncorrected retained softmax
 *   (the logit offset -ln pi dropped, the ablation arm of Sec. 5 and App. "Experimental
 *   details"), while vhat, b and r stay the Hajek certificate of the same retained set;
 *   costs a second pass over the retained rows.
 */
#define EBD_F_NO_OFFSET 1u

typedef struct ebd_attend_params {
    int32_t num_units;
    int32_t group;
    int32_t head_dim;
    int32_t split_rows;
    int64_t max_rows;
    const int64_t *cap_off;
    float scale;
    float delta;
    float eps0;
    uint32_t flags;
} ebd_attend_params;

/*
 * ebd_attend_certify -- one decode step of certified attention over the retained rows.
 *   q [U, G, 128] bf16; Kc, Vc, pic, count as written by ebd_evict.  The step sees the first
 *   min(count[u], capacity, max_rows) rows of unit u; what it cannot see is reported in status.
 *   Outputs per (unit, query head), fp32:
 *     y      [U, G, 128]  Hajek output yhat = sum_S (a/pi) v / sum_S (a/pi)      (eq. (3))
 *     vhat   [U, G]       variance estimate of Theorem 2
 *     lse    [U, G]       ln Nhat, Nhat = sum_S a/pi (a = exp(scale q.k)); -inf if S empty
 *     brange [U, G]       range term b of eq. (4) (exact maximum), or NULL
 *     radius [U, G]       radius r of eq. (4), or NULL
 *     status [U] uint32 or NULL, written (not or-ed): EBD_ST_CAP_OVERFLOW when count[u] exceeds
 *            the unit's capacity (rows past the capacity were never stored and are not seen),
 *            EBD_ST_BAD_LAYOUT when the unit holds more rows than max_rows (the rows past
 *            max_rows are not seen); 0 otherwise.  The outputs then cover the rows seen.
 *   vhat is accumulated in the same pass as C2 - 2 yhat.Cv + |yhat|^2 C0 (C0 = sum c,
 *   Cv = sum c v, C2 = sum c |v|^2, c = (1 - pi) (a/pi)^2), with each head's largest-weight
 *   row kept out of these sums and added back in closed form, so that one tail row dominating
 *   both yhat and the variance does not make them cancel; a head where the other rows still
 *   cancel (several identical dominating rows) is summed again directly over the unit's rows,
 *   sum c |v - yhat|^2, in the same call.
 *   workspace: at least ebd_workspace_size(EBD_WS_ATTEND, p) bytes, 256-byte aligned; y must
 *   be 16-byte aligned.  After the call the workspace starts with two uint32 counts per (unit,
 *   block of 8 query heads): the 512-row chunks re-read to make the range term exact (0 when
 *   the kept candidates already decide it), then the heads whose vhat was summed directly.
 *   Then, when units span several splits, one partial record per (unit, split, query head).
 *   A unit of up to 4 splits runs them as the waves of one work-group, the last of which
 *   finalizes it, so the step is one kernel; units of more splits take a second kernel that
 *   combines the records.  When every unit fits one split the workspace holds only the counts.
 */
ebd_status ebd_attend_certify(const ebd_attend_params *p, const uint16_t *q, const uint16_t *Kc,
                              const uint16_t *Vc, const float *pic, const int32_t *count,
                              float *y, float *vhat, float *lse, float *brange, float *radius,
                              uint32_t *status, void *workspace, size_t ws_bytes, void *stream);

/*
 * ebd_attend_certify_noalloc -- ebd_attend_certify for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * same arguments, outputs and kernels, without the workspace argument.  The workspace is a fixed
 * device array inside the library of EBD_NOALLOC_SCRATCH_BYTES (64 MiB), one copy per GPU that
 * loads the library, held until the process ends.  The call allocates nothing and frees nothing
 * (host or device), and is not recorded by the kernel timing below.
 *   Returns EBD_ERR_UNSUPPORTED when the launch needs more than EBD_NOALLOC_SCRATCH_BYTES, i.e.
 *   when ebd_workspace_size(EBD_WS_ATTEND, p) exceeds it (nothing is launched); use
 *   ebd_attend_certify with a caller workspace for such launches.  Launches whose units are
 *   each one split need only 8 bytes per (unit, block of 8 query heads).
 *   Every call on one GPU uses that GPU's one array: calls that overlap on the same GPU (on
 *   several streams or from several host threads) race and must be ordered by the caller, e.g.
 *   issued on one stream.  The array keeps the last call's contents; nothing in it has to be
 *   cleared between calls.  The diagnostic counts that ebd_attend_certify leaves at the start
 *   of its workspace stay inside the library here.
 */
#define EBD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

ebd_status ebd_attend_certify_noalloc(const ebd_attend_params *p, const uint16_t *q,
                                      const uint16_t *Kc, const uint16_t *Vc, const float *pic,
                                      const int32_t *count, float *y, float *vhat, float *lse,
                                      float *brange, float *radius, uint32_t *status,
                                      void *stream);

/*
 * ebd_append_certain -- append one decode token per unit to its retained set with pi = 1
 * (a recency-certainty token; the sampled draw is reused across steps, App. A.2).
 *   k_new, v_new [U, 128] bf16; pos_new [U] int32 original positions or NULL (idx = -1).
 *   The row goes to slot count[u] of unit u and count[u] is incremented; if the unit is
 *   full, nothing is written, count is unchanged and EBD_ST_CAP_OVERFLOW is set in
 *   status[u] (status may be NULL).
 */
ebd_status ebd_append_certain(int32_t num_units, int32_t head_dim, const int64_t *cap_off,
                              int32_t *count, const uint16_t *k_new, const uint16_t *v_new,
                              const int32_t *pos_new, uint16_t *Kc, uint16_t *Vc, float *pic,
                              int32_t *idxc, uint32_t *status, void *stream);

/*
 * Importance scores from accumulated attention (App. "Experimental details", Harness: the
 * sampler's scores come from the attention that prefill queries, or a window of observation
 * queries, pay to each cached key).  For unit u and its W queries q_w (bf16 [U, W, 128]):
 *     score_i = sum_w softmax_w(scale q_w . k)_i
 * where query w sees rows 0 .. qpos[u * W + w] of the unit (a prefill query at that
 * position; a negative position sees nothing), or every row of the unit when qpos is NULL
 * (an observation window placed after the cache).  Each query's softmax sums to 1 over the
 * rows it sees, so the scores of a unit sum to the number of queries that see a row.
 *   seq_off [U+1] device int64: unit u owns rows seq_off[u] .. seq_off[u+1]-1 of K and of
 *            `scores` (fp32, written; with EBD_SCORES_ACCUMULATE added to instead, so that
 *            more than 64 queries can be spread over several calls).
 *   num_queries W: 1 .. 64.  max_rows >= the longest unit (sizes the split grid; rows of a
 *   longer unit past the planned splits are neither seen nor written).
 *   scale: logit scale (0 means 1/sqrt(head_dim)); split_rows: rows per split, one wave
 *   each (0 = library choice; else a multiple of 16 in [16, 65536]).
 *   workspace: at least ebd_workspace_size(EBD_WS_SCORES, p) bytes, 256-byte aligned.
 * Two passes over K: per split, each query's running max and exp-sum; then, with the
 * unit's combined normalisers, the scores.
 */
#define EBD_SCORES_ACCUMULATE 1u

typedef struct ebd_scores_params {
    int32_t num_units;
    int32_t head_dim;
    int32_t num_queries;
    int32_t split_rows;
    int64_t max_rows;
    const int64_t *seq_off;
    const int32_t *qpos;
    float scale;
    uint32_t flags;
} ebd_scores_params;

ebd_status ebd_scores(const ebd_scores_params *p, const uint16_t *q, const uint16_t *K,
                      float *scores, void *workspace, size_t ws_bytes, void *stream);

/*
 * Fine-grained attribution (Sec. 6 "Finer grains"; App. "Experimental details", the
 * fine-grained probe): the variance contribution of each retained row j to each query head h,
 *     kappa_hj = (1 - pi_j) / pi_j^2 * a_hj^2 |v_j - yhat_h|^2 / Nhat_h^2
 * (the summand of Theorem 2, so sum_j kappa_hj = vhat_h), summed over the unit's query heads
 * and over the rows whose original position idxc[j] falls in each block of block_rows
 * positions:  blocks[u * nblocks + b] = sum_h sum_{j: idxc_j / block_rows = b} kappa_hj.
 * Evicted blocks ranked by this sum are the retrieval targets of the paper's probe.
 *   q, Kc, Vc, pic, idxc, count: as given to / written by ebd_attend_certify and ebd_evict;
 *   y, lse: the outputs of ebd_attend_certify for the same q (yhat and ln Nhat).
 *   Rows with pi = 1, with idxc < 0 (appended decode rows) or past the last block add nothing.
 *   block_rows >= 1; 1 <= nblocks <= 8192; max_rows as for ebd_attend_certify (rows of a unit
 *   beyond it are ignored), below 2^24 (else EBD_ERR_UNSUPPORTED).  blocks [U, nblocks] fp32
 *   is written.  No workspace.
 */
typedef struct ebd_blocks_params {
    int32_t num_units;
    int32_t group;
    int32_t head_dim;
    int32_t block_rows;
    int64_t nblocks;
    int64_t max_rows;
    const int64_t *cap_off;
    float scale;
} ebd_blocks_params;

ebd_status ebd_block_contributions(const ebd_blocks_params *p, const uint16_t *q,
                                   const uint16_t *Kc, const uint16_t *Vc, const float *pic,
                                   const int32_t *idxc, const int32_t *count, const float *y,
                                   const float *lse, float *blocks, void *stream);

/*
 * Deployed certificate, one decode step (App. "Experimental details": eq. (4) at delta = 0.1 on
 * every fourth head of every layer over the first six decode steps, averaged, then maximized
 * over the steps).  For every sequence s: the mean of radius[u, g] over the units with
 * unit_seq[u] = s and the query heads g whose index (unit_head0[u] + g) is a multiple of
 * head_stride; cert[s] = max(cert[s], mean) (the caller sets cert before the first step);
 * mean_out[s] (or NULL) receives the mean.  A sequence without sampled pairs keeps cert[s]
 * and gets mean 0.  unit_seq [U] device int32 (negative: not counted); unit_head0 [U] device
 * int32 >= 0 or NULL (all 0); radius [U, G] as written by ebd_attend_certify.  U G < 2^31
 * (else EBD_ERR_INVALID_ARG).  The sums are taken in a fixed order (deterministic).
 */
typedef struct ebd_cert_params {
    int32_t num_units;
    int32_t group;
    int32_t num_seqs;
    int32_t head_stride;
    const int32_t *unit_seq;
    const int32_t *unit_head0;
} ebd_cert_params;

ebd_status ebd_certificate_step(const ebd_cert_params *p, const float *radius, float *cert,
                                float *mean_out, void *stream);

/* which-values for ebd_workspace_size */
#define EBD_WS_EVICT 0
#define EBD_WS_ATTEND 1
#define EBD_WS_SCORES 2

/*
 * Workspace bytes needed by ebd_evict (which = EBD_WS_EVICT, params = ebd_evict_params*),
 * ebd_attend_certify (EBD_WS_ATTEND, ebd_attend_params*) or ebd_scores (EBD_WS_SCORES,
 * ebd_scores_params*).  Depends only on the host fields of the params.  Returns 0 on
 * invalid arguments.
 */
size_t ebd_workspace_size(int32_t which, const void *params);

/* Static description of a status code; never NULL. */
const char *ebd_status_string(ebd_status s);

/* Library version string, e.g. "ebd-gfx950 0.1.0". */
const char *ebd_version(void);

/*
 * Kernel timing (a process-wide profiling aid, off by default).  While enabled, every kernel
 * launch of the library is bracketed by HIP events recorded on its own launch stream.
 * ebd_timing_read() waits for the recorded events, and adds the elapsed times of kernel `name`
 * ("evict_select", "evict_copy", "attend_split", "attend_finalize", "append_certain",
 * "scores_stats", "scores_accum", "block_contrib", "cert_step") to *total_ms and its launch
 * count to *launches; it then clears that kernel's record.  The switch is an atomic flag and the
 * records are guarded by a lock, so both calls may come from any host thread; while timing is
 * off no event is created and launches take no lock.
 */
ebd_status ebd_timing_enable(int32_t enable);
ebd_status ebd_timing_read(const char *name, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* EBD_H */
