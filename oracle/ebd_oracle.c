/*
 * ebd_oracle.c -- plain fp64 CPU oracle for the eviction-by-design (EBD) hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the parity oracle for the HIP library.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load or call it.  It shares no code, header, table or constant generator with
 * the GPU path; it was written directly from the paper's definitions:
 *
 *   "Error Certificates for KV-Cache Eviction via Randomized Design"
 *     Sec. 3.1  eq. (1)  full-cache attention  y = sum a_i v_i / sum a_i
 *     Sec. 3.3  eq. (2)  inclusion probabilities pi_i = clip(m s_i / sum_T s, eps, 1)
 *               certainty set: protected positions + tokens clipped at 1
 *               Poisson (independent Bernoulli) retention on the tail T
 *     Sec. 3.3  eq. (3)  Hajek estimator  yhat = sum_S (a/pi) v / sum_S a/pi
 *     Sec. 3.3  Theorem 2  Vhat = Nhat^-2 sum_{S cap T} (1-pi)/pi^2 a^2 |v - yhat|^2
 *     Sec. 3.4  eq. (4)  radius r = (sqrt(2 Vhat ln(1/delta)) + b ln(1/delta)) / (|yhat| + eps0)
 *                        b = max_{S cap T} sqrt((1-pi)/pi^2) a |v - yhat| / Nhat
 *   Sec. 6 "Finer grains" and the fine-grained probe: per-token variance contributions
 *     pooled into blocks of original positions; the deployed certificate (mean radius
 *     over sampled heads, maximum over decode steps)
 *   App. "Experimental details", Harness: importance scores from accumulated attention
 *     (strided prefill queries) or an observation window of queries: per query, the
 *     softmax over the keys it sees, summed over the queries
 *   Counter-based RNG: Philox4x32-10, Salmon, Moraes, Dror & Shaw,
 *     "Parallel random numbers: as easy as 1, 2, 3", SC 2011.
 *
 * Readings of points the paper leaves open (each also listed in the design notes):
 *   - The tail budget m is solved for: lambda with sum_T clip(lambda s_i, eps, 1) = m,
 *     so the expected tail size equals m exactly (eq. (2) read as a budget solve;
 *     the literal lambda = m / sum_T s is kept as pi_mode 1).
 *   - m = f n - |P| (the budget counts protected tokens), real valued.
 *   - Non-finite or negative scores are treated as 0 (pi = eps) and flagged.
 *   - Retention of token i of unit u: x_i = word (i mod 4) of
 *     Philox4x32-10(counter = (i / 4, u, epoch, 0x45424431), key = (seed lo, seed hi));
 *     retained iff x_i < pi32_i * 2^32, compared exactly in fp64.
 *   - Retained tokens keep ascending original order.
 *   - The offset -ln(pi) applies to every retained token (0 when pi = 1).
 *
 *   - Fixed-size systematic design: integer weights a_i = ceil(pi32_i 2^32) (the
 *     Poisson test's exact inclusion probability), cumulative sums C_i, start
 *     u = word 0 of Philox4x32-10(counter = (0, u, epoch, 0x45424453), key = seed);
 *     position i is kept iff a point u + k 2^32 falls in [C_{i-1}, C_i).
 *   - Top-k comparison design: the protected positions and the k = floor(m + 1/2)
 *     largest cleaned tail scores, ties to the lower position, kept with pi = 1.
 *   - Uniform comparison design: every tail score taken as 1 (pi = clip(m/|T|, eps, 1)).
 *
 * Everything is fp64 except the stored per-token pi, which is rounded once to
 * fp32 (the stored design), exactly as the library stores it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define REF_ST_CAP_OVERFLOW 1u
#define REF_ST_BUDGET_FLOOR 2u
#define REF_ST_NO_EVICTION 4u
#define REF_ST_BAD_SCORE 8u

#define REF_PHILOX_TAG 0x45424431u     /* "EBD1": the per-token Poisson stream */
#define REF_SYSTEMATIC_TAG 0x45424453u /* "EBDS": the per-unit systematic start */

/* Sampling designs (Sec. 3.3 Poisson; App. "Experimental details": fixed-size systematic
   sampling at the same pi; the deterministic top-k and uniform comparison arms). */
#define REF_DESIGN_POISSON 0
#define REF_DESIGN_SYSTEMATIC 1
#define REF_DESIGN_TOPK 2
#define REF_DESIGN_UNIFORM 3

/* ------------------------------------------------------------------ */
/* bf16 bits -> double (exact: bf16 is the top half of an fp32)        */
/* ------------------------------------------------------------------ */
static double ref_bf16(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* ------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon et al. 2011): ten rounds of the 4x32 Philox   */
/* S-box, key bumped by the Weyl constants between rounds.             */
/* ------------------------------------------------------------------ */
void ebd_ref_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const uint32_t mul0 = 0xD2511F53u, mul1 = 0xCD9E8D57u;
    const uint32_t weyl0 = 0x9E3779B9u, weyl1 = 0xBB67AE85u;
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += weyl0;
            k1 += weyl1;
        }
        uint64_t p0 = (uint64_t)mul0 * c0;
        uint64_t p1 = (uint64_t)mul1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The 32-bit uniform word that decides token i of unit u. */
uint32_t ebd_ref_token_word(uint64_t seed, uint32_t unit, uint32_t epoch, int64_t i)
{
    uint32_t ctr[4] = {(uint32_t)(i >> 2), unit, epoch, REF_PHILOX_TAG};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    ebd_ref_philox4x32_10(ctr, key, out);
    return out[i & 3];
}

/* ------------------------------------------------------------------ */
/* Sec. 3.3: partition into protected P and tail T                     */
/* ------------------------------------------------------------------ */
static int ref_is_protected(int64_t i, int64_t n, int32_t n_sink, int32_t n_recent)
{
    return i < (int64_t)n_sink || i >= n - (int64_t)n_recent;
}

/* g(lambda) = sum_T clip(lambda s_i, eps, 1): the expected tail size under eq. (2). */
static double ref_tail_mass(int64_t n, const double *s, const unsigned char *tail, double lam, double eps)
{
    double g = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        if (!tail[i]) continue;
        double p = lam * s[i];
        if (p < eps) p = eps;
        if (p > 1.0) p = 1.0;
        g += p;
    }
    return g;
}

/*
 * Inclusion probabilities for one unit (Sec. 3.3, eq. (2), certainty set).
 *   budget_frac f: total expected resident tokens = f n, protected tokens included.
 *   pi_mode 0: lambda solves sum_T clip(lambda s, eps, 1) = m by plain bisection in fp64.
 *   pi_mode 1: lambda = m / sum_T s, eq. (2) verbatim.
 * Writes pi (fp64) for every position and returns the status bits.
 */
uint32_t ebd_ref_inclusion_probs(int64_t n, const float *scores, int32_t n_sink, int32_t n_recent,
                                 double budget_frac, double pi_min, int pi_mode,
                                 double *lambda_out, double *pi_out)
{
    uint32_t status = 0;
    double *s = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    unsigned char *tail = (unsigned char *)malloc((size_t)(n > 0 ? n : 1));
    int64_t n_prot = 0, n_tail = 0, n_pos = 0, n_zero = 0;
    double sum_tail = 0.0, s_min_pos = INFINITY;

    for (int64_t i = 0; i < n; ++i) {
        double v = (double)scores[i];
        if (!isfinite(v) || v < 0.0) {
            status |= REF_ST_BAD_SCORE;
            v = 0.0;
        }
        s[i] = v;
        tail[i] = !ref_is_protected(i, n, n_sink, n_recent);
        if (tail[i]) {
            n_tail++;
            sum_tail += v;
            if (v > 0.0) {
                n_pos++;
                if (v < s_min_pos) s_min_pos = v;
            } else {
                n_zero++;
            }
        } else {
            n_prot++;
        }
    }

    const double eps = pi_min;
    const double m = budget_frac * (double)n - (double)n_prot;
    double lam = 0.0;

    if (n_tail == 0) {
        lam = 0.0;
    } else if (pi_mode == 1) {
        /* eq. (2) verbatim: lambda = m / sum_T score; only the clip applies */
        lam = (sum_tail > 0.0 && m > 0.0) ? m / sum_tail : 0.0;
        if (m <= eps * (double)n_tail) status |= REF_ST_BUDGET_FLOOR;
    } else if (m <= eps * (double)n_tail) {
        /* the floor alone already spends the budget: every tail pi = eps */
        lam = 0.0;
        status |= REF_ST_BUDGET_FLOOR;
    } else if (m >= (double)n_pos + eps * (double)n_zero) {
        /* budget covers every positive-score token: no eviction among them */
        lam = INFINITY;
        status |= REF_ST_NO_EVICTION;
    } else {
        /* g(0) = eps |T| < m <= g(1 / s_min_pos): bisect on [0, 1 / s_min_pos]. */
        double lo = 0.0, hi = 1.0 / s_min_pos;
        for (int it = 0; it < 4000; ++it) {
            double mid = 0.5 * (lo + hi);
            if (mid <= lo || mid >= hi) break;
            if (ref_tail_mass(n, s, tail, mid, eps) < m) lo = mid;
            else hi = mid;
        }
        lam = 0.5 * (lo + hi);
    }

    for (int64_t i = 0; i < n; ++i) {
        if (!tail[i]) {
            pi_out[i] = 1.0;
        } else if (isinf(lam)) {
            pi_out[i] = s[i] > 0.0 ? 1.0 : eps;
        } else {
            double p = lam * s[i];
            if (p < eps) p = eps;
            if (p > 1.0) p = 1.0;
            pi_out[i] = p;
        }
    }
    if (lambda_out) *lambda_out = lam;
    free(s);
    free(tail);
    return status;
}

/* Poisson retention (Sec. 3.3): I_i = [x_i < pi32_i 2^32], exact fp64 compare. Returns |S|. */
int64_t ebd_ref_mask(int64_t n, const float *pi32, uint64_t seed, uint32_t unit, uint32_t epoch,
                     uint8_t *mask)
{
    int64_t kept = 0;
    for (int64_t i = 0; i < n; ++i) {
        double x = (double)ebd_ref_token_word(seed, unit, epoch, i);
        double thr = (double)pi32[i] * 4294967296.0;
        mask[i] = x < thr ? 1 : 0;
        kept += mask[i];
    }
    return kept;
}

/* ------------------------------------------------------------------ */
/* Fixed-size systematic sampling at the same inclusion probabilities  */
/* (App. "Experimental details"; Hajek 1964): one uniform start per    */
/* unit, points u + k 2^32 on the cumulative integer weights.          */
/* ------------------------------------------------------------------ */
uint32_t ebd_ref_systematic_start(uint64_t seed, uint32_t unit, uint32_t epoch)
{
    const uint32_t ctr[4] = {0u, unit, epoch, REF_SYSTEMATIC_TAG};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    ebd_ref_philox4x32_10(ctr, key, out);
    return out[0];
}

/* Number of points u + k 2^32 (k >= 0) strictly below C. */
static uint64_t ref_points_below(uint64_t C, uint32_t u)
{
    return C > (uint64_t)u ? ((C - (uint64_t)u - 1u) >> 32) + 1u : 0u;
}

int64_t ebd_ref_mask_systematic(int64_t n, const float *pi32, uint64_t seed, uint32_t unit,
                                uint32_t epoch, uint8_t *mask)
{
    const uint32_t u = ebd_ref_systematic_start(seed, unit, epoch);
    uint64_t C = 0;
    int64_t kept = 0;
    for (int64_t i = 0; i < n; ++i) {
        /* pi32 * 2^32 is exact in fp64; its ceiling is the Poisson test's integer threshold */
        const uint64_t a = (uint64_t)ceil((double)pi32[i] * 4294967296.0);
        const uint64_t Cn = C + a;
        mask[i] = (uint8_t)(ref_points_below(Cn, u) - ref_points_below(C, u));
        kept += mask[i];
        C = Cn;
    }
    return kept;
}

/* ------------------------------------------------------------------ */
/* Comparison designs: deterministic top-k and uniform tail sampling.  */
/* ------------------------------------------------------------------ */
static const double *ref_sort_scores;
static int ref_by_score_desc(const void *x, const void *y)
{
    int64_t i = *(const int64_t *)x, j = *(const int64_t *)y;
    double a = ref_sort_scores[i], b = ref_sort_scores[j];
    if (a > b) return -1;
    if (a < b) return 1;
    return i < j ? -1 : (i > j ? 1 : 0);
}

/* Top-k: pi = 1 on P and on the k = floor(m + 1/2) best tail positions, 0 elsewhere. */
uint32_t ebd_ref_topk_probs(int64_t n, const float *scores, int32_t n_sink, int32_t n_recent,
                            double budget_frac, double *pi_out)
{
    uint32_t status = 0;
    double *s = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    int64_t *idx = (int64_t *)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    int64_t n_tail = 0, n_prot = 0;
    for (int64_t i = 0; i < n; ++i) {
        double v = (double)scores[i];
        if (!isfinite(v) || v < 0.0) {
            status |= REF_ST_BAD_SCORE;
            v = 0.0;
        }
        s[i] = v;
        if (ref_is_protected(i, n, n_sink, n_recent)) {
            pi_out[i] = 1.0;
            n_prot++;
        } else {
            pi_out[i] = 0.0;
            idx[n_tail++] = i;
        }
    }
    double m = budget_frac * (double)n - (double)n_prot;
    int64_t k = (int64_t)floor(m + 0.5);
    if (k < 0) k = 0;
    if (k >= n_tail) {
        k = n_tail;
        if (n_tail > 0) status |= REF_ST_NO_EVICTION;
    }
    /* qsort is not reentrant with a file-scope key: callers run one unit per thread, so the
       sort is done under a critical section */
#ifdef _OPENMP
#pragma omp critical(ref_topk_sort)
#endif
    {
        ref_sort_scores = s;
        qsort(idx, (size_t)n_tail, sizeof(int64_t), ref_by_score_desc);
        ref_sort_scores = NULL;
    }
    for (int64_t r = 0; r < k; ++r) pi_out[idx[r]] = 1.0;
    free(s);
    free(idx);
    return status;
}

/*
 * Stable compaction of the retained set (Sec. 3.1: evicted tokens are deleted;
 * Sec. 3.3: one stored pi per retained token).  Rows beyond `cap` are not
 * written; the return value is always the true |S|.
 */
int64_t ebd_ref_compact(int64_t n, int32_t d, const uint8_t *mask, const float *pi32,
                        const uint16_t *K, const uint16_t *V, int64_t cap,
                        uint16_t *Kc, uint16_t *Vc, float *pic, int32_t *idx)
{
    int64_t r = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (!mask[i]) continue;
        if (r < cap) {
            memcpy(Kc + r * d, K + i * d, (size_t)d * sizeof(uint16_t));
            memcpy(Vc + r * d, V + i * d, (size_t)d * sizeof(uint16_t));
            pic[r] = pi32[i];
            idx[r] = (int32_t)i;
        }
        r++;
    }
    return r;
}

/*
 * Hajek output and certificate for the G query heads of one unit
 * (Sec. 3.3 eq. (3), Theorem 2; Sec. 3.4 eq. (4)).
 *   q [G, d] bf16 bits; Kc, Vc [count, d] bf16 bits; pic [count] stored pi.
 *   a_j = exp(s_j - M) with s_j = scale q.k_j and M = max_j s_j (the common
 *   factor exp(-M) cancels in yhat, Vhat, b and r; it is added back in lse).
 *   use_offset = 0: y and lse are those of the uncorrected retained softmax (weights a_j,
 *   no 1/pi), while Vhat, b and r stay the Hajek certificate of the same retained set
 *   (App. "Experimental details": runs with the uncorrected softmax computed the
 *   certificate as the Hajek radius).
 * Outputs per head: y [G, d], vhat, lse = ln Nhat, brange, radius.
 */
void ebd_ref_attend_certify(int32_t G, int32_t d, int64_t count, const uint16_t *q,
                            const uint16_t *Kc, const uint16_t *Vc, const float *pic,
                            double scale, double delta, double eps0, int use_offset,
                            double *y, double *vhat, double *lse, double *brange, double *radius)
{
    double *s = (double *)malloc((size_t)(count > 0 ? count : 1) * sizeof(double));
    double *a = (double *)malloc((size_t)(count > 0 ? count : 1) * sizeof(double));
    double *qd = (double *)malloc((size_t)d * sizeof(double));
    double *yhaj = (double *)malloc((size_t)d * sizeof(double));
    const double log_inv_delta = log(1.0 / delta);

    for (int32_t h = 0; h < G; ++h) {
        double *yh = yhaj; /* the Hajek output, for the certificate */
        for (int32_t c = 0; c < d; ++c) {
            qd[c] = ref_bf16(q[(int64_t)h * d + c]);
            yh[c] = 0.0;
        }
        for (int32_t c = 0; c < d; ++c) y[(int64_t)h * d + c] = 0.0;
        if (count == 0) {
            vhat[h] = 0.0;
            lse[h] = -INFINITY;
            if (brange) brange[h] = 0.0;
            if (radius) radius[h] = 0.0;
            continue;
        }
        /* scores s_j = q^T k_j / sqrt(d) (Sec. 3.1) */
        double M = -INFINITY;
        for (int64_t j = 0; j < count; ++j) {
            double dot = 0.0;
            for (int32_t c = 0; c < d; ++c) dot += qd[c] * ref_bf16(Kc[j * d + c]);
            s[j] = scale * dot;
            if (s[j] > M) M = s[j];
        }
        /* a_j (scaled by exp(-M)); Nhat = sum_S a_j / pi_j (eq. (3) denominator) */
        double Nhat = 0.0;
        for (int64_t j = 0; j < count; ++j) {
            a[j] = exp(s[j] - M);
            Nhat += a[j] / (double)pic[j];
        }
        /* yhat = sum_S (a_j / pi_j) v_j / Nhat (eq. (3)) */
        for (int64_t j = 0; j < count; ++j) {
            double wj = a[j] / (double)pic[j] / Nhat;
            for (int32_t c = 0; c < d; ++c) yh[c] += wj * ref_bf16(Vc[j * d + c]);
        }
        /* Theorem 2 and eq. (4): sums over S cap T (pi < 1; pi = 1 terms vanish) */
        double V = 0.0, bmax = 0.0;
        for (int64_t j = 0; j < count; ++j) {
            double pj = (double)pic[j];
            if (!(pj < 1.0)) continue;
            double dist2 = 0.0;
            for (int32_t c = 0; c < d; ++c) {
                double e = ref_bf16(Vc[j * d + c]) - yh[c];
                dist2 += e * e;
            }
            V += (1.0 - pj) / (pj * pj) * a[j] * a[j] * dist2 / (Nhat * Nhat);
            double bj = sqrt((1.0 - pj) / (pj * pj)) * a[j] * sqrt(dist2) / Nhat;
            if (bj > bmax) bmax = bj;
        }
        double ynorm = 0.0;
        for (int32_t c = 0; c < d; ++c) ynorm += yh[c] * yh[c];
        ynorm = sqrt(ynorm);
        vhat[h] = V;
        if (brange) brange[h] = bmax;
        if (radius) radius[h] = (sqrt(2.0 * V * log_inv_delta) + bmax * log_inv_delta) / (ynorm + eps0);
        double *yo = y + (int64_t)h * d;
        if (use_offset) {
            for (int32_t c = 0; c < d; ++c) yo[c] = yh[c];
            lse[h] = M + log(Nhat);
        } else {
            /* uncorrected retained softmax: weights a_j, normaliser sum_S a_j */
            double N0 = 0.0;
            for (int64_t j = 0; j < count; ++j) N0 += a[j];
            for (int64_t j = 0; j < count; ++j) {
                double wj = a[j] / N0;
                for (int32_t c = 0; c < d; ++c) yo[c] += wj * ref_bf16(Vc[j * d + c]);
            }
            lse[h] = M + log(N0);
        }
    }
    free(s);
    free(a);
    free(qd);
    free(yhaj);
}

/* Full-cache head output, eq. (1): y = sum_C a_i v_i / sum_C a_i, for G heads. */
void ebd_ref_full_attention(int32_t G, int32_t d, int64_t n, const uint16_t *q, const uint16_t *K,
                            const uint16_t *V, double scale, double *y)
{
    double *s = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    double *qd = (double *)malloc((size_t)d * sizeof(double));
    for (int32_t h = 0; h < G; ++h) {
        double *yh = y + (int64_t)h * d;
        for (int32_t c = 0; c < d; ++c) {
            qd[c] = ref_bf16(q[(int64_t)h * d + c]);
            yh[c] = 0.0;
        }
        if (n == 0) continue;
        double M = -INFINITY;
        for (int64_t i = 0; i < n; ++i) {
            double dot = 0.0;
            for (int32_t c = 0; c < d; ++c) dot += qd[c] * ref_bf16(K[i * d + c]);
            s[i] = scale * dot;
            if (s[i] > M) M = s[i];
        }
        double N = 0.0;
        for (int64_t i = 0; i < n; ++i) N += exp(s[i] - M);
        for (int64_t i = 0; i < n; ++i) {
            double w = exp(s[i] - M) / N;
            for (int32_t c = 0; c < d; ++c) yh[c] += w * ref_bf16(V[i * d + c]);
        }
    }
    free(s);
    free(qd);
}

/* ------------------------------------------------------------------ */
/* Fine-grained attribution (Sec. 6 "Finer grains"; App. "Experimental */
/* details", fine-grained probe): the variance contribution of each    */
/* retained token, kappa_hj = (1-pi_j)/pi_j^2 a_hj^2 |v_j - yhat_h|^2 / */
/* Nhat_h^2 (the summand of Theorem 2), summed over the unit's query   */
/* heads and over the retained tokens whose original position lies in  */
/* each block of `block_rows` positions.  yhat and ln Nhat are inputs  */
/* (the outputs of the certified attention).                           */
/* ------------------------------------------------------------------ */
void ebd_ref_block_contributions(int32_t G, int32_t d, int64_t count, const uint16_t *q,
                                 const uint16_t *Kc, const uint16_t *Vc, const float *pic,
                                 const int32_t *idx, const double *yhat, const double *lse,
                                 double scale, int32_t block_rows, int64_t nblocks, double *out)
{
    double *qd = (double *)malloc((size_t)d * sizeof(double));
    for (int64_t b = 0; b < nblocks; ++b) out[b] = 0.0;
    for (int32_t h = 0; h < G; ++h) {
        for (int32_t c = 0; c < d; ++c) qd[c] = ref_bf16(q[(int64_t)h * d + c]);
        const double *yh = yhat + (int64_t)h * d;
        for (int64_t j = 0; j < count; ++j) {
            if (idx[j] < 0) continue;  /* appended without a position (pi = 1: no term) */
            const int64_t b = (int64_t)idx[j] / block_rows;
            if (b >= nblocks) continue;
            const double pj = (double)pic[j];
            if (!(pj < 1.0)) continue;
            double dot = 0.0, dist2 = 0.0;
            for (int32_t c = 0; c < d; ++c) {
                dot += qd[c] * ref_bf16(Kc[j * d + c]);
                const double e = ref_bf16(Vc[j * d + c]) - yh[c];
                dist2 += e * e;
            }
            /* a/(pi Nhat) = exp(scale q.k - ln pi - ln Nhat) */
            const double wn = exp(scale * dot - log(pj) - lse[h]);
            out[b] += (1.0 - pj) * wn * wn * dist2;
        }
    }
    free(qd);
}

/* Deployed certificate (App. "Experimental details"): per sequence, the mean radius over the  */
/* sampled (unit, query head) pairs -- query head index head0[u] + g a multiple of head_stride */
/* -- folded into a running maximum over decode steps.  A sequence with no sampled pair keeps */
/* its maximum; mean_out gets 0 for it.                                                      */
void ebd_ref_certificate_step(int32_t U, int32_t G, int32_t S, int32_t head_stride,
                              const int32_t *unit_seq, const int32_t *unit_head0,
                              const float *radius, double *cert, double *mean_out)
{
    for (int32_t sq = 0; sq < S; ++sq) {
        double sum = 0.0;
        int64_t cnt = 0;
        for (int32_t u = 0; u < U; ++u) {
            if (unit_seq[u] != sq) continue;
            for (int32_t g = 0; g < G; ++g) {
                const int64_t hidx = (int64_t)(unit_head0 ? unit_head0[u] : 0) + g;
                if (hidx % head_stride != 0) continue;
                sum += (double)radius[(int64_t)u * G + g];
                cnt++;
            }
        }
        const double mean = cnt > 0 ? sum / (double)cnt : 0.0;
        if (mean_out) mean_out[sq] = mean;
        if (cnt > 0 && mean > cert[sq]) cert[sq] = mean;
    }
}

/* ------------------------------------------------------------------ */
/* Importance scores (App. "Experimental details", Harness): the       */
/* attention mass each key receives from a set of queries.  Query w     */
/* sees keys 0..qpos[w] (a prefill query at position qpos[w]), or every */
/* key when qpos is NULL (an observation window placed after the        */
/* cache).  score_i = sum_w softmax_w(scale q_w . k)_i over those keys. */
/* ------------------------------------------------------------------ */
void ebd_ref_window_scores(int64_t n, int32_t d, int32_t W, const uint16_t *K, const uint16_t *Q,
                           const int32_t *qpos, double scale, double *out)
{
    double *lg = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    double *qd = (double *)malloc((size_t)d * sizeof(double));
    for (int64_t i = 0; i < n; ++i) out[i] = 0.0;
    for (int32_t w = 0; w < W; ++w) {
        int64_t seen = n;
        if (qpos) {
            seen = (int64_t)qpos[w] + 1;
            if (seen > n) seen = n;
        }
        if (seen <= 0) continue;
        for (int32_t c = 0; c < d; ++c) qd[c] = ref_bf16(Q[(int64_t)w * d + c]);
        double M = -INFINITY;
        for (int64_t i = 0; i < seen; ++i) {
            double dot = 0.0;
            for (int32_t c = 0; c < d; ++c) dot += qd[c] * ref_bf16(K[i * d + c]);
            lg[i] = scale * dot;
            if (lg[i] > M) M = lg[i];
        }
        double Z = 0.0;
        for (int64_t i = 0; i < seen; ++i) Z += exp(lg[i] - M);
        for (int64_t i = 0; i < seen; ++i) out[i] += exp(lg[i] - M) / Z;
    }
    free(lg);
    free(qd);
}

/* ------------------------------------------------------------------ */
/* Batched drivers over independent units (one KV head cache each).   */
/* Units are independent, so they are split across threads.          */
/* ------------------------------------------------------------------ */

/*
 * Whole sampler for U units: pi (eq. (2)), Poisson mask, stable compaction.
 *   seq_off [U+1]: unit u owns full-cache rows seq_off[u] .. seq_off[u+1]-1.
 *   cap_off [U+1]: unit u owns compacted rows cap_off[u] .. cap_off[u+1]-1.
 *   budget_per_unit [U] (fractions) overrides budget_frac when non-NULL.
 *   seed_per_unit [U] overrides seed when non-NULL.
 *   pi_full [rows] (optional) receives the fp32 pi of every position.
 *   pi_given [rows] (optional): use these fp32 pi instead of solving (parity of
 *   the mask and compaction given the same pi).
 *   unit_ids [U] (optional): the unit word of each unit's Philox counter (default u), so that
 *   a sample of units drawn from a larger batch gets the same streams as in that batch.
 */
void ebd_ref_evict_batch(int32_t U, int32_t d, const int64_t *seq_off, const int64_t *cap_off,
                         const float *scores, const uint16_t *K, const uint16_t *V,
                         int32_t n_sink, int32_t n_recent, double budget_frac,
                         const float *budget_per_unit, double pi_min, uint64_t seed,
                         const uint64_t *seed_per_unit, uint32_t epoch, int32_t pi_mode,
                         int32_t design, const float *pi_given, const uint32_t *unit_ids,
                         uint16_t *Kc, uint16_t *Vc, float *pic, int32_t *idxc, int32_t *count,
                         double *lambda_out, float *pi_full, uint32_t *status, int32_t nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int32_t u = 0; u < U; ++u) {
        int64_t base = seq_off[u], n = seq_off[u + 1] - seq_off[u];
        int64_t cbase = cap_off[u], cap = cap_off[u + 1] - cap_off[u];
        double *pi64 = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
        float *pi32 = (float *)malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
        uint8_t *mask = (uint8_t *)malloc((size_t)(n > 0 ? n : 1));
        uint32_t st = 0;
        double lam = 0.0;
        if (pi_given) {
            memcpy(pi32, pi_given + base, (size_t)n * sizeof(float));
        } else {
            double f = budget_per_unit ? (double)budget_per_unit[u] : budget_frac;
            if (design == REF_DESIGN_TOPK) {
                st = ebd_ref_topk_probs(n, scores + base, n_sink, n_recent, f, pi64);
            } else if (design == REF_DESIGN_UNIFORM) {
                float *ones = (float *)malloc((size_t)(n > 0 ? n : 1) * sizeof(float));
                for (int64_t i = 0; i < n; ++i) ones[i] = 1.0f;
                st = ebd_ref_inclusion_probs(n, ones, n_sink, n_recent, f, pi_min, pi_mode, &lam,
                                             pi64);
                free(ones);
            } else {
                st = ebd_ref_inclusion_probs(n, scores + base, n_sink, n_recent, f, pi_min,
                                             pi_mode, &lam, pi64);
            }
            for (int64_t i = 0; i < n; ++i) pi32[i] = (float)pi64[i];
        }
        uint64_t sd = seed_per_unit ? seed_per_unit[u] : seed;
        uint32_t uid = unit_ids ? unit_ids[u] : (uint32_t)u;
        if (design == REF_DESIGN_SYSTEMATIC)
            ebd_ref_mask_systematic(n, pi32, sd, uid, epoch, mask);
        else
            ebd_ref_mask(n, pi32, sd, uid, epoch, mask);
        int64_t kept = ebd_ref_compact(n, d, mask, pi32, K + base * d, V + base * d, cap,
                                       Kc + cbase * d, Vc + cbase * d, pic + cbase, idxc + cbase);
        if (kept > cap) st |= REF_ST_CAP_OVERFLOW;
        count[u] = (int32_t)kept;
        if (lambda_out) lambda_out[u] = lam;
        if (pi_full) memcpy(pi_full + base, pi32, (size_t)n * sizeof(float));
        if (status) status[u] = st;
        free(pi64);
        free(pi32);
        free(mask);
    }
}

/* Certified decode attention for U units of G query heads (q [U, G, d]). */
void ebd_ref_attend_batch(int32_t U, int32_t G, int32_t d, const int64_t *cap_off,
                          const int32_t *count, const uint16_t *q, const uint16_t *Kc,
                          const uint16_t *Vc, const float *pic, double scale, double delta,
                          double eps0, int32_t use_offset, double *y, double *vhat, double *lse,
                          double *brange, double *radius, int32_t nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int32_t u = 0; u < U; ++u) {
        int64_t cbase = cap_off[u];
        int64_t cnt = count[u];
        int64_t cap = cap_off[u + 1] - cap_off[u];
        if (cnt > cap) cnt = cap;
        ebd_ref_attend_certify(G, d, cnt, q + (int64_t)u * G * d, Kc + cbase * d, Vc + cbase * d,
                               pic + cbase, scale, delta, eps0, use_offset,
                               y + (int64_t)u * G * d, vhat + (int64_t)u * G, lse + (int64_t)u * G,
                               brange ? brange + (int64_t)u * G : NULL,
                               radius ? radius + (int64_t)u * G : NULL);
    }
}

/* Full-cache outputs for U units (coverage reference). */
void ebd_ref_full_batch(int32_t U, int32_t G, int32_t d, const int64_t *seq_off, const uint16_t *q,
                        const uint16_t *K, const uint16_t *V, double scale, double *y, int32_t nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int32_t u = 0; u < U; ++u) {
        int64_t base = seq_off[u], n = seq_off[u + 1] - seq_off[u];
        ebd_ref_full_attention(G, d, n, q + (int64_t)u * G * d, K + base * d, V + base * d, scale,
                               y + (int64_t)u * G * d);
    }
}

/* Importance scores for U units: Q [U, W, d], qpos [U, W] or NULL, out [rows]. */
void ebd_ref_window_scores_batch(int32_t U, int32_t d, int32_t W, const int64_t *seq_off,
                                 const uint16_t *K, const uint16_t *Q, const int32_t *qpos,
                                 double scale, double *out, int32_t nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int32_t u = 0; u < U; ++u) {
        int64_t base = seq_off[u], n = seq_off[u + 1] - seq_off[u];
        ebd_ref_window_scores(n, d, W, K + base * d, Q + (int64_t)u * W * d,
                              qpos ? qpos + (int64_t)u * W : NULL, scale, out + base);
    }
}

int32_t ebd_ref_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
