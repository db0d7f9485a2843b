/*
 * ECOKV CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, double-precision implementation of the prefill-time KV-cache
 * eviction pass of "ECOKV: Geometry-Aware KV Cache Eviction via Complementary
 * Diversity Metrics" (arXiv 2609.06663):
 *   - importance from an observation window of the last w queries (Sec. 3;
 *     SnapKV baseline, Appendix A.1), averaged over the window (Sec. 5.2) and
 *     average-pooled with kernel 5 (Table 6);
 *   - composite diversity S_div = alpha s_E + (1 - alpha) s_C (Sec. 5.1,
 *     Eqs. (1)-(3); MixKV cosine term, Appendix A.1; Appendix C, Algorithm 1);
 *   - head-adaptive redundancy lambda = beta r_E + (1 - beta) r_C
 *     (Sec. 5.2, Eqs. (4)-(6));
 *   - rescaled diversity and final score S (Sec. 5.2, Eq. (7));
 *   - top-k over the non-window tokens plus the whole window (Sec. 3),
 *     per head or flattened across the heads of a layer (AdaKV, Appendix A.1);
 *   - the first sweep's key sums and window softmax statistics in the form a
 *     prefill can hand them over (ora_prefill_unit);
 *   - gather of the kept K/V rows;
 *   - decode attention of one new query per head over the kept rows (the
 *     generation step that reads the compressed cache, Sec. 3).
 *
 * Who may use it: the test-suite, the package smoke check and the benchmark's
 * CPU-baseline leg.  The HIP library never links, loads or calls this file and
 * the two share no source, header, table or helper.
 *
 * Readings of points the paper leaves open are marked "Reading:" below.
 * Parity unpinned: the sigmoid that maps the MAD-scaled deviation to s_E
 * (ECOKV_NORM_MAD, an alternative of Sec. 6.3); the paper gives no formula
 * or value for it, so it rests on that reading alone.
 * Inputs are the exact bytes the GPU consumes (bf16 bit patterns or fp32),
 * decoded exactly to double; everything is accumulated in double with plain
 * loops, in the order the paper states the steps.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORA_BF16 = 0, ORA_F32 = 1 };
enum { ORA_PER_HEAD = 0, ORA_LAYER_FLAT = 1, ORA_HEAD_BUDGETS = 2 };

/* Per-head statistics written by ora_score_unit (indices into stats[ORA_NSTATS]). */
enum {
    ORA_LAMBDA = 0,    /* lambda, Eq. (6) (or the override)                    */
    ORA_RC = 1,        /* cosine redundancy r_C (Appendix A.1, MixKV)          */
    ORA_RE = 2,        /* Euclidean redundancy r_E, Eq. (5)                    */
    ORA_DE = 3,        /* mean distance D_E, Eq. (4)                           */
    ORA_DMIN = 4,      /* min of d_E over the non-window tokens                */
    ORA_DMAX = 5,      /* max of d_E over the non-window tokens                */
    ORA_SDMIN = 6,     /* min of S_div                                         */
    ORA_SDMAX = 7,     /* max of S_div                                         */
    ORA_IMPMEAN = 8,   /* mean of S_imp over the non-window tokens             */
    ORA_SBARMEAN = 9,  /* mean of the min-max normalised S_div                 */
    ORA_MUNORM2 = 10,  /* |mu|^2                                               */
    ORA_SCALE = 11,    /* mean(S_imp) / (mean(S_bar) + eps)                    */
    ORA_NSTATS = 12
};

typedef struct {
    double alpha;            /* Euclidean weight in S_div, Eq. (3); 0.8 (Table 6)  */
    double beta;             /* Euclidean weight in lambda, Eq. (6); 0.6 (Table 6) */
    double eps;              /* stabiliser of the min-max / mean ratios           */
    double tau;              /* temperature of Eq. (5); <= 0 means sqrt(D)        */
    int pool_kernel;         /* average-pool width (odd), 5 in Table 6            */
    int causal;              /* window query j sees keys <= P + j                 */
    double lambda_override;  /* NaN: use Eq. (6); else use this value (tests)     */
    int imp_mode;            /* 0: S_imp = pooled attention; 1: times |v_i|_2     */
    int norm_mode;           /* s_E: 0 min-max (Eq. (2)), 1 winsorised, 2 MAD     */
    double winsor_q;         /* winsorised min-max: clip at quantiles q, 1 - q    */
    double mad_tau;          /* MAD scaling temperature                           */
    int redundancy;          /* 0: r_E (Eq. (5)); 1: r_std (Appendix D)           */
    int centroid_scope;      /* 0: kbar over all T keys; 1: over the P non-window */
} ora_params;

/* Optional per-unit intermediates (any pointer may be NULL). */
typedef struct {
    double *a;       /* [P] window-mean attention, before pooling     */
    double *imp;     /* [P] pooled importance S_imp                   */
    double *dE;      /* [T] distance of each key to the centroid      */
    double *cosmu;   /* [P] normalised key . mu                       */
    double *sC;      /* [P] cosine diversity                          */
    double *sE;      /* [P] Euclidean diversity, Eq. (2)              */
    double *sdiv;    /* [P] composite diversity, Eq. (3)              */
    double *sbar;    /* [P] min-max normalised S_div                  */
    double *stilde;  /* [P] rescaled diversity                        */
    double *kbar;    /* [D] centroid                                  */
    double *mu;      /* [D] mean of the normalised keys               */
    double *rowmass; /* [G*w] softmax mass of each window row         */
} ora_trace;

static int ora_dbl_cmp(const void *x, const void *y)
{
    const double a = *(const double *)x, b = *(const double *)y;
    return a < b ? -1 : (a > b ? 1 : 0);
}

/* The q quantile of x[0..n) (n >= 1) by linear interpolation between the order
 * statistics at ranks floor(h) and floor(h) + 1, h = q (n - 1) (the usual
 * definition, as numpy's default).  Sorts a copy. */
static double ora_quantile(const double *x, int n, double q)
{
    double *c = malloc((size_t)n * sizeof(double));
    if (!c) return NAN;
    memcpy(c, x, (size_t)n * sizeof(double));
    qsort(c, (size_t)n, sizeof(double), ora_dbl_cmp);
    const double h = q * (double)(n - 1);
    const int j = (int)floor(h);
    const double r = j + 1 < n ? c[j] + (h - j) * (c[j + 1] - c[j]) : c[j];
    free(c);
    return r;
}

static double ora_get(const void *base, int dtype, size_t i)
{
    if (dtype == ORA_BF16) {
        uint32_t u = (uint32_t)((const uint16_t *)base)[i] << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return (double)((const float *)base)[i];
}

/*
 * Score one (layer, KV head, sequence) unit.
 *   K: T x D rows of this unit (element type dtype).
 *   V: T x D value rows of this unit; read only when p->imp_mode == 1.
 *   Q: the window queries of the G query heads mapped to this KV head; query
 *      head g, window row j is at Q + (g * q_gstride + j * D) elements.
 *   S: [P] output scores, P = T - w.   stats: [ORA_NSTATS] output.
 * Returns 0, or -1 on invalid sizes.
 */
int ora_score_unit_v(const void *K, const void *V, const void *Q, size_t q_gstride, int dtype,
                     int T, int D, int G, int w, const ora_params *p,
                     double *S, double *stats, const ora_trace *tr)
{
    if (T < 2 || w < 1 || w >= T || D < 1 || G < 1 || p->pool_kernel < 1 || (p->pool_kernel % 2) == 0)
        return -1;
    if (p->imp_mode != 0 && (p->imp_mode != 1 || !V)) return -1;
    if (p->norm_mode < 0 || p->norm_mode > 2 || p->redundancy < 0 || p->redundancy > 1 ||
        p->centroid_scope < 0 || p->centroid_scope > 1)
        return -1;
    const int P = T - w;
    const double inv_sqrt_d = 1.0 / sqrt((double)D);

    double *a = calloc((size_t)P, sizeof(double));
    double *imp = calloc((size_t)P, sizeof(double));
    double *logit = malloc((size_t)T * sizeof(double));
    double *kbar = calloc((size_t)D, sizeof(double));
    double *mu = calloc((size_t)D, sizeof(double));
    double *dE = malloc((size_t)T * sizeof(double));
    double *cosmu = malloc((size_t)P * sizeof(double));
    double *sdiv = malloc((size_t)P * sizeof(double));
    double *sE = malloc((size_t)P * sizeof(double));
    double *sC = malloc((size_t)P * sizeof(double));
    if (!a || !imp || !logit || !kbar || !mu || !dE || !cosmu || !sdiv || !sE || !sC) {
        free(a); free(imp); free(logit); free(kbar); free(mu); free(dE);
        free(cosmu); free(sdiv); free(sE); free(sC);
        return -2;
    }

    /* Steps 1-2. Observation-window importance (Sec. 3; Appendix A.1, SnapKV).
     * Each window query attends to the keys with softmax(q k^T / sqrt(d_k))
     * (Sec. 3 attention); the attention each non-window key receives is
     * averaged over the window rows (Sec. 5.2: "average attention score").
     * Reading: causal window (row j sees keys 0..P+j); the G query heads that
     * share this KV head are averaged together with the window rows. */
    for (int g = 0; g < G; ++g) {
        for (int j = 0; j < w; ++j) {
            const size_t qoff = (size_t)g * q_gstride + (size_t)j * D;
            const int last = p->causal ? P + j : T - 1;
            double m = -INFINITY;
            for (int i = 0; i <= last; ++i) {
                double dot = 0.0;
                for (int d = 0; d < D; ++d)
                    dot += ora_get(Q, dtype, qoff + d) * ora_get(K, dtype, (size_t)i * D + d);
                logit[i] = dot * inv_sqrt_d;
                if (logit[i] > m) m = logit[i];
            }
            double z = 0.0;
            for (int i = 0; i <= last; ++i) z += exp(logit[i] - m);
            double mass = 0.0;
            for (int i = 0; i <= last; ++i) {
                const double att = exp(logit[i] - m) / z;
                mass += att;
                if (i < P) a[i] += att;
            }
            if (tr && tr->rowmass) tr->rowmass[g * w + j] = mass;
        }
    }
    for (int i = 0; i < P; ++i) a[i] /= (double)(G * w);

    /* Step 3. 1-D average pooling of the importance (Table 6: kernel 5,
     * average pool).  Reading: zero padding of half the kernel on both sides
     * and a fixed divisor equal to the kernel width. */
    const int half = p->pool_kernel / 2;
    for (int i = 0; i < P; ++i) {
        double acc = 0.0;
        for (int t = -half; t <= half; ++t)
            if (i + t >= 0 && i + t < P) acc += a[i + t];
        imp[i] = acc / (double)p->pool_kernel;
    }

    /* Step 3'. Value-norm importance (imp_mode 1): the importance combines the
     * l2 norm of the value vector with the window-mean attention (Sec. 5.2;
     * VNorm, Sec. 2).  Reading: the product of the pooled attention and
     * |v_i|_2; the norm is not pooled. */
    if (p->imp_mode == 1) {
        for (int i = 0; i < P; ++i) {
            double n2 = 0.0;
            for (int d = 0; d < D; ++d) {
                const double v = ora_get(V, dtype, (size_t)i * D + d);
                n2 += v * v;
            }
            imp[i] *= sqrt(n2);
        }
    }

    /* Step 4. Anchors over all T keys: the centroid kbar (Eq. (1)) and the mean
     * of the normalised keys mu (Appendix A.1, MixKV; Algorithm 1, cosine
     * branch).  Reading: a zero key normalises to zero (norm floored at 1e-12). */
    for (int i = 0; i < T; ++i) {
        double n2 = 0.0;
        for (int d = 0; d < D; ++d) {
            const double v = ora_get(K, dtype, (size_t)i * D + d);
            n2 += v * v;
            kbar[d] += v;
        }
        const double nrm = fmax(sqrt(n2), 1e-12);
        for (int d = 0; d < D; ++d) mu[d] += ora_get(K, dtype, (size_t)i * D + d) / nrm;
    }
    for (int d = 0; d < D; ++d) {
        kbar[d] /= (double)T;
        mu[d] /= (double)T;
    }
    /* Alternative (Appendix B.6): the centroid over the non-window keys only;
     * mu keeps all T keys (the alternative concerns the Euclidean step). */
    if (p->centroid_scope == 1) {
        for (int d = 0; d < D; ++d) {
            kbar[d] = 0.0;
            for (int i = 0; i < P; ++i) kbar[d] += ora_get(K, dtype, (size_t)i * D + d);
            kbar[d] /= (double)P;
        }
    }

    /* Step 5. Cosine diversity of each non-window key (Appendix A.1, MixKV:
     * negative similarity to mu).  Reading: mapped to [0, 1] as (1 - khat.mu)/2,
     * so that a larger value means a more diverse key. */
    for (int i = 0; i < P; ++i) {
        double n2 = 0.0, dot = 0.0;
        for (int d = 0; d < D; ++d) {
            const double v = ora_get(K, dtype, (size_t)i * D + d);
            n2 += v * v;
            dot += v * mu[d];
        }
        cosmu[i] = dot / fmax(sqrt(n2), 1e-12);
        sC[i] = (1.0 - cosmu[i]) / 2.0;
    }

    /* Step 6. Cosine redundancy: the mean off-diagonal pairwise cosine,
     * r_C = (T |mu|^2 - 1) / (T - 1) (Appendix A.1, MixKV; Algorithm 1). */
    double mu2 = 0.0;
    for (int d = 0; d < D; ++d) mu2 += mu[d] * mu[d];
    const double rC = ((double)T * mu2 - 1.0) / ((double)T - 1.0);

    /* Step 7. Euclidean distance of every key to the centroid, Eq. (1), taken as
     * a direct difference; min-max normalised over the non-window keys, Eq. (2). */
    for (int i = 0; i < T; ++i) {
        double s2 = 0.0;
        for (int d = 0; d < D; ++d) {
            const double diff = ora_get(K, dtype, (size_t)i * D + d) - kbar[d];
            s2 += diff * diff;
        }
        dE[i] = sqrt(s2);
    }
    double dmin = dE[0], dmax = dE[0];
    for (int i = 1; i < P; ++i) {
        if (dE[i] < dmin) dmin = dE[i];
        if (dE[i] > dmax) dmax = dE[i];
    }
    if (p->norm_mode == 0) {
        for (int i = 0; i < P; ++i) sE[i] = (dE[i] - dmin) / (dmax - dmin + p->eps);
    } else if (p->norm_mode == 1) {
        /* Winsorised min-max (Sec. 6.3, Table 4): d_E clipped to its q and
         * 1 - q quantiles over the non-window keys, then min-max between them. */
        const double lo = ora_quantile(dE, P, p->winsor_q), hi = ora_quantile(dE, P, 1.0 - p->winsor_q);
        for (int i = 0; i < P; ++i) {
            const double c = dE[i] < lo ? lo : (dE[i] > hi ? hi : dE[i]);
            sE[i] = (c - lo) / (hi - lo + p->eps);
        }
    } else {
        /* Per-head MAD scaling (Sec. 6.3, Table 4), temperature mad_tau.
         * Reading: the deviation from the median in units of the median
         * absolute deviation, mapped to (0, 1) by a sigmoid so that it blends
         * with s_C as the min-max value does.  Parity unpinned: the paper
         * names the method but not the mapping, so no pin can fix the sigmoid
         * (the median and MAD themselves are pinned to numpy). */
        const double med = ora_quantile(dE, P, 0.5);
        for (int i = 0; i < P; ++i) sE[i] = fabs(dE[i] - med);  /* the deviations, then s_E */
        const double mad = ora_quantile(sE, P, 0.5);
        for (int i = 0; i < P; ++i) sE[i] = 1.0 / (1.0 + exp(-(dE[i] - med) / (p->mad_tau * mad + p->eps)));
    }

    /* Step 8. Mean distance over all T keys, Eq. (4), and the magnitude-aware
     * redundancy r_E = 2 - 2 sigmoid(D_E / tau), Eq. (5), tau = sqrt(d_k). */
    double DE = 0.0;
    for (int i = 0; i < T; ++i) DE += dE[i];
    DE /= (double)T;
    const double tau = p->tau > 0.0 ? p->tau : sqrt((double)D);
    double rE = 2.0 - 2.0 / (1.0 + exp(-DE / tau));
    if (p->redundancy == 1) {
        /* Alternative (Appendix D): the standard deviation of the keys,
         * D_std = sqrt(mean_T |k_i - kbar|^2), and r_std = 1 - sigmoid(D_std / tau)
         * in place of r_E. */
        double ss = 0.0;
        for (int i = 0; i < T; ++i) ss += dE[i] * dE[i];
        const double Dstd = sqrt(ss / (double)T);
        rE = 1.0 - 1.0 / (1.0 + exp(-Dstd / tau));
    }

    /* Step 9. Head-adaptive weight, Eq. (6). */
    double lambda = p->beta * rE + (1.0 - p->beta) * rC;
    if (!isnan(p->lambda_override)) lambda = p->lambda_override;

    /* Step 10. Composite diversity, Eq. (3); min-max normalisation and the
     * rescale to the magnitude of the importance (Sec. 5.2).  Reading: the
     * denominator mean is that of the normalised composite diversity, and
     * eps guards both ratios. */
    double smin = 0.0, smax = 0.0;
    for (int i = 0; i < P; ++i) {
        sdiv[i] = p->alpha * sE[i] + (1.0 - p->alpha) * sC[i];
        if (i == 0 || sdiv[i] < smin) smin = sdiv[i];
        if (i == 0 || sdiv[i] > smax) smax = sdiv[i];
    }
    double imp_mean = 0.0, sbar_mean = 0.0;
    for (int i = 0; i < P; ++i) imp_mean += imp[i];
    imp_mean /= (double)P;
    for (int i = 0; i < P; ++i) sbar_mean += (sdiv[i] - smin) / (smax - smin + p->eps);
    sbar_mean /= (double)P;
    const double scale = imp_mean / (sbar_mean + p->eps);

    /* Step 11. Final score, Eq. (7). */
    for (int i = 0; i < P; ++i) {
        const double sbar = (sdiv[i] - smin) / (smax - smin + p->eps);
        const double stilde = sbar * scale;
        S[i] = lambda * stilde + (1.0 - lambda) * imp[i];
        if (tr) {
            if (tr->sbar) tr->sbar[i] = sbar;
            if (tr->stilde) tr->stilde[i] = stilde;
        }
    }

    if (stats) {
        stats[ORA_LAMBDA] = lambda;
        stats[ORA_RC] = rC;
        stats[ORA_RE] = rE;
        stats[ORA_DE] = DE;
        stats[ORA_DMIN] = dmin;
        stats[ORA_DMAX] = dmax;
        stats[ORA_SDMIN] = smin;
        stats[ORA_SDMAX] = smax;
        stats[ORA_IMPMEAN] = imp_mean;
        stats[ORA_SBARMEAN] = sbar_mean;
        stats[ORA_MUNORM2] = mu2;
        stats[ORA_SCALE] = scale;
    }
    if (tr) {
        if (tr->a) memcpy(tr->a, a, (size_t)P * sizeof(double));
        if (tr->imp) memcpy(tr->imp, imp, (size_t)P * sizeof(double));
        if (tr->dE) memcpy(tr->dE, dE, (size_t)T * sizeof(double));
        if (tr->cosmu) memcpy(tr->cosmu, cosmu, (size_t)P * sizeof(double));
        if (tr->sC) memcpy(tr->sC, sC, (size_t)P * sizeof(double));
        if (tr->sE) memcpy(tr->sE, sE, (size_t)P * sizeof(double));
        if (tr->sdiv) memcpy(tr->sdiv, sdiv, (size_t)P * sizeof(double));
        if (tr->kbar) memcpy(tr->kbar, kbar, (size_t)D * sizeof(double));
        if (tr->mu) memcpy(tr->mu, mu, (size_t)D * sizeof(double));
    }
    free(a); free(imp); free(logit); free(kbar); free(mu); free(dE);
    free(cosmu); free(sdiv); free(sE); free(sC);
    return 0;
}

int ora_score_unit(const void *K, const void *Q, size_t q_gstride, int dtype,
                   int T, int D, int G, int w, const ora_params *p,
                   double *S, double *stats, const ora_trace *tr)
{
    return ora_score_unit_v(K, NULL, Q, q_gstride, dtype, T, D, G, w, p, S, stats, tr);
}

/* ---------------------------------------------------------------------------
 * Selection (Sec. 3): the k = b - w highest-scoring non-window tokens plus the
 * whole window.  Reading: equal scores rank the smaller position first; the
 * output lists the chosen positions in ascending order followed by the window;
 * a budget b >= T keeps every token.  NaN scores rank below every number.
 * ------------------------------------------------------------------------- */
typedef struct {
    double s;
    int64_t key; /* flattened (head, position) order used to break ties */
} ora_item;

static int ora_rank_cmp(const void *x, const void *y)
{
    const ora_item *a = x, *b = y;
    const int na = isnan(a->s), nb = isnan(b->s);
    if (na != nb) return na ? 1 : -1;
    if (!na && a->s != b->s) return a->s > b->s ? -1 : 1;
    return a->key < b->key ? -1 : (a->key > b->key ? 1 : 0);
}

static int ora_int_cmp(const void *x, const void *y)
{
    const int32_t a = *(const int32_t *)x, b = *(const int32_t *)y;
    return a < b ? -1 : (a > b ? 1 : 0);
}

/* Per-head selection for one unit; writes min(b, T) positions, returns that count. */
int ora_select_unit(const double *S, int T, int w, int b, int32_t *idx)
{
    if (w < 1 || w >= T || b < w) return -1;
    if (b >= T) {
        for (int i = 0; i < T; ++i) idx[i] = i;
        return T;
    }
    const int P = T - w, k = b - w;
    ora_item *it = malloc((size_t)P * sizeof(ora_item));
    if (!it) return -2;
    for (int i = 0; i < P; ++i) {
        it[i].s = S[i];
        it[i].key = i;
    }
    qsort(it, (size_t)P, sizeof(ora_item), ora_rank_cmp);
    for (int r = 0; r < k; ++r) idx[r] = (int32_t)it[r].key;
    qsort(idx, (size_t)k, sizeof(int32_t), ora_int_cmp);
    for (int j = 0; j < w; ++j) idx[k + j] = P + j;
    free(it);
    return b;
}

/* Layer-flat selection (AdaKV budget sharing, Appendix A.1): the scores of the
 * H heads of one (layer, sequence) compete for H * (b - w) places; ties rank
 * the smaller (head, position) first; every head keeps its window.  Head h's
 * scores are at S + h * hstride.  Output: head-major, each head's chosen
 * positions ascending then its window; counts[h] = entries of head h.
 * Returns the total (H * min(b, T)). */
int ora_select_flat(const double *S, size_t hstride, int H, int T, int w, int b,
                    int32_t *idx, int32_t *counts)
{
    if (w < 1 || w >= T || b < w || H < 1) return -1;
    if (b >= T) {
        for (int h = 0; h < H; ++h) {
            for (int i = 0; i < T; ++i) idx[(size_t)h * T + i] = i;
            counts[h] = T;
        }
        return H * T;
    }
    const int P = T - w;
    const int64_t ktot = (int64_t)H * (b - w);
    const int64_t n = (int64_t)H * P;
    ora_item *it = malloc((size_t)n * sizeof(ora_item));
    uint8_t *chosen = calloc((size_t)n, 1);
    if (!it || !chosen) {
        free(it); free(chosen);
        return -2;
    }
    for (int h = 0; h < H; ++h)
        for (int i = 0; i < P; ++i) {
            it[(int64_t)h * P + i].s = S[(size_t)h * hstride + i];
            it[(int64_t)h * P + i].key = (int64_t)h * P + i;
        }
    qsort(it, (size_t)n, sizeof(ora_item), ora_rank_cmp);
    for (int64_t r = 0; r < ktot; ++r) chosen[it[r].key] = 1;
    int64_t o = 0;
    for (int h = 0; h < H; ++h) {
        const int64_t start = o;
        for (int i = 0; i < P; ++i)
            if (chosen[(int64_t)h * P + i]) idx[o++] = i;
        for (int j = 0; j < w; ++j) idx[o++] = P + j;
        counts[h] = (int32_t)(o - start);
    }
    free(it);
    free(chosen);
    return (int)o;
}

/* ---------------------------------------------------------------------------
 * Whole-tensor drivers (layouts as the HIP library's, written independently):
 *   K, V   [L][Hkv][Ttot][D]   rows of sequence s at cu[s] .. cu[s+1]-1
 *   Q      [L][Hq][B][w][D]    query head q belongs to KV head q / (Hq/Hkv)
 *   S      [L][Hkv][Ptot]      Ptot = Ttot - B*w; sequence s at cu[s] - s*w
 *   stats  [L][Hkv][B][ORA_NSTATS]
 * ------------------------------------------------------------------------- */
int ora_score_v(const void *K, const void *V, const void *Q, int dtype, int L, int Hq, int Hkv, int B,
                const int32_t *cu, int D, int w, const ora_params *p,
                double *S, double *stats, int nthreads)
{
    if (L < 0 || Hkv < 1 || Hq % Hkv != 0 || B < 1) return -1;
    const int G = Hq / Hkv;
    const int64_t Ttot = cu[B];
    const int64_t Ptot = Ttot - (int64_t)B * w;
    const size_t es = dtype == ORA_BF16 ? 2 : 4;
    const int64_t U = (int64_t)L * Hkv * B;
    int bad = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) reduction(|| : bad)
#endif
    for (int64_t u = 0; u < U; ++u) {
        const int s = (int)(u % B);
        const int h = (int)((u / B) % Hkv);
        const int l = (int)(u / ((int64_t)B * Hkv));
        const int T = cu[s + 1] - cu[s];
        const size_t krow = ((size_t)l * Hkv + h) * (size_t)Ttot + (size_t)cu[s];
        const char *Ku = (const char *)K + krow * (size_t)D * es;
        const char *Vu = V ? (const char *)V + krow * (size_t)D * es : NULL;
        const char *Qu = (const char *)Q + ((((size_t)l * Hq + (size_t)h * G) * B + s) * (size_t)w * D) * es;
        double *Su = S + ((size_t)l * Hkv + h) * (size_t)Ptot + (size_t)(cu[s] - s * w);
        double *st = stats ? stats + (size_t)u * ORA_NSTATS : NULL;
        if (ora_score_unit_v(Ku, Vu, Qu, (size_t)B * w * D, dtype, T, D, G, w, p, Su, st, NULL) != 0) bad = 1;
    }
    (void)nthreads;
    return bad ? -1 : 0;
}

int ora_score(const void *K, const void *Q, int dtype, int L, int Hq, int Hkv, int B,
              const int32_t *cu, int D, int w, const ora_params *p,
              double *S, double *stats, int nthreads)
{
    return ora_score_v(K, NULL, Q, dtype, L, Hq, Hkv, B, cu, D, w, p, S, stats, nthreads);
}

/* ---------------------------------------------------------------------------
 * The first sweep's results for one unit, in the form a prefill hands them
 * to the pass (what the KV-cache write and the window rows of the prefill's
 * attention can produce as it runs), pre[2D + 2R]:
 *   [0, D)          sum over the T keys of k_i (the centroid of Eq. (1)
 *                   before its division by T);
 *   [D, 2D)         sum over the T keys of k_i / |k_i| (the mean normalised
 *                   key mu of the cosine term, Appendix A.1, before its
 *                   division by T; a zero key counts as zero, as above);
 *   [2D + r]        for window row r = g w + j (query head g of the group,
 *                   window position j): the largest q.k / sqrt(D) over the
 *                   keys that row sees (Sec. 3 attention; keys 0 .. P + j
 *                   when causal, all T otherwise);
 *   [2D + R + r]    the sum over those keys of exp(q.k / sqrt(D) - largest).
 * Returns 0, or -1 on invalid sizes.
 * ------------------------------------------------------------------------- */
int ora_prefill_unit(const void *K, const void *Q, size_t q_gstride, int dtype, int T, int D, int G, int w,
                     int causal, double *pre)
{
    if (T < 2 || w < 1 || w >= T || D < 1 || G < 1) return -1;
    const int R = G * w, P = T - w;
    const double inv_sqrt_d = 1.0 / sqrt((double)D);
    for (int c = 0; c < 2 * D + 2 * R; ++c) pre[c] = 0.0;
    for (int i = 0; i < T; ++i) {
        double n2 = 0.0;
        for (int d = 0; d < D; ++d) {
            const double x = ora_get(K, dtype, (size_t)i * D + d);
            n2 += x * x;
        }
        const double nrm = fmax(sqrt(n2), 1e-12);
        for (int d = 0; d < D; ++d) {
            const double x = ora_get(K, dtype, (size_t)i * D + d);
            pre[d] += x;
            pre[D + d] += x / nrm;
        }
    }
    double *lg = malloc((size_t)T * sizeof(double));
    if (!lg) return -2;
    for (int g = 0; g < G; ++g) {
        for (int j = 0; j < w; ++j) {
            const size_t qoff = (size_t)g * q_gstride + (size_t)j * D;
            const int seen = causal ? P + j : T - 1;  /* last key the row sees */
            double m = -INFINITY;
            for (int i = 0; i <= seen; ++i) {
                double dot = 0.0;
                for (int d = 0; d < D; ++d) dot += ora_get(Q, dtype, qoff + d) * ora_get(K, dtype, (size_t)i * D + d);
                lg[i] = dot * inv_sqrt_d;
                m = fmax(m, lg[i]);
            }
            double z = 0.0;
            for (int i = 0; i <= seen; ++i) z += exp(lg[i] - m);
            pre[2 * D + g * w + j] = m;
            pre[2 * D + R + g * w + j] = z;
        }
    }
    free(lg);
    return 0;
}

/* ora_prefill_unit over every unit; K, Q laid out as for ora_score_v,
 * pre [L][Hkv][B][2D + 2R]. */
int ora_prefill_sums(const void *K, const void *Q, int dtype, int L, int Hq, int Hkv, int B, const int32_t *cu,
                     int D, int w, int causal, double *pre, int nthreads)
{
    if (L < 0 || Hkv < 1 || Hq % Hkv != 0 || B < 1) return -1;
    const int G = Hq / Hkv;
    const int64_t Ttot = cu[B];
    const size_t es = dtype == ORA_BF16 ? 2 : 4;
    const size_t width = (size_t)2 * D + (size_t)2 * G * w;
    const int64_t U = (int64_t)L * Hkv * B;
    int bad = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) reduction(|| : bad)
#endif
    for (int64_t u = 0; u < U; ++u) {
        const int s = (int)(u % B);
        const int h = (int)((u / B) % Hkv);
        const int l = (int)(u / ((int64_t)B * Hkv));
        const int T = cu[s + 1] - cu[s];
        const size_t krow = ((size_t)l * Hkv + h) * (size_t)Ttot + (size_t)cu[s];
        const char *Ku = (const char *)K + krow * (size_t)D * es;
        const char *Qu = (const char *)Q + ((((size_t)l * Hq + (size_t)h * G) * B + s) * (size_t)w * D) * es;
        if (ora_prefill_unit(Ku, Qu, (size_t)B * w * D, dtype, T, D, G, w, causal, pre + (size_t)u * width) != 0)
            bad = 1;
    }
    (void)nthreads;
    return bad ? -1 : 0;
}

/* idx layout: PER_HEAD -- unit (l, h, s) owns min(b_s, T_s) entries, units in
 * (l, h, s) order.  LAYER_FLAT -- group (l, s) owns Hkv * min(b_s, T_s)
 * entries, groups in (l, s) order, heads in order inside a group.
 * HEAD_BUDGETS -- budget is [L][Hkv] (a budget per layer and head, as the
 * PyramidKV layer schedule and the SparseMM head budgets of Appendix A.1
 * assign them): unit (l, h, s) owns min(b[l][h], T_s) entries, units in
 * (l, h, s) order.  counts and offsets ([L][Hkv][B]) give each unit's entry
 * count and start. */
int ora_select(const double *S, int L, int Hkv, int B, const int32_t *cu, int w,
               const int32_t *budget, int mode, int32_t *idx, int32_t *counts,
               int32_t *offsets, int nthreads)
{
    const int64_t Ttot = cu[B];
    const int64_t Ptot = Ttot - (int64_t)B * w;
    int bad = 0;
    if (mode == ORA_HEAD_BUDGETS) {
        for (int s = 0; s < B; ++s)
            if (w >= cu[s + 1] - cu[s]) return -1;
        for (int64_t lh = 0; lh < (int64_t)L * Hkv; ++lh)
            if (budget[lh] < w) return -1;
        const int64_t U = (int64_t)L * Hkv * B;
        int64_t *start = malloc((size_t)(U > 0 ? U : 1) * sizeof(int64_t));
        if (!start) return -2;
        int64_t o = 0;
        for (int64_t u = 0; u < U; ++u) {
            const int s = (int)(u % B);
            const int T = cu[s + 1] - cu[s];
            const int32_t b = budget[u / B];
            start[u] = o;
            o += b < T ? b : T;
        }
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) reduction(|| : bad)
#endif
        for (int64_t u = 0; u < U; ++u) {
            const int s = (int)(u % B);
            const int64_t lh = u / B;
            const int T = cu[s + 1] - cu[s];
            const int n = ora_select_unit(S + lh * Ptot + (cu[s] - s * w), T, w, budget[lh], idx + start[u]);
            if (n < 0) bad = 1;
            if (counts) counts[u] = n;
            if (offsets) offsets[u] = (int32_t)start[u];
        }
        free(start);
        (void)nthreads;
        return bad ? -1 : 0;
    }
    int64_t per_layer_head = 0; /* sum over s of min(b_s, T_s) */
    for (int s = 0; s < B; ++s) {
        const int T = cu[s + 1] - cu[s];
        if (budget[s] < w || w >= T) return -1;
        per_layer_head += budget[s] < T ? budget[s] : T;
    }
    if (mode == ORA_PER_HEAD) {
        const int64_t U = (int64_t)L * Hkv * B;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) reduction(|| : bad)
#endif
        for (int64_t u = 0; u < U; ++u) {
            const int s = (int)(u % B);
            const int64_t lh = u / B;
            int64_t off = lh * per_layer_head;
            for (int t = 0; t < s; ++t) {
                const int Tt = cu[t + 1] - cu[t];
                off += budget[t] < Tt ? budget[t] : Tt;
            }
            const int T = cu[s + 1] - cu[s];
            const int n = ora_select_unit(S + lh * Ptot + (cu[s] - s * w), T, w, budget[s], idx + off);
            if (n < 0) bad = 1;
            if (counts) counts[u] = n;
            if (offsets) offsets[u] = (int32_t)off;
        }
    } else if (mode == ORA_LAYER_FLAT) {
        const int64_t NG = (int64_t)L * B;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1) reduction(|| : bad)
#endif
        for (int64_t gi = 0; gi < NG; ++gi) {
            const int l = (int)(gi / B), s = (int)(gi % B);
            int64_t off = (int64_t)l * Hkv * per_layer_head;
            for (int t = 0; t < s; ++t) {
                const int Tt = cu[t + 1] - cu[t];
                off += (int64_t)Hkv * (budget[t] < Tt ? budget[t] : Tt);
            }
            const int T = cu[s + 1] - cu[s];
            int32_t cnt[1024];
            if (Hkv > 1024) { bad = 1; continue; }
            const int n = ora_select_flat(S + (size_t)l * Hkv * Ptot + (cu[s] - s * w), (size_t)Ptot,
                                          Hkv, T, w, budget[s], idx + off, cnt);
            if (n < 0) { bad = 1; continue; }
            int64_t o = off;
            for (int h = 0; h < Hkv; ++h) {
                const int64_t u = ((int64_t)l * Hkv + h) * B + s;
                if (counts) counts[u] = cnt[h];
                if (offsets) offsets[u] = (int32_t)o;
                o += cnt[h];
            }
        }
    } else {
        return -1;
    }
    (void)nthreads;
    return bad ? -1 : 0;
}

/* Gather of the kept rows: Kc[offsets[u] + j] = K[unit u row idx[offsets[u] + j]]. */
int ora_compact(const void *K, const void *V, int esize, int L, int Hkv, int B,
                const int32_t *cu, int D, const int32_t *idx, const int32_t *counts,
                const int32_t *offsets, void *Kc, void *Vc)
{
    const int64_t Ttot = cu[B];
    const size_t row = (size_t)D * (size_t)esize;
    for (int l = 0; l < L; ++l)
        for (int h = 0; h < Hkv; ++h)
            for (int s = 0; s < B; ++s) {
                const int64_t u = ((int64_t)l * Hkv + h) * B + s;
                const size_t base = ((size_t)l * Hkv + h) * (size_t)Ttot + (size_t)cu[s];
                const int T = cu[s + 1] - cu[s];
                for (int j = 0; j < counts[u]; ++j) {
                    const int32_t i = idx[offsets[u] + j];
                    if (i < 0 || i >= T) return -1;
                    memcpy((char *)Kc + ((size_t)offsets[u] + j) * row, (const char *)K + (base + i) * row, row);
                    memcpy((char *)Vc + ((size_t)offsets[u] + j) * row, (const char *)V + (base + i) * row, row);
                }
            }
    return 0;
}

/* Decode attention over the compressed cache (Sec. 3: generation attends to
 * the kept rows).  For layer l, query head q (KV head h = q / G) and sequence
 * s, unit u = (l, h, s) owns the n = counts[u] rows offsets[u] .. of Kc / Vc:
 *   x_j = q . Kc[j] / sqrt(D),  O = sum_j softmax(x)_j Vc[j],
 *   lse = log sum_j exp(x_j)  (max-subtracted).
 * Q [L][Hq][B][D] (dtype), O [L][Hq][B][D], lse [L][Hq][B].  A unit with no
 * rows gives O = 0 and lse = -inf. */
int ora_decode(const void *Q, const void *Kc, const void *Vc, int dtype, int L, int Hq, int Hkv, int B, int D,
               const int32_t *counts, const int32_t *offsets, double *O, double *lse)
{
    if (L < 0 || Hkv < 1 || Hq % Hkv != 0 || B < 1 || D < 1) return -1;
    const int G = Hq / Hkv;
    const double inv_sqrt_d = 1.0 / sqrt((double)D);
    for (int l = 0; l < L; ++l)
        for (int q = 0; q < Hq; ++q)
            for (int s = 0; s < B; ++s) {
                const int h = q / G;
                const int64_t u = ((int64_t)l * Hkv + h) * B + s;
                const int64_t r = ((int64_t)l * Hq + q) * B + s;
                const int n = counts[u];
                double *o = O + (size_t)r * D;
                for (int d = 0; d < D; ++d) o[d] = 0.0;
                if (n <= 0) {
                    lse[r] = -INFINITY;
                    continue;
                }
                double *x = malloc((size_t)n * sizeof(double));
                if (!x) return -2;
                double m = -INFINITY;
                for (int j = 0; j < n; ++j) {
                    double dot = 0.0;
                    for (int d = 0; d < D; ++d)
                        dot += ora_get(Q, dtype, (size_t)r * D + d) *
                               ora_get(Kc, dtype, ((size_t)offsets[u] + j) * D + d);
                    x[j] = dot * inv_sqrt_d;
                    if (x[j] > m) m = x[j];
                }
                double z = 0.0;
                for (int j = 0; j < n; ++j) z += exp(x[j] - m);
                for (int j = 0; j < n; ++j) {
                    const double pj = exp(x[j] - m) / z;
                    for (int d = 0; d < D; ++d) o[d] += pj * ora_get(Vc, dtype, ((size_t)offsets[u] + j) * D + d);
                }
                lse[r] = m + log(z);
                free(x);
            }
    return 0;
}
