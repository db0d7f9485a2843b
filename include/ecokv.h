/*
 * ecokv.h -- C ABI of libecokv.so, the gfx950 (MI355X) implementation of the
 * prefill-time KV-cache eviction pass of ECOKV ("Geometry-Aware KV Cache
 * Eviction via Complementary Diversity Metrics", arXiv 2609.06663).
 *
 * The pass, for every (layer, KV head, sequence) "unit":
 *   ecokv_score   importance of each non-window key from the observation window
 *                 (Sec. 3; SnapKV, Appendix A.1; mean over the window, Sec. 5.2;
 *                 average pool, Table 6), composite diversity (Sec. 5.1,
 *                 Eqs. (1)-(3)), head redundancy weight lambda (Sec. 5.2,
 *                 Eqs. (4)-(6)) and the final score S (Sec. 5.2, Eq. (7)).
 *   ecokv_select  top-k of S over the non-window keys plus the whole window
 *                 (Sec. 3), per head or shared across the heads of a layer
 *                 (AdaKV budget sharing, Appendix A.1).
 *   ecokv_compact gather of the kept K/V rows into the compressed cache
 *                 (Sec. 3, selected subset).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers unless stated; the caller
 *    allocates and owns every buffer (inputs, outputs, workspace).  The library
 *    never allocates or frees device memory and never synchronises outside
 *    ecokv_stage_times() and ecokv_workspace_status().  Its only process-wide
 *    state is per-device caches of the number of blocks of the split
 *    epilogues the device holds at once and the optional stage timer; calls
 *    on different streams with different workspaces may run concurrently,
 *    and a call captured in a HIP graph may be replayed.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    Work is enqueued asynchronously; results are valid once the stream has
 *    been synchronised.
 *  - Return value: ECOKV_OK, or a negative error code.  Every argument check
 *    runs on the host before anything is enqueued, so an error leaves every
 *    output untouched.  ecokv_last_error() describes the last failure of the
 *    calling thread.  Device faults surface at the caller's next synchronise.
 *  - Layouts are row-major and contiguous:
 *      K, V   [L][H_kv][Ttot][D]   sequence s of a (varlen) batch occupies
 *                                  rows cu_seqlens[s] .. cu_seqlens[s+1]-1
 *      Q_win  [L][H_q][B][w][D]    the last w query rows of every query head;
 *                                  query head q belongs to KV head q / (H_q/H_kv)
 *      scores [L][H_kv][Ptot]      Ptot = Ttot - B*w; sequence s starts at
 *                                  cu_seqlens[s] - s*w (non-window keys only)
 *      per-unit arrays [L][H_kv][B] (unit u = (l*H_kv + h)*B + s)
 *  - Positions stored in idx are relative to the start of their sequence.
 */
#ifndef ECOKV_H
#define ECOKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ECOKV_OK 0
#define ECOKV_EINVAL (-1)       /* bad shape, parameter or NULL pointer          */
#define ECOKV_EWORKSPACE (-2)   /* workspace smaller than ecokv_workspace_size   */
#define ECOKV_EUNSUPPORTED (-3) /* valid request the library does not implement  */
#define ECOKV_EHIP (-4)         /* the HIP runtime refused a launch              */
#define ECOKV_ETIMEOUT (-5)     /* a bounded wait between blocks gave up (see    */
                                /* ecokv_workspace_status)                        */

#define ECOKV_BF16 0 /* bfloat16 elements (2 bytes) */
#define ECOKV_F32 1  /* float32 elements  (4 bytes) */

#define ECOKV_PER_HEAD 0   /* each unit keeps exactly min(b_s, T_s) tokens    */
#define ECOKV_LAYER_FLAT 1 /* the H_kv heads of (layer, sequence) share       */
                           /* H_kv*min(b_s, T_s) places (AdaKV, App. A.1)     */
#define ECOKV_HEAD_BUDGETS 2 /* head h of layer l keeps min(b^l_h, T_s) tokens */
                             /* per sequence: a caller-chosen budget for each */
                             /* (layer, KV head), as PyramidKV's layer        */
                             /* schedule and SparseMM's head budgets assign   */
                             /* them (App. A.1)                               */

#define ECOKV_IMP_ATTN 0       /* S_imp: pooled window-mean attention (SnapKV)   */
#define ECOKV_IMP_ATTN_VNORM 1 /* S_imp: that times |v_i|_2 (Sec. 5.2; VNorm)    */

/* Normalisation of d_E into s_E (the Eq. (2) step; Sec. 6.3, Table 4). */
#define ECOKV_NORM_MINMAX 0  /* (d - min) / (max - min + eps), Eq. (2)           */
#define ECOKV_NORM_WINSOR 1  /* d clipped to its q and 1-q quantiles, then       */
                             /* min-max between them                            */
#define ECOKV_NORM_MAD 2     /* sigmoid((d - median) / (mad_tau * MAD + eps))    */

/* Redundancy in lambda (Eq. (6)). */
#define ECOKV_RED_EUCLID 0   /* r_E = 2 - 2 sigmoid(D_E / tau), Eq. (5)          */
#define ECOKV_RED_STD 1      /* r_std = 1 - sigmoid(D_std / tau), Appendix D     */

/* Keys averaged into the centroid kbar (Eq. (1)). */
#define ECOKV_CENTROID_ALL 0    /* all T keys                                   */
#define ECOKV_CENTROID_PREFIX 1 /* the P non-window keys (Appendix B.6)         */

#define ECOKV_MAX_SEQS 64   /* sequences per call                              */
#define ECOKV_MAX_ROWS 64   /* window rows per KV head, (H_q/H_kv)*w           */

/* Per-unit statistics written by ecokv_score when `stats` is non-NULL. */
#define ECOKV_STAT_LAMBDA 0    /* lambda = beta r_E + (1-beta) r_C, Eq. (6)      */
#define ECOKV_STAT_RC 1        /* cosine redundancy (T|mu|^2-1)/(T-1), App. A.1  */
#define ECOKV_STAT_RE 2        /* the redundancy in lambda: r_E, Eq. (5), or r_std */
#define ECOKV_STAT_DE 3        /* mean distance to the centroid, Eq. (4)         */
#define ECOKV_STAT_DMIN 4      /* min / max of d_E over the non-window keys      */
#define ECOKV_STAT_DMAX 5
#define ECOKV_STAT_SDIV_MIN 6  /* min / max of S_div, Eq. (3)                    */
#define ECOKV_STAT_SDIV_MAX 7
#define ECOKV_STAT_IMP_MEAN 8  /* mean of the pooled importance S_imp            */
#define ECOKV_STAT_SBAR_MEAN 9 /* mean of the min-max normalised S_div           */
#define ECOKV_STAT_MU_NORM2 10 /* |mu|^2                                         */
#define ECOKV_STAT_SCALE 11    /* mean(S_imp) / (mean(S_bar) + eps)              */
#define ECOKV_NSTATS 12

/* Shape of one call.  cu_seqlens is a HOST array of num_seqs+1 nondecreasing
 * offsets with cu_seqlens[0] = 0; a fixed-length batch of one sequence of T
 * tokens is {0, T}.  Every sequence needs 1 <= window < T_s. */
typedef struct ecokv_shape {
    int32_t num_layers;         /* L >= 0 (0: nothing to do)                     */
    int32_t num_q_heads;        /* H_q, a multiple of H_kv                       */
    int32_t num_kv_heads;       /* H_kv >= 1                                     */
    int32_t head_dim;           /* D: 64 or 128                                  */
    int32_t window;             /* w >= 1, the observation window (Sec. 5.3)     */
    int32_t num_seqs;           /* B in [1, ECOKV_MAX_SEQS]                      */
    const int32_t *cu_seqlens;  /* host, [B+1]                                   */
} ecokv_shape;

/* Hyper-parameters (Table 6 defaults via ecokv_default_params). */
typedef struct ecokv_params {
    float alpha;            /* Euclidean weight of S_div, Eq. (3); 0.8            */
    float beta;             /* Euclidean weight of lambda, Eq. (6); 0.6           */
    float eps;              /* guard of the min-max and mean ratios; 1e-6         */
    float tau;              /* temperature of Eq. (5); <= 0 selects sqrt(D)       */
    int32_t pool_kernel;    /* odd average-pool width for S_imp; 5                */
    int32_t causal;         /* 1: window row j sees keys <= T-w+j; 0: all keys    */
    float lambda_override;  /* NaN: lambda from Eq. (6); else this fixed value    */
    int32_t imp_mode;       /* ECOKV_IMP_ATTN or ECOKV_IMP_ATTN_VNORM             */
    int32_t norm_mode;      /* ECOKV_NORM_MINMAX / _WINSOR / _MAD                 */
    float winsor_q;         /* ECOKV_NORM_WINSOR: lower quantile q in [0, 0.5)    */
    float mad_tau;          /* ECOKV_NORM_MAD: temperature (> 0); 1               */
    int32_t redundancy;     /* ECOKV_RED_EUCLID or ECOKV_RED_STD                  */
    int32_t centroid_scope; /* ECOKV_CENTROID_ALL or ECOKV_CENTROID_PREFIX        */
} ecokv_params;

/* Fills *p with the paper's defaults: alpha 0.8, beta 0.6, eps 1e-6,
 * tau sqrt(D), pool 5, causal, no override, ECOKV_IMP_ATTN, min-max
 * normalisation (winsor_q 0.01 and mad_tau 1 for the alternatives), r_E, the
 * centroid over all T keys.  Returns ECOKV_OK.
 * Quantiles (ECOKV_NORM_WINSOR, ECOKV_NORM_MAD) are taken over the P
 * non-window keys of a unit, interpolating linearly between the two nearest
 * order statistics at rank q (P - 1); the median is the 0.5 quantile and MAD
 * the median of |d_E - median|.  D_std = sqrt(mean over the T keys of
 * |k - kbar|^2).  With ECOKV_CENTROID_PREFIX only kbar changes (mu, D_E and
 * D_std still average over all T keys). */
int ecokv_default_params(ecokv_params *p);

/* Bytes of device workspace ecokv_score / ecokv_score_v need for this shape
 * and these parameters (select and compact need none; ECOKV_IMP_ATTN_VNORM
 * adds one float per non-window key).  The workspace is scratch, except for
 * its first 4 bytes, a status word (see ecokv_workspace_status) that must be
 * zero before the workspace's first use: allocate it zero-filled, or call
 * ecokv_workspace_status once; the next 4 bytes count the calls made on it
 * (any initial value will do).  It must not be shared by calls that may
 * overlap. */
int ecokv_workspace_size(const ecokv_shape *shape, const ecokv_params *params, size_t *bytes);

/* Status of the score calls enqueued on `workspace` since the last query.
 * The only failure a score call can meet after its launch is a bounded wait
 * between two blocks of its final step that gives up (see ecokv_score); it
 * then writes NaN lambda and scores for the units concerned and sets the
 * workspace's status word.  This query synchronises `stream` (which must be
 * the stream of those calls, or ordered after them), reads the word, clears
 * it and returns ECOKV_ETIMEOUT if it was set, else ECOKV_OK. */
int ecokv_workspace_status(void *workspace, void *stream);

/* Score every unit (Sec. 3 and Sec. 5, Eqs. (1)-(7)).
 *   K      [L][H_kv][Ttot][D]  keys, element type `dtype`
 *   Q_win  [L][H_q][B][w][D]   window queries, element type `dtype`
 *   scores [L][H_kv][Ptot]     float32 output S for the non-window keys
 *   lambda [L][H_kv][B]        float32 output, may be NULL
 *   stats  [L][H_kv][B][ECOKV_NSTATS] float32 output, may be NULL
 *   workspace, workspace_bytes: device scratch of ecokv_workspace_size bytes,
 *   256-byte aligned.
 * Arithmetic: fp32 accumulation of bf16/fp32 inputs.
 * For sequences of at most 65536 + w tokens the final step runs as groups
 * of 2 to 8 blocks per (layer, KV head, sequence) that exchange sums once and
 * wait for each other, when the device can hold all of them at once (no
 * waits when a unit has at most 4096 non-window keys, nor when the device
 * cannot hold the groups: one block per unit then, or two launches past 32768
 * keys); if one ever
 * waits for another for seconds (the device taken by other work all that
 * time), that unit's lambda and scores come out NaN and the workspace's status
 * word records it: check with ecokv_workspace_status.  (The environment
 * variable ECOKV_SPIN_LIMIT, read at each call, sets how many times such a
 * wait polls before it gives up; values <= 0 give up at once.  It exists for
 * tests.)
 * params->imp_mode must be ECOKV_IMP_ATTN here (the value norm needs V:
 * ecokv_score_v). */
int ecokv_score(const void *K, const void *Q_win, int dtype, const ecokv_shape *shape,
                const ecokv_params *params, float *scores, float *lambda, float *stats,
                void *workspace, size_t workspace_bytes, void *stream);

/* ecokv_score with the values V [L][H_kv][Ttot][D] (element type `dtype`).
 * With params->imp_mode == ECOKV_IMP_ATTN_VNORM the importance of key i < P
 * combines the l2 norm of its value vector with the window-mean attention
 * (Sec. 5.2; VNorm, Sec. 2) as the product S_imp(i) = pool(a)(i) * |v_i|_2
 * (the pooled attention times the norm; the norm is not pooled); V is read
 * once, in one extra pass over the non-window rows.  With ECOKV_IMP_ATTN, V
 * is not read and may be NULL. */
int ecokv_score_v(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                  const ecokv_params *params, float *scores, float *lambda, float *stats,
                  void *workspace, size_t workspace_bytes, void *stream);

/* ecokv_score_v with the results of the first sweep over K supplied by the
 * caller, so that K is read only once.  A prefill that runs flash attention
 * over the window queries has each window row's softmax max and sum as a
 * by-product of its epilogue, and the pass that writes K into the cache can
 * accumulate the two key sums; passing them here skips the first sweep
 * (Sec. 3 window attention; Eq. (1) centroid; Appendix A.1 mu).
 *   pre  DEVICE [L][H_kv][B][2D + 2R] float32, per unit u:
 *          [0, D)          sum over its T keys of k_i
 *          [D, 2D)         sum over its T keys of k_i / max(|k_i|, 1e-12)
 *          [2D, 2D+R)      per window row r = g w + j (query head g of the
 *                          group, window row j): a reference m_r, and
 *          [2D+R, 2D+2R)   z_r, the sum over its visible keys of
 *                          exp(q.k / sqrt(D) - m_r)
 *        (visible: keys <= T - w + j when causal, all T otherwise).  Only
 *        m_r + log(z_r), the row's log-sum-exp, is used: m_r is usually the
 *        row's largest logit, and a prefill's flash attention can pass its
 *        log-sum-exp output as m_r with z_r = 1.
 * Everything else as ecokv_score_v; the two-sweep path's second sweep and
 * epilogue run as usual.  pre == NULL is ecokv_score_v. */
int ecokv_score_pre(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                    const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
                    void *workspace, size_t workspace_bytes, void *stream);

/* ecokv_score_pre for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid it): no
 * workspace argument.  Its scratch is a 96 MiB device array that the library
 * holds on every device it runs on until the process ends, shared by all
 * calls on that device: calls that may overlap on one device race.  A call
 * whose scratch (ecokv_workspace_size for its shape) would exceed 96 MiB is
 * refused with ECOKV_EWORKSPACE before anything is enqueued (the 28-layer,
 * 4-KV-head, 32768-token stack needs 77 MiB).  The final step runs one block
 * per (layer, KV head, sequence), so no block waits for another and there is
 * no status to query.  The current device must be the stream's device.  No
 * allocation, no memset, no synchronisation. */
int ecokv_score_noalloc(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                        const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
                        void *stream);

/* The KV-cache write of a prefill with the first sweep over K as its
 * by-product (Sec. 3 window attention; Eq. (1) centroid; Appendix A.1 mu), so
 * that the pass reads K once (ecokv_score_pre).  It copies the new K and V
 * rows from the token-major layout a projection writes into the head-major
 * layout the pass reads, and while K streams through it accumulates the two
 * key sums and runs the window rows' online softmax over the keys:
 *   K_new, V_new      DEVICE [L][T_total][H_kv][D] dtype (token-major: row
 *                     cu[s] + t holds token t of sequence s for every KV head)
 *   Q_win             DEVICE as for ecokv_score
 *   params            only params->causal is read (which keys a window row sees)
 *   K_cache, V_cache  DEVICE [L][H_kv][T_total][D] dtype, the K and V layout of
 *                     ecokv_score; written, every row
 *   pre               DEVICE [L][H_kv][B][2D + 2R] float32, written in the
 *                     layout ecokv_score_pre reads; the reference m_r of a
 *                     window row is at most its largest logit and within
 *                     16 ln 2 of it (the sweep moves it lazily)
 *   workspace         DEVICE, >= ecokv_prefill_workspace_size bytes, 256-byte
 *                     aligned; no initial contents needed
 * V_new and V_cache are both NULL (keys only) or both non-NULL.  The four row
 * buffers must be 16-byte aligned and the new rows must not overlap the
 * cache.  Errors: ECOKV_EINVAL for NULL, misaligned or overlapping buffers,
 * ECOKV_EWORKSPACE for a short workspace, ECOKV_EUNSUPPORTED as ecokv_score;
 * nothing is enqueued then.  No allocation, no synchronisation. */
int ecokv_prefill_write(const void *K_new, const void *V_new, const void *Q_win, int dtype, const ecokv_shape *shape,
                        const ecokv_params *params, void *K_cache, void *V_cache, float *pre, void *workspace,
                        size_t workspace_bytes, void *stream);

/* Workspace bytes of ecokv_prefill_write for this shape (either element type). */
int ecokv_prefill_workspace_size(const ecokv_shape *shape, size_t *bytes);

/* Number of int32 entries ecokv_select writes to idx:
 * L * H_kv * sum_s min(budget[s], T_s) (ECOKV_PER_HEAD and ECOKV_LAYER_FLAT). */
int ecokv_index_count(const ecokv_shape *shape, const int32_t *budget, int64_t *count);

/* The same for any mode: `budget` is laid out as ecokv_select takes it in
 * that mode ([B], or [L][H_kv] for ECOKV_HEAD_BUDGETS, where the count is
 * sum over (l, h, s) of min(budget[l][h], T_s)). */
int ecokv_index_count_mode(const ecokv_shape *shape, int mode, const int32_t *budget, int64_t *count);

/* Bytes of device workspace ecokv_select needs for this shape and mode (the
 * budgets do not change it).  Like the score workspace it must be zero-filled
 * before its first use; ecokv_select leaves it zero-filled, so one workspace
 * serves any number of calls of this or a smaller shape, one at a time. */
int ecokv_select_workspace_size(const ecokv_shape *shape, int mode, size_t *bytes);

/* Select the kept positions (Sec. 3; AdaKV, PyramidKV and SparseMM budgets,
 * Appendix A.1).
 *   scores  [L][H_kv][Ptot] float32, as written by ecokv_score
 *   budget  HOST [B]: b_s = tokens kept per head for sequence s, window
 *           included, b_s >= w.  b_s >= T_s keeps every token.
 *           ECOKV_HEAD_BUDGETS: HOST [L][H_kv] instead, b^l_h = tokens kept
 *           by head h of layer l in every sequence (window included, >= w,
 *           >= T_s keeps every token).
 *   mode    ECOKV_PER_HEAD: unit (l,h,s) keeps the b_s - w highest scores
 *           (equal scores: smaller position first), listed ascending, then the
 *           window T_s-w .. T_s-1.  Units are laid out in (l, h, s) order.
 *           ECOKV_LAYER_FLAT: the H_kv heads of (l, s) compete for
 *           H_kv*(b_s - w) places (equal scores: smaller (head, position)
 *           first); each head lists its chosen positions ascending, then its
 *           window.  Groups are laid out in (l, s) order, heads in order.
 *           ECOKV_HEAD_BUDGETS: as ECOKV_PER_HEAD with unit (l,h,s) keeping
 *           min(b^l_h, T_s) tokens; units in (l, h, s) order.
 *   idx     output, ecokv_index_count entries
 *   counts  [L][H_kv][B] output: entries of each unit (may be NULL, except in
 *           LAYER_FLAT)
 *   offsets [L][H_kv][B] output: start of each unit in idx (may be NULL,
 *           except in LAYER_FLAT)
 *   workspace, workspace_bytes: device scratch of at least
 *           ecokv_select_workspace_size bytes, 256-byte aligned, zero-filled
 *           before its first use (left so); not shared by calls that may
 *           overlap.  A selection group (a unit, or the heads of a (layer,
 *           sequence) in LAYER_FLAT) of more than 32768 keys is split over
 *           many blocks: its radix-select histograms and per-slice counts
 *           live there, or, for single-head groups whose budget is small,
 *           each 8192-key slice's own largest keys and their positions.
 * NaN scores rank below every number; -0 ranks equal to +0.
 * ECOKV_EUNSUPPORTED: LAYER_FLAT with more than 256 KV heads, or with
 * H_kv * Ptot * 4 > 2^31 - 1 bytes of scores per layer; a sequence with
 * (T_s - w) * 4 > 2^31 - 1 bytes of scores. */
int ecokv_select(const float *scores, const ecokv_shape *shape, int mode, const int32_t *budget,
                 int32_t *idx, int32_t *counts, int32_t *offsets, void *workspace, size_t workspace_bytes,
                 void *stream);

/* Gather Kc[e] = K[row of entry e], Vc[e] = V[row of entry e] for every idx
 * entry e, bit-exact (Sec. 3).  `mode` and `budget` as given to ecokv_select;
 * counts and offsets are required for ECOKV_LAYER_FLAT (device arrays written
 * by ecokv_select) and ignored for ECOKV_PER_HEAD and ECOKV_HEAD_BUDGETS.
 * Kc, Vc have ecokv_index_count_mode rows of D elements. */
int ecokv_compact(const void *K, const void *V, int dtype, const ecokv_shape *shape, int mode,
                  const int32_t *budget, const int32_t *idx, const int32_t *counts,
                  const int32_t *offsets, void *Kc, void *Vc, void *stream);

/* Workspace bytes of ecokv_decode for this shape and max_count (>= 1). */
int ecokv_decode_workspace_size(const ecokv_shape *shape, int32_t max_count, size_t *bytes);

/* Decode attention over the compressed cache: the generation step that reads
 * the kept rows (Sec. 3).  For layer l, query head q (KV head h = q / G, G =
 * H_q / H_kv) and sequence s, unit u = (l, h, s) owns rows offsets[u] ..
 * offsets[u] + counts[u] - 1 of Kc / Vc, and
 *   O[l][q][s] = sum_j softmax_j(Q_dec[l][q][s] . Kc[j] / sqrt(D)) Vc[j],
 *   lse[l][q][s] = log sum_j exp(Q_dec[l][q][s] . Kc[j] / sqrt(D)).
 *   Q_dec   [L][H_q][B][D]  one new query per head and sequence (dtype)
 *   Kc, Vc  [entries][D]    as written by ecokv_compact (dtype)
 *   counts, offsets  DEVICE [L][H_kv][B], as written by ecokv_select (any mode)
 *   max_count  an upper bound of every counts[u] (e.g. the largest budget);
 *           the work is split into chunks of rows up to it.  A unit with more
 *           rows gets NaN outputs.
 *   O       [L][H_q][B][D] float32 output;  lse [L][H_q][B] float32, may be NULL
 *   workspace of ecokv_decode_workspace_size bytes, 256-byte aligned.
 * Q_dec, Kc and Vc must be 16-byte aligned.  Arithmetic: fp32 accumulation;
 * the softmax is computed online per row chunk and the chunks are merged by
 * their log-sum-exp. */
int ecokv_decode(const void *Q_dec, const void *Kc, const void *Vc, int dtype, const ecokv_shape *shape,
                 const int32_t *counts, const int32_t *offsets, int32_t max_count, float *O, float *lse,
                 void *workspace, size_t workspace_bytes, void *stream);

/* PyramidKV's layer schedule (Appendix A.1), host only: for m = num_layers
 * layers sharing `total` tokens per head, the last layer gets
 * b^{m-1} = total / (beta m), the first b^0 = 2 total / m - b^{m-1}, and the
 * layers between follow the straight line b^l = b^0 - (b^0 - b^{m-1}) l / (m-1)
 * (one layer: b^0 = total).  Each value is rounded down, so the sum is at most
 * `total`.  out: HOST [num_layers].  ECOKV_EINVAL if num_layers < 1, total or
 * beta is not a positive finite number, or a value would fall below
 * `window` (>= 1) or exceed INT32_MAX.  To give every KV head of a layer its
 * layer's budget, repeat each value H_kv times for ECOKV_HEAD_BUDGETS. */
int ecokv_pyramid_budgets(int num_layers, double total, double beta, int window, int32_t *out);

/* Message for the calling thread's last failed call ("" if none). */
const char *ecokv_last_error(void);

/*
 * Optional per-kernel timing, for benchmarks.  While the environment variable
 * ECOKV_STAGE_TIMING is set to 1 at the time of a call, ecokv_score,
 * ecokv_select and ecokv_compact bracket every kernel they launch with HIP
 * events on the call's stream (which adds a little launch overhead).
 * ecokv_stage_times() waits for the recorded events, writes up to `max`
 * entries (one per kernel name, in order of first launch) to `out` and their
 * number to `*count`, and clears the record.  Host arrays; returns ECOKV_OK or
 * ECOKV_EINVAL / ECOKV_EHIP.
 */
typedef struct {
    char name[48];    /* kernel name                                      */
    double ms;        /* summed duration of its launches, milliseconds     */
    int64_t launches; /* number of launches                               */
} ecokv_stage_time;

int ecokv_stage_times(ecokv_stage_time *out, int max, int *count);

#ifdef __cplusplus
}
#endif
#endif /* ECOKV_H */
