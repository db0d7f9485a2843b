// C entry points of libecokv: host-side argument checks, workspace layout and
// launches.  Every check completes before anything is enqueued.
#include <math.h>
#include <stdlib.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "ecokv_internal.h"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

struct ShapeInfo {
    int L, Hq, Hkv, G, D, w, B, R;
    int64_t Ttot, Ptot;
    int maxT, maxP;
};

int check_shape(const ecokv_shape *sh, ShapeInfo *o)
{
    if (!sh) return fail(ECOKV_EINVAL, "shape is NULL");
    if (sh->num_layers < 0) return fail(ECOKV_EINVAL, "num_layers %d < 0", sh->num_layers);
    if (sh->num_kv_heads < 1) return fail(ECOKV_EINVAL, "num_kv_heads %d < 1", sh->num_kv_heads);
    if (sh->num_q_heads < sh->num_kv_heads || sh->num_q_heads % sh->num_kv_heads != 0)
        return fail(ECOKV_EINVAL, "num_q_heads %d is not a positive multiple of num_kv_heads %d", sh->num_q_heads,
                    sh->num_kv_heads);
    if (sh->head_dim != 64 && sh->head_dim != 128)
        return fail(ECOKV_EUNSUPPORTED, "head_dim %d (supported: 64, 128)", sh->head_dim);
    if (sh->window < 1) return fail(ECOKV_EINVAL, "window %d < 1", sh->window);
    if (sh->num_seqs < 1 || sh->num_seqs > ECOKV_MAX_SEQS)
        return fail(ECOKV_EINVAL, "num_seqs %d outside [1, %d]", sh->num_seqs, ECOKV_MAX_SEQS);
    if (!sh->cu_seqlens) return fail(ECOKV_EINVAL, "cu_seqlens is NULL");
    if (sh->cu_seqlens[0] != 0) return fail(ECOKV_EINVAL, "cu_seqlens[0] = %d, must be 0", sh->cu_seqlens[0]);
    o->maxT = 0;
    for (int s = 0; s < sh->num_seqs; ++s) {
        const int64_t T = (int64_t)sh->cu_seqlens[s + 1] - sh->cu_seqlens[s];
        if (T <= sh->window)
            return fail(ECOKV_EINVAL, "sequence %d has %lld tokens; the window %d must be shorter", s, (long long)T,
                        sh->window);
        if (T > o->maxT) o->maxT = (int)T;
    }
    o->L = sh->num_layers;
    o->Hq = sh->num_q_heads;
    o->Hkv = sh->num_kv_heads;
    o->G = o->Hq / o->Hkv;
    o->D = sh->head_dim;
    o->w = sh->window;
    o->B = sh->num_seqs;
    o->R = o->G * o->w;
    o->Ttot = sh->cu_seqlens[o->B];
    o->Ptot = o->Ttot - (int64_t)o->B * o->w;
    o->maxP = o->maxT - o->w;
    if ((int64_t)o->L * o->Hkv * o->B > (int64_t)INT32_MAX / 8)
        return fail(ECOKV_EINVAL, "too many (layer, head, sequence) units");
    return ECOKV_OK;
}

int check_params(const ecokv_params *p)
{
    if (!p) return fail(ECOKV_EINVAL, "params is NULL");
    if (!(isfinite(p->alpha) && isfinite(p->beta) && isfinite(p->eps) && isfinite(p->tau)))
        return fail(ECOKV_EINVAL, "alpha, beta, eps and tau must be finite");
    if (p->eps < 0.f) return fail(ECOKV_EINVAL, "eps %g < 0", (double)p->eps);
    if (p->pool_kernel < 1 || p->pool_kernel % 2 == 0)
        return fail(ECOKV_EINVAL, "pool_kernel %d must be odd and >= 1", p->pool_kernel);
    if (p->causal != 0 && p->causal != 1) return fail(ECOKV_EINVAL, "causal must be 0 or 1");
    if (isinf(p->lambda_override)) return fail(ECOKV_EINVAL, "lambda_override must be NaN or finite");
    if (p->imp_mode != ECOKV_IMP_ATTN && p->imp_mode != ECOKV_IMP_ATTN_VNORM)
        return fail(ECOKV_EINVAL, "imp_mode %d", p->imp_mode);
    if (p->norm_mode < ECOKV_NORM_MINMAX || p->norm_mode > ECOKV_NORM_MAD)
        return fail(ECOKV_EINVAL, "norm_mode %d", p->norm_mode);
    if (!(p->winsor_q >= 0.f && p->winsor_q < 0.5f))
        return fail(ECOKV_EINVAL, "winsor_q %g outside [0, 0.5)", (double)p->winsor_q);
    if (!(isfinite(p->mad_tau) && p->mad_tau > 0.f)) return fail(ECOKV_EINVAL, "mad_tau %g", (double)p->mad_tau);
    if (p->redundancy != ECOKV_RED_EUCLID && p->redundancy != ECOKV_RED_STD)
        return fail(ECOKV_EINVAL, "redundancy %d", p->redundancy);
    if (p->centroid_scope != ECOKV_CENTROID_ALL && p->centroid_scope != ECOKV_CENTROID_PREFIX)
        return fail(ECOKV_EINVAL, "centroid_scope %d", p->centroid_scope);
    return ECOKV_OK;
}

int fill_seqtab(const ecokv_shape *sh, const int32_t *budget, int w, ecokv::SeqTab *t, int64_t *per_lh)
{
    memset(t, 0, sizeof *t);
    t->nseq = sh->num_seqs;
    for (int s = 0; s <= sh->num_seqs; ++s) t->cu[s] = sh->cu_seqlens[s];
    int64_t acc = 0;
    t->boff[0] = 0;
    for (int s = 0; s < sh->num_seqs; ++s) {
        const int T = sh->cu_seqlens[s + 1] - sh->cu_seqlens[s];
        int b = T;
        if (budget) {
            if (budget[s] < w)
                return fail(ECOKV_EINVAL, "budget[%d] = %d is below the window %d", s, budget[s], w);
            b = budget[s] < T ? budget[s] : T;
        }
        t->beff[s] = b;
        acc += b;
        if (acc > INT32_MAX) return fail(ECOKV_EINVAL, "budget sum overflows");
        t->boff[s + 1] = (int)acc;
    }
    if (per_lh) *per_lh = acc;
    return ECOKV_OK;
}

// Per-(layer, KV head) budgets (ECOKV_HEAD_BUDGETS): checks every budget and
// counts the idx entries, sum over (l, h, s) of min(b^l_h, T_s).
int head_budget_total(const ecokv_shape *sh, const ShapeInfo &si, const int32_t *budget, int64_t *total)
{
    const int64_t n = (int64_t)si.L * si.Hkv;
    int64_t acc = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (budget[j] < si.w)
            return fail(ECOKV_EINVAL, "budget[%lld] = %d is below the window %d", (long long)j, budget[j], si.w);
        for (int s = 0; s < si.B; ++s) {
            const int T = sh->cu_seqlens[s + 1] - sh->cu_seqlens[s];
            acc += budget[j] < T ? budget[j] : T;
        }
        if (acc > INT32_MAX) return fail(ECOKV_EINVAL, "index count overflows int32");
    }
    *total = acc;
    return ECOKV_OK;
}

// The table of pairs lh0 .. lh0+n-1 (n <= kLhChunk) whose entries start at
// idx offset e0; returns the offset just past them.
int64_t fill_lhtab(const ecokv_shape *sh, int B, const int32_t *budget, int64_t lh0, int n, int64_t e0,
                   ecokv::LhTab *t)
{
    t->lh0 = (int)lh0;
    t->n = n;
    int64_t e = e0;
    for (int j = 0; j < n; ++j) {
        const int b = budget[lh0 + j];
        t->b[j] = b;
        t->start[j] = (int)e;
        for (int s = 0; s < B; ++s) {
            const int T = sh->cu_seqlens[s + 1] - sh->cu_seqlens[s];
            e += b < T ? b : T;
        }
    }
    t->start[n] = (int)e;
    return e;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(ECOKV_EHIP, "%s: %s", what, hipGetErrorString(e));
}

struct StageRec {
    const char *name;
    hipEvent_t start, stop;
};
std::mutex g_stage_mu;
std::vector<StageRec> g_stages;
thread_local const char *g_stage_name = nullptr;
thread_local hipEvent_t g_stage_start = nullptr;

// Groups of the largest select launch and keys of the largest group, which
// size the select workspace.
void select_dims(const ShapeInfo &si, const ecokv_shape *sh, int mode, int64_t *groups, int64_t *maxn)
{
    const int64_t pairs = (int64_t)si.L * si.Hkv;
    *groups = mode == ECOKV_HEAD_BUDGETS ? (pairs < ecokv::kLhChunk ? pairs : ecokv::kLhChunk) * si.B
              : mode == ECOKV_LAYER_FLAT ? (int64_t)si.L * si.B
                                         : pairs * si.B;
    *maxn = (int64_t)si.maxP * (mode == ECOKV_LAYER_FLAT ? si.Hkv : 1);
    (void)sh;
}

int check_select_mode(const ShapeInfo &si, int mode)
{
    if (mode != ECOKV_PER_HEAD && mode != ECOKV_LAYER_FLAT && mode != ECOKV_HEAD_BUDGETS)
        return fail(ECOKV_EINVAL, "mode %d", mode);
    if (mode == ECOKV_LAYER_FLAT) {
        if (si.Hkv > ecokv::select_max_flat_heads())
            return fail(ECOKV_EUNSUPPORTED, "LAYER_FLAT supports at most %d KV heads", ecokv::select_max_flat_heads());
        // (a selection group's scores are read through one 32-bit-addressed buffer descriptor)
        if ((int64_t)si.Hkv * si.Ptot * 4 > INT32_MAX)
            return fail(ECOKV_EUNSUPPORTED, "LAYER_FLAT: H_kv x P_total scores of a layer exceed 2^31 bytes");
    }
    if ((int64_t)si.maxP * 4 > INT32_MAX)
        return fail(ECOKV_EUNSUPPORTED, "a sequence's scores exceed 2^31 bytes");
    return ECOKV_OK;
}

// Checks the caller's select workspace and points the launch at it.
int select_workspace(const ShapeInfo &si, const ecokv_shape *shape, int mode, void *workspace, size_t workspace_bytes,
                     ecokv::SelectArgs *a)
{
    int64_t groups = 0, maxn = 0;
    select_dims(si, shape, mode, &groups, &maxn);
    const size_t need = ecokv::select_ws_layout(groups, maxn, mode != ECOKV_LAYER_FLAT).total;
    if (!workspace) return fail(ECOKV_EINVAL, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(ECOKV_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(ECOKV_EWORKSPACE, "select workspace has %zu bytes, needs %zu", workspace_bytes, need);
    a->mb_groups = groups;
    a->mb_maxn = maxn;
    return ECOKV_OK;
}

int score_impl(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
               const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
               void *workspace, size_t workspace_bytes, void *stream, bool noalloc);

// Scratch of ecokv_score_noalloc: a file-scope device array, one copy on
// every device the library runs on, kept until the process ends.  In host
// code `scratch` names a host-side stand-in, not device memory: its device
// address comes from hipGetSymbolAddress, taken once per device (with that
// device current) on the entry point's first call there and kept here.
constexpr size_t kNoAllocBytes = (size_t)96 << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace {

// The scratch's device address on the current device, which must be the
// stream's device.
int noalloc_scratch(hipStream_t stream, void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "ecokv_score_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(ECOKV_EUNSUPPORTED, "ecokv_score_noalloc: device %d", dev);
    if (stream) {
        hipDevice_t sdev = -1;
        if ((e = hipStreamGetDevice(stream, &sdev)) != hipSuccess)
            return hip_fail(e, "ecokv_score_noalloc: hipStreamGetDevice");
        if ((int)sdev != dev)
            return fail(ECOKV_EINVAL, "ecokv_score_noalloc: the stream belongs to device %d, device %d is current",
                        (int)sdev, dev);
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess)
            return hip_fail(e, "ecokv_score_noalloc: hipGetSymbolAddress");
        if (!p || ((uintptr_t)p & 255u) != 0) return fail(ECOKV_EHIP, "ecokv_score_noalloc: bad scratch address");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return ECOKV_OK;
}

}  // namespace

namespace ecokv {

bool stage_timing_on()
{
    const char *v = getenv("ECOKV_STAGE_TIMING");
    return v && v[0] == '1' && v[1] == 0;
}

void stage_begin(const char *name, hipStream_t st)
{
    g_stage_name = nullptr;
    if (!stage_timing_on()) return;
    if (hipEventCreate(&g_stage_start) != hipSuccess) return;
    if (hipEventRecord(g_stage_start, st) != hipSuccess) {
        (void)hipEventDestroy(g_stage_start);
        return;
    }
    g_stage_name = name;
}

void stage_end(hipStream_t st)
{
    if (!g_stage_name) return;
    hipEvent_t stop;
    if (hipEventCreate(&stop) != hipSuccess || hipEventRecord(stop, st) != hipSuccess) {
        (void)hipEventDestroy(g_stage_start);
        g_stage_name = nullptr;
        return;
    }
    std::lock_guard<std::mutex> lk(g_stage_mu);
    g_stages.push_back({g_stage_name, g_stage_start, stop});
    g_stage_name = nullptr;
}

}  // namespace ecokv

extern "C" {

int ecokv_stage_times(ecokv_stage_time *out, int max, int *count)
{
    if (!count || (max > 0 && !out) || max < 0) return fail(ECOKV_EINVAL, "ecokv_stage_times: bad arguments");
    std::vector<StageRec> recs;
    {
        std::lock_guard<std::mutex> lk(g_stage_mu);
        recs.swap(g_stages);
    }
    int n = 0, rc = ECOKV_OK;
    for (const StageRec &r : recs) {
        float ms = 0.f;
        hipError_t e = hipEventSynchronize(r.stop);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
        if (e != hipSuccess) {
            rc = hip_fail(e, "ecokv_stage_times");
            continue;
        }
        int k = 0;
        while (k < n && strcmp(out[k].name, r.name) != 0) ++k;
        if (k == n) {
            if (n >= max) continue;
            memset(&out[n], 0, sizeof out[n]);
            strncpy(out[n].name, r.name, sizeof out[n].name - 1);
            ++n;
        }
        out[k].ms += ms;
        out[k].launches += 1;
    }
    *count = n;
    return rc;
}


int ecokv_default_params(ecokv_params *p)
{
    if (!p) return fail(ECOKV_EINVAL, "params is NULL");
    p->alpha = 0.8f;
    p->beta = 0.6f;
    p->eps = 1e-6f;
    p->tau = 0.f;
    p->pool_kernel = 5;
    p->causal = 1;
    p->lambda_override = NAN;
    p->imp_mode = ECOKV_IMP_ATTN;
    p->norm_mode = ECOKV_NORM_MINMAX;
    p->winsor_q = 0.01f;
    p->mad_tau = 1.f;
    p->redundancy = ECOKV_RED_EUCLID;
    p->centroid_scope = ECOKV_CENTROID_ALL;
    return ECOKV_OK;
}

int ecokv_workspace_size(const ecokv_shape *shape, const ecokv_params *params, size_t *bytes)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((rc = check_params(params))) return rc;
    if (!bytes) return fail(ECOKV_EINVAL, "bytes is NULL");
    if (si.R > ECOKV_MAX_ROWS)
        return fail(ECOKV_EUNSUPPORTED, "(H_q/H_kv)*window = %d exceeds %d", si.R, ECOKV_MAX_ROWS);
    *bytes = 0;  // the size depends on the element type; report the larger layout
    {
        const bool vn = params->imp_mode == ECOKV_IMP_ATTN_VNORM;
        const size_t b0 = ecokv::score_ws_layout(si.L, si.Hkv, si.B, si.D, si.R, si.Ptot, si.maxT, true, vn).total;
        const size_t b1 = ecokv::score_ws_layout(si.L, si.Hkv, si.B, si.D, si.R, si.Ptot, si.maxT, false, vn).total;
        *bytes = b0 > b1 ? b0 : b1;
    }
    return ECOKV_OK;
}

int ecokv_score(const void *K, const void *Q_win, int dtype, const ecokv_shape *shape, const ecokv_params *params,
                float *scores, float *lambda, float *stats, void *workspace, size_t workspace_bytes, void *stream)
{
    if (params && params->imp_mode != ECOKV_IMP_ATTN)
        return fail(ECOKV_EINVAL, "imp_mode %d needs the values: use ecokv_score_v", params->imp_mode);
    return ecokv_score_v(K, nullptr, Q_win, dtype, shape, params, scores, lambda, stats, workspace,
                         workspace_bytes, stream);
}

int ecokv_score_v(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                  const ecokv_params *params, float *scores, float *lambda, float *stats, void *workspace,
                  size_t workspace_bytes, void *stream)
{
    return ecokv_score_pre(K, V, Q_win, dtype, shape, params, nullptr, scores, lambda, stats, workspace,
                           workspace_bytes, stream);
}

int ecokv_score_pre(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                    const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
                    void *workspace, size_t workspace_bytes, void *stream)
{
    return score_impl(K, V, Q_win, dtype, shape, params, pre, scores, lambda, stats, workspace, workspace_bytes,
                      stream, false);
}

int ecokv_score_noalloc(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
                        const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
                        void *stream)
{
    void *ws = nullptr;
    const int rc = noalloc_scratch(static_cast<hipStream_t>(stream), &ws);
    if (rc) return rc;
    return score_impl(K, V, Q_win, dtype, shape, params, pre, scores, lambda, stats, ws, kNoAllocBytes, stream,
                      true);
}

}  // extern "C"

namespace {

int score_impl(const void *K, const void *V, const void *Q_win, int dtype, const ecokv_shape *shape,
               const ecokv_params *params, const float *pre, float *scores, float *lambda, float *stats,
               void *workspace, size_t workspace_bytes, void *stream, bool noalloc)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((rc = check_params(params))) return rc;
    if (dtype != ECOKV_BF16 && dtype != ECOKV_F32) return fail(ECOKV_EUNSUPPORTED, "dtype %d", dtype);
    if (si.R > ECOKV_MAX_ROWS)
        return fail(ECOKV_EUNSUPPORTED, "(H_q/H_kv)*window = %d exceeds %d", si.R, ECOKV_MAX_ROWS);
    if (si.L == 0) return ECOKV_OK;
    if (!K || !Q_win || !scores) return fail(ECOKV_EINVAL, "K, Q_win and scores must be non-NULL");
    const bool vnorm = params->imp_mode == ECOKV_IMP_ATTN_VNORM;
    if (vnorm && !V) return fail(ECOKV_EINVAL, "imp_mode ECOKV_IMP_ATTN_VNORM needs V");
    const ecokv::WsLayout lay =
        ecokv::score_ws_layout(si.L, si.Hkv, si.B, si.D, si.R, si.Ptot, si.maxT, dtype == ECOKV_BF16, vnorm);
    if (!workspace) return fail(ECOKV_EINVAL, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(ECOKV_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes < lay.total)
        return noalloc ? fail(ECOKV_EWORKSPACE,
                              "ecokv_score_noalloc: this call needs %zu bytes of scratch, the library holds %zu "
                              "per device; split it (fewer layers per call)", lay.total, workspace_bytes)
                       : fail(ECOKV_EWORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, lay.total);

    ecokv::ScoreArgs a;
    memset(&a, 0, sizeof a);
    a.K = K;
    a.V = vnorm ? V : nullptr;
    a.vnorm = vnorm ? 1 : 0;
    a.Q = Q_win;
    a.scores = scores;
    a.lambda = lambda;
    a.stats = stats;
    a.L = si.L;
    a.Hq = si.Hq;
    a.Hkv = si.Hkv;
    a.G = si.G;
    a.D = si.D;
    a.w = si.w;
    a.R = si.R;
    a.B = si.B;
    a.Ttot = si.Ttot;
    a.Ptot = si.Ptot;
    a.alpha = params->alpha;
    a.beta = params->beta;
    a.eps = params->eps;
    a.tau = params->tau > 0.f ? params->tau : sqrtf((float)si.D);
    a.inv_sqrt_d = 1.f / sqrtf((float)si.D);
    a.use_override = isnan(params->lambda_override) ? 0 : 1;
    a.lambda_override = a.use_override ? params->lambda_override : 0.f;
    a.pool_half = params->pool_kernel / 2;
    a.causal = params->causal;
    a.kbf16 = dtype == ECOKV_BF16;
    a.norm_mode = params->norm_mode;
    a.mad_tau = params->mad_tau;
    a.red_std = params->redundancy == ECOKV_RED_STD;
    a.centroid_prefix = params->centroid_scope == ECOKV_CENTROID_PREFIX;
    a.winsor_q = params->winsor_q;
    a.pre = pre;
    if (pre && ((uintptr_t)pre & 3u) != 0) return fail(ECOKV_EINVAL, "pre must be 4-byte aligned");
    // bounded waits between blocks poll up to this many times; ECOKV_SPIN_LIMIT
    // lowers it so that tests can make a wait give up (every kernel still ends)
    a.spin_limit = 1 << 20;
    if (const char *sl = getenv("ECOKV_SPIN_LIMIT")) a.spin_limit = atoi(sl);
    a.no_wait = noalloc ? 1 : 0;  // (its final step runs one block per unit: no waits, no status word)
    if ((rc = fill_seqtab(shape, nullptr, si.w, &a.seq, nullptr))) return rc;
    const hipError_t e = ecokv::score_launch(a, static_cast<char *>(workspace), lay, si.maxT,
                                             static_cast<hipStream_t>(stream), dtype == ECOKV_BF16);
    if (e != hipSuccess) return hip_fail(e, "ecokv_score launch");
    return ECOKV_OK;
}

}  // namespace

extern "C" {

int ecokv_prefill_workspace_size(const ecokv_shape *shape, size_t *bytes)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if (!bytes) return fail(ECOKV_EINVAL, "bytes is NULL");
    if (si.R > ECOKV_MAX_ROWS)
        return fail(ECOKV_EUNSUPPORTED, "(H_q/H_kv)*window = %d exceeds %d", si.R, ECOKV_MAX_ROWS);
    // the element type changes the key block; report the larger
    const size_t b0 = ecokv::prefill_ws_bytes(si.L, si.Hkv, si.B, si.D, si.R, si.maxT, true);
    const size_t b1 = ecokv::prefill_ws_bytes(si.L, si.Hkv, si.B, si.D, si.R, si.maxT, false);
    *bytes = b0 > b1 ? b0 : b1;
    return ECOKV_OK;
}

int ecokv_prefill_write(const void *K_new, const void *V_new, const void *Q_win, int dtype, const ecokv_shape *shape,
                        const ecokv_params *params, void *K_cache, void *V_cache, float *pre, void *workspace,
                        size_t workspace_bytes, void *stream)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((rc = check_params(params))) return rc;
    if (dtype != ECOKV_BF16 && dtype != ECOKV_F32) return fail(ECOKV_EUNSUPPORTED, "dtype %d", dtype);
    if (si.R > ECOKV_MAX_ROWS)
        return fail(ECOKV_EUNSUPPORTED, "(H_q/H_kv)*window = %d exceeds %d", si.R, ECOKV_MAX_ROWS);
    if (si.L == 0) return ECOKV_OK;
    if (!K_new || !Q_win || !K_cache || !pre) return fail(ECOKV_EINVAL, "K_new, Q_win, K_cache and pre must be non-NULL");
    if ((V_new == nullptr) != (V_cache == nullptr)) return fail(ECOKV_EINVAL, "V_new and V_cache: both or neither");
    const uintptr_t al = (uintptr_t)K_new | (uintptr_t)K_cache | (uintptr_t)V_new | (uintptr_t)V_cache;
    if ((al & 15u) != 0) return fail(ECOKV_EINVAL, "K_new, V_new, K_cache and V_cache must be 16-byte aligned");
    if (((uintptr_t)pre & 3u) != 0) return fail(ECOKV_EINVAL, "pre must be 4-byte aligned");
    // the copies read and write different memory
    const size_t es = dtype == ECOKV_BF16 ? 2 : 4;
    const size_t nb = (size_t)si.L * si.Hkv * (size_t)si.Ttot * si.D * es;
    auto overlap = [nb](const void *x, const void *y) {
        const uintptr_t a = (uintptr_t)x, b = (uintptr_t)y;
        return a < b + nb && b < a + nb;
    };
    if (overlap(K_new, K_cache) || (V_new && (overlap(V_new, V_cache) || overlap(K_new, V_cache) ||
                                             overlap(V_new, K_cache) || overlap(K_cache, V_cache))))
        return fail(ECOKV_EINVAL, "the new rows and the cache must not overlap");
    const bool bf16 = dtype == ECOKV_BF16;
    const size_t need = ecokv::prefill_ws_bytes(si.L, si.Hkv, si.B, si.D, si.R, si.maxT, bf16);
    if (!workspace) return fail(ECOKV_EINVAL, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(ECOKV_EINVAL, "workspace must be 256-byte aligned");
    if (workspace_bytes < need) return fail(ECOKV_EWORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);

    ecokv::ScoreArgs a;
    memset(&a, 0, sizeof a);
    a.K = K_cache;
    a.Ksrc = K_new;
    a.Q = Q_win;
    a.pre_out = pre;
    a.L = si.L;
    a.Hq = si.Hq;
    a.Hkv = si.Hkv;
    a.G = si.G;
    a.D = si.D;
    a.w = si.w;
    a.R = si.R;
    a.B = si.B;
    a.Ttot = si.Ttot;
    a.Ptot = si.Ptot;
    a.inv_sqrt_d = 1.f / sqrtf((float)si.D);
    a.causal = params->causal;
    a.kbf16 = bf16;
    if ((rc = fill_seqtab(shape, nullptr, si.w, &a.seq, nullptr))) return rc;
    const hipError_t e = ecokv::prefill_launch(a, V_new, V_cache, static_cast<char *>(workspace), si.maxT,
                                               static_cast<hipStream_t>(stream), bf16);
    if (e != hipSuccess) return hip_fail(e, "ecokv_prefill_write launch");
    return ECOKV_OK;
}

int ecokv_workspace_status(void *workspace, void *stream)
{
    if (!workspace) return fail(ECOKV_EINVAL, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(ECOKV_EINVAL, "workspace must be 256-byte aligned");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    unsigned word = 0u;
    hipError_t e = hipMemcpyAsync(&word, workspace, sizeof word, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "ecokv_workspace_status");
    if (word == 0u) return ECOKV_OK;
    if ((e = ecokv::status_clear(static_cast<unsigned *>(workspace), st)) != hipSuccess)
        return hip_fail(e, "ecokv_workspace_status");
    return fail(ECOKV_ETIMEOUT,
                "a wait between the blocks of an ecokv_score call on this workspace gave up: that call's lambda "
                "and scores of the affected units are NaN");
}

int ecokv_index_count(const ecokv_shape *shape, const int32_t *budget, int64_t *count)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if (!budget || !count) return fail(ECOKV_EINVAL, "budget and count must be non-NULL");
    ecokv::SeqTab t;
    int64_t per_lh = 0;
    if ((rc = fill_seqtab(shape, budget, si.w, &t, &per_lh))) return rc;
    *count = (int64_t)si.L * si.Hkv * per_lh;
    return ECOKV_OK;
}

int ecokv_index_count_mode(const ecokv_shape *shape, int mode, const int32_t *budget, int64_t *count)
{
    if (mode == ECOKV_PER_HEAD || mode == ECOKV_LAYER_FLAT) return ecokv_index_count(shape, budget, count);
    if (mode != ECOKV_HEAD_BUDGETS) return fail(ECOKV_EINVAL, "mode %d", mode);
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((!budget && (int64_t)si.L * si.Hkv > 0) || !count) return fail(ECOKV_EINVAL, "budget and count must be non-NULL");
    int64_t total = 0;
    if ((rc = head_budget_total(shape, si, budget, &total))) return rc;
    *count = total;
    return ECOKV_OK;
}

int ecokv_select_workspace_size(const ecokv_shape *shape, int mode, size_t *bytes)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((rc = check_select_mode(si, mode))) return rc;
    if (!bytes) return fail(ECOKV_EINVAL, "bytes is NULL");
    int64_t groups = 0, maxn = 0;
    select_dims(si, shape, mode, &groups, &maxn);
    *bytes = ecokv::select_ws_layout(groups, maxn, mode != ECOKV_LAYER_FLAT).total;
    return ECOKV_OK;
}

int ecokv_select(const float *scores, const ecokv_shape *shape, int mode, const int32_t *budget,
                            int32_t *idx, int32_t *counts, int32_t *offsets, void *workspace,
                            size_t workspace_bytes, void *stream)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if ((rc = check_select_mode(si, mode))) return rc;
    if (!budget && (mode != ECOKV_HEAD_BUDGETS || (int64_t)si.L * si.Hkv > 0))
        return fail(ECOKV_EINVAL, "budget is NULL");
    ecokv::SelectArgs a;
    memset(&a, 0, sizeof a);
    int64_t per_lh = 0;
    if (mode == ECOKV_HEAD_BUDGETS) {
        int64_t total = 0;
        if ((rc = head_budget_total(shape, si, budget, &total))) return rc;
        if ((rc = fill_seqtab(shape, nullptr, si.w, &a.seq, &per_lh))) return rc;
        if (si.L == 0) return ECOKV_OK;
        if (!scores || !idx) return fail(ECOKV_EINVAL, "scores and idx must be non-NULL");
        if ((rc = select_workspace(si, shape, mode, workspace, workspace_bytes, &a))) return rc;
        a.scores = scores;
        a.idx = idx;
        a.counts = counts;
        a.offsets = offsets;
        a.L = si.L;
        a.Hkv = si.Hkv;
        a.B = si.B;
        a.w = si.w;
        a.Ptot = si.Ptot;
        a.heads = 1;
        // one launch per kLhChunk (layer, head) pairs, each with its table
        const int64_t npairs = (int64_t)si.L * si.Hkv;
        int64_t e0 = 0;
        for (int64_t lh0 = 0; lh0 < npairs; lh0 += ecokv::kLhChunk) {
            const int n = (int)(npairs - lh0 < ecokv::kLhChunk ? npairs - lh0 : ecokv::kLhChunk);
            e0 = fill_lhtab(shape, si.B, budget, lh0, n, e0, &a.lht);
            const hipError_t e = ecokv::select_launch(a, static_cast<char *>(workspace),
                                                      static_cast<hipStream_t>(stream));
            if (e != hipSuccess) return hip_fail(e, "ecokv_select launch");
        }
        return ECOKV_OK;
    }
    if ((rc = fill_seqtab(shape, budget, si.w, &a.seq, &per_lh))) return rc;
    if ((int64_t)si.L * si.Hkv * per_lh > INT32_MAX) return fail(ECOKV_EINVAL, "index count overflows int32");
    if (mode == ECOKV_LAYER_FLAT && (!counts || !offsets))
        return fail(ECOKV_EINVAL, "LAYER_FLAT needs counts and offsets");
    if (si.L == 0) return ECOKV_OK;
    if (!scores || !idx) return fail(ECOKV_EINVAL, "scores and idx must be non-NULL");
    if ((rc = select_workspace(si, shape, mode, workspace, workspace_bytes, &a))) return rc;
    a.scores = scores;
    a.idx = idx;
    a.counts = counts;
    a.offsets = offsets;
    a.L = si.L;
    a.Hkv = si.Hkv;
    a.B = si.B;
    a.w = si.w;
    a.Ptot = si.Ptot;
    a.per_lh = per_lh;
    a.flat = mode == ECOKV_LAYER_FLAT;
    const hipError_t e = ecokv::select_launch(a, static_cast<char *>(workspace), static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ecokv_select launch");
    return ECOKV_OK;
}

int ecokv_compact(const void *K, const void *V, int dtype, const ecokv_shape *shape, int mode, const int32_t *budget,
                  const int32_t *idx, const int32_t *counts, const int32_t *offsets, void *Kc, void *Vc,
                  void *stream)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if (dtype != ECOKV_BF16 && dtype != ECOKV_F32) return fail(ECOKV_EUNSUPPORTED, "dtype %d", dtype);
    if (mode != ECOKV_PER_HEAD && mode != ECOKV_LAYER_FLAT && mode != ECOKV_HEAD_BUDGETS)
        return fail(ECOKV_EINVAL, "mode %d", mode);
    if (!budget && (mode != ECOKV_HEAD_BUDGETS || (int64_t)si.L * si.Hkv > 0))
        return fail(ECOKV_EINVAL, "budget is NULL");
    ecokv::CompactArgs a;
    memset(&a, 0, sizeof a);
    int64_t per_lh = 0;
    if (mode == ECOKV_HEAD_BUDGETS) {
        int64_t total = 0;
        if ((rc = head_budget_total(shape, si, budget, &total))) return rc;
        if ((rc = fill_seqtab(shape, nullptr, si.w, &a.seq, &per_lh))) return rc;
        if (si.L == 0) return ECOKV_OK;
        if (!K || !V || !idx || !Kc || !Vc) return fail(ECOKV_EINVAL, "K, V, idx, Kc and Vc must be non-NULL");
        a.K = static_cast<const char *>(K);
        a.V = static_cast<const char *>(V);
        a.Kc = static_cast<char *>(Kc);
        a.Vc = static_cast<char *>(Vc);
        a.idx = idx;
        a.L = si.L;
        a.Hkv = si.Hkv;
        a.B = si.B;
        a.heads = 1;
        a.Ttot = si.Ttot;
        a.row_bytes = si.D * (dtype == ECOKV_BF16 ? 2 : 4);
        a.segs = a.row_bytes / 16;
        const int64_t npairs = (int64_t)si.L * si.Hkv;
        int64_t e0 = 0;
        for (int64_t lh0 = 0; lh0 < npairs; lh0 += ecokv::kLhChunk) {
            const int n = (int)(npairs - lh0 < ecokv::kLhChunk ? npairs - lh0 : ecokv::kLhChunk);
            a.e0 = e0;
            a.total = e0 = fill_lhtab(shape, si.B, budget, lh0, n, e0, &a.lht);
            const hipError_t e = ecokv::compact_launch(a, static_cast<hipStream_t>(stream));
            if (e != hipSuccess) return hip_fail(e, "ecokv_compact launch");
        }
        return ECOKV_OK;
    }
    if ((rc = fill_seqtab(shape, budget, si.w, &a.seq, &per_lh))) return rc;
    if (mode == ECOKV_LAYER_FLAT && !offsets) return fail(ECOKV_EINVAL, "LAYER_FLAT needs offsets");
    (void)counts;
    if (si.L == 0) return ECOKV_OK;
    if (!K || !V || !idx || !Kc || !Vc) return fail(ECOKV_EINVAL, "K, V, idx, Kc and Vc must be non-NULL");
    a.K = static_cast<const char *>(K);
    a.V = static_cast<const char *>(V);
    a.Kc = static_cast<char *>(Kc);
    a.Vc = static_cast<char *>(Vc);
    a.idx = idx;
    a.offsets = offsets;
    a.L = si.L;
    a.Hkv = si.Hkv;
    a.B = si.B;
    a.flat = mode == ECOKV_LAYER_FLAT;
    a.Ttot = si.Ttot;
    a.row_bytes = si.D * (dtype == ECOKV_BF16 ? 2 : 4);
    a.segs = a.row_bytes / 16;
    a.total = (int64_t)si.L * si.Hkv * per_lh;
    a.per_lh = per_lh;
    const hipError_t e = ecokv::compact_launch(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ecokv_compact launch");
    return ECOKV_OK;
}

int ecokv_decode_workspace_size(const ecokv_shape *shape, int32_t max_count, size_t *bytes)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if (!bytes) return fail(ECOKV_EINVAL, "bytes is NULL");
    if (max_count < 1) return fail(ECOKV_EINVAL, "max_count %d < 1", max_count);
    *bytes = sizeof(float) * (size_t)si.L * si.Hq * si.B * (size_t)ecokv::decode_parts(max_count) * (si.D + 2);
    return ECOKV_OK;
}

int ecokv_decode(const void *Q_dec, const void *Kc, const void *Vc, int dtype, const ecokv_shape *shape,
                 const int32_t *counts, const int32_t *offsets, int32_t max_count, float *O, float *lse,
                 void *workspace, size_t workspace_bytes, void *stream)
{
    ShapeInfo si;
    int rc = check_shape(shape, &si);
    if (rc) return rc;
    if (dtype != ECOKV_BF16 && dtype != ECOKV_F32) return fail(ECOKV_EUNSUPPORTED, "dtype %d", dtype);
    if (max_count < 1) return fail(ECOKV_EINVAL, "max_count %d < 1", max_count);
    size_t need = 0;
    if ((rc = ecokv_decode_workspace_size(shape, max_count, &need))) return rc;
    if (si.L == 0) return ECOKV_OK;
    if (!Q_dec || !Kc || !Vc || !counts || !offsets || !O)
        return fail(ECOKV_EINVAL, "Q_dec, Kc, Vc, counts, offsets and O must be non-NULL");
    if (!workspace) return fail(ECOKV_EINVAL, "workspace is NULL");
    if (((uintptr_t)workspace & 255u) != 0) return fail(ECOKV_EINVAL, "workspace must be 256-byte aligned");
    if (((uintptr_t)Q_dec & 15u) != 0 || ((uintptr_t)Kc & 15u) != 0 || ((uintptr_t)Vc & 15u) != 0)
        return fail(ECOKV_EINVAL, "Q_dec, Kc and Vc must be 16-byte aligned");
    if (workspace_bytes < need)
        return fail(ECOKV_EWORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
    ecokv::DecodeArgs a;
    memset(&a, 0, sizeof a);
    a.Q = Q_dec;
    a.Kc = Kc;
    a.Vc = Vc;
    a.counts = counts;
    a.offsets = offsets;
    a.O = O;
    a.lse = lse;
    a.part = static_cast<float *>(workspace);
    a.L = si.L;
    a.Hq = si.Hq;
    a.Hkv = si.Hkv;
    a.G = si.G;
    a.B = si.B;
    a.D = si.D;
    a.max_count = max_count;
    a.nparts = ecokv::decode_parts(max_count);
    a.qscale = 1.4426950408889634f / sqrtf((float)si.D);
    const hipError_t e = ecokv::decode_launch(a, dtype == ECOKV_BF16, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ecokv_decode launch");
    return ECOKV_OK;
}

int ecokv_pyramid_budgets(int num_layers, double total, double beta, int window, int32_t *out)
{
    if (num_layers < 1 || !out) return fail(ECOKV_EINVAL, "num_layers %d < 1 or out is NULL", num_layers);
    if (!(isfinite(total) && total > 0.0) || !(isfinite(beta) && beta > 0.0))
        return fail(ECOKV_EINVAL, "total %g and beta %g must be positive and finite", total, beta);
    if (window < 1) return fail(ECOKV_EINVAL, "window %d < 1", window);
    const int m = num_layers;
    const double last = total / (beta * m), first = 2.0 * total / m - last;
    // every value checked before any is written
    for (int pass = 0; pass < 2; ++pass)
        for (int l = 0; l < m; ++l) {
            const double v = m == 1 ? total : first - (first - last) * l / (m - 1);
            // rounded down; a value within 1e-9 below an integer is that integer
            const double f = floor(v + 1e-9);
            if (pass == 0 && !(f >= window && f <= (double)INT32_MAX))
                return fail(ECOKV_EINVAL, "layer %d budget %g is outside [window %d, INT32_MAX]", l, v, window);
            if (pass == 1) out[l] = (int32_t)f;
        }
    return ECOKV_OK;
}

const char *ecokv_last_error(void) { return g_err; }

}  // extern "C"
