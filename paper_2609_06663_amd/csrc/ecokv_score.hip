// ecokv_score kernels (gfx950): importance, diversity, redundancy and the
// final score of every (layer, KV head, sequence) unit.
//
// Stages, in stream order:
//   pass1  one sweep over K: column sums of k and of k/|k| (anchors kbar, mu,
//          Eq. (1) and the MixKV cosine anchor of Appendix A.1) and, per
//          window row, the chunk's softmax max and sum of exponentials
//          (Sec. 3 attention).  The last block of a unit combines the chunks.
//   pass2  second sweep over K: per key d_E = |k - kbar| (Eq. (1)), khat.mu,
//          and the window-mean attention a_i (Sec. 5.2, "average attention
//          score").  The last block forms D_E (Eq. (4)), r_E (Eq. (5)),
//          r_C (Appendix A.1) and lambda (Eq. (6)).
//   epi1   per non-window key: pooled S_imp (Table 6), s_E (Eq. (2)),
//          s_C, S_div (Eq. (3)); block min/max/sums, last block forms the
//          rescale of Sec. 5.2.
//   epi2   S = lambda * S_tilde + (1 - lambda) * S_imp (Eq. (7)).
//
// Lane layout of the sweeps: 16 lanes per key row, each lane holding D/16
// consecutive elements, so one wave reads 4 whole rows per instruction
// (coalesced 1 KiB for bf16, D = 128) and row reductions stay inside a
// 16-lane segment.
#include "ecokv_internal.h"

namespace ecokv {

constexpr int kThreads = 256;
constexpr int kCh = 128;       // key rows per block in the sweeps
constexpr int kEpi = 256;      // non-window keys per block in the epilogues

__device__ __forceinline__ const char *unit_krow0(const ScoreArgs &a, const Unit &un, int esz)
{
    const int64_t row = ((int64_t)un.l * a.Hkv + un.h) * a.Ttot + a.seq.cu[un.s];
    return static_cast<const char *>(a.K) + row * (int64_t)a.D * esz;
}

// Window row r = (g, j) of unit `un` as float into LDS q[r][D].
template <int D, bool BF>
__device__ void load_window_rows(const ScoreArgs &a, const Unit &un, float *q)
{
    for (int idx = threadIdx.x; idx < a.R * D; idx += blockDim.x) {
        const int r = idx / D, d = idx % D;
        const int g = r / a.w, j = r % a.w;
        const int64_t qrow = (((int64_t)un.l * a.Hq + (int64_t)un.h * a.G + g) * a.B + un.s) * a.w + j;
        float v;
        if constexpr (BF)
            v = bf16_to_f32(static_cast<const uint16_t *>(a.Q)[qrow * D + d]);
        else
            v = static_cast<const float *>(a.Q)[qrow * D + d];
        q[r * D + d] = v;
    }
}

template <int D, bool BF>
__global__ __launch_bounds__(kThreads) void k_pass1(ScoreArgs a)
{
    constexpr int VEC = D / 16;
    constexpr int ESZ = BF ? 2 : 4;
    __shared__ float q_lds[ECOKV_MAX_ROWS * D];
    __shared__ float lg[ECOKV_MAX_ROWS * (kCh + 1)];
    __shared__ float red[2][16][D];
    __shared__ int flag;

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row0 = blockIdx.x * kCh;
    if (row0 >= T) return;
    const int nch = (T + kCh - 1) / kCh;

    load_window_rows<D, BF>(a, un, q_lds);
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = lane & 15, sub = lane >> 4;
    const char *k0 = unit_krow0(a, un, ESZ);
    float sk[VEC], skh[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) sk[e] = skh[e] = 0.f;

    for (int it = 0; it < kCh / 16; ++it) {
        const int rl = it * 16 + wv * 4 + sub;
        const int i = row0 + rl;
        const bool valid = i < T;
        float v[VEC];
        if (valid) {
            load_seg<D, BF>(k0 + (int64_t)i * D * ESZ, c, v);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[e] = 0.f;
        }
        float n2 = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) n2 += v[e] * v[e];
        n2 = seg16_sum(n2);
        const float inv = 1.f / fmaxf(sqrtf(n2), 1e-12f);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            sk[e] += v[e];
            skh[e] += v[e] * inv;
        }
        for (int r = 0; r < a.R; ++r) {
            const float *qr = q_lds + r * D + c * VEC;
            float d = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) d += qr[e] * v[e];
            d = seg16_sum(d);
            const int j = r % a.w;
            const bool vis = valid && (!a.causal || i <= P + j);
            if (c == 0) lg[r * (kCh + 1) + rl] = vis ? d * a.inv_sqrt_d : -INFINITY;
        }
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        red[0][wv * 4 + sub][c * VEC + e] = sk[e];
        red[1][wv * 4 + sub][c * VEC + e] = skh[e];
    }
    __syncthreads();

    const int stride = 2 * D + 2 * a.R;
    float *part = a.part1 + ((int64_t)u * a.nch1 + blockIdx.x) * stride;
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
        float m = -INFINITY;
        for (int t = 0; t < kCh; ++t) m = fmaxf(m, lg[r * (kCh + 1) + t]);
        float s = 0.f;
        if (m > -INFINITY)
            for (int t = 0; t < kCh; ++t) s += __expf(lg[r * (kCh + 1) + t] - m);
        part[2 * D + r] = m;
        part[2 * D + a.R + r] = s;
    }
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        float s0 = 0.f, s1 = 0.f;
        for (int g = 0; g < 16; ++g) {
            s0 += red[0][g][d];
            s1 += red[1][g][d];
        }
        part[d] = s0;
        part[D + d] = s1;
    }

    if (!last_block_arrives(a.counters + u * 4 + 0, nch, &flag)) return;

    const float* pu = a.part1 + (int64_t)u * a.nch1 * stride;
    float *anc = a.anchors + (int64_t)u * stride;
    for (int d = threadIdx.x; d < 2 * D; d += blockDim.x) {
        float s = 0.f;
        for (int ch = 0; ch < nch; ++ch) s += pu[(int64_t)ch * stride + d];
        anc[d] = s / (float)T;
    }
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
        float m = -INFINITY;
        for (int ch = 0; ch < nch; ++ch) m = fmaxf(m, pu[(int64_t)ch * stride + 2 * D + r]);
        float s = 0.f;
        for (int ch = 0; ch < nch; ++ch) {
            const float pm = pu[(int64_t)ch * stride + 2 * D + r];
            if (pm > -INFINITY) s += pu[(int64_t)ch * stride + 2 * D + a.R + r] * __expf(pm - m);
        }
        anc[2 * D + r] = m;
        anc[2 * D + a.R + r] = s;
    }
    if (threadIdx.x == 0) a.counters[u * 4 + 0] = 0;
}

template <int D, bool BF>
__global__ __launch_bounds__(kThreads) void k_pass2(ScoreArgs a)
{
    constexpr int VEC = D / 16;
    constexpr int ESZ = BF ? 2 : 4;
    __shared__ float q_lds[ECOKV_MAX_ROWS * D];
    __shared__ float kb[D], mu[D], rm[ECOKV_MAX_ROWS], rs_inv[ECOKV_MAX_ROWS];
    __shared__ float wred[3][kThreads / kWave];
    __shared__ int flag;

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row0 = blockIdx.x * kCh;
    if (row0 >= T) return;
    const int nch = (T + kCh - 1) / kCh;
    const int stride = 2 * D + 2 * a.R;
    const float *anc = a.anchors + (int64_t)u * stride;

    load_window_rows<D, BF>(a, un, q_lds);
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        kb[d] = anc[d];
        mu[d] = anc[D + d];
    }
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
        rm[r] = anc[2 * D + r];
        rs_inv[r] = 1.f / anc[2 * D + a.R + r];
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = lane & 15, sub = lane >> 4;
    const char *k0 = unit_krow0(a, un, ESZ);
    const int64_t obase = ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - un.s * a.w);
    const float inv_r = 1.f / (float)a.R;
    float dsum = 0.f, dmin = INFINITY, dmax = -INFINITY;

    for (int it = 0; it < kCh / 16; ++it) {
        const int i = row0 + it * 16 + wv * 4 + sub;
        const bool valid = i < T;
        float v[VEC];
        if (valid) {
            load_seg<D, BF>(k0 + (int64_t)i * D * ESZ, c, v);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) v[e] = 0.f;
        }
        float d2 = 0.f, n2 = 0.f, km = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const float df = v[e] - kb[c * VEC + e];
            d2 += df * df;
            n2 += v[e] * v[e];
            km += v[e] * mu[c * VEC + e];
        }
        d2 = seg16_sum(d2);
        n2 = seg16_sum(n2);
        km = seg16_sum(km);
        const float dE = sqrtf(d2);
        const float cm = km / fmaxf(sqrtf(n2), 1e-12f);
        float att = 0.f;
        for (int r = 0; r < a.R; ++r) {
            const float *qr = q_lds + r * D + c * VEC;
            float d = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) d += qr[e] * v[e];
            d = seg16_sum(d);
            att += __expf(d * a.inv_sqrt_d - rm[r]) * rs_inv[r];
        }
        if (valid) {
            dsum += (c == 0) ? dE : 0.f;
            if (i < P) {
                dmin = fminf(dmin, dE);
                dmax = fmaxf(dmax, dE);
                if (c == 0) {
                    a.bufA[obase + i] = dE;
                    a.bufB[obase + i] = cm;
                    a.bufC[obase + i] = att * inv_r;
                }
            }
        }
    }
    dsum = wave_sum(dsum);
    dmin = wave_min(dmin);
    dmax = wave_max(dmax);
    if (lane == 0) {
        wred[0][wv] = dsum;
        wred[1][wv] = dmin;
        wred[2][wv] = dmax;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float s = 0.f, mn = INFINITY, mx = -INFINITY;
        for (int k = 0; k < kThreads / kWave; ++k) {
            s += wred[0][k];
            mn = fminf(mn, wred[1][k]);
            mx = fmaxf(mx, wred[2][k]);
        }
        float *pp = a.part2 + ((int64_t)u * a.nch1 + blockIdx.x) * 4;
        pp[0] = s;
        pp[1] = mn;
        pp[2] = mx;
    }

    if (!last_block_arrives(a.counters + u * 4 + 1, nch, &flag)) return;
    if (threadIdx.x == 0) {
        const float *pp = a.part2 + (int64_t)u * a.nch1 * 4;
        float s = 0.f, mn = INFINITY, mx = -INFINITY;
        for (int ch = 0; ch < nch; ++ch) {
            s += pp[ch * 4 + 0];
            mn = fminf(mn, pp[ch * 4 + 1]);
            mx = fmaxf(mx, pp[ch * 4 + 2]);
        }
        float mu2 = 0.f;
        for (int d = 0; d < D; ++d) mu2 += mu[d] * mu[d];
        const float DE = s / (float)T;
        const float rE = 2.f - 2.f / (1.f + expf(-DE / a.tau));
        const float rC = ((float)T * mu2 - 1.f) / ((float)T - 1.f);
        const float lam = a.use_override ? a.lambda_override : a.beta * rE + (1.f - a.beta) * rC;
        float *hs = a.hstat + (int64_t)u * HS_COUNT;
        hs[HS_LAMBDA] = lam;
        hs[HS_RC] = rC;
        hs[HS_RE] = rE;
        hs[HS_DE] = DE;
        hs[HS_DMIN] = mn;
        hs[HS_DMAX] = mx;
        hs[HS_MU2] = mu2;
        a.counters[u * 4 + 1] = 0;
    }
}

__global__ __launch_bounds__(kEpi) void k_epi1(ScoreArgs a)
{
    __shared__ float wred[4][kEpi / kWave];
    __shared__ int flag;
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int i0 = blockIdx.x * kEpi;
    if (i0 >= P) return;
    const int nblk = (P + kEpi - 1) / kEpi;
    const int64_t obase = ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - un.s * a.w);
    const float *hs = a.hstat + (int64_t)u * HS_COUNT;
    const float dmin = hs[HS_DMIN], dden = hs[HS_DMAX] - hs[HS_DMIN] + a.eps;
    const int i = i0 + threadIdx.x;
    float sdiv = 0.f, imp = 0.f, mn = INFINITY, mx = -INFINITY;
    if (i < P) {
        float acc = 0.f;
        for (int t = -a.pool_half; t <= a.pool_half; ++t) {
            const int k = i + t;
            if (k >= 0 && k < P) acc += a.bufC[obase + k];
        }
        imp = acc / (float)(2 * a.pool_half + 1);
        const float sE = (a.bufA[obase + i] - dmin) / dden;
        const float sC = (1.f - a.bufB[obase + i]) * 0.5f;
        sdiv = a.alpha * sE + (1.f - a.alpha) * sC;
        mn = mx = sdiv;
        a.bufA[obase + i] = sdiv;
        a.bufB[obase + i] = imp;
    }
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const float s1 = wave_sum(sdiv), s2 = wave_sum(imp);
    mn = wave_min(mn);
    mx = wave_max(mx);
    if (lane == 0) {
        wred[0][wv] = mn;
        wred[1][wv] = mx;
        wred[2][wv] = s1;
        wred[3][wv] = s2;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float a0 = INFINITY, a1 = -INFINITY, a2 = 0.f, a3 = 0.f;
        for (int k = 0; k < kEpi / kWave; ++k) {
            a0 = fminf(a0, wred[0][k]);
            a1 = fmaxf(a1, wred[1][k]);
            a2 += wred[2][k];
            a3 += wred[3][k];
        }
        float *pp = a.part3 + ((int64_t)u * a.nch3 + blockIdx.x) * 4;
        pp[0] = a0;
        pp[1] = a1;
        pp[2] = a2;
        pp[3] = a3;
    }
    if (!last_block_arrives(a.counters + u * 4 + 2, nblk, &flag)) return;
    if (threadIdx.x == 0) {
        const float *pp = a.part3 + (int64_t)u * a.nch3 * 4;
        float a0 = INFINITY, a1 = -INFINITY, a2 = 0.f, a3 = 0.f;
        for (int k = 0; k < nblk; ++k) {
            a0 = fminf(a0, pp[k * 4 + 0]);
            a1 = fmaxf(a1, pp[k * 4 + 1]);
            a2 += pp[k * 4 + 2];
            a3 += pp[k * 4 + 3];
        }
        float *h = a.hstat + (int64_t)u * HS_COUNT;
        const float sdmean = a2 / (float)P;
        const float impmean = a3 / (float)P;
        const float sbarmean = (sdmean - a0) / (a1 - a0 + a.eps);
        h[HS_SDMIN] = a0;
        h[HS_SDMAX] = a1;
        h[HS_IMPMEAN] = impmean;
        h[HS_SBARMEAN] = sbarmean;
        h[HS_SCALE] = impmean / (sbarmean + a.eps);
        a.counters[u * 4 + 2] = 0;
    }
}

__global__ __launch_bounds__(kEpi) void k_epi2(ScoreArgs a)
{
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int i0 = blockIdx.x * kEpi;
    if (i0 >= P) return;
    const int64_t obase = ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - un.s * a.w);
    const float *hs = a.hstat + (int64_t)u * HS_COUNT;
    const float lam = hs[HS_LAMBDA], smin = hs[HS_SDMIN];
    const float sden = hs[HS_SDMAX] - smin + a.eps, scale = hs[HS_SCALE];
    const int i = i0 + threadIdx.x;
    if (i < P) {
        const float sbar = (a.bufA[obase + i] - smin) / sden;
        a.scores[obase + i] = lam * (sbar * scale) + (1.f - lam) * a.bufB[obase + i];
    }
    if (blockIdx.x == 0 && threadIdx.x < ECOKV_NSTATS) {
        if (a.stats) a.stats[(int64_t)u * ECOKV_NSTATS + threadIdx.x] = hs[threadIdx.x];
        if (a.lambda && threadIdx.x == 0) a.lambda[u] = lam;
    }
}

__global__ void k_zero_u32(unsigned *p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

template <int D, bool BF>
static hipError_t launch_sweeps(const ScoreArgs &a, int U, int maxT, hipStream_t st)
{
    const dim3 g1((maxT + kCh - 1) / kCh, U);
    hipLaunchKernelGGL((k_pass1<D, BF>), g1, dim3(kThreads), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_pass2<D, BF>), g1, dim3(kThreads), 0, st, a);
    return hipGetLastError();
}



static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout score_ws_layout(int L, int Hkv, int B, int D, int R, int64_t Ptot, int maxT, int maxP)
{
    WsLayout w{};
    const int64_t U = (int64_t)L * Hkv * B;
    const int64_t nch1 = (maxT + kCh - 1) / kCh;
    const int64_t nch3 = (maxP + kEpi - 1) / kEpi;
    const int64_t stride = 2 * D + 2 * R;
    size_t o = 0;
    w.part1 = o; o = align256(o + sizeof(float) * U * nch1 * stride);
    w.anchors = o; o = align256(o + sizeof(float) * U * stride);
    w.part2 = o; o = align256(o + sizeof(float) * U * nch1 * 4);
    w.hstat = o; o = align256(o + sizeof(float) * U * HS_COUNT);
    w.bufA = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.bufB = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.bufC = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.part3 = o; o = align256(o + sizeof(float) * U * nch3 * 4);
    w.counters = o; o = align256(o + sizeof(unsigned) * U * 4);
    w.total = o;
    return w;
}

hipError_t score_launch(ScoreArgs a, char *ws, const WsLayout &lay, int maxT, int maxP, hipStream_t st,
                        bool bf16)
{
    const int U = a.L * a.Hkv * a.B;
    a.part1 = reinterpret_cast<float *>(ws + lay.part1);
    a.anchors = reinterpret_cast<float *>(ws + lay.anchors);
    a.part2 = reinterpret_cast<float *>(ws + lay.part2);
    a.hstat = reinterpret_cast<float *>(ws + lay.hstat);
    a.bufA = reinterpret_cast<float *>(ws + lay.bufA);
    a.bufB = reinterpret_cast<float *>(ws + lay.bufB);
    a.bufC = reinterpret_cast<float *>(ws + lay.bufC);
    a.part3 = reinterpret_cast<float *>(ws + lay.part3);
    a.counters = reinterpret_cast<unsigned *>(ws + lay.counters);
    a.nch1 = (maxT + kCh - 1) / kCh;
    a.nch3 = (maxP + kEpi - 1) / kEpi;

    const int64_t ncnt = (int64_t)U * 4;
    hipLaunchKernelGGL(k_zero_u32, dim3((unsigned)((ncnt + 255) / 256)), dim3(256), 0, st, a.counters, ncnt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    if (bf16) {
        e = a.D == 128 ? launch_sweeps<128, true>(a, U, maxT, st) : launch_sweeps<64, true>(a, U, maxT, st);
    } else {
        e = a.D == 128 ? launch_sweeps<128, false>(a, U, maxT, st) : launch_sweeps<64, false>(a, U, maxT, st);
    }
    if (e != hipSuccess) return e;
    const dim3 ge((maxP + kEpi - 1) / kEpi, U);
    hipLaunchKernelGGL(k_epi1, ge, dim3(kEpi), 0, st, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_epi2, ge, dim3(kEpi), 0, st, a);
    return hipGetLastError();
}

}  // namespace ecokv
