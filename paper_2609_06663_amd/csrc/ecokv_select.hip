// ecokv_select kernels (gfx950): exact top-k of the scores of each unit
// (ECOKV_PER_HEAD, ECOKV_HEAD_BUDGETS) or of all heads of a (layer, sequence)
// (ECOKV_LAYER_FLAT, AdaKV budget sharing, Appendix A.1), plus the
// always-kept window (Sec. 3); and the order statistics of d_E that the
// winsorised and MAD normalisations need (Sec. 6.3, Table 4).
//
// The k-th largest score is found exactly by a most-significant-digit radix
// select over order-preserving 32-bit keys.  An ordered pass then emits the
// chosen positions in ascending order: keys above the threshold are always
// taken, keys equal to it are taken in position order until the budget is
// met, so equal scores favour the smaller position.
#include "ecokv_internal.h"

namespace ecokv {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kMaxFlatHeads = 256;


// Selection group gi of a launch: layer l, heads h0 .. h0+nh-1 of sequence
// s, min(budget, T_s) entries per head, first entry at out_base.
struct SelGroup {
    int l, h0, s, nh, beff;
    int64_t out_base;
};
__device__ __forceinline__ SelGroup sel_group(const SelectArgs &a, int gi)
{
    SelGroup g;
    if (a.heads) {
        // one unit per group, (layer, head) pair lh0 + j of the launch's table
        const int j = gi / a.B;
        g.s = gi - j * a.B;
        const int lh = a.lht.lh0 + j;
        g.l = lh / a.Hkv;
        g.h0 = lh - g.l * a.Hkv;
        g.nh = 1;
        g.beff = min(a.lht.b[j], a.seq.cu[g.s + 1] - a.seq.cu[g.s]);
        g.out_base = a.lht.start[j] + lh_seq_offset(a.lht, a.seq, j, g.s);
    } else if (a.flat) {
        g.l = gi / a.B;
        g.s = gi % a.B;
        g.h0 = 0;
        g.nh = a.Hkv;
        g.beff = a.seq.beff[g.s];
        g.out_base = (int64_t)g.l * a.Hkv * a.per_lh + (int64_t)a.Hkv * a.seq.boff[g.s];
    } else {
        const Unit un = unit_of(gi, a.Hkv, a.B);
        g.l = un.l;
        g.s = un.s;
        g.h0 = un.h;
        g.nh = 1;
        g.beff = a.seq.beff[g.s];
        g.out_base = ((int64_t)g.l * a.Hkv + g.h0) * a.per_lh + a.seq.boff[g.s];
    }
    return g;
}

// f(v, key) for every v in [0, n) with v = tid (mod blockDim.x); eight keys
// are fetched before any is used so that loads overlap.
template <class Src, class F>
__device__ __forceinline__ void for_each_key(const Src &key, int64_t n, F &&f)
{
    const int64_t step = blockDim.x;
    for (int64_t base = threadIdx.x; base < n; base += 8 * step) {
        uint32_t kk[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int64_t v = base + q * step;
            kk[q] = v < n ? key(v) : 0u;
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int64_t v = base + q * step;
            if (v < n) f(v, kk[q]);
        }
    }
}

__device__ __forceinline__ uint32_t wave_min_u(uint32_t x) { return wave_min_u32(x); }
__device__ __forceinline__ uint32_t wave_max_u(uint32_t x) { return wave_max_u32(x); }

// Exact radix select of the k-th largest key (k >= 1) among n keys whose
// extremes are kmin, kmax: digits of up to 8 bits, starting just below the
// common prefix of kmin and kmax so that the first histogram is spread out.
// Returns the threshold key and how many keys equal to it are taken.
template <class Src>
__device__ void radix_threshold(const Src &key, int64_t n, int64_t k, uint32_t kmin, uint32_t kmax, uint32_t *hist,
                                uint32_t *bc, uint32_t *thr_out, int64_t *need_eq_out)
{
    const uint32_t diff = kmin ^ kmax;
    if (diff == 0) {
        *thr_out = kmin;
        *need_eq_out = k;
        return;
    }
    int hi = 31 - __clz(diff);
    uint32_t mask = hi == 31 ? 0u : ~((2u << hi) - 1u);
    uint32_t prefix = kmin & mask;
    int64_t rem = k;
    while (hi >= 0) {
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t nb = 1u << (hi - lo + 1);
        for (int b = threadIdx.x; b < kSelWaves * 256; b += blockDim.x) hist[b] = 0;
        __syncthreads();
        uint32_t *const myh = hist + (threadIdx.x >> 6) * 256;
        for_each_key(key, n, [&](int64_t, uint32_t kk) {
            if ((kk & mask) == prefix) atomicAdd(&myh[(kk >> lo) & (nb - 1u)], 1u);
        });
        __syncthreads();
        if (threadIdx.x < 256) {
            // fold the wave histograms into the first (each thread its own bin)
            uint32_t c = 0;
#pragma unroll
            for (int w2 = 0; w2 < kSelWaves; ++w2) c += hist[w2 * 256 + threadIdx.x];
            hist[threadIdx.x] = c;
        }
        __syncthreads();
        if (threadIdx.x < kWave) {
            // lane l owns bins 255-4l .. 252-4l (descending order of digit)
            const int lane = threadIdx.x;
            uint32_t c4[4], loc = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                c4[q] = hist[255 - 4 * lane - q];
                loc += c4[q];
            }
            uint32_t inc = wave_incl_scan(loc);
            const uint32_t before = inc - loc;
            if ((int64_t)before < rem && rem <= (int64_t)inc) {
                uint32_t cum = before;
                for (int q = 0; q < 4; ++q) {
                    if ((int64_t)(cum + c4[q]) >= rem) {
                        bc[0] = 255u - 4u * lane - q;
                        bc[1] = cum;
                        break;
                    }
                    cum += c4[q];
                }
            }
        }
        __syncthreads();
        const uint32_t digit = bc[0];
        rem -= bc[1];
        prefix |= digit << lo;
        mask |= (nb - 1u) << lo;
        hi = lo - 1;
        __syncthreads();
    }
    *thr_out = prefix;
    *need_eq_out = rem;
}

// radix_threshold for the streaming select of large groups, with the later
// digits over a gathered list: after the first digit, the keys that keep the
// chosen prefix (usually a small part of the group) are written to cand (one
// LDS atomic per wave and load, positions by mbcnt), and the later digits
// count only them into the first histogram, which the scanning wave reads
// directly.  If more than cap keys keep the prefix, every digit reads all

// ---------------------------------------------------------------------------
// Register-resident radix select: thread t holds keys kk[0..KPT) at positions
// v0 .. v0+KPT-1 of n (positions >= n are not keys).
// ---------------------------------------------------------------------------
// Block-wide min and max of the keys (mm: LDS, 2 x kSelWaves).
template <int KPT>
__device__ __forceinline__ void reg_extremes(const uint32_t (&kk)[KPT], int v0, int n, uint32_t (*mm)[kSelWaves],
                                             uint32_t *kmin_out, uint32_t *kmax_out)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
    for (int q = 0; q < KPT; ++q)
        if (v0 + q < n) {
            kmin = min(kmin, kk[q]);
            kmax = max(kmax, kk[q]);
        }
    kmin = wave_min_u(kmin);
    kmax = wave_max_u(kmax);
    if (lane == 0) {
        mm[0][wv] = kmin;
        mm[1][wv] = kmax;
    }
    __syncthreads();
    kmin = mm[0][0];
    kmax = mm[1][0];
    for (int q = 1; q < kSelWaves; ++q) {
        kmin = min(kmin, mm[0][q]);
        kmax = max(kmax, mm[1][q]);
    }
    *kmin_out = kmin;
    *kmax_out = kmax;
}

// The k-th largest key (k >= 1): digits of up to 8 bits below the common
// prefix of kmin and kmax, one LDS histogram of 256 counters per wave (hist:
// kSelWaves of them), three barriers per pass (the histograms are cleared by
// the threads that fold them, and the chosen digit alternates between two
// slots).  Returns the threshold and how many keys equal to it are taken.
template <int KPT>
__device__ __forceinline__ void reg_radix_select(const uint32_t (&kk)[KPT], int v0, int n, int k, uint32_t kmin,
                                                 uint32_t kmax, uint32_t *hist, uint32_t *hsum,
                                                 uint32_t (*bc)[2], uint32_t *thr_out, int *need_eq_out)
{
    constexpr int HS = 256;
    constexpr int NH = kSelWaves;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    uint32_t *const myh = hist + wv * HS;
    const uint32_t diff = kmin ^ kmax;
    if (diff == 0) {
        *thr_out = kmin;
        *need_eq_out = k;
        return;
    }
    int hi = 31 - __clz(diff);
    uint32_t mask = hi == 31 ? 0u : ~((2u << hi) - 1u);
    uint32_t prefix = kmin & mask;
    int rem = k;
    for (int b = tid; b < NH * HS; b += blockDim.x) hist[b] = 0;
    __syncthreads();
    int par = 0;
    while (hi >= 0) {
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t nb = 1u << (hi - lo + 1);
#pragma unroll
        for (int q = 0; q < KPT; ++q)
            if (v0 + q < n && (kk[q] & mask) == prefix) atomicAdd(&myh[(kk[q] >> lo) & (nb - 1u)], 1u);
        __syncthreads();
        if (tid < 256) {
            uint32_t c = 0;
#pragma unroll
            for (int w2 = 0; w2 < NH; ++w2) {
                c += hist[w2 * HS + tid];
                hist[w2 * HS + tid] = 0;
            }
            hsum[tid] = c;
        }
        __syncthreads();
        if (tid < kWave) {
            // lane owns bins 255-4l .. 252-4l (descending digit order)
            uint32_t c4[4], loc = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                c4[q] = hsum[255 - 4 * lane - q];
                loc += c4[q];
            }
            uint32_t inc = wave_incl_scan(loc);
            const uint32_t before = inc - loc;
            if ((int)before < rem && rem <= (int)inc) {
                uint32_t cum = before;
                for (int q = 0; q < 4; ++q) {
                    if ((int)(cum + c4[q]) >= rem) {
                        bc[par][0] = 255u - 4u * lane - q;
                        bc[par][1] = cum;
                        break;
                    }
                    cum += c4[q];
                }
            }
        }
        __syncthreads();
        prefix |= bc[par][0] << lo;
        rem -= (int)bc[par][1];
        mask |= (nb - 1u) << lo;
        hi = lo - 1;
        par ^= 1;
    }
    *thr_out = prefix;
    *need_eq_out = rem;
}

// ---------------------------------------------------------------------------
// Order statistics of d_E for the winsorised and MAD normalisations (Sec. 6.3,
// Table 4): per unit, its q and 1 - q quantiles, or its median and the median
// of |d_E - median|, over the P non-window keys.  A quantile interpolates
// linearly between the order statistics at ranks floor(h) and floor(h) + 1,
// h = q (P - 1).  One block per unit; the lower order statistic is an exact
// radix select (the unit's values are re-read from the cache in every pass),
// the upper one either equals it (ties) or is the smallest key above it.
// ---------------------------------------------------------------------------
struct DistKey {
    const float *d;
    float c;   // with dev: the key of v is |d[v] - c|
    bool dev;
    __device__ __forceinline__ uint32_t operator()(int64_t v) const { return score_key(dev ? fabsf(d[v] - c) : d[v]); }
};

// The value of an order-preserving key (inverse of score_key for numbers).
__device__ __forceinline__ float key_value(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Block-wide min and max of the keys.
template <class Src>
__device__ void key_extremes(const Src &key, int64_t n, uint32_t *red, uint32_t *kmin, uint32_t *kmax)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t mn = 0xffffffffu, mx = 0u;
    for_each_key(key, n, [&](int64_t, uint32_t kk) {
        mn = min(mn, kk);
        mx = max(mx, kk);
    });
    mn = wave_min_u(mn);
    mx = wave_max_u(mx);
    if (lane == 0) {
        red[wv] = mn;
        red[kSelWaves + wv] = mx;
    }
    __syncthreads();
    mn = red[0];
    mx = red[kSelWaves];
    for (int q = 1; q < kSelWaves; ++q) {
        mn = min(mn, red[q]);
        mx = max(mx, red[kSelWaves + q]);
    }
    __syncthreads();
    *kmin = mn;
    *kmax = mx;
}

// The q quantile (linear interpolation) of n >= 1 keys with extremes kmin, kmax.
template <class Src>
__device__ float key_quantile(const Src &key, int64_t n, double q, uint32_t kmin, uint32_t kmax, uint32_t *hist,
                              uint32_t *bc, uint32_t *red)
{
    const double h = q * (double)(n - 1);
    const int64_t j = (int64_t)floor(h);
    // x_(j), the (n - j)-th largest; need_eq counts its copies among the n - j largest
    uint32_t thr;
    int64_t need_eq;
    radix_threshold(key, n, n - j, kmin, kmax, hist, bc, &thr, &need_eq);
    __syncthreads();
    const float x = key_value(thr);
    if (j + 1 >= n || need_eq >= 2) return x;  // x_(j+1) = x_(j), or no x_(j+1)
    uint32_t m = 0xffffffffu;
    for_each_key(key, n, [&](int64_t, uint32_t kk) {
        if (kk > thr) m = min(m, kk);
    });
    m = wave_min_u(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    m = red[0];
    for (int w2 = 1; w2 < kSelWaves; ++w2) m = min(m, red[w2]);
    __syncthreads();
    return x + (float)(h - (double)j) * (key_value(m) - x);
}

__global__ __launch_bounds__(kSelThreads) void k_dquant(DQuantArgs a)
{
    __shared__ uint32_t hist[kSelWaves * 256];  // one histogram per wave
    __shared__ uint32_t bc[2];
    __shared__ uint32_t red[2 * kSelWaves];
    const Unit un = unit_of(blockIdx.x, a.Hkv, a.B);
    const int P = a.seq.cu[un.s + 1] - a.seq.cu[un.s] - a.w;
    const float *d = a.d + ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - (int64_t)un.s * a.w);
    const DistKey key{d, 0.f, false};
    uint32_t kmin, kmax;
    key_extremes(key, P, red, &kmin, &kmax);
    float o0, o1;
    if (a.mode == ECOKV_NORM_WINSOR) {
        o0 = key_quantile(key, P, (double)a.q, kmin, kmax, hist, bc, red);
        o1 = key_quantile(key, P, 1.0 - (double)a.q, kmin, kmax, hist, bc, red);
    } else {
        o0 = key_quantile(key, P, 0.5, kmin, kmax, hist, bc, red);  // median
        const DistKey dev{d, o0, true};
        key_extremes(dev, P, red, &kmin, &kmax);
        o1 = key_quantile(dev, P, 0.5, kmin, kmax, hist, bc, red);  // median absolute deviation
    }
    if (threadIdx.x == 0) {
        a.out[2 * (int64_t)blockIdx.x] = o0;
        a.out[2 * (int64_t)blockIdx.x + 1] = o1;
    }
}

// The q quantile of the keys held in registers (extremes kmin, kmax; mm as
// in reg_extremes).
template <int KPT>
__device__ float reg_quantile(const uint32_t (&kk)[KPT], int v0, int n, double q, uint32_t kmin, uint32_t kmax,
                              uint32_t (*hist)[256], uint32_t *hsum, uint32_t (*bc)[2], uint32_t (*mm)[kSelWaves])
{
    const double h = q * (double)(n - 1);
    const int j = (int)floor(h);
    uint32_t thr;
    int need_eq;
    reg_radix_select<KPT>(kk, v0, n, n - j, kmin, kmax, &hist[0][0], hsum, bc, &thr, &need_eq);
    const float x = key_value(thr);
    if (j + 1 >= n || need_eq >= 2) return x;  // x_(j+1) = x_(j), or no x_(j+1)
    uint32_t m = 0xffffffffu;
#pragma unroll
    for (int k = 0; k < KPT; ++k)
        if (v0 + k < n && kk[k] > thr) m = min(m, kk[k]);
    m = wave_min_u(m);
    if ((threadIdx.x & 63) == 0) mm[0][threadIdx.x >> 6] = m;
    __syncthreads();
    m = mm[0][0];
    for (int w2 = 1; w2 < kSelWaves; ++w2) m = min(m, mm[0][w2]);
    __syncthreads();
    return x + (float)(h - (double)j) * (key_value(m) - x);
}

// Register-resident form for units of at most 32 Ki non-window keys: thread t
// holds d_E of keys 32t .. 32t+31 for every pass.
constexpr int kDqKeys = 32 * kSelThreads;

__global__ __launch_bounds__(kSelThreads) void k_dquant_reg(DQuantArgs a)
{
    constexpr int KPT = 32;
    __shared__ uint32_t hist[kSelWaves][256];
    __shared__ uint32_t hsum[256];
    __shared__ uint32_t bc[2][2];
    __shared__ uint32_t mm[2][kSelWaves];
    const Unit un = unit_of(blockIdx.x, a.Hkv, a.B);
    const int P = a.seq.cu[un.s + 1] - a.seq.cu[un.s] - a.w;  // <= kDqKeys (checked on the host)
    const float *d = a.d + ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - (int64_t)un.s * a.w);
    const int v0 = threadIdx.x * KPT;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(uniform_ptr(d)), (short)0, uniform_i32(P) * 4, 0x00020000);
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    float dv[KPT];
    uint32_t kk[KPT];
#pragma unroll
    for (int q = 0; q < KPT / 4; ++q) {
        const f32x4_t x = __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (v0 + 4 * q) * 4, 0, 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) dv[4 * q + e] = x[e];
    }
#pragma unroll
    for (int q = 0; q < KPT; ++q) kk[q] = score_key(dv[q]);
    uint32_t kmin, kmax;
    reg_extremes<KPT>(kk, v0, P, mm, &kmin, &kmax);
    float o0, o1;
    if (a.mode == ECOKV_NORM_WINSOR) {
        o0 = reg_quantile<KPT>(kk, v0, P, (double)a.q, kmin, kmax, hist, hsum, bc, mm);
        o1 = reg_quantile<KPT>(kk, v0, P, 1.0 - (double)a.q, kmin, kmax, hist, hsum, bc, mm);
    } else {
        o0 = reg_quantile<KPT>(kk, v0, P, 0.5, kmin, kmax, hist, hsum, bc, mm);  // median
#pragma unroll
        for (int q = 0; q < KPT; ++q) kk[q] = score_key(fabsf(dv[q] - o0));
        reg_extremes<KPT>(kk, v0, P, mm, &kmin, &kmax);
        o1 = reg_quantile<KPT>(kk, v0, P, 0.5, kmin, kmax, hist, hsum, bc, mm);  // median absolute deviation
    }
    if (threadIdx.x == 0) {
        a.out[2 * (int64_t)blockIdx.x] = o0;
        a.out[2 * (int64_t)blockIdx.x + 1] = o1;
    }
}

hipError_t dquant_launch(const DQuantArgs &a, hipStream_t st)
{
    const unsigned units = (unsigned)(a.L * a.Hkv * a.B);
    if (units == 0) return hipSuccess;
    int maxP = 0;
    for (int s = 0; s < a.B; ++s) maxP = max(maxP, a.seq.cu[s + 1] - a.seq.cu[s] - a.w);
    if (maxP <= kDqKeys)
        ECOKV_TIMED("dquant", st, hipLaunchKernelGGL(k_dquant_reg, dim3(units), dim3(kSelThreads), 0, st, a));
    else
        ECOKV_TIMED("dquant", st, hipLaunchKernelGGL(k_dquant, dim3(units), dim3(kSelThreads), 0, st, a));
    return hipGetLastError();
}


// Exclusive block-wide scan of two uint32 per thread (independent sums);
// returns the exclusive prefixes and the block totals.
__device__ __forceinline__ void block_exscan2(uint32_t x0, uint32_t x1, uint32_t *wsum, uint32_t &e0, uint32_t &e1,
                                              uint32_t &t0, uint32_t &t1)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const uint32_t i0 = wave_incl_scan(x0), i1 = wave_incl_scan(x1);
    if (lane == kWave - 1) {
        wsum[wv] = i0;
        wsum[kSelWaves + 1 + wv] = i1;
    }
    __syncthreads();
    if (wv == 0) {
        uint32_t a0 = lane < kSelWaves ? wsum[lane] : 0u;
        uint32_t a1 = lane < kSelWaves ? wsum[kSelWaves + 1 + lane] : 0u;
        const uint32_t c0 = wave_incl_scan(a0), c1 = wave_incl_scan(a1);  // (lanes past the waves add 0)
        if (lane < kSelWaves) {
            wsum[lane] = c0 - a0;
            wsum[kSelWaves + 1 + lane] = c1 - a1;
        }
        if (lane == kSelWaves - 1) {
            wsum[kSelWaves] = c0;
            wsum[2 * kSelWaves + 1] = c1;
        }
    }
    __syncthreads();
    e0 = wsum[wv] + i0 - x0;
    e1 = wsum[kSelWaves + 1 + wv] + i1 - x1;
    t0 = wsum[kSelWaves];
    t1 = wsum[2 * kSelWaves + 1];
    __syncthreads();
}

// Scores of one selection group: head h's non-window scores at base + h * hstride

// (a single head in per-head mode: no division on that path; a group has at
// most kMaxFlatHeads * 2^31 keys, so the head index fits 32 bits).
struct GroupView {
    const float *base;
    int64_t hstride;
    int P;
    int nh;
    __device__ __forceinline__ float get(int64_t v) const
    {
        if (nh == 1) return base[v];
        const int h = v < 0x7fffffff ? (int)((uint32_t)v / (uint32_t)P) : (int)(v / P);
        return base[(int64_t)h * hstride + (v - (int64_t)h * P)];
    }
};


// The selection group of this block: layer l, heads h0 .. h0+nh-1 of


// Wave 0 (all 64 lanes): the digit of the rem-th largest key from a 256-bin
// histogram h, counts above it into slot[1]; with clear, the bins are zeroed.
__device__ __forceinline__ void pick_digit(uint32_t *h, bool clear, int rem, uint32_t *slot)
{
    const int lane = threadIdx.x & 63;
    // lane owns bins 255-4l .. 252-4l (descending digit order)
    uint32_t c4[4], loc = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        c4[q] = h[255 - 4 * lane - q];
        if (clear) h[255 - 4 * lane - q] = 0u;
        loc += c4[q];
    }
    uint32_t inc = wave_incl_scan(loc);
    const uint32_t before = inc - loc;
    if ((int)before < rem && rem <= (int)inc) {
        uint32_t cum = before;
        for (int q = 0; q < 4; ++q) {
            if ((int)(cum + c4[q]) >= rem) {
                slot[0] = 255u - 4u * lane - q;
                slot[1] = cum;
                break;
            }
            cum += c4[q];
        }
    }
}

// The k-th largest key, as reg_radix_select, for a block whose 128 KiB
// stage (lds) is free during the selection:
//  * first digit: four histograms per wave (lane l of wave w counts into
//    histogram 4 w + l % 4; 257 words apart, so lanes that share a digit hit
//    different banks), folded by 256 threads;
//  * then the keys that still carry the chosen prefix -- usually a small part
//    of the group -- are gathered into the stage (a wave scan of the
//    per-thread counts and one LDS atomic per wave place them), and the later
//    digits count only them, into one shared histogram that the scanning wave
//    reads and clears: two barriers per digit and no fold.  When they do not
//    fit, the later digits count the registers into that histogram instead.
constexpr int kStHistC = 4;
constexpr int kStHistWords = kSelWaves * kStHistC * 257;
constexpr int kStCandOff = kStHistWords + 256;
constexpr int kStCandCap = 32 * kSelThreads - kStCandOff;

template <int KPT>
__device__ __forceinline__ void reg_radix_select_staged(const uint32_t (&kk)[KPT], int v0, int n, int k,
                                                        uint32_t kmin, uint32_t kmax, uint32_t *lds,
                                                        uint32_t *hsum, uint32_t (*bc)[2], uint32_t *ccount,
                                                        uint32_t *thr_out, int *need_eq_out)
{
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const uint32_t diff = kmin ^ kmax;
    if (diff == 0) {
        *thr_out = kmin;
        *need_eq_out = k;
        return;
    }
    int hi = 31 - __clz(diff);
    uint32_t mask = hi == 31 ? 0u : ~((2u << hi) - 1u);
    uint32_t prefix = kmin & mask;
    int rem = k;
    uint32_t *const h1 = lds + kStHistWords;
    uint32_t *const cand = lds + kStCandOff;
    for (int b = tid; b < kStHistWords + 256; b += blockDim.x) lds[b] = 0u;
    if (tid == 0) *ccount = 0u;
    __syncthreads();
    {
        // first digit (every key lies in [kmin, kmax], so all carry the prefix)
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t nb = 1u << (hi - lo + 1);
        uint32_t *const myh = lds + (wv * kStHistC + (lane & (kStHistC - 1))) * 257;
#pragma unroll
        for (int q = 0; q < KPT; ++q)
            if (v0 + q < n) atomicAdd(&myh[(kk[q] >> lo) & (nb - 1u)], 1u);
        __syncthreads();
        if (tid < 256) {
            uint32_t c = 0;
#pragma unroll 8
            for (int w2 = 0; w2 < kSelWaves * kStHistC; ++w2) c += lds[w2 * 257 + tid];
            hsum[tid] = c;
        }
        __syncthreads();
        if (tid < kWave) pick_digit(hsum, false, rem, bc[0]);
        __syncthreads();
        prefix |= bc[0][0] << lo;
        rem -= (int)bc[0][1];
        mask |= (nb - 1u) << lo;
        hi = lo - 1;
    }
    if (hi >= 0) {
        // gather the keys that carry the prefix
        uint32_t cnt = 0;
#pragma unroll
        for (int q = 0; q < KPT; ++q) cnt += (v0 + q < n && (kk[q] & mask) == prefix) ? 1u : 0u;
        uint32_t inc = wave_incl_scan(cnt);
        const uint32_t wtot = (uint32_t)__builtin_amdgcn_readlane((int)inc, kWave - 1);
        uint32_t base = 0;
        if (lane == kWave - 1 && wtot > 0) base = atomicAdd(ccount, wtot);
        base = (uint32_t)__builtin_amdgcn_readlane((int)base, kWave - 1);
        uint32_t pos = base + inc - cnt;
#pragma unroll
        for (int q = 0; q < KPT; ++q)
            if (v0 + q < n && (kk[q] & mask) == prefix) {
                if (pos < (uint32_t)kStCandCap) cand[pos] = kk[q];
                ++pos;
            }
        __syncthreads();
        const uint32_t ncand = *ccount;
        const bool use_cand = ncand <= (uint32_t)kStCandCap;
        int par = 1;
        while (hi >= 0) {
            const int lo = hi >= 7 ? hi - 7 : 0;
            const uint32_t nb = 1u << (hi - lo + 1);
            if (use_cand) {
                for (uint32_t i = tid; i < ncand; i += kSelThreads) {
                    const uint32_t key = cand[i];
                    if ((key & mask) == prefix) atomicAdd(&h1[(key >> lo) & (nb - 1u)], 1u);
                }
            } else {
#pragma unroll
                for (int q = 0; q < KPT; ++q)
                    if (v0 + q < n && (kk[q] & mask) == prefix) atomicAdd(&h1[(kk[q] >> lo) & (nb - 1u)], 1u);
            }
            __syncthreads();
            if (tid < kWave) pick_digit(h1, true, rem, bc[par]);
            __syncthreads();
            prefix |= bc[par][0] << lo;
            rem -= (int)bc[par][1];
            mask |= (nb - 1u) << lo;
            hi = lo - 1;
            par ^= 1;
        }
    }
    *thr_out = prefix;
    *need_eq_out = rem;
}


// Ordered emission of one head's chosen keys from the registers (thread t
// holds keys v0 .. v0+KPT-1 of n): bit q of gtm[c] / eqm[c] marks key
// v0 + 32 c + q above / equal to the threshold; the thread's taken keys go to
// consecutive slots from the number taken before its run, put(slot, key
// index); equal keys are taken in key order while fewer than need_eq precede
// them.
template <int KPT, class F>
__device__ __forceinline__ void emit_ordered(const uint32_t (&kk)[KPT], int v0, int n, uint32_t thr, int need_eq,
                                             uint32_t *wsum, F &&put)
{
    constexpr int NC = (KPT + 31) / 32;      // 32-key words per thread
    constexpr int QW = KPT < 32 ? KPT : 32;  // keys per word
    uint32_t gtm[NC], eqm[NC];
    uint32_t cg = 0, ce = 0;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        gtm[c] = 0u;
        eqm[c] = 0u;
#pragma unroll
        for (int q = 0; q < QW; ++q)
            if (v0 + 32 * c + q < n) {
                gtm[c] |= kk[32 * c + q] > thr ? 1u << q : 0u;
                eqm[c] |= kk[32 * c + q] == thr ? 1u << q : 0u;
            }
        cg += (uint32_t)__builtin_popcount(gtm[c]);
        ce += (uint32_t)__builtin_popcount(eqm[c]);
    }
    uint32_t eg, ee, tg, te;
    block_exscan2(cg, ce, wsum, eg, ee, tg, te);
    (void)tg;
    (void)te;
    const int eq_take = min((int)ce, max(need_eq - (int)ee, 0));
    uint32_t take[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) take[c] = gtm[c];
    for (int r = 0; r < eq_take; ++r) {
        bool done = false;
#pragma unroll
        for (int c = 0; c < NC; ++c)
            if (!done && eqm[c]) {
                const uint32_t low = eqm[c] & (~eqm[c] + 1u);
                take[c] |= low;
                eqm[c] ^= low;
                done = true;
            }
    }
    int o = (int)eg + min((int)ee, need_eq);
#pragma unroll
    for (int c = 0; c < NC; ++c)
        while (take[c]) {
            const int q = 32 * c + __builtin_ctz(take[c]);
            take[c] &= take[c] - 1u;
            put(o, v0 + q);
            ++o;
        }
}

// ---------------------------------------------------------------------------
// One block per group, for groups of up to 32 Ki keys (each a handful of
// launches' worth of work for the multi-block form below): thread t owns the
// contiguous run [t*KPT, t*KPT + KPT) of the group's keys in registers
// (16-byte loads in per-head mode), the radix passes histogram them into one
// LDS copy per wave, and the ordered emission walks the registers.
// ---------------------------------------------------------------------------

template <int KPT>
__global__ __launch_bounds__(kSelThreads) void k_select_reg(SelectArgs a)
{
    // the radix histograms and the gathered keys live in stg
    __shared__ uint32_t hsum[256];
    __shared__ uint32_t bc[2][2];
    __shared__ uint32_t wsum[2 * kSelWaves + 2];
    __shared__ uint32_t mm[2][kSelWaves];
    __shared__ uint32_t ccount;
    __shared__ int64_t through[kMaxFlatHeads];
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    // 128 KiB: with KPT == 32 the stage of the coalesced score load, then of
    // the radix histograms and gathered keys, then of the output (the
    // barriers of the extremes and of the radix passes separate the three
    // uses); with KPT == 64 the radix scratch only
    __shared__ u32x4_t stg[8 * kSelThreads];
    static_assert(kStCandCap > 0, "histograms must fit the stage");

    const SelGroup grp = sel_group(a, blockIdx.x);
    const int l = grp.l, h0 = grp.h0, s = grp.s, nh = grp.nh;
    const int T = a.seq.cu[s + 1] - a.seq.cu[s];
    const int P = T - a.w;
    const int beff = grp.beff;
    const int64_t out_base = grp.out_base;
    int32_t *out = a.idx + out_base;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    if (beff >= T) {  // keep every token
        for (int64_t e = tid; e < (int64_t)nh * T; e += blockDim.x) out[e] = (int32_t)(e % T);
        if (tid < nh && (a.counts || a.offsets)) {
            const int64_t u = ((int64_t)l * a.Hkv + h0 + tid) * a.B + s;
            if (a.counts) a.counts[u] = T;
            if (a.offsets) a.offsets[u] = (int32_t)(out_base + (int64_t)tid * T);
        }
        return;
    }

    GroupView g;
    g.base = a.scores + ((int64_t)l * a.Hkv + h0) * a.Ptot + (a.seq.cu[s] - s * a.w);
    g.hstride = a.Ptot;
    g.P = P;
    g.nh = nh;
    const int n = nh * P;  // <= KPT * kSelThreads (chosen on the host)
    const int k = nh * (beff - a.w);
    const int v0 = tid * KPT;

    for (int h = tid; h < nh; h += blockDim.x) through[h] = 0;
    uint32_t kk[KPT];
    bool ext_done = false;  // the extremes are in mm (reduced with the load's barrier)
    if (nh == 1 && KPT == 32) {
        // Coalesced load through LDS: the block reads the group's scores as
        // consecutive 16-byte pieces (1 KiB per wave instruction) into a
        // swizzled stage (piece g at g ^ ((g >> 3) & 7)), then each thread takes
        // its 32 consecutive scores from it.
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(uniform_ptr(g.base)), (short)0, uniform_i32(n) * 4, 0x00020000);
        u32x4_t x[KPT / 4];
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q)
            x[q] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (q * kSelThreads + tid) * 16, 0, 0));
        // the extremes of the loaded keys (the same set as the thread's run
        // after the stage) ride on the stage's barrier
        uint32_t lmin = 0xffffffffu, lmax = 0u;
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if ((q * kSelThreads + tid) * 4 + e < n) {
                    const uint32_t kv = score_key(__uint_as_float(x[q][e]));
                    lmin = min(lmin, kv);
                    lmax = max(lmax, kv);
                }
        lmin = wave_min_u(lmin);
        lmax = wave_max_u(lmax);
        if (lane == 0) {
            mm[0][wv] = lmin;
            mm[1][wv] = lmax;
        }
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) stg[q * kSelThreads + (tid ^ ((tid >> 3) & 7))] = x[q];
        lds_barrier();
        ext_done = true;
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) {
            const u32x4_t y = stg[(KPT / 4) * tid + (q ^ (tid & 7))];
#pragma unroll
            for (int e = 0; e < 4; ++e) kk[4 * q + e] = score_key(__uint_as_float(y[e]));
        }
    } else if (nh == 1) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(uniform_ptr(g.base)), (short)0, uniform_i32(n) * 4, 0x00020000);
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) {
            const u32x4_t x = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (v0 + 4 * q) * 4, 0, 0));
#pragma unroll
            for (int e = 0; e < 4; ++e) kk[4 * q + e] = score_key(__uint_as_float(x[e]));
        }
    } else {
#pragma unroll
        for (int q = 0; q < KPT; ++q) kk[q] = v0 + q < n ? score_key(g.get(v0 + q)) : 0u;
    }

    // KPT == 32: the ordered output is assembled in LDS and written out in
    // consecutive 4-byte pieces (instead of each thread's scattered stores)
    uint32_t *ost = reinterpret_cast<uint32_t *>(stg);
    const bool staged = KPT == 32 && k + nh * a.w <= KPT * kSelThreads;
    uint32_t thr = 0xffffffffu;
    int need_eq = 0;
    if (k > 0) {
        uint32_t kmin, kmax;
        if (ext_done) {
            kmin = mm[0][0];
            kmax = mm[1][0];
            for (int q = 1; q < kSelWaves; ++q) {
                kmin = min(kmin, mm[0][q]);
                kmax = max(kmax, mm[1][q]);
            }
        } else {
            reg_extremes<KPT>(kk, v0, n, mm, &kmin, &kmax);
        }
        // radix select of the k-th largest key
        reg_radix_select_staged<KPT>(kk, v0, n, k, kmin, kmax, reinterpret_cast<uint32_t *>(stg), hsum, bc, &ccount,
                                     &thr, &need_eq);
    }
    if (k > 0 && nh == 1) {
        // ordered emission of one head
        emit_ordered<KPT>(kk, v0, n, thr, need_eq, wsum, [&](int o, int v) {
            if (staged) ost[o] = (uint32_t)v;
            else out[o] = v;
        });
        if (tid == 0) through[0] = k;
    } else if (k > 0) {
        // ordered emission from the registers (several heads)
        uint32_t cg = 0, ce = 0;
#pragma unroll
        for (int q = 0; q < KPT; ++q)
            if (v0 + q < n) {
                cg += kk[q] > thr;
                ce += kk[q] == thr;
            }
        uint32_t eg, ee, tg, te;
        block_exscan2(cg, ce, wsum, eg, ee, tg, te);
        (void)tg;
        (void)te;
        int gt_before = (int)eg, eq_before = (int)ee;
        int h = nh == 1 ? 0 : (v0 < n ? v0 / P : nh);
        int pos = v0 - h * P;
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
            if (v0 + q < n) {
                const bool gt = kk[q] > thr, eq = kk[q] == thr;
                const bool take = gt || (eq && eq_before < need_eq);
                if (take) {
                    const int64_t o = gt_before + min(eq_before, need_eq) + (int64_t)h * a.w;
                    if (staged) ost[o] = (uint32_t)pos;
                    else out[o] = pos;
                }
                gt_before += gt;
                eq_before += eq;
                if (++pos == P) {
                    through[h] = gt_before + min(eq_before, need_eq);
                    pos = 0;
                    ++h;
                }
            }
        }
    }
    __syncthreads();
    // windows, counts and offsets
    for (int e = tid; e < nh * a.w; e += blockDim.x) {
        const int hh = e / a.w, j = e % a.w;
        const int64_t o = through[hh] + (int64_t)hh * a.w + j;
        if (staged) ost[o] = (uint32_t)(P + j);
        else out[o] = P + j;
    }
    if (staged) {
        __syncthreads();
        for (int e = tid; e < k + nh * a.w; e += blockDim.x) out[e] = (int32_t)ost[e];
    }
    if (tid < nh && (a.counts || a.offsets)) {
        const int hh = tid;
        const int64_t prev = hh > 0 ? through[hh - 1] : 0;
        const int64_t u = ((int64_t)l * a.Hkv + h0 + hh) * a.B + s;
        if (a.counts) a.counts[u] = (int32_t)(through[hh] - prev + a.w);
        if (a.offsets) a.offsets[u] = (int32_t)(out_base + prev + (int64_t)hh * a.w);
    }
}

// ---------------------------------------------------------------------------
// Two-stage selection of single-head groups longer than one block's registers
// when their budget is small.  The group's k chosen keys are the k largest
// under the order (key descending, position ascending); restricted to one
// slice they are that slice's largest, at most min(k, slice) of them.  So:
//   stage 1  one block per slice of kCandSlice keys selects the slice's own
//            min(k, n_slice) largest (the radix select and tie rule of the
//            one-block form) and writes their keys and positions, ascending;
//   stage 2  one block per group reads its slices' candidates in slice
//            order -- ascending position, so equal keys still favour the
//            smaller position -- selects the k largest among them and writes
//            their positions.
// Used when the candidates of every group fit one block's registers (32-head
// layer of 65536 tokens, budget 2048: 8 slices of 2040 candidates).
// ---------------------------------------------------------------------------
constexpr int kCandKPT = 8;
constexpr int kCandSlice = kCandKPT * kSelThreads;  // 8192 keys

// The scores of single-head group grp.
__device__ __forceinline__ const float *head_scores(const SelectArgs &a, const SelGroup &grp)
{
    return a.scores + ((int64_t)grp.l * a.Hkv + grp.h0) * a.Ptot + (a.seq.cu[grp.s] - grp.s * a.w);
}

__global__ __launch_bounds__(kSelThreads) void k_sel_cand(SelectArgs a)
{
    __shared__ uint32_t hsum[256];
    __shared__ uint32_t bc[2][2];
    __shared__ uint32_t wsum[2 * kSelWaves + 2];
    __shared__ uint32_t mm[2][kSelWaves];
    __shared__ uint32_t ccount;
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    __shared__ u32x4_t stg[8 * kSelThreads];  // the radix scratch
    const int gi = blockIdx.x / a.c_slices, j = blockIdx.x - gi * a.c_slices;
    const SelGroup grp = sel_group(a, gi);
    const int T = a.seq.cu[grp.s + 1] - a.seq.cu[grp.s];
    const int P = T - a.w;
    const int k = grp.beff - a.w;
    const int s0 = j * kCandSlice;
    if (grp.beff >= T || k <= 0 || s0 >= P) return;  // (stage 2 writes those groups)
    const int n = min(kCandSlice, P - s0);
    const int tid = threadIdx.x, v0 = tid * kCandKPT;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(uniform_ptr(head_scores(a, grp) + s0)), (short)0, uniform_i32(n) * 4, 0x00020000);
    uint32_t kk[kCandKPT];
#pragma unroll
    for (int q = 0; q < kCandKPT / 4; ++q) {
        const u32x4_t x = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (v0 + 4 * q) * 4, 0, 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) kk[4 * q + e] = score_key(__uint_as_float(x[e]));
    }
    uint32_t kmin, kmax, thr;
    int need_eq;
    reg_extremes<kCandKPT>(kk, v0, n, mm, &kmin, &kmax);
    reg_radix_select_staged<kCandKPT>(kk, v0, n, min(k, n), kmin, kmax, reinterpret_cast<uint32_t *>(stg), hsum, bc,
                                      &ccount, &thr, &need_eq);
    // the keys through LDS (free again after the selection), so that the
    // emission can write each chosen key beside its position
    uint32_t *kst = reinterpret_cast<uint32_t *>(stg);
#pragma unroll
    for (int q = 0; q < kCandKPT; ++q) kst[v0 + q] = kk[q];
    __syncthreads();
    // slice j's candidates follow those of the slices before it (each but
    // the last has min(k, kCandSlice) of them)
    const int64_t cb = (int64_t)gi * a.c_slices * kCandSlice + (int64_t)j * min(k, kCandSlice);
    int32_t *cp = a.c_pos + cb;
    uint32_t *ck = a.c_key + cb;
    emit_ordered<kCandKPT>(kk, v0, n, thr, need_eq, wsum, [&](int o, int v) {
        cp[o] = s0 + v;
        ck[o] = kst[v];
    });
}

template <int KPT>
__global__ __launch_bounds__(kSelThreads) void k_sel_final(SelectArgs a)
{
    __shared__ uint32_t hsum[256];
    __shared__ uint32_t bc[2][2];
    __shared__ uint32_t wsum[2 * kSelWaves + 2];
    __shared__ uint32_t mm[2][kSelWaves];
    __shared__ uint32_t ccount;
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    __shared__ u32x4_t stg[8 * kSelThreads];  // the radix scratch
    const int gi = blockIdx.x;
    const SelGroup grp = sel_group(a, gi);
    const int T = a.seq.cu[grp.s + 1] - a.seq.cu[grp.s];
    const int P = T - a.w;
    int32_t *out = a.idx + grp.out_base;
    const int tid = threadIdx.x;
    const int64_t u = ((int64_t)grp.l * a.Hkv + grp.h0) * a.B + grp.s;
    if (grp.beff >= T) {  // keep every token
        for (int e = tid; e < T; e += blockDim.x) out[e] = e;
        if (tid == 0) {
            if (a.counts) a.counts[u] = T;
            if (a.offsets) a.offsets[u] = (int32_t)grp.out_base;
        }
        return;
    }
    const int k = grp.beff - a.w;
    if (k > 0) {
        const int ns = (P + kCandSlice - 1) / kCandSlice;
        const int kfull = min(k, kCandSlice);                        // candidates of each slice but the last
        const int nc = (ns - 1) * kfull + min(k, P - (ns - 1) * kCandSlice);  // <= KPT * kSelThreads (host)
        // the candidates lie contiguously, in slice order: thread t takes
        // candidates KPT t .. KPT t + KPT - 1 with 16-byte loads
        const int64_t cb = (int64_t)gi * a.c_slices * kCandSlice;
        const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
            uniform_ptr(a.c_key + cb), (short)0, uniform_i32(nc) * 4, 0x00020000);
        const int v0 = tid * KPT;
        uint32_t kk[KPT];
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) {
            const u32x4_t x = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rk, (v0 + 4 * q) * 4, 0, 0));
#pragma unroll
            for (int e = 0; e < 4; ++e) kk[4 * q + e] = x[e];
        }
        uint32_t kmin, kmax, thr;
        int need_eq;
        reg_extremes<KPT>(kk, v0, nc, mm, &kmin, &kmax);
        reg_radix_select_staged<KPT>(kk, v0, nc, k, kmin, kmax, reinterpret_cast<uint32_t *>(stg), hsum, bc, &ccount,
                                     &thr, &need_eq);
        emit_ordered<KPT>(kk, v0, nc, thr, need_eq, wsum, [&](int o, int v) { out[o] = a.c_pos[cb + v]; });
    }
    // the window, count and offset
    for (int e = tid; e < a.w; e += blockDim.x) out[max(k, 0) + e] = P + e;
    if (tid == 0) {
        if (a.counts) a.counts[u] = max(k, 0) + a.w;
        if (a.offsets) a.offsets[u] = (int32_t)grp.out_base;
    }
}

// ---------------------------------------------------------------------------
// Selection over many blocks per group.  A group's n keys, in (head,
// position) order, are cut into slices of kMbThreads * KPT keys, one block
// each; thread t of a slice owns KPT consecutive keys.  Five launches in
// stream order, in which no block ever waits for another:
//   digit 0..2  every block histograms one digit (key bits 31..21, 20..10,
//               9..0) of its keys that carry the prefix found so far into
//               LDS and adds the histogram into the group's global one with
//               atomics; the blocks of the next launch each read that
//               histogram and derive the same digit of the k-th largest key,
//               and block 0 of the group records the state;
//   count       per slice, the keys above and equal to the threshold (per
//               head too, in layer-flat groups);
//   emit        each slice adds up the counts of the slices before it and
//               writes its taken positions in order; block 0 of the group
//               writes the windows, counts and offsets.
// A global histogram and the per-head counts are cleared by the launch after
// their last reader, so the workspace ends as zero-filled as it started.
// When the chosen bin of a digit is taken whole, the later digits are
// skipped and the key class under the prefix so far is the threshold class.
// ---------------------------------------------------------------------------
constexpr int kMbThreads = 256;
constexpr int kMbWaves = kMbThreads / kWave;
constexpr int kMbHistWords = 2048 + 2048 + 1024;  // global histogram words per group

__device__ __forceinline__ int mb_bins(int d) { return d == 2 ? 1024 : 2048; }
__device__ __forceinline__ int mb_lo(int d) { return d == 0 ? 21 : (d == 1 ? 10 : 0); }
__device__ __forceinline__ int mb_hoff(int d) { return d == 0 ? 0 : (d == 1 ? 2048 : 4096); }

// Geometry of the group of this block.
struct MbGroup {
    SelGroup sg;
    int T, P;
    int64_t n, k;       // keys of the group and how many of them are taken
    const float *base;  // head h0's scores; head h0 + h at base + h * hstride
    int64_t hstride;
    __amdgpu_buffer_rsrc_t rs;  // every score of the group
};

__device__ __forceinline__ MbGroup mb_group(const SelectArgs &a, int gi)
{
    MbGroup g;
    g.sg = sel_group(a, gi);
    g.T = a.seq.cu[g.sg.s + 1] - a.seq.cu[g.sg.s];
    g.P = g.T - a.w;
    g.n = (int64_t)g.sg.nh * g.P;
    g.k = (int64_t)g.sg.nh * (g.sg.beff - a.w);
    g.base = a.scores + ((int64_t)g.sg.l * a.Hkv + g.sg.h0) * a.Ptot + (a.seq.cu[g.sg.s] - g.sg.s * a.w);
    g.hstride = a.Ptot;
    // bytes from base to the end of the last head's scores (< 2^31, checked on the host)
    const int bytes = (int)(((int64_t)(g.sg.nh - 1) * g.hstride + g.P) * 4);
    g.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(uniform_ptr(g.base)), (short)0, uniform_i32(bytes),
                                             0x00020000);
    return g;
}

typedef float f32x4s __attribute__((ext_vector_type(4)));

// Keys r0 .. r0+KPT-1 of the group (those at or past n are marked invalid and
// read as 0), and the (head, position) of r0.
template <int KPT>
__device__ __forceinline__ void mb_load(const MbGroup &g, int64_t r0, uint32_t (&kk)[KPT], int &h0, int &i0)
{
    int h = g.sg.nh == 1 ? 0 : (int)(r0 / g.P);
    int i = (int)(r0 - (int64_t)h * g.P);
    h0 = h;
    i0 = i;
    if (i + KPT <= g.P && r0 + KPT <= g.n) {
        // one head, all keys valid: 16-byte loads
        const int off = (int)((int64_t)h * g.hstride + i) * 4;
#pragma unroll
        for (int q = 0; q < KPT / 4; ++q) {
            const f32x4s x = __builtin_bit_cast(f32x4s, __builtin_amdgcn_raw_buffer_load_b128(g.rs, off + 16 * q, 0, 0));
#pragma unroll
            for (int e = 0; e < 4; ++e) kk[4 * q + e] = score_key(x[e]);
        }
    } else {
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
            if (r0 + q < g.n) {
                const float x = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(g.rs, (int)((int64_t)h * g.hstride + i) * 4, 0, 0));
                kk[q] = score_key(x);
                if (++i == g.P) {
                    i = 0;
                    ++h;
                }
            } else {
                kk[q] = 0u;
            }
        }
    }
}

// Exclusive scan of one uint32 per thread over the block (kMbThreads
// threads); returns the thread's prefix, *total the block total.
__device__ __forceinline__ uint32_t mb_exscan(uint32_t x, uint32_t *ws, uint32_t *total)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t inc = wave_incl_scan(x);
    if (lane == kWave - 1) ws[wv] = inc;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int w2 = 0; w2 < kMbWaves; ++w2) {
        const uint32_t v = ws[w2];
        before += w2 < wv ? v : 0u;
        tot += v;
    }
    __syncthreads();
    *total = tot;
    return before + inc - x;
}

// The selection state after digit d (0..2) from the state before it and the
// group's global histogram of digit d: the digit holding the rem-th largest
// key of the class under the prefix.  Every block derives the same state.
// st: x prefix, y mask, z keys still to take from the class, w 1 when the
// chosen bin is taken whole (the later digits are then skipped).
__device__ uint4 mb_advance(uint4 st, const uint32_t *gh, int d, uint32_t *sh)
{
    const int nb = mb_bins(d), per = nb / kMbThreads;
    const int t = threadIdx.x;
    // thread t: bins nb-1-per*t .. nb-per*(t+1), in descending digit order,
    // read as 16-byte pieces (the histogram was completed by an earlier launch;
    // read before st is looked at, so that these loads overlap the state's)
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    const u32x4_t *src = reinterpret_cast<const u32x4_t *>(gh + nb - per * (t + 1));
    u32x4_t v0 = src[0], v1 = per == 8 ? src[1] : (u32x4_t){0u, 0u, 0u, 0u};
    if (st.w) return st;
    // descending order: the last bin of the piece first
    uint32_t c[8] = {per == 8 ? v1[3] : v0[3], per == 8 ? v1[2] : v0[2], per == 8 ? v1[1] : v0[1],
                     per == 8 ? v1[0] : v0[0], v0[3], v0[2], v0[1], v0[0]};
    if (per == 4) c[4] = c[5] = c[6] = c[7] = 0u;
    uint32_t loc = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) loc += c[q];
    uint32_t total;
    const uint32_t before = mb_exscan(loc, sh, &total);
    const uint32_t rem = st.z;
    if (before < rem && rem <= before + loc) {
        uint32_t cum = before;
        for (int q = 0; q < per; ++q) {
            if (cum + c[q] >= rem) {
                sh[kMbWaves] = (uint32_t)(nb - 1 - per * t - q);  // digit
                sh[kMbWaves + 1] = cum;                          // keys of the class above the bin
                sh[kMbWaves + 2] = c[q];                         // keys in the bin
                break;
            }
            cum += c[q];
        }
    }
    __syncthreads();
    const uint32_t dig = sh[kMbWaves], above = sh[kMbWaves + 1], inbin = sh[kMbWaves + 2];
    __syncthreads();
    uint4 r;
    r.x = st.x | (dig << mb_lo(d));
    r.y = st.y | ((uint32_t)(nb - 1) << mb_lo(d));
    r.z = rem - above;
    r.w = r.z == inbin ? 1u : 0u;
    return r;
}

// Clear this block's share of global histogram d of group gi (slices ns).
__device__ __forceinline__ void mb_clear(const SelectArgs &a, int gi, int j, int ns, int d)
{
    uint32_t *gh = a.mb_hist + (int64_t)gi * kMbHistWords + mb_hoff(d);
    const int nb = mb_bins(d);
    for (int b = j * kMbThreads + threadIdx.x; b < nb; b += ns * kMbThreads) gh[b] = 0u;
}

// The state before digit DIG (DIG = 0 .. 3): derived from the histogram of
// digit DIG-1 and the state recorded before it; block 0 records it.
template <int DIG>
__device__ __forceinline__ uint4 mb_state(const SelectArgs &a, int gi, int j, int64_t k, uint32_t *sh)
{
    uint4 st = {0u, 0u, (uint32_t)k, 0u};
    if constexpr (DIG > 0) {
        if (DIG > 1) st = a.mb_state[(int64_t)(DIG - 2) * a.mb_groups + gi];
        st = mb_advance(st, a.mb_hist + (int64_t)gi * kMbHistWords + mb_hoff(DIG - 1), DIG - 1, sh);
        if (j == 0 && threadIdx.x == 0) a.mb_state[(int64_t)(DIG - 1) * a.mb_groups + gi] = st;
    }
    return st;
}

// Slices of group g (of kMbThreads * KPT keys).
template <int KPT>
__device__ __forceinline__ int mb_slices(const MbGroup &g)
{
    return (int)((g.n + kMbThreads * KPT - 1) / (kMbThreads * KPT));
}

// Histogram of digit DIG of the keys that carry the prefix.
template <int KPT, int DIG>
__global__ __launch_bounds__(kMbThreads) void k_sel_digit(SelectArgs a)
{
    __shared__ __attribute__((aligned(16))) uint32_t hist[kMbWaves][2048];
    __shared__ uint32_t sh[kMbWaves + 4];
    const int gi = blockIdx.x / a.mb_slices, j = blockIdx.x - gi * a.mb_slices;
    const MbGroup g = mb_group(a, gi);
    if (g.sg.beff >= g.T || g.k <= 0) return;
    const int ns = mb_slices<KPT>(g);
    if (j >= ns) return;
    const int t = threadIdx.x, wv = t >> 6;
    // the keys first, so that their loads overlap those of the state and histogram
    const int64_t r0 = (int64_t)j * kMbThreads * KPT + (int64_t)t * KPT;
    uint32_t kk[KPT];
    int hh, ii;
    if (r0 < g.n) mb_load<KPT>(g, r0, kk, hh, ii);
    // the LDS histograms are cleared while the keys and the state are in
    // flight (the state's block scan orders the clear before the counts)
    {
        typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
        u32x4_t *h4 = reinterpret_cast<u32x4_t *>(&hist[0][0]);
        for (int b = t; b < kMbWaves * 2048 / 4; b += kMbThreads) h4[b] = (u32x4_t){0u, 0u, 0u, 0u};
    }
    const uint4 st = mb_state<DIG>(a, gi, j, g.k, sh);
    if (DIG == 2) mb_clear(a, gi, j, ns, 0);  // digit 0's histogram: its last reader was the previous launch
    if (st.w) return;
    const int nb = mb_bins(DIG), lo = mb_lo(DIG);
    if (DIG == 0) __syncthreads();
    if (r0 < g.n) {
#pragma unroll
        for (int q = 0; q < KPT; ++q)
            if (r0 + q < g.n && (kk[q] & st.y) == st.x) atomicAdd(&hist[wv][(kk[q] >> lo) & (uint32_t)(nb - 1)], 1u);
    }
    __syncthreads();
    uint32_t *gh = a.mb_hist + (int64_t)gi * kMbHistWords + mb_hoff(DIG);
    for (int b = t; b < nb; b += kMbThreads) {
        uint32_t c = 0;
#pragma unroll
        for (int w2 = 0; w2 < kMbWaves; ++w2) c += hist[w2][b];
        if (c) __hip_atomic_fetch_add(&gh[b], c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The final threshold; per slice the keys above and equal to it; in
// layer-flat groups the same per head.
template <int KPT>
__global__ __launch_bounds__(kMbThreads) void k_sel_count(SelectArgs a)
{
    __shared__ uint32_t sh[kMbWaves + 4];
    __shared__ uint32_t hc[kMaxFlatHeads][2];
    const int gi = blockIdx.x / a.mb_slices, j = blockIdx.x - gi * a.mb_slices;
    const MbGroup g = mb_group(a, gi);
    if (g.sg.beff >= g.T || g.k <= 0) return;
    const int ns = mb_slices<KPT>(g);
    if (j >= ns) return;
    const int t = threadIdx.x;
    const int64_t r0 = (int64_t)j * kMbThreads * KPT + (int64_t)t * KPT;
    uint32_t kk[KPT];
    int h = 0, i = 0;
    if (r0 < g.n) mb_load<KPT>(g, r0, kk, h, i);  // (overlaps the state's loads)
    const uint4 st = mb_state<3>(a, gi, j, g.k, sh);
    mb_clear(a, gi, j, ns, 1);  // digit 1's histogram: last read by the previous launch
    const bool flat = g.sg.nh > 1;
    if (flat)
        for (int hh = t; hh < g.sg.nh; hh += kMbThreads) hc[hh][0] = hc[hh][1] = 0u;
    __syncthreads();
    uint32_t cg = 0, ce = 0, hg = 0, he = 0;
    if (r0 < g.n) {
#pragma unroll
        for (int q = 0; q < KPT; ++q) {
            if (r0 + q >= g.n) break;
            const uint32_t m = kk[q] & st.y;
            const uint32_t gt = m > st.x, eq = m == st.x;
            cg += gt;
            ce += eq;
            if (flat) {
                hg += gt;
                he += eq;
                if (++i == g.P || r0 + q + 1 == g.n || q == KPT - 1) {
                    if (hg) atomicAdd(&hc[h][0], hg);
                    if (he) atomicAdd(&hc[h][1], he);
                    hg = he = 0;
                    if (i == g.P) {
                        i = 0;
                        ++h;
                    }
                }
            }
        }
    }
    uint32_t tg, te;
    (void)mb_exscan(cg, sh, &tg);
    (void)mb_exscan(ce, sh, &te);
    if (t == 0) {
        uint32_t *c = a.mb_cnt + ((int64_t)gi * a.mb_slices + j) * 2;
        c[0] = tg;
        c[1] = te;
    }
    if (flat) {
        __syncthreads();
        uint32_t *gc = a.mb_head + (int64_t)gi * kMaxFlatHeads * 2;
        for (int hh = t; hh < g.sg.nh; hh += kMbThreads) {
            if (hc[hh][0]) __hip_atomic_fetch_add(&gc[2 * hh], hc[hh][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (hc[hh][1]) __hip_atomic_fetch_add(&gc[2 * hh + 1], hc[hh][1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Ordered emission of the taken positions; windows, counts and offsets.
template <int KPT>
__global__ __launch_bounds__(kMbThreads) void k_sel_emit(SelectArgs a)
{
    __shared__ uint32_t sh[kMbWaves + 4];
    __shared__ uint32_t red[2][kMbWaves];
    __shared__ int64_t through[kMaxFlatHeads];
    const int gi = blockIdx.x / a.mb_slices, j = blockIdx.x - gi * a.mb_slices;
    const MbGroup g = mb_group(a, gi);
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int nh = g.sg.nh, T = g.T, P = g.P, w = a.w;
    int32_t *out = a.idx + g.sg.out_base;
    const int ns = max(1, mb_slices<KPT>(g));
    if (j >= ns) return;
    auto unit_of_head = [&](int hh) { return ((int64_t)g.sg.l * a.Hkv + g.sg.h0 + hh) * a.B + g.sg.s; };
    if (g.sg.beff >= T) {  // keep every token
        for (int64_t e = (int64_t)j * kMbThreads + t; e < (int64_t)nh * T; e += (int64_t)ns * kMbThreads)
            out[e] = (int32_t)(e % T);
        if (j == 0 && t < nh) {
            if (a.counts) a.counts[unit_of_head(t)] = T;
            if (a.offsets) a.offsets[unit_of_head(t)] = (int32_t)(g.sg.out_base + (int64_t)t * T);
        }
        return;
    }
    if (g.k > 0) {
        mb_clear(a, gi, j, ns, 2);  // digit 2's histogram: last read by the count launch
        const uint4 st = a.mb_state[2 * (int64_t)a.mb_groups + gi];
        const int64_t need_eq = st.z;
        const int64_t nentries = g.k + (int64_t)nh * w;
        // keys above / equal to the threshold in the slices before this one
        uint32_t pg = 0, pe = 0;
        for (int q = t; q < j; q += kMbThreads) {
            const uint32_t *c = a.mb_cnt + ((int64_t)gi * a.mb_slices + q) * 2;
            pg += c[0];
            pe += c[1];
        }
        pg = wave_sum_u32(pg);
        pe = wave_sum_u32(pe);
        if (lane == 0) {
            red[0][wv] = pg;
            red[1][wv] = pe;
        }
        const int64_t r0 = (int64_t)j * kMbThreads * KPT + (int64_t)t * KPT;
        uint32_t kk[KPT];
        int h = 0, i = 0;
        if (r0 < g.n) mb_load<KPT>(g, r0, kk, h, i);
        __syncthreads();
        int64_t gbase = 0, ebase = 0;
#pragma unroll
        for (int w2 = 0; w2 < kMbWaves; ++w2) {
            gbase += red[0][w2];
            ebase += red[1][w2];
        }
        uint32_t cg = 0, ce = 0;
        if (r0 < g.n) {
#pragma unroll
            for (int q = 0; q < KPT; ++q)
                if (r0 + q < g.n) {
                    const uint32_t m = kk[q] & st.y;
                    cg += m > st.x;
                    ce += m == st.x;
                }
        }
        uint32_t tg, te;
        int64_t gt_before = gbase + mb_exscan(cg, sh, &tg);
        int64_t eq_before = ebase + mb_exscan(ce, sh, &te);
        if (r0 < g.n) {
#pragma unroll
            for (int q = 0; q < KPT; ++q) {
                if (r0 + q >= g.n) break;
                const uint32_t m = kk[q] & st.y;
                const bool gt = m > st.x, eq = m == st.x;
                const int64_t o = gt_before + min(eq_before, need_eq) + (int64_t)h * w;
                // (o < nentries always; the bound keeps a wrong count from writing past the group)
                if ((gt || (eq && eq_before < need_eq)) && o < nentries) out[o] = i;
                gt_before += gt;
                eq_before += eq;
                if (++i == P) {
                    i = 0;
                    ++h;
                }
            }
        }
    }
    if (j != 0) return;
    // block 0: entries taken through each head (layer-flat: from the per-head
    // counts, equal keys in (head, position) order), then the windows, counts
    // and offsets; the per-head counts are cleared for the next call
    if (nh == 1) {
        if (t == 0) through[0] = g.k;
    } else {
        const uint4 st = g.k > 0 ? a.mb_state[2 * (int64_t)a.mb_groups + gi] : uint4{0u, 0u, 0u, 0u};
        uint32_t *gc = a.mb_head + (int64_t)gi * kMaxFlatHeads * 2;
        uint32_t hgt = 0, heq = 0;
        if (t < nh && g.k > 0) {  // (completed by the count launch)
            hgt = gc[2 * t];
            heq = gc[2 * t + 1];
        }
        uint32_t tot;
        const int64_t g_incl = (int64_t)mb_exscan(hgt, sh, &tot) + hgt;
        const int64_t e_incl = (int64_t)mb_exscan(heq, sh, &tot) + heq;
        if (t < nh) {
            through[t] = g_incl + min(e_incl, (int64_t)st.z);
            if (g.k > 0) {
                gc[2 * t] = 0u;
                gc[2 * t + 1] = 0u;
            }
        }
    }
    __syncthreads();
    for (int e = t; e < nh * w; e += kMbThreads) {
        const int hh = e / w, jj = e - (e / w) * w;
        out[through[hh] + (int64_t)hh * w + jj] = P + jj;
    }
    if (t < nh && (a.counts || a.offsets)) {
        const int64_t prev = t > 0 ? through[t - 1] : 0;
        if (a.counts) a.counts[unit_of_head(t)] = (int32_t)(through[t] - prev + w);
        if (a.offsets) a.offsets[unit_of_head(t)] = (int32_t)(g.sg.out_base + prev + (int64_t)t * w);
    }
}

// Keys per thread of the selection kernels for a call whose largest group has
// maxn keys (16 when that still gives 512 blocks or more, else 4).
static int mb_kpt(int64_t groups, int64_t maxn)
{
    const int64_t blocks16 = groups * ((maxn + kMbThreads * 16 - 1) / (kMbThreads * 16));
    return blocks16 >= 512 ? 16 : 4;
}

SelWsLayout select_ws_layout(int64_t groups, int64_t maxn, bool per_head)
{
    SelWsLayout w{};
    const int64_t slices = max((int64_t)1, (maxn + kMbThreads * 4 - 1) / (kMbThreads * 4));
    // the two-stage form's candidate positions (single-head groups past one block)
    const int64_t cand = per_head && maxn > 32 * kSelThreads ? (maxn + kCandSlice - 1) / kCandSlice * kCandSlice : 0;
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    size_t o = 0;
    w.state = o; o = al(o + sizeof(uint4) * 3 * groups);
    w.hist = o; o = al(o + sizeof(uint32_t) * kMbHistWords * groups);
    w.head = o; o = al(o + sizeof(uint32_t) * 2 * kMaxFlatHeads * groups);
    w.cnt = o; o = al(o + sizeof(uint32_t) * 2 * slices * groups);
    w.cand = o; o = al(o + (sizeof(int32_t) + sizeof(uint32_t)) * cand * groups);
    w.total = o;
    return w;
}

template <int KPT>
static hipError_t select_launch_kpt(const SelectArgs &a, unsigned blocks, hipStream_t st)
{
    ECOKV_TIMED("select", st, hipLaunchKernelGGL((k_sel_digit<KPT, 0>), dim3(blocks), dim3(kMbThreads), 0, st, a));
    ECOKV_TIMED("select", st, hipLaunchKernelGGL((k_sel_digit<KPT, 1>), dim3(blocks), dim3(kMbThreads), 0, st, a));
    ECOKV_TIMED("select", st, hipLaunchKernelGGL((k_sel_digit<KPT, 2>), dim3(blocks), dim3(kMbThreads), 0, st, a));
    ECOKV_TIMED("select", st, hipLaunchKernelGGL((k_sel_count<KPT>), dim3(blocks), dim3(kMbThreads), 0, st, a));
    ECOKV_TIMED("select", st, hipLaunchKernelGGL((k_sel_emit<KPT>), dim3(blocks), dim3(kMbThreads), 0, st, a));
    return hipGetLastError();
}

hipError_t select_launch(SelectArgs a, char *ws, hipStream_t st)
{
    const int64_t groups = a.heads ? (int64_t)a.lht.n * a.B : a.flat ? (int64_t)a.L * a.B : (int64_t)a.L * a.Hkv * a.B;
    if (groups == 0) return hipSuccess;
    int64_t maxn = 0;
    for (int s = 0; s < a.B; ++s) {
        const int64_t P = (int64_t)(a.seq.cu[s + 1] - a.seq.cu[s]) - a.w;
        maxn = max(maxn, P * (a.flat ? a.Hkv : 1));
    }
    if (maxn <= 32 * kSelThreads) {
        // one block per group: for groups this small, one launch beats five
        // short ones (28-layer stack, 112 groups of 32764 keys: 29 against 46 us;
        // one layer, 4 groups: 25 against 33 us).  Keys per thread by group
        // size, so that a small group's per-key work spreads over every wave
        if (maxn <= 8 * kSelThreads)
            ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select_reg<8>, dim3((unsigned)groups), dim3(kSelThreads),
                                                         0, st, a));
        else if (maxn <= 16 * kSelThreads)
            ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select_reg<16>, dim3((unsigned)groups), dim3(kSelThreads),
                                                         0, st, a));
        else
            ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select_reg<32>, dim3((unsigned)groups), dim3(kSelThreads),
                                                         0, st, a));
        return hipGetLastError();
    }
    const SelWsLayout lay = select_ws_layout(a.mb_groups, a.mb_maxn, !a.flat);
    if (!a.flat) {
        // single-head groups: two stages when every group's candidates (the
        // largest min(k, slice) keys of each slice) fit one block's registers
        // (groups kept whole need none)
        int kmax = 0;
        for (int s = 0; s < a.B; ++s) {
            const int Ts = a.seq.cu[s + 1] - a.seq.cu[s];
            if (a.heads) {
                for (int j = 0; j < a.lht.n; ++j)
                    if (a.lht.b[j] < Ts) kmax = max(kmax, a.lht.b[j] - a.w);
            } else if (a.seq.beff[s] < Ts) {
                kmax = max(kmax, a.seq.beff[s] - a.w);
            }
        }
        const int ns = (int)((maxn + kCandSlice - 1) / kCandSlice);
        const int64_t ncmax = (int64_t)ns * min(kmax, kCandSlice);
        if (ncmax <= 32 * kSelThreads) {
            a.c_slices = ns;
            const int64_t nslots = (a.mb_maxn + kCandSlice - 1) / kCandSlice * kCandSlice * a.mb_groups;
            a.c_pos = reinterpret_cast<int32_t *>(ws + lay.cand);
            a.c_key = reinterpret_cast<uint32_t *>(ws + lay.cand + sizeof(int32_t) * nslots);
            ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_sel_cand, dim3((unsigned)(groups * ns)), dim3(kSelThreads), 0,
                                                         st, a));
            if (ncmax <= 8 * kSelThreads)
                ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_sel_final<8>, dim3((unsigned)groups), dim3(kSelThreads),
                                                             0, st, a));
            else if (ncmax <= 16 * kSelThreads)
                ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_sel_final<16>, dim3((unsigned)groups),
                                                             dim3(kSelThreads), 0, st, a));
            else
                ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_sel_final<32>, dim3((unsigned)groups),
                                                             dim3(kSelThreads), 0, st, a));
            return hipGetLastError();
        }
    }
    a.mb_state = reinterpret_cast<uint4 *>(ws + lay.state);
    a.mb_hist = reinterpret_cast<uint32_t *>(ws + lay.hist);
    a.mb_head = reinterpret_cast<uint32_t *>(ws + lay.head);
    a.mb_cnt = reinterpret_cast<uint32_t *>(ws + lay.cnt);
    const int kpt = mb_kpt(groups, maxn);
    a.mb_slices = (int)max((int64_t)1, (maxn + kMbThreads * kpt - 1) / (kMbThreads * kpt));
    const unsigned blocks = (unsigned)(groups * a.mb_slices);
    return kpt == 16 ? select_launch_kpt<16>(a, blocks, st) : select_launch_kpt<4>(a, blocks, st);
}

int select_max_flat_heads() { return kMaxFlatHeads; }

}  // namespace ecokv
