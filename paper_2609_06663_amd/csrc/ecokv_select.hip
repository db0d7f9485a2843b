// ecokv_select kernels (gfx950): exact top-k of the scores of each unit
// (ECOKV_PER_HEAD) or of all heads of a (layer, sequence) (ECOKV_LAYER_FLAT,
// AdaKV budget sharing, Appendix A.1), plus the always-kept window (Sec. 3).
//
// One 1024-thread block per selection group.  The k-th largest score is found
// exactly by a most-significant-digit radix select over order-preserving
// 32-bit keys (4 passes of 8 bits, LDS histograms).  A single ordered pass then
// emits the chosen positions in ascending order: keys above the threshold are
// always taken, keys equal to it are taken in position order until the budget
// is met, so equal scores favour the smaller position.
#include "ecokv_internal.h"

namespace ecokv {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kMaxFlatHeads = 256;



// Exclusive block-wide scan of two uint32 per thread (independent sums);
// returns the exclusive prefixes and the block totals.
__device__ __forceinline__ void block_exscan2(uint32_t x0, uint32_t x1, uint32_t *wsum, uint32_t &e0, uint32_t &e1,
                                              uint32_t &t0, uint32_t &t1)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t i0 = x0, i1 = x1;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t y0 = __shfl_up(i0, d, kWave), y1 = __shfl_up(i1, d, kWave);
        if (lane >= d) {
            i0 += y0;
            i1 += y1;
        }
    }
    if (lane == kWave - 1) {
        wsum[wv] = i0;
        wsum[kSelWaves + 1 + wv] = i1;
    }
    __syncthreads();
    if (wv == 0) {
        uint32_t a0 = lane < kSelWaves ? wsum[lane] : 0u;
        uint32_t a1 = lane < kSelWaves ? wsum[kSelWaves + 1 + lane] : 0u;
        uint32_t c0 = a0, c1 = a1;
#pragma unroll
        for (int d = 1; d < kSelWaves; d <<= 1) {
            const uint32_t y0 = __shfl_up(c0, d, kWave), y1 = __shfl_up(c1, d, kWave);
            if (lane >= d) {
                c0 += y0;
                c1 += y1;
            }
        }
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
// sequence s, min(budget, T_s) entries per head, first entry at out_base.
struct SelGroup {
    int l, h0, s, nh, beff;
    int64_t out_base;
};
__device__ __forceinline__ SelGroup sel_group(const SelectArgs &a)
{
    SelGroup g;
    if (a.heads) {
        // one unit per block, (layer, head) pair lh0 + j of the launch's table
        const int j = blockIdx.x / a.B;
        g.s = blockIdx.x - j * a.B;
        const int lh = a.lht.lh0 + j;
        g.l = lh / a.Hkv;
        g.h0 = lh - g.l * a.Hkv;
        g.nh = 1;
        g.beff = min(a.lht.b[j], a.seq.cu[g.s + 1] - a.seq.cu[g.s]);
        g.out_base = a.lht.start[j] + lh_seq_offset(a.lht, a.seq, j, g.s);
    } else if (a.flat) {
        g.l = blockIdx.x / a.B;
        g.s = blockIdx.x % a.B;
        g.h0 = 0;
        g.nh = a.Hkv;
        g.beff = a.seq.beff[g.s];
        g.out_base = (int64_t)g.l * a.Hkv * a.per_lh + (int64_t)a.Hkv * a.seq.boff[g.s];
    } else {
        const Unit un = unit_of(blockIdx.x, a.Hkv, a.B);
        g.l = un.l;
        g.s = un.s;
        g.h0 = un.h;
        g.nh = 1;
        g.beff = a.seq.beff[g.s];
        g.out_base = ((int64_t)g.l * a.Hkv + g.h0) * a.per_lh + a.seq.boff[g.s];
    }
    return g;
}

template <bool RESIDENT>
struct KeySource {
    const GroupView &g;
    const uint32_t *lds;
    __device__ __forceinline__ uint32_t operator()(int64_t v) const
    {
        if constexpr (RESIDENT)
            return lds[v];
        else
            return score_key(g.get(v));
    }
};

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

// The same over the scores in memory, head by head (v = h P + i): no index
// division per key; lane l reads scores 4l .. 4l+3 of each 4096-score round
// with one 16-byte buffer load, four rounds in flight (the head's descriptor
// ends at P, so loads past it read zero).
typedef float f32x4s __attribute__((ext_vector_type(4)));
template <class F>
__device__ __forceinline__ void for_each_key(const KeySource<false> &key, int64_t n, F &&f)
{
    const GroupView &g = key.g;
    constexpr int U = 4;
    const int step = 4 * blockDim.x;
    for (int h = 0; h < g.nh; ++h) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(uniform_ptr(g.base + (int64_t)h * g.hstride)), (short)0, uniform_i32(g.P) * 4,
            0x00020000);
        const int64_t vh = (int64_t)h * g.P;
        for (int base = 4 * (int)threadIdx.x; base < g.P; base += U * step) {
            f32x4s x[U];
#pragma unroll
            for (int u = 0; u < U; ++u)
                x[u] = __builtin_bit_cast(f32x4s, __builtin_amdgcn_raw_buffer_load_b128(rs, (base + u * step) * 4, 0, 0));
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = base + u * step + e;
                    if (i < g.P) f(vh + i, score_key(x[u][e]));
                }
        }
    }
    (void)n;
}

__device__ __forceinline__ uint32_t wave_min_u(uint32_t x)
{
    for (int m = 32; m >= 1; m >>= 1) x = min(x, (uint32_t)__shfl_xor(x, m, kWave));
    return x;
}
__device__ __forceinline__ uint32_t wave_max_u(uint32_t x)
{
    for (int m = 32; m >= 1; m >>= 1) x = max(x, (uint32_t)__shfl_xor(x, m, kWave));
    return x;
}

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
            uint32_t inc = loc;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const uint32_t y = __shfl_up(inc, d, kWave);
                if (lane >= d) inc += y;
            }
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
// keys.  hist: kSelWaves x 256 counters.
constexpr int kCandKeys = 32768;  // gathered keys (128 KiB of LDS)

__device__ void radix_threshold_gather(const KeySource<false> &key, int64_t n, int64_t k, uint32_t kmin, uint32_t kmax,
                                       uint32_t *hist, uint32_t *bc, uint32_t *cand, uint32_t *ccount,
                                       uint32_t *thr_out, int64_t *need_eq_out)
{
    const uint32_t diff = kmin ^ kmax;
    if (diff == 0) {
        *thr_out = kmin;
        *need_eq_out = k;
        return;
    }
    const int lane = threadIdx.x & 63;
    int hi = 31 - __clz(diff);
    uint32_t mask = hi == 31 ? 0u : ~((2u << hi) - 1u);
    uint32_t prefix = kmin & mask;
    int64_t rem = k;
    bool first = true, listed = false;
    uint32_t ncand = 0;
    while (hi >= 0) {
        const int lo = hi >= 7 ? hi - 7 : 0;
        const uint32_t nb = 1u << (hi - lo + 1);
        for (int b = threadIdx.x; b < kSelWaves * 256; b += blockDim.x) hist[b] = 0;
        __syncthreads();
        if (listed) {
            for (uint32_t i = threadIdx.x; i < ncand; i += blockDim.x) {
                const uint32_t kk = cand[i];
                if ((kk & mask) == prefix) atomicAdd(&hist[(kk >> lo) & (nb - 1u)], 1u);
            }
        } else {
            uint32_t *const myh = hist + (threadIdx.x >> 6) * 256;
            for_each_key(key, n, [&](int64_t, uint32_t kk) {
                if ((kk & mask) == prefix) atomicAdd(&myh[(kk >> lo) & (nb - 1u)], 1u);
            });
        }
        __syncthreads();
        if (!listed && threadIdx.x < 256) {
            // fold the wave histograms into the first (each thread its own bin)
            uint32_t c = 0;
#pragma unroll
            for (int w2 = 0; w2 < kSelWaves; ++w2) c += hist[w2 * 256 + threadIdx.x];
            hist[threadIdx.x] = c;
        }
        __syncthreads();
        if (threadIdx.x < kWave) {
            // lane l owns bins 255-4l .. 252-4l (descending order of digit)
            uint32_t c4[4], loc = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                c4[q] = hist[255 - 4 * lane - q];
                loc += c4[q];
            }
            uint32_t inc = loc;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const uint32_t y = __shfl_up(inc, d, kWave);
                if (lane >= d) inc += y;
            }
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
        if (first && hi >= 0) {
            // gather the keys that keep the prefix
            first = false;
            if (threadIdx.x == 0) *ccount = 0u;
            __syncthreads();
            for_each_key(key, n, [&](int64_t, uint32_t kk) {
                const bool m = (kk & mask) == prefix;
                const unsigned long long bal = __ballot(m);
                if (bal) {
                    const int leader = __ffsll((long long)bal) - 1;
                    uint32_t base = 0;
                    if (lane == leader) base = atomicAdd(ccount, (uint32_t)__popcll(bal));
                    base = __shfl(base, leader, kWave);
                    const uint32_t pos = base + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
                    if (m && pos < (uint32_t)kCandKeys) cand[pos] = kk;
                }
            });
            __syncthreads();
            ncand = *ccount;
            listed = ncand <= (uint32_t)kCandKeys;
        }
    }
    *thr_out = prefix;
    *need_eq_out = rem;
}

__global__ __launch_bounds__(kSelThreads) void k_select(SelectArgs a)
{
    __shared__ uint32_t hist[kSelWaves * 256];  // one histogram per wave
    __shared__ uint32_t cand[kCandKeys];
    __shared__ uint32_t ccount;
    __shared__ uint32_t bc[2];
    __shared__ uint32_t wsum[2 * kSelWaves + 2];
    __shared__ uint32_t mm[2][kSelWaves];
    __shared__ int64_t through[kMaxFlatHeads];

    const SelGroup grp = sel_group(a);
    const int l = grp.l, h0 = grp.h0, s = grp.s, nh = grp.nh;
    const int T = a.seq.cu[s + 1] - a.seq.cu[s];
    const int P = T - a.w;
    const int beff = grp.beff;
    const int64_t out_base = grp.out_base;
    int32_t *out = a.idx + out_base;

    if (beff >= T) {  // keep every token
        for (int64_t e = threadIdx.x; e < (int64_t)nh * T; e += blockDim.x) out[e] = (int32_t)(e % T);
        if (threadIdx.x < nh && (a.counts || a.offsets)) {
            const int64_t u = ((int64_t)l * a.Hkv + h0 + threadIdx.x) * a.B + s;
            if (a.counts) a.counts[u] = T;
            if (a.offsets) a.offsets[u] = (int32_t)(out_base + (int64_t)threadIdx.x * T);
        }
        return;
    }

    GroupView g;
    g.base = a.scores + ((int64_t)l * a.Hkv + h0) * a.Ptot + (a.seq.cu[s] - s * a.w);
    g.hstride = a.Ptot;
    g.P = P;
    g.nh = nh;
    const int64_t n = (int64_t)nh * P;
    const int64_t k = (int64_t)nh * (beff - a.w);
    const KeySource<false> key{g, nullptr};
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    for (int h = tid; h < nh; h += blockDim.x) through[h] = 0;
    uint32_t thr = 0xffffffffu;
    int64_t need_eq = 0;
    if (k > 0) {
        // the keys' extremes
        uint32_t kmin = 0xffffffffu, kmax = 0u;
        for_each_key(key, n, [&](int64_t, uint32_t kk) {
            kmin = min(kmin, kk);
            kmax = max(kmax, kk);
        });
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
        radix_threshold_gather(key, n, k, kmin, kmax, hist, bc, cand, &ccount, &thr, &need_eq);
    }
    __syncthreads();

    if (k > 0) {
        // ordered emission: thread t owns the contiguous run [v0, v1); its
        // keys are read by (head, position), stepped along the run (one
        // division per thread), sixteen at a time: four 16-byte loads while
        // they lie in one head, else one load per key.  One descriptor spans
        // the group's scores (head h at h hstride).
        const int64_t per = (n + blockDim.x - 1) / blockDim.x;
        const int64_t v0 = min((int64_t)tid * per, n), v1 = min(v0 + per, n);
        const int h_0 = nh == 1 ? 0 : (int)(v0 / P);
        const int pos_0 = (int)(v0 - (int64_t)h_0 * P);
        const __amdgpu_buffer_rsrc_t rg = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(uniform_ptr(g.base)), (short)0,
            uniform_i32((int)(((int64_t)(nh - 1) * g.hstride + P) * 4)), 0x00020000);
        auto load16 = [&](int hh, int pp, int64_t b, uint32_t (&kk)[16]) {
            const int off = (int)((int64_t)hh * g.hstride + pp);
            if (pp + 16 <= P && b + 16 <= v1) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const f32x4s x = __builtin_bit_cast(f32x4s, __builtin_amdgcn_raw_buffer_load_b128(rg, (off + 4 * u) * 4, 0, 0));
#pragma unroll
                    for (int e = 0; e < 4; ++e) kk[4 * u + e] = score_key(x[e]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    kk[q] = b + q < v1 ? score_key(__builtin_bit_cast(
                                             float, __builtin_amdgcn_raw_buffer_load_b32(
                                                        rg, (int)((int64_t)hh * g.hstride + pp) * 4, 0, 0)))
                                       : 0u;
                    if (++pp == P) {
                        pp = 0;
                        ++hh;
                    }
                }
            }
        };
        uint32_t cg = 0, ce = 0;
        {
            int hh = h_0, pp = pos_0;
            for (int64_t b = v0; b < v1; b += 16) {
                uint32_t kk[16];
                load16(hh, pp, b, kk);
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    if (b + q < v1) {
                        cg += kk[q] > thr;
                        ce += kk[q] == thr;
                    }
                    if (++pp == P) {
                        pp = 0;
                        ++hh;
                    }
                }
            }
        }
        uint32_t eg, ee, tg, te;
        block_exscan2(cg, ce, wsum, eg, ee, tg, te);
        (void)tg;
        (void)te;
        int64_t gt_before = eg, eq_before = ee;
        int h = h_0, pos = pos_0;
        for (int64_t b = v0; b < v1; b += 16) {
            // the run's next sixteen keys (second read of the cache-resident scores)
            uint32_t kk[16];
            load16(h, pos, b, kk);
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                if (b + q >= v1) break;
                const bool gt = kk[q] > thr, eq = kk[q] == thr;
                const bool take = gt || (eq && eq_before < need_eq);
                if (take) out[gt_before + min(eq_before, need_eq) + (int64_t)h * a.w] = (int32_t)pos;
                gt_before += gt;
                eq_before += eq;
                if (++pos == P) {
                    if (nh > 1) through[h] = gt_before + min(eq_before, need_eq);
                    pos = 0;
                    ++h;
                }
            }
        }
        if (nh == 1 && tid == 0) through[0] = k;
    }
    __syncthreads();
    // windows, counts and offsets
    for (int e = tid; e < nh * a.w; e += blockDim.x) {
        const int h = e / a.w, j = e % a.w;
        out[through[h] + (int64_t)h * a.w + j] = P + j;
    }
    if (tid < nh && (a.counts || a.offsets)) {
        const int h = tid;
        const int64_t prev = h > 0 ? through[h - 1] : 0;
        const int64_t u = ((int64_t)l * a.Hkv + h0 + h) * a.B + s;
        if (a.counts) a.counts[u] = (int32_t)(through[h] - prev + a.w);
        if (a.offsets) a.offsets[u] = (int32_t)(out_base + prev + (int64_t)h * a.w);
    }
}

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
            uint32_t inc = loc;
#pragma unroll
            for (int d = 1; d < kWave; d <<= 1) {
                const uint32_t y = __shfl_up(inc, d, kWave);
                if (lane >= d) inc += y;
            }
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
    uint32_t inc = loc;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t y = __shfl_up(inc, d, kWave);
        if (lane >= d) inc += y;
    }
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
        uint32_t inc = cnt;
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const uint32_t y = __shfl_up(inc, d, kWave);
            if (lane >= d) inc += y;
        }
        const uint32_t wtot = __shfl(inc, kWave - 1, kWave);
        uint32_t base = 0;
        if (lane == kWave - 1 && wtot > 0) base = atomicAdd(ccount, wtot);
        base = __shfl(base, kWave - 1, kWave);
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

// ---------------------------------------------------------------------------
// Register-resident variant for groups of up to 64 Ki keys: thread t owns the
// contiguous run [t*KPT, t*KPT + KPT) of the group's keys in registers
// (16-byte loads in per-head mode), the radix passes histogram them into one
// LDS copy per wave, and the ordered emission walks the registers.
// ---------------------------------------------------------------------------
constexpr int kRegMaxKeys = 64 * kSelThreads;

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

    const SelGroup grp = sel_group(a);
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
    const int n = nh * P;  // <= kRegMaxKeys (checked on the host)
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
        // ordered emission of one head: bit q of gtm[c] / eqm[c] marks key
        // v0 + 32 c + q above / equal to the threshold; the thread's taken
        // keys go to consecutive slots from the number taken before its run
        constexpr int NC = KPT / 32;  // 32-key words per thread
        uint32_t gtm[NC], eqm[NC];
        uint32_t cg = 0, ce = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            gtm[c] = 0u;
            eqm[c] = 0u;
#pragma unroll
            for (int q = 0; q < 32; ++q)
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
        // equal keys are taken in position order while fewer than need_eq precede them
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
                if (staged) ost[o] = (uint32_t)(v0 + q);
                else out[o] = v0 + q;
                ++o;
            }
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

hipError_t select_launch(const SelectArgs &a, hipStream_t st)
{
    const unsigned groups = a.heads  ? (unsigned)(a.lht.n * a.B)
                            : a.flat ? (unsigned)(a.L * a.B)
                                     : (unsigned)(a.L * a.Hkv * a.B);
    // largest group: every head's non-window keys in layer-flat mode
    int64_t maxn = 0;
    for (int s = 0; s < a.B; ++s) {
        const int64_t P = (int64_t)(a.seq.cu[s + 1] - a.seq.cu[s]) - a.w;
        maxn = P * (a.flat ? a.Hkv : 1) > maxn ? P * (a.flat ? a.Hkv : 1) : maxn;
    }
    if (maxn <= 32 * kSelThreads)
        ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select_reg<32>, dim3(groups), dim3(kSelThreads), 0, st, a));
    else if (maxn <= kRegMaxKeys)
        ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select_reg<64>, dim3(groups), dim3(kSelThreads), 0, st, a));
    else
        ECOKV_TIMED("select", st, hipLaunchKernelGGL(k_select, dim3(groups), dim3(kSelThreads), 0, st, a));
    return hipGetLastError();
}

int select_max_flat_heads() { return kMaxFlatHeads; }

}  // namespace ecokv
