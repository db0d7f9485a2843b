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



// Exclusive block-wide scan of one uint32 per thread; returns the exclusive
// prefix and writes the block total to *total (all threads).
__device__ __forceinline__ uint32_t block_exscan(uint32_t x, uint32_t *wsum, uint32_t *total)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    uint32_t inc = x;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const uint32_t y = __shfl_up(inc, d, kWave);
        if (lane >= d) inc += y;
    }
    if (lane == kWave - 1) wsum[wv] = inc;
    __syncthreads();
    if (wv == 0) {
        uint32_t t = lane < kSelWaves ? wsum[lane] : 0u;
        uint32_t ti = t;
#pragma unroll
        for (int d = 1; d < kSelWaves; d <<= 1) {
            const uint32_t y = __shfl_up(ti, d, kWave);
            if (lane >= d) ti += y;
        }
        if (lane < kSelWaves) wsum[lane] = ti - t;  // exclusive wave offsets
        if (lane == kSelWaves - 1) wsum[kSelWaves] = ti;
    }
    __syncthreads();
    const uint32_t r = wsum[wv] + inc - x;
    *total = wsum[kSelWaves];
    __syncthreads();
    return r;
}

// Score of virtual element v of the group.
struct GroupView {
    const float *base;  // first score of head 0
    int64_t hstride;    // distance between heads (Ptot)
    int P;
    __device__ __forceinline__ float get(int64_t v) const
    {
        const int64_t h = v / P;
        return base[h * hstride + (v - h * P)];
    }
};

// Radix select: the key of the k-th largest element (k >= 1) and how many
// elements equal to it must be taken.
__device__ void radix_threshold(const GroupView &g, int64_t n, int64_t k, uint32_t *hist, uint32_t *bc,
                                uint32_t *thr_out, int64_t *need_eq_out)
{
    uint32_t prefix = 0, mask = 0;
    int64_t rem = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int b = threadIdx.x; b < 256; b += blockDim.x) hist[b] = 0;
        __syncthreads();
        for (int64_t v = threadIdx.x; v < n; v += blockDim.x) {
            const uint32_t key = score_key(g.get(v));
            if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (threadIdx.x < kWave) {
            // lane l owns bins 255-4l .. 252-4l (descending); suffix counts in
            // descending digit order locate the bin holding the rem-th key.
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
            const uint32_t before = inc - loc;  // keys in higher digits than this lane's bins
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
        prefix |= digit << shift;
        mask |= 255u << shift;
        __syncthreads();
    }
    *thr_out = prefix;
    *need_eq_out = rem;
}

__global__ __launch_bounds__(kSelThreads) void k_select(SelectArgs a)
{
    __shared__ uint32_t hist[256];
    __shared__ uint32_t bc[2];
    __shared__ uint32_t wsum[kSelWaves + 1];
    __shared__ int64_t through[kMaxFlatHeads];

    int l, h0, s, nh;
    if (a.flat) {
        l = blockIdx.x / a.B;
        s = blockIdx.x % a.B;
        h0 = 0;
        nh = a.Hkv;
    } else {
        const Unit un = unit_of(blockIdx.x, a.Hkv, a.B);
        l = un.l;
        s = un.s;
        h0 = un.h;
        nh = 1;
    }
    const int T = a.seq.cu[s + 1] - a.seq.cu[s];
    const int P = T - a.w;
    const int beff = a.seq.beff[s];
    const int64_t out_base = a.flat ? ((int64_t)l * a.Hkv * a.per_lh + (int64_t)a.Hkv * a.seq.boff[s])
                                    : (((int64_t)l * a.Hkv + h0) * a.per_lh + a.seq.boff[s]);
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
    const int64_t n = (int64_t)nh * P;
    const int64_t k = (int64_t)nh * (beff - a.w);

    for (int h = threadIdx.x; h < nh; h += blockDim.x) through[h] = 0;
    uint32_t thr = 0xffffffffu;
    int64_t need_eq = 0;
    if (k > 0) radix_threshold(g, n, k, hist, bc, &thr, &need_eq);
    __syncthreads();

    if (k > 0) {
        int64_t run_gt = 0, run_eq = 0;
        for (int64_t b0 = 0; b0 < n; b0 += blockDim.x) {
            const int64_t v = b0 + threadIdx.x;
            uint32_t key = 0;
            if (v < n) key = score_key(g.get(v));
            const bool gt = v < n && key > thr;
            const bool eq = v < n && key == thr;
            uint32_t total;
            const uint32_t ex = block_exscan((gt ? 1u : 0u) | (eq ? 0x10000u : 0u), wsum, &total);
            const int64_t gt_before = run_gt + (ex & 0xffffu);
            const int64_t eq_before = run_eq + (ex >> 16);
            const bool take = gt || (eq && eq_before < need_eq);
            const int64_t pos = gt_before + (eq_before < need_eq ? eq_before : need_eq);
            if (v < n) {
                const int64_t h = v / P;
                if (take) out[pos + h * a.w] = (int32_t)(v - h * P);
                if (nh > 1 && v - h * P == P - 1) through[h] = pos + (take ? 1 : 0);
            }
            run_gt += total & 0xffffu;
            run_eq += total >> 16;
        }
        if (nh == 1 && threadIdx.x == 0) through[0] = k;
    }
    __syncthreads();
    // windows, counts and offsets
    for (int e = threadIdx.x; e < nh * a.w; e += blockDim.x) {
        const int h = e / a.w, j = e % a.w;
        out[through[h] + (int64_t)h * a.w + j] = P + j;
    }
    if (threadIdx.x < nh && (a.counts || a.offsets)) {
        const int h = threadIdx.x;
        const int64_t prev = h > 0 ? through[h - 1] : 0;
        const int64_t u = ((int64_t)l * a.Hkv + h0 + h) * a.B + s;
        if (a.counts) a.counts[u] = (int32_t)(through[h] - prev + a.w);
        if (a.offsets) a.offsets[u] = (int32_t)(out_base + prev + (int64_t)h * a.w);
    }
}

hipError_t select_launch(const SelectArgs &a, hipStream_t st)
{
    const unsigned groups = a.flat ? (unsigned)(a.L * a.B) : (unsigned)(a.L * a.Hkv * a.B);
    hipLaunchKernelGGL(k_select, dim3(groups), dim3(kSelThreads), 0, st, a);
    return hipGetLastError();
}

int select_max_flat_heads() { return kMaxFlatHeads; }

}  // namespace ecokv
