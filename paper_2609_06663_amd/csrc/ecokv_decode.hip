// ecokv_decode kernels (gfx950): attention of one new query per (layer, query
// head, sequence) over the compressed cache written by ecokv_compact -- the
// generation step that reads the kept rows (Sec. 3).
//
// Split over rows (flash-decoding): block (c, u, z) takes chunk c of unit u's
// rows for query heads QG z .. QG z + QG - 1 of the unit's G; each of its
// waves takes kWaveRows consecutive rows.  Two forms of the wave's work:
//  * k_decode_mx (bf16): q.k on the matrix cores, 16 rows per MFMA tile, P
//    through LDS into the layout of the coalesced V loads, P.V by fp32 FMAs,
//    the next tile's rows loading while one is used;
//  * k_decode (fp32): S = row_bytes / 16 lanes cover a row with 16-byte
//    loads (64 / S rows per instruction); the S lanes of a row add their
//    partial dot products by DPP butterflies; P.V as above.
// Both keep the online softmax in base 2.  A block merges its waves in LDS
// and writes one (max, sum, acc[D]) per query to the workspace;
// k_decode_merge combines a query row's chunks.
#include "ecokv_internal.h"

namespace ecokv {

typedef unsigned int u32x4d __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2d __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8d __attribute__((ext_vector_type(8)));

constexpr int kDecThreads = 256;
constexpr int kDecWaves = kDecThreads / kWave;
constexpr int kWaveRows = 192;  // rows per wave (96, 128 and 256 measured no faster)
constexpr int kDecChunk = kDecWaves * kWaveRows;
constexpr int kDecQG = 8;       // query heads per block at most

// a.lo * b.lo + a.hi * b.hi + c for packed bf16 pairs, fp32 accumulation.
// (The words are passed by value: a bit cast applied to a vector element
// inside an unrolled loop has compiled to element 0 for every index.)
__device__ __forceinline__ float dot2_bf16(unsigned a, unsigned b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2d, a), __builtin_bit_cast(bf16x2d, b), c, false);
}

// Max over the 64 / S row groups of a value that is uniform within each group.
template <int S>
__device__ __forceinline__ float groups_max(float v)
{
    float M = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
#pragma unroll
    for (int r = 1; r < kWave / S; ++r) M = fmaxf(M, __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), r * S)));
    return M;
}

template <bool BF16>
__device__ __forceinline__ void unpack(const u32x4d &x, float (&f)[BF16 ? 8 : 4])
{
    if constexpr (BF16) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            f[2 * c] = __uint_as_float(x[c] << 16);
            f[2 * c + 1] = __uint_as_float(x[c] & 0xffff0000u);
        }
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) f[c] = __uint_as_float(x[c]);
    }
}

template <bool BF16, int D, int QG>
__global__ __launch_bounds__(kDecThreads) void k_decode(DecodeArgs a)
{
    constexpr int E = BF16 ? 2 : 4;
    constexpr int RB = D * E;       // row bytes
    constexpr int S = RB / 16;      // lanes per row
    constexpr int RPI = kWave / S;  // rows per load instruction
    constexpr int EL = 16 / E;      // elements per lane
    constexpr int NR = 4;           // load instructions per batch
    constexpr int BR = NR * RPI;    // rows per batch
    __shared__ float cm[kDecWaves][QG], cl[kDecWaves][QG];
    __shared__ float cacc[kDecWaves][QG][D];
    const int c = blockIdx.x, u = blockIdx.y, z = blockIdx.z;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int lane = threadIdx.x & 63, wv = uniform_i32(threadIdx.x >> 6);
    const int seg = lane % S;
    // (u is the block's: the unit's count and offset are the same in every lane)
    const int n = uniform_i32(min(a.counts[u], a.max_count));  // more rows than max_count: the merge writes NaN
    const int64_t off = uniform_i32(a.offsets[u]);
    const int row0 = (c * kDecWaves + wv) * a.wave_rows;
    const int nrows = max(0, min(n - row0, a.wave_rows));
    const int nq = min(QG, a.G - z * QG);

    // this lane's 16-byte segment of every query (the logit scale
    // log2(e) / sqrt(D) is applied after the dot product)
    u32x4d qw[QG];
#pragma unroll
    for (int g = 0; g < QG; ++g) {
        qw[g] = (u32x4d){0u, 0u, 0u, 0u};
        if (g < nq) {
            const int64_t qrow = ((int64_t)un.l * a.Hq + un.h * a.G + z * QG + g) * a.B + un.s;
            qw[g] = *reinterpret_cast<const u32x4d *>(static_cast<const char *>(a.Q) + qrow * RB + seg * 16);
        }
    }

    const int64_t base = (off + row0) * RB;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char *>(uniform_ptr(static_cast<const char *>(a.Kc) + base)), (short)0, uniform_i32(nrows * RB),
        0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char *>(uniform_ptr(static_cast<const char *>(a.Vc) + base)), (short)0, uniform_i32(nrows * RB),
        0x00020000);

    float m[QG], ls[QG], acc[QG][EL];
#pragma unroll
    for (int g = 0; g < QG; ++g) {
        m[g] = -INFINITY;
        ls[g] = 0.f;
#pragma unroll
        for (int e = 0; e < EL; ++e) acc[g][e] = 0.f;
    }

    // lane l covers row l / S of an instruction's rows, bytes 16 (l % S): offset
    // 16 l; nontemporal (the rows are read once)
    auto load = [&](u32x4d (&kx)[NR], u32x4d (&vx)[NR], int b0) {
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            const int o = (b0 + i * RPI) * RB + lane * 16;
            kx[i] = __builtin_bit_cast(u32x4d, __builtin_amdgcn_raw_buffer_load_b128(rk, o, 0, 2));
            vx[i] = __builtin_bit_cast(u32x4d, __builtin_amdgcn_raw_buffer_load_b128(rv, o, 0, 2));
        }
    };
    for (int b0 = 0; b0 < nrows; b0 += BR) {
        u32x4d kx[NR], vx[NR];
        load(kx, vx, b0);
        __builtin_amdgcn_sched_barrier(0);
        float x[NR][QG];
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            const bool valid = b0 + i * RPI + lane / S < nrows;
            float kf[EL];
            if constexpr (!BF16) unpack<BF16>(kx[i], kf);
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                float pd = 0.f;
                if constexpr (BF16) {
#pragma unroll
                    for (int w = 0; w < 4; ++w) pd = dot2_bf16(qw[g][w], kx[i][w], pd);
                } else {
#pragma unroll
                    for (int e = 0; e < EL; ++e) pd += __uint_as_float(qw[g][e]) * kf[e];
                }
                pd = row_sum<S>(pd);
                x[i][g] = valid ? pd * a.qscale : -INFINITY;
            }
        }
#pragma unroll
        for (int g = 0; g < QG; ++g) {
            float mb = x[0][g];
#pragma unroll
            for (int i = 1; i < NR; ++i) mb = fmaxf(mb, x[i][g]);
            mb = groups_max<S>(mb);
            const float mn = fmaxf(m[g], mb);  // finite: row b0 of the batch is valid
            const float sc = __builtin_amdgcn_exp2f(m[g] - mn);
            m[g] = mn;
            ls[g] *= sc;
#pragma unroll
            for (int e = 0; e < EL; ++e) acc[g][e] *= sc;
        }
#pragma unroll
        for (int i = 0; i < NR; ++i) {
            float vf[EL];
            unpack<BF16>(vx[i], vf);
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                const float p = __builtin_amdgcn_exp2f(x[i][g] - m[g]);
                ls[g] += p;
#pragma unroll
                for (int e = 0; e < EL; ++e) acc[g][e] += p * vf[e];
            }
        }

    }

    // the rows of a wave are spread over its 64 / S row groups: add them up,
    // then merge the block's waves through LDS (fixed order)
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int msk = S; msk < kWave; msk <<= 1) {
            ls[g] += __shfl_xor(ls[g], msk, kWave);
#pragma unroll
            for (int e = 0; e < EL; ++e) acc[g][e] += __shfl_xor(acc[g][e], msk, kWave);
        }
    if (lane < S) {
#pragma unroll
        for (int g = 0; g < QG; ++g) {
#pragma unroll
            for (int e = 0; e < EL; ++e) cacc[wv][g][seg * EL + e] = acc[g][e];
            if (lane == 0) {
                cm[wv][g] = m[g];
                cl[wv][g] = ls[g];
            }
        }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < nq * D; t += kDecThreads) {
        const int g = t / D, d = t - g * D;
        float M = cm[0][g];
        for (int w2 = 1; w2 < kDecWaves; ++w2) M = fmaxf(M, cm[w2][g]);
        float L = 0.f, A = 0.f;
        if (M != -INFINITY)
            for (int w2 = 0; w2 < kDecWaves; ++w2) {
                const float wt = exp2f(cm[w2][g] - M);
                L += cl[w2][g] * wt;
                A += cacc[w2][g][d] * wt;
            }
        const int64_t qrow = ((int64_t)un.l * a.Hq + un.h * a.G + z * QG + g) * a.B + un.s;
        float *pp = a.part + (qrow * a.nparts + c) * (D + 2);
        pp[2 + d] = A;
        if (d == 0) {
            pp[0] = M;
            pp[1] = L;
        }
    }
}

// bf16 rows: Q.K^T on the matrix cores, P.V on the vector ALUs in fp32.
// (The dot products by v_dot2 with DPP row sums cost about as many vector
// instructions as the fp32 P.V itself, which left the kernel bound by issue.)
//  * Tile of 16 rows: v_mfma_f32_16x16x32_bf16 with the rows as A (lane l:
//    row l % 16, 16 bytes at 64 st + 16 (l / 16) of the row for step st, so
//    each load instruction reads 64 contiguous bytes of 16 rows) and the
//    block's query heads as B (lane l: head l % 16, the same bytes; heads
//    >= nq are zero).  Both operands take dimension j of a row from the same
//    lane group and element, so the contraction is exact whatever order the
//    instruction sums its 32 products in.  Lane l then holds the logits of
//    rows 4 (l / 16) .. +3 against head l % 16.
//  * Online softmax per head, base 2, with a lazy reference: the running
//    maximum m moves only when a batch exceeds it by more than 2^8, so the
//    fp32 P.V accumulators are rescaled rarely (one wave-uniform branch).
//  * P goes through a wave-private LDS tile into the V layout (lane l: row
//    RPI i + l / S, bytes 16 (l % S)) and P.V accumulates as in k_decode.
constexpr float kDecRebase = 8.f;
constexpr int kDecTB = 1;  // 16-row tiles per batch (two measured no faster)
// Double-buffered rows (69 vs 73 us on the 28-layer cache), within 168
// registers so that three waves share a SIMD (the launch bound asks for it).
constexpr bool kDecPrefetch = true;

template <int D, int QG, int TB>
__global__ __launch_bounds__(kDecThreads, 3) void k_decode_mx(DecodeArgs a)
{
    constexpr int RB = 2 * D;           // row bytes
    constexpr int KS = D / 32;          // MFMA steps over the head dimension
    constexpr int S = RB / 16;          // lanes per row in the V layout
    constexpr int RPI = kWave / S;      // V rows per load instruction
    constexpr int NV = 16 / RPI;        // V load instructions per 16-row tile
    constexpr int BR = 16 * TB;         // rows per batch
    constexpr int QP = QG < 4 ? 4 : QG; // floats per row of the P tile
    typedef float f32x4d __attribute__((ext_vector_type(4)));
    __shared__ float cm[kDecWaves][QG], cl[kDecWaves][QG];
    __shared__ float cacc[kDecWaves][QG][D];
    __shared__ __attribute__((aligned(16))) float pt[kDecWaves][BR][QP];
    const int c = blockIdx.x, u = blockIdx.y, z = blockIdx.z;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int lane = threadIdx.x & 63, wv = uniform_i32(threadIdx.x >> 6);
    const int r16 = lane & 15, kg = lane >> 4, seg = lane % S, rg = lane / S;
    const int n = uniform_i32(min(a.counts[u], a.max_count));  // more rows than max_count: the merge writes NaN
    const int64_t off = uniform_i32(a.offsets[u]);
    const int row0 = (c * kDecWaves + wv) * a.wave_rows;
    const int nrows = max(0, min(n - row0, a.wave_rows));
    const int nq = min(QG, a.G - z * QG);

    u32x4d qb[KS];
    {
        const int64_t qrow = ((int64_t)un.l * a.Hq + un.h * a.G + z * QG + min(r16, nq - 1)) * a.B + un.s;
        const char *qp = static_cast<const char *>(a.Q) + qrow * RB + 16 * kg;
#pragma unroll
        for (int st = 0; st < KS; ++st)
            qb[st] = r16 < nq ? *reinterpret_cast<const u32x4d *>(qp + 64 * st) : (u32x4d){0u, 0u, 0u, 0u};
    }

    const int64_t base = (off + row0) * RB;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char *>(uniform_ptr(static_cast<const char *>(a.Kc) + base)), (short)0, uniform_i32(nrows * RB),
        0x00020000);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char *>(uniform_ptr(static_cast<const char *>(a.Vc) + base)), (short)0, uniform_i32(nrows * RB),
        0x00020000);

    // m, ls: head r16's reference maximum and this lane's part of its sum
    float m = -INFINITY, ls = 0.f, acc[QG][8];
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[g][e] = 0.f;
    float *ptw = &pt[wv][0][0];

    // every load is unconditional: rows past nrows read zero.  A Kc load
    // instruction covers 64 of a row's bytes, so two instructions share each
    // 128-byte line: those loads keep the default cache policy, and the
    // second finds the line the first brought in (nontemporal Kc loads took
    // 68 us instead of 62 on the 28-layer cache); the Vc loads cover whole
    // lines and stream nontemporally.
    auto load = [&](u32x4d (&kx)[TB][KS], u32x4d (&vx)[TB][NV], int b0) {
#pragma unroll
        for (int t = 0; t < TB; ++t) {
#pragma unroll
            for (int st = 0; st < KS; ++st)
                kx[t][st] = __builtin_bit_cast(
                    u32x4d, __builtin_amdgcn_raw_buffer_load_b128(rk, (b0 + 16 * t + r16) * RB + 64 * st + 16 * kg, 0, 0));
#pragma unroll
            for (int i = 0; i < NV; ++i)
                vx[t][i] = __builtin_bit_cast(
                    u32x4d, __builtin_amdgcn_raw_buffer_load_b128(rv, (b0 + 16 * t + RPI * i) * RB + lane * 16, 0, 2));
        }
    };
    auto batch = [&](const u32x4d (&kx)[TB][KS], const u32x4d (&vx)[TB][NV], int b0) {
        float x[TB][4];
        float mb = -INFINITY;
#pragma unroll
        for (int t = 0; t < TB; ++t) {
            f32x4d cc = (f32x4d){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int st = 0; st < KS; ++st)
                cc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8d, kx[t][st]),
                                                            __builtin_bit_cast(bf16x8d, qb[st]), cc, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                x[t][r] = b0 + 16 * t + 4 * kg + r < nrows ? cc[r] * a.qscale : -INFINITY;
                mb = fmaxf(mb, x[t][r]);
            }
        }
        mb = fmaxf(mb, __shfl_xor(mb, 16, kWave));
        mb = fmaxf(mb, __shfl_xor(mb, 32, kWave));  // finite: row b0 is valid
        const bool move = mb > m + kDecRebase;      // (always in the first batch: m = -inf)
        if (__builtin_amdgcn_ballot_w64(move)) {
            const float nm = move ? mb : m;
            const float sc = __builtin_amdgcn_exp2f(m - nm);  // 0 while m = -inf
            ls *= sc;
            m = nm;
#pragma unroll
            for (int g = 0; g < QG; ++g) {
                const float sg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sc), g));
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[g][e] *= sg;
            }
        }
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float p = __builtin_amdgcn_exp2f(x[t][r] - m);
                ls += p;
                if (r16 < QG) ptw[(16 * t + 4 * kg + r) * QP + r16] = p;
            }
        // (a wave's own LDS accesses are ordered)
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const float *prow = ptw + (16 * t + RPI * i + rg) * QP;
                float pv[QP];
#pragma unroll
                for (int q4 = 0; q4 < QP / 4; ++q4) {
                    const f32x4d y = *reinterpret_cast<const f32x4d *>(prow + 4 * q4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) pv[4 * q4 + e] = y[e];
                }
                float vf[8];
                unpack<true>(vx[t][i], vf);
#pragma unroll
                for (int g = 0; g < QG; ++g)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[g][e] = fmaf(pv[g], vf[e], acc[g][e]);
            }
    };
    if constexpr (kDecPrefetch) {
        // two register buffers: the next batch's rows load while this one is used
        u32x4d ka[TB][KS], va[TB][NV], kb[TB][KS], vb[TB][NV];
        if (nrows > 0) load(ka, va, 0);
        for (int b0 = 0; b0 < nrows; b0 += 2 * BR) {
            load(kb, vb, b0 + BR);
            __builtin_amdgcn_sched_barrier(0);
            batch(ka, va, b0);
            if (b0 + BR >= nrows) break;
            load(ka, va, b0 + 2 * BR);
            __builtin_amdgcn_sched_barrier(0);
            batch(kb, vb, b0 + BR);
        }
    } else {
        for (int b0 = 0; b0 < nrows; b0 += BR) {
            u32x4d kx[TB][KS], vx[TB][NV];
            load(kx, vx, b0);
            __builtin_amdgcn_sched_barrier(0);
            batch(kx, vx, b0);
        }
    }

    // P.V: add the row groups of the V layout; sums: add the four lane groups
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
        for (int msk = S; msk < kWave; msk <<= 1)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[g][e] += __shfl_xor(acc[g][e], msk, kWave);
    ls += __shfl_xor(ls, 16, kWave);
    ls += __shfl_xor(ls, 32, kWave);
    if (lane < S) {
#pragma unroll
        for (int g = 0; g < QG; ++g)
#pragma unroll
            for (int e = 0; e < 8; ++e) cacc[wv][g][seg * 8 + e] = acc[g][e];
    }
    if (lane < QG) {
        cm[wv][lane] = m;
        cl[wv][lane] = ls;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < nq * D; t += kDecThreads) {
        const int g = t / D, d = t - g * D;
        float M = cm[0][g];
        for (int w2 = 1; w2 < kDecWaves; ++w2) M = fmaxf(M, cm[w2][g]);
        float L = 0.f, A = 0.f;
        if (M != -INFINITY)
            for (int w2 = 0; w2 < kDecWaves; ++w2) {
                const float wt = exp2f(cm[w2][g] - M);
                L += cl[w2][g] * wt;
                A += cacc[w2][g][d] * wt;
            }
        const int64_t qrow = ((int64_t)un.l * a.Hq + un.h * a.G + z * QG + g) * a.B + un.s;
        float *pp = a.part + (qrow * a.nparts + c) * (D + 2);
        pp[2 + d] = A;
        if (d == 0) {
            pp[0] = M;
            pp[1] = L;
        }
    }
}

constexpr int kMergeRegs = 16;  // chunks a merge thread holds in registers

// One block per query row (D threads): the log-sum-exp merge of its chunks.
__global__ __launch_bounds__(128) void k_decode_merge(DecodeArgs a)
{
    const int64_t qrow = blockIdx.x;
    const int t = threadIdx.x;
    const int s = (int)(qrow % a.B), q = (int)((qrow / a.B) % a.Hq), l = (int)(qrow / ((int64_t)a.B * a.Hq));
    const int64_t u = ((int64_t)l * a.Hkv + q / a.G) * a.B + s;
    const int n = a.counts[u];
    const float *pp = a.part + qrow * a.nparts * (a.D + 2);
    const int chunk = kDecWaves * a.wave_rows;
    const int used = min((min(n, a.max_count) + chunk - 1) / chunk, a.nparts);
    float M = -INFINITY, L = 0.f, o = 0.f;
    const int tt = min(t, a.D - 1);
    if (used <= kMergeRegs) {
        // every chunk's (max, sum, acc) loaded at once: one round of latency
        float cmx[kMergeRegs], csm[kMergeRegs], cac[kMergeRegs];
#pragma unroll
        for (int p = 0; p < kMergeRegs; ++p) {
            const float *r = pp + (int64_t)min(p, max(used - 1, 0)) * (a.D + 2);
            cmx[p] = p < used ? r[0] : -INFINITY;
            csm[p] = r[1];
            cac[p] = r[2 + tt];
        }
#pragma unroll
        for (int p = 0; p < kMergeRegs; ++p) M = fmaxf(M, cmx[p]);
        if (M != -INFINITY) {
#pragma unroll
            for (int p = 0; p < kMergeRegs; ++p) {
                const float w = p < used ? exp2f(cmx[p] - M) : 0.f;
                L += csm[p] * w;
                o += cac[p] * w;
            }
        }
    } else {
        // (unrolled so that the chunks' loads are in flight together)
#pragma unroll 8
        for (int p = 0; p < used; ++p) M = fmaxf(M, pp[(int64_t)p * (a.D + 2)]);
        if (M != -INFINITY) {
#pragma unroll 8
            for (int p = 0; p < used; ++p) {
                const float *r = pp + (int64_t)p * (a.D + 2);
                const float w = exp2f(r[0] - M);
                L += r[1] * w;
                o += r[2 + tt] * w;
            }
        }
    }
    const bool bad = n > a.max_count || n < 0;
    if (t < a.D) a.O[qrow * a.D + t] = bad ? NAN : (M == -INFINITY ? 0.f : o / L);
    if (t == 0 && a.lse)
        a.lse[qrow] = bad ? NAN : (M == -INFINITY ? -INFINITY : (M + log2f(L)) * 0.69314718055994531f);
}

// Query heads per block: all of G up to 8 (so that Kc / Vc are read once),
// rounded up to 1, 2, 4 or 8; larger G takes several blocks of 8.
static int decode_qg(int G) { return G > 4 ? kDecQG : G > 2 ? 4 : G; }

template <int D>
static void launch_dec_mx(const DecodeArgs &a, dim3 grid, hipStream_t st)
{
    constexpr int TB = kDecTB;
    const int qg = decode_qg(a.G);
    if (qg == 8) hipLaunchKernelGGL((k_decode_mx<D, 8, TB>), grid, dim3(kDecThreads), 0, st, a);
    else if (qg == 4) hipLaunchKernelGGL((k_decode_mx<D, 4, TB>), grid, dim3(kDecThreads), 0, st, a);
    else if (qg == 2) hipLaunchKernelGGL((k_decode_mx<D, 2, TB>), grid, dim3(kDecThreads), 0, st, a);
    else hipLaunchKernelGGL((k_decode_mx<D, 1, TB>), grid, dim3(kDecThreads), 0, st, a);
}

template <bool BF16, int D>
static void launch_dec(const DecodeArgs &a, dim3 grid, hipStream_t st)
{
    const int qg = decode_qg(a.G);
    if (qg == 8) hipLaunchKernelGGL((k_decode<BF16, D, 8>), grid, dim3(kDecThreads), 0, st, a);
    else if (qg == 4) hipLaunchKernelGGL((k_decode<BF16, D, 4>), grid, dim3(kDecThreads), 0, st, a);
    else if (qg == 2) hipLaunchKernelGGL((k_decode<BF16, D, 2>), grid, dim3(kDecThreads), 0, st, a);
    else hipLaunchKernelGGL((k_decode<BF16, D, 1>), grid, dim3(kDecThreads), 0, st, a);
}

int decode_parts(int max_count) { return (max_count + kDecChunk - 1) / kDecChunk; }

hipError_t decode_launch(DecodeArgs a, bool bf16, hipStream_t st)
{
    const int U = a.L * a.Hkv * a.B;
    if (U == 0) return hipSuccess;
    const int qg = decode_qg(a.G);
    const int zg = (a.G + qg - 1) / qg;
    // chunks of kDecWaves waves of kWaveRows rows (longer chunks that fit the
    // grid into fewer rounds of resident blocks measured slower: the kernel
    // is bound by the rows each wave has in flight, not by the last round)
    a.wave_rows = kWaveRows;
    a.nparts = decode_parts(a.max_count);
    const dim3 grid(a.nparts, U, zg);
    if (bf16 && a.D == 128) ECOKV_TIMED("decode", st, (launch_dec_mx<128>(a, grid, st)));
    else if (bf16) ECOKV_TIMED("decode", st, (launch_dec_mx<64>(a, grid, st)));
    else if (a.D == 128) ECOKV_TIMED("decode", st, (launch_dec<false, 128>(a, grid, st)));
    else ECOKV_TIMED("decode", st, (launch_dec<false, 64>(a, grid, st)));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned rows = (unsigned)((int64_t)a.L * a.Hq * a.B);
    ECOKV_TIMED("decode_merge", st, hipLaunchKernelGGL(k_decode_merge, dim3(rows), dim3(128), 0, st, a));
    return hipGetLastError();
}

}  // namespace ecokv
