// ecokv_score kernels (gfx950): importance, diversity, redundancy and the
// final score of every (layer, KV head, sequence) unit.
//
// Stages, in stream order:
//   sweep1   one pass over K per block of rows: column sums of k and of k/|k|
//            (centroid kbar, Eq. (1); mean normalised key mu, Appendix A.1)
//            and, for every window row, the block's softmax maximum and sum of
//            exponentials of q.k/sqrt(d_k) (Sec. 3 attention, causal window).
//   reduce1  per unit: combine the block partials into kbar, mu and the
//            per-row softmax maximum and normaliser.
//   sweep2   second pass over K: per key d_E = |k - kbar| (Eq. (1)), khat.mu
//            and the window-mean attention a_i (Sec. 5.2: average attention
//            score over the window); block partials of sum/min/max d_E.
//   epilogue per unit: D_E (Eq. (4)), r_E (Eq. (5)), r_C (Appendix A.1),
//            lambda (Eq. (6)); pooled S_imp (Table 6), s_E (Eq. (2)), s_C,
//            S_div (Eq. (3)); the rescale of Sec. 5.2 and S (Eq. (7)).
//
// Two implementations of the sweeps:
//   * bf16 with head_dim 128 (the shapes of the paper's models): a 128-key
//     tile is staged through LDS (XOR-swizzled 16-byte chunks, conflict free
//     for both read patterns).  Geometry runs on the VALU with 16 lanes per
//     key row (DPP row reductions); the window logits run on the matrix
//     cores, v_mfma_f32_32x32x16_bf16 with the window rows as the 32-row A
//     operand and 32 keys per wave as the B operand.
//   * any other case (fp32 inputs, head_dim 64): a plain VALU sweep with 16
//     lanes per key row and window dot products reduced across the row.
#include <stdlib.h>
#include <string.h>

#include "ecokv_fast.h"

namespace ecokv {

constexpr int kThreads = 256;
constexpr int kCh = 128;        // key rows per block, generic sweeps

// Component c of kbar from the sum of the unit's T keys: divided by T, or,
// with the centroid over the non-window keys, the w window rows taken out
// and divided by P.
__device__ __forceinline__ float centroid_component(const ScoreArgs &a, const Unit &un, int T, int c, float s)
{
    if (!a.centroid_prefix) return s / (float)T;
    const int64_t r0 = unit_row0(a, un) + (T - a.w);
    float ws = 0.f;
    for (int j = 0; j < a.w; ++j) {
        const int64_t off = (r0 + j) * a.D + c;
        ws += a.kbf16 ? __uint_as_float((uint32_t)static_cast<const uint16_t *>(a.K)[off] << 16)
                      : static_cast<const float *>(a.K)[off];
    }
    return (s - ws) / (float)(T - a.w);
}

// Anchor column c of unit u (the layout of a.anchors: kbar, mu, the window
// rows' base-2 references and sums): from the workspace after the first sweep,
// or converted from the sums a prefill handed over (ecokv_score_pre: plain
// sums over the T keys, references in natural units).
__device__ __forceinline__ float anchor_value(const ScoreArgs &a, const Unit &un, int u, int T, int c)
{
    const int64_t at = (int64_t)u * (2 * a.D + 2 * a.R) + c;
    if (!a.pre) return a.anchors[at];
    const float v = a.pre[at];
    if (c < a.D) return centroid_component(a, un, T, c, v);
    if (c < 2 * a.D) return v / (float)T;
    if (c < 2 * a.D + a.R) return v * kLog2e;
    return v;
}

// The unit's anchors for a sweep-2 block: the workspace row after the first
// sweep, or, with handed-over sums, the converted row staged in `lds` (every
// thread of the block calls it; a.pre is the same for the whole launch).
__device__ __forceinline__ const float *unit_anchors(const ScoreArgs &a, const Unit &un, int u, int T, float *lds)
{
    if (!a.pre) return a.anchors + (int64_t)u * (2 * a.D + 2 * a.R);
    for (int c = threadIdx.x; c < 2 * a.D + 2 * a.R; c += blockDim.x) lds[c] = anchor_value(a, un, u, T, c);
    __syncthreads();
    return lds;
}

// ---------------------------------------------------------------------------
// Generic sweeps (fp32 or head_dim 64): 16 lanes per key row.
// ---------------------------------------------------------------------------
template <int D, bool BF>
__device__ void load_window_rows(const ScoreArgs &a, const Unit &un, float *q)
{
    for (int idx = threadIdx.x; idx < a.R * D; idx += blockDim.x) {
        const int r = idx / D, d = idx % D;
        const int64_t qrow = window_row(a, un, r);
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

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row0 = blockIdx.x * kCh;
    if (row0 >= T) return;

    load_window_rows<D, BF>(a, un, q_lds);
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = lane & 15, sub = lane >> 4;
    const char *k0 = static_cast<const char *>(a.K) + unit_row0(a, un) * D * ESZ;
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
            if (c == 0) lg[r * (kCh + 1) + rl] = vis ? d * (a.inv_sqrt_d * kLog2e) : -INFINITY;
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
            for (int t = 0; t < kCh; ++t) s += exp2f(lg[r * (kCh + 1) + t] - m);
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
}

// The workspace's exchange tag, bumped once per score call by the second
// sweep's first block and read by the split epilogue after it, so that every
// call (every replay of a captured call included) tags its exchanges afresh
// and never reads an older call's words (0 is skipped: the status word
// records the tag of a call whose wait gave up).
__device__ __forceinline__ void bump_call_tag(const ScoreArgs &a)
{
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {
        const unsigned t = *a.tagw + 1u;
        *a.tagw = t ? t : 1u;
    }
}

template <int D, bool BF>
__global__ __launch_bounds__(kThreads) void k_pass2(ScoreArgs a)
{
    bump_call_tag(a);
    constexpr int VEC = D / 16;
    constexpr int ESZ = BF ? 2 : 4;
    __shared__ float q_lds[ECOKV_MAX_ROWS * D];
    __shared__ float kb[D], mu[D], rm[ECOKV_MAX_ROWS], rs_inv[ECOKV_MAX_ROWS];
    __shared__ float wred[4][kThreads / kWave];

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row0 = blockIdx.x * kCh;
    if (row0 >= T) return;
    load_window_rows<D, BF>(a, un, q_lds);
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        kb[d] = anchor_value(a, un, u, T, d);
        mu[d] = anchor_value(a, un, u, T, D + d);
    }
    for (int r = threadIdx.x; r < a.R; r += blockDim.x) {
        rm[r] = anchor_value(a, un, u, T, 2 * D + r);
        rs_inv[r] = 1.f / anchor_value(a, un, u, T, 2 * D + a.R + r);
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int c = lane & 15, sub = lane >> 4;
    const char *k0 = static_cast<const char *>(a.K) + unit_row0(a, un) * D * ESZ;
    const int64_t obase = unit_out_base(a, un);
    const float inv_r = 1.f / (float)a.R;
    float dsum = 0.f, dsq = 0.f, dmin = INFINITY, dmax = -INFINITY;

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
            if (i < P) att += exp2f(d * (a.inv_sqrt_d * kLog2e) - rm[r]) * rs_inv[r];
        }
        if (valid) {
            dsum += (c == 0) ? dE : 0.f;
            dsq += (c == 0) ? dE * dE : 0.f;
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
    dsq = wave_sum(dsq);
    dmin = wave_min(dmin);
    dmax = wave_max(dmax);
    if (lane == 0) {
        wred[0][wv] = dsum;
        wred[1][wv] = dmin;
        wred[2][wv] = dmax;
        wred[3][wv] = dsq;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        float s = 0.f, s2 = 0.f, mn = INFINITY, mx = -INFINITY;
        for (int k = 0; k < kThreads / kWave; ++k) {
            s += wred[0][k];
            mn = fminf(mn, wred[1][k]);
            mx = fmaxf(mx, wred[2][k]);
            s2 += wred[3][k];
        }
        float *pp = a.part2 + ((int64_t)u * a.nch2 + blockIdx.x) * 4;
        pp[0] = s;
        pp[1] = mn;
        pp[2] = mx;
        pp[3] = s2;
    }
}

// ---------------------------------------------------------------------------
// bf16, head_dim 128: LDS-staged tiles, matrix-core window logits and
// projections.
// ---------------------------------------------------------------------------
namespace fast {

constexpr float kRebase = 16.f;       // log2 headroom of a lazily moved softmax reference
constexpr int kTilesPerBlock = 8;  // tiles per block (1024 keys)
constexpr int kSweep1Depth = 2;    // tiles in flight ahead of the one in use
constexpr int kSweep2Depth = 2;
constexpr int kRows = kTile * kTilesPerBlock;
constexpr int kSmallRows = 2 * kTile;  // keys per block when 1024-key blocks would be too few to fill the device

// One 128-key tile into registers: 16 lanes per 256-byte row, coalesced.
// Rows outside the descriptor's range come back as zero.
__device__ __forceinline__ void tile_load(u32x4 (&pf)[8], __amdgpu_buffer_rsrc_t rs, int tr0, int g, int c)
{
#pragma unroll
    for (int j = 0; j < 8; ++j)
        pf[j] = __builtin_amdgcn_raw_buffer_load_b128(rs, (tr0 + j * 16 + g) * (kD * 2) + c * 16, 0, 2);  // nt: read once
}

__device__ __forceinline__ void tile_store(u32x4 *kt, const u32x4 (&pf)[8], int g, int c)
{
#pragma unroll
    for (int j = 0; j < 8; ++j) kt[sw(j * 16 + g, c)] = pf[j];
}

// The first DEPTH 128-key tiles of a block into registers: issued before the
// block's set-up loads (window rows, anchors), so that their latencies overlap.
template <int DEPTH>
__device__ __forceinline__ void tile_prefetch(u32x4 (&pf)[DEPTH][8], __amdgpu_buffer_rsrc_t rs, int row_base, int g,
                                              int c)
{
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) tile_load(pf[d], rs, row_base + d * kTile, g, c);
}

// Calls body(tr0) for each of the block's `ntiles` 128-key tiles with the tile
// in kt, the first DEPTH of them already in pf (tile_prefetch).  DEPTH tiles
// are in flight in registers while one is processed.  The prefetch is
// unconditional (the descriptor ends at the block's last row), so every
// barrier waits only for LDS and the oldest tile.
template <int DEPTH, class F>
__device__ __forceinline__ void tile_pipeline(u32x4 (&pf)[DEPTH][8], u32x4 *kt, __amdgpu_buffer_rsrc_t rs,
                                              int row_base, int ntiles, int g, int c, F &&body)
{
    // The loop over groups of DEPTH tiles is kept rolled (code size); the
    // loads are unconditional, so the outstanding-load count is the same on
    // every path and each barrier waits only for the oldest tile.
    // Whole groups only: a tile past the block's range reads as zeros from the
    // descriptor and adds nothing (callers mask keys at or past T), so every
    // iteration is identical and no path re-enters the loop with fewer loads
    // in flight.
    const int ngroups = (ntiles + DEPTH - 1) / DEPTH;
#pragma unroll 1
    for (int grp = 0; grp < ngroups; ++grp) {
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int tile = grp * DEPTH + d;
            tile_store(kt, pf[d], g, c);
            lds_barrier();
            tile_load(pf[d], rs, row_base + (tile + DEPTH) * kTile, g, c);
            body(row_base + tile * kTile);
            lds_barrier();
        }
    }
}

// Window rows 32t + (lane & 31) as MFMA A operands (zero beyond R): for k-step
// s the lane holds elements 8*(2s + lane/32) .. +7.
template <int MT>
__device__ __forceinline__ void load_query_operands(const ScoreArgs &a, const Unit &un, int lane, bf16x8 (&aq)[MT][8])
{
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const int r = 32 * t + (lane & 31);
        const bool ok = r < a.R;
        const uint16_t *qp = static_cast<const uint16_t *>(a.Q) + window_row(a, un, ok ? r : 0) * kD;
        u32x4 q[8];
#pragma unroll
        for (int s = 0; s < 8; ++s) q[s] = *reinterpret_cast<const u32x4 *>(qp + 8 * (2 * s + (lane >> 5)));
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const u32x4 z = {0u, 0u, 0u, 0u};
            aq[t][s] = __builtin_bit_cast(bf16x8, ok ? q[s] : z);
        }
    }
}

// Sweep 1, per block of a.rpb1 keys (kRows, or kSmallRows for calls with few blocks):
//  * window logits on the matrix cores (window rows x 32 keys per wave) with
//    per-row online softmax statistics, x = log2(e) q.k / sqrt(d_k);
//  * |k|^2 from v_dot2 on the same B registers, and 1/|k| per key;
//  * the column sums sum_k k and sum_k k/|k| also on the matrix cores: the
//    A operand rows are (1, 1/|k| high bf16, 1/|k| remainder) over 16 keys and
//    the B operand is 16 keys x 32 dimensions, read transposed from the LDS
//    tile with ds_read_b64_tr_b16 (each 16-lane group returns the 4 x 4
//    transpose of the 8-byte pieces its lanes address).
template <int MT>
__global__ __launch_bounds__(256, MT == 1 ? 2 : 1) void k_fs1(ScoreArgs a)
{
    __shared__ u32x4 kt[kTile * kChunks];                   // 32 KiB key tile
    __shared__ __attribute__((aligned(16))) uint16_t aw[4][kTile];  // ones, 1/|k| high, remainder, zeros

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row_base = blockIdx.x * a.rpb1;
    if (row_base >= T) return;

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int c = tid & 15, g = tid >> 4, h = lane >> 5;
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const float sc = a.inv_sqrt_d * kLog2e;
    const __amdgpu_buffer_rsrc_t rs = key_rows_rsrc(krow0, min(T, row_base + a.rpb1));
    u32x4 pf[kSweep1Depth][8];
    tile_prefetch(pf, rs, row_base, g, c);

    bf16x8 aq[MT][8];
    load_query_operands<MT>(a, un, lane, aq);
    for (int i = tid; i < kTile; i += blockDim.x) {
        aw[0][i] = 0x3f80;  // 1.0
        aw[3][i] = 0;
    }

    // Per-lane addresses of the transposed reads (constant over the block):
    // lane X reads 4 dimensions 32 wv + 16 ((X/16) % 2) + 4 (X % 4) of key
    // 8 (X/32) + ((X % 16) / 4) (+4 for the second read) of each 16-key step.
    const int tr_key = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int tr_dim = 32 * wv + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int aw_row = (lane & 31) < 3 ? (lane & 31) : 3;

    float ms[MT][16], ss[MT][16];
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            ms[t][i] = -INFINITY;
            ss[t][i] = 0.f;
        }
    f32x16 csum = (f32x16){};

    const int ntiles = min(a.rpb1 / kTile, (T - row_base + kTile - 1) / kTile);
    tile_pipeline(pf, kt, rs, row_base, ntiles, g, c, [&](int tr0) {
        // window logits and |k|^2 of this wave's 32 keys
        f32x16 acc[MT];
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = (f32x16){};
        float n2 = 0.f;
        {
            const int r = 32 * wv + (lane & 31);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const u32x4 bq = kt[sw(r, 2 * s + h)];
                n2 = dot2sq(bq[0], dot2sq(bq[1], dot2sq(bq[2], dot2sq(bq[3], n2))));
                const bf16x8 b = __builtin_bit_cast(bf16x8, bq);
#pragma unroll
                for (int t = 0; t < MT; ++t)
                    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[t][s], b, acc[t], 0, 0, 0);
            }
        }
        n2 += __shfl_xor(n2, 32, kWave);
        if (h == 0) {
            const float inv = __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
            const unsigned hi = bf16_rne(inv);
            aw[1][32 * wv + lane] = (uint16_t)hi;
            aw[2][32 * wv + lane] = (uint16_t)bf16_rne(inv - __uint_as_float(hi << 16));
        }

        // online softmax statistics.  (ms, ss) keeps ss = sum 2^(x - ms) over the
        // values seen so far, where ms is a reference that stays within
        // kRebase of the running maximum instead of tracking it exactly: the
        // reference moves only when a value exceeds it by more than kRebase,
        // so after the first tile almost every tile takes the cheap branch.
        const int gi = tr0 + 32 * wv + (lane & 31);
        if (tr0 + kTile <= P) {
            // every key of the tile is a non-window key, visible to every row
            if (tr0 == row_base) {
                // first tile of the block: each value is its own reference
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        ms[t][i] = acc[t][i] * sc;
                        ss[t][i] = 1.f;
                    }
            } else {
                float d[MT][16];
                float dmax = -INFINITY;
#pragma unroll
                for (int t = 0; t < MT; ++t)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        d[t][i] = fmaf(acc[t][i], sc, -ms[t][i]);
                        dmax = fmaxf(dmax, d[t][i]);
                    }
                if (!__any(dmax > kRebase)) {
#pragma unroll
                    for (int t = 0; t < MT; ++t)
#pragma unroll
                        for (int i = 0; i < 16; ++i) ss[t][i] += fast_exp2(d[t][i]);
                } else {
#pragma unroll
                    for (int t = 0; t < MT; ++t)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            if (d[t][i] > kRebase) {
                                ss[t][i] = fmaf(ss[t][i], fast_exp2(-d[t][i]), 1.f);
                                ms[t][i] = acc[t][i] * sc;
                            } else {
                                ss[t][i] += fast_exp2(d[t][i]);
                            }
                        }
                }
            }
        } else {
#pragma unroll
            for (int t = 0; t < MT; ++t)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int m = 32 * t + 8 * (i >> 2) + 4 * h + (i & 3);
                    const bool ok = gi < T && (!a.causal || gi <= P + (m % a.w));
                    const float x = acc[t][i] * sc;
                    const float dd = x - ms[t][i];
                    const float e = fast_exp2(-fabsf(dd));
                    const float s_new = dd > 0.f ? fmaf(ss[t][i], e, 1.f) : ss[t][i] + e;
                    if (ok) {
                        ss[t][i] = s_new;
                        ms[t][i] = fmaxf(ms[t][i], x);
                    }
                }
        }
        lds_barrier();  // 1/|k| of the tile is in aw

        // column sums on the matrix cores: this wave's 32 dimensions, 8 steps of 16 keys
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const bf16x8 wa = *reinterpret_cast<const bf16x8 *>(&aw[aw_row][16 * ks + 8 * h]);
            const int key0 = 16 * ks + tr_key;
            typedef short s16x4 __attribute__((ext_vector_type(4)));
            const uint16_t *p0 = reinterpret_cast<const uint16_t *>(kt) + key0 * kD +
                                 (((tr_dim >> 3) ^ (key0 & 15)) << 3) + (tr_dim & 7);
            const uint16_t *p1 = reinterpret_cast<const uint16_t *>(kt) + (key0 + 4) * kD +
                                 (((tr_dim >> 3) ^ ((key0 + 4) & 15)) << 3) + (tr_dim & 7);
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p0)));
            const s16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p1)));
            const short __attribute__((ext_vector_type(8))) kb8 = {lo[0], lo[1], lo[2], lo[3],
                                                                    hi4[0], hi4[1], hi4[2], hi4[3]};
            csum = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa, __builtin_bit_cast(bf16x8, kb8), csum, 0, 0, 0);
        }
    });

    const int stride = 2 * kD + 2 * a.R;
    float *part = a.part1 + ((int64_t)u * a.nch1 + blockIdx.x) * stride;
    if (h == 0) {
        part[32 * wv + lane] = csum[0];              // sum of k
        part[kD + 32 * wv + lane] = csum[1] + csum[2];  // sum of k / |k|
    }
    // per-row softmax partials: a row's 128 (reference, sum) pairs (32 lanes
    // of each of the 4 waves) go through the key tile, free now, and 8 threads
    // per row merge 16 of them each, then by a 3-step DPP butterfly: the
    // row's largest reference, each sum moved onto it, summed.  (Butterflies
    // over the 32 lanes that hold a row, one row at a time, took 5 of this
    // block's 12 us on one 8192-token layer: 64 dependent chains in 4 waves.)
    // (pair p of row r at r * 128 + (p ^ 8 (r % 8)): the 8 rows a wave reads at
    // once fall on different banks)
    float2 *scr = reinterpret_cast<float2 *>(kt);  // [32 rows][4 waves x 32 lanes]
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t) lds_barrier();  // the previous rows' readers are done
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = 8 * (i >> 2) + 4 * h + (i & 3);
            scr[r * 128 + ((32 * wv + (lane & 31)) ^ (8 * (r & 7)))] = make_float2(ms[t][i], ss[t][i]);
        }
        lds_barrier();
        const int row = tid >> 3, q = tid & 7;
        float2 v[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) v[j] = scr[row * 128 + ((8 * j + q) ^ (8 * (row & 7)))];
        float m = -INFINITY, s = 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) m = fmaxf(m, v[j].x);
#pragma unroll
        for (int j = 0; j < 16; ++j) s += v[j].x == -INFINITY ? 0.f : v[j].y * fast_exp2(v[j].x - m);
        const float mg = row_reduce<8>(m, OpMax{});
        s = row_reduce<8>(m == -INFINITY ? 0.f : s * fast_exp2(m - mg), OpAdd{});
        if (q == 0 && 32 * t + row < a.R) {
            part[2 * kD + 32 * t + row] = mg;
            part[2 * kD + a.R + 32 * t + row] = s;
        }
    }
}

// Sweep 2.  The A operand carries the window rows and, in its last two rows,
// mu split into a bf16 high part and a bf16 remainder, so that one MFMA chain
// gives q.k for the window rows together with k.mu to about 2^-17 relative.
// |k|^2 comes from v_dot2 on the same B registers; khat.mu = k.mu / |k|.
// d_E = |k - kbar| is summed directly from the differences in fp32 (each lane
// over the 64 dimensions it holds): the expansion |k|^2 - 2 k.kbar + |kbar|^2
// would lose the distance to cancellation when the keys share a large common
// offset (mean cosine near 1, Sec. 4).
template <int MT>
__global__ __launch_bounds__(256, MT == 1 ? 2 : 1) void k_fs2(ScoreArgs a)
{
    bump_call_tag(a);
    constexpr int kAnc = 32 * MT - 2;  // first anchor row of the A operand
    __shared__ u32x4 kt[kTile * kChunks];
    __shared__ float rowM[32 * MT], rowIS[32 * MT];
    __shared__ float wred[4][4];

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row_base = blockIdx.x * a.rpb2;
    if (row_base >= T) return;

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int c = tid & 15, g = tid >> 4, h = lane >> 5;
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const int64_t obase = unit_out_base(a, un);
    const __amdgpu_buffer_rsrc_t rs = key_rows_rsrc(krow0, min(T, row_base + a.rpb2));
    u32x4 pf[kSweep2Depth][8];
    tile_prefetch(pf, rs, row_base, g, c);
    __shared__ __attribute__((aligned(16))) float sanc[2 * kD + 2 * ECOKV_MAX_ROWS];
    const float *anc = unit_anchors(a, un, u, T, sanc);
    const float sc = a.inv_sqrt_d * kLog2e;

    bf16x8 aq[MT][8];
    load_query_operands<MT>(a, un, lane, aq);
    {
        // anchor rows: kAnc + 0: mu high, +1: mu remainder
        const int rr = 32 * (MT - 1) + (lane & 31);
        if (rr >= kAnc) mu_operand(anc + kD, rr - kAnc, h, aq[MT - 1]);
    }
    float kbv[8][8];  // kbar at the 64 dimensions this lane holds
    centroid_lane(anc, h, kbv);
    if (tid < 32 * MT) {
        const bool ok = tid < a.R;
        rowM[tid] = ok ? anc[2 * kD + tid] : 0.f;
        rowIS[tid] = ok ? 1.f / anc[2 * kD + a.R + tid] : 0.f;
    }

    float dsum = 0.f, dsq = 0.f, dmn = INFINITY, dmx = -INFINITY;
    const float inv_r = 1.f / (float)a.R;
    const int ntiles = min(a.rpb2 / kTile, (T - row_base + kTile - 1) / kTile);
    tile_pipeline(pf, kt, rs, row_base, ntiles, g, c, [&](int tr0) {

        f32x16 acc[MT];
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = (f32x16){};
        float n2 = 0.f;
        {
            const int r = 32 * wv + (lane & 31);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const u32x4 bq = kt[sw(r, 2 * s + h)];
                n2 = dot2sq(bq[0], dot2sq(bq[1], dot2sq(bq[2], dot2sq(bq[3], n2))));
                const bf16x8 b = __builtin_bit_cast(bf16x8, bq);
#pragma unroll
                for (int t = 0; t < MT; ++t)
                    acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[t][s], b, acc[t], 0, 0, 0);
            }
        }
        float att = 0.f;
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = 32 * t + 8 * (i >> 2) + 4 * h + (i & 3);
                if (m < a.R) att = fmaf(fast_exp2(fmaf(acc[t][i], sc, -rowM[m])), rowIS[m], att);
            }
        float kmu = h ? acc[MT - 1][14] + acc[MT - 1][15] : 0.f;
        float d2;
        {
            const int r = 32 * wv + (lane & 31);
            u32x4 bq[8];
#pragma unroll
            for (int s = 0; s < 8; ++s) bq[s] = kt[sw(r, 2 * s + h)];
            d2 = dist2_lane(bq, kbv);
        }
        n2 += __shfl_xor(n2, 32, kWave);
        att += __shfl_xor(att, 32, kWave);
        kmu += __shfl_xor(kmu, 32, kWave);
        d2 += __shfl_xor(d2, 32, kWave);
        const float dE = __builtin_amdgcn_sqrtf(d2);
        const float cm = kmu * __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
        const int gi = tr0 + 32 * wv + (lane & 31);
        if (h == 0) {
            if (gi < T) {
                dsum += dE;
                dsq += dE * dE;
            }
            if (gi < P) {
                dmn = fminf(dmn, dE);
                dmx = fmaxf(dmx, dE);
                a.bufA[obase + gi] = dE;
                a.bufB[obase + gi] = cm;
                a.bufC[obase + gi] = att * inv_r;
            }
        }
    });

    dsum = wave_sum(dsum);
    dsq = wave_sum(dsq);
    dmn = wave_min(dmn);
    dmx = wave_max(dmx);
    if (lane == 0) {
        wred[0][wv] = dsum;
        wred[1][wv] = dmn;
        wred[2][wv] = dmx;
        wred[3][wv] = dsq;
    }
    lds_barrier();
    if (tid == 0) {
        float s = 0.f, s2 = 0.f, mn = INFINITY, mx = -INFINITY;
        for (int k = 0; k < 4; ++k) {
            s += wred[0][k];
            mn = fminf(mn, wred[1][k]);
            mx = fmaxf(mx, wred[2][k]);
            s2 += wred[3][k];
        }
        float *pp = a.part2 + ((int64_t)u * a.nch2 + blockIdx.x) * 4;
        pp[0] = s;
        pp[1] = mn;
        pp[2] = mx;
        pp[3] = s2;
    }
}

// Sweep 2, streaming form (window rows + 2 rows of mu in one 32-row operand,
// i.e. G*w <= 30): no LDS tile and no barrier in the key loop.  Each wave
// streams its own 512 keys in groups of 32 from HBM into registers (three
// groups in flight), re-lays them out through a wave-private LDS stage into
// MFMA B operands (lane l: key l % 32, 16-byte chunks 2s + l / 32).  The
// attention of row m is 2^(x - M'_m) with M'_m = M_m + log2(S_m), the
// normaliser folded into the shift.  2048-key blocks (1024 and 4096 measured
// no better); 1024- or 512-key blocks when a call has too few keys to fill
// the device with 2048-key ones (one layer, say).
constexpr int kS2Waves = 4;
constexpr int kS2Keys = 2048;       // keys per block
constexpr int kS2KeysMid = 1024;    // keys per block for calls with fewer blocks
constexpr int kS2KeysSmall = 512;   // keys per block for calls with few blocks

// Coalesced load of 32 key rows: instruction i covers rows 4i .. 4i+3, lane l
// chunk l % 16 of row 4i + l / 16 (four whole 256-byte rows per instruction).
// Nontemporal (cache policy nt): K streams through once per sweep, and keeping
// it out of the caches makes both sweeps 15-20 us faster.
__device__ __forceinline__ void group_load(u32x4 (&b)[8], __amdgpu_buffer_rsrc_t rs, int key0, int lane)
{
#pragma unroll
    for (int i = 0; i < 8; ++i)
        b[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (key0 + 4 * i + (lane >> 4)) * (kD * 2) + (lane & 15) * 16, 0, 2);
}

template <int KEYS>
__global__ __launch_bounds__(256, 2) void k_fs2s(ScoreArgs a)
{
    bump_call_tag(a);
    constexpr int kS2Groups = KEYS / (32 * kS2Waves);  // 32-key groups per wave
    __shared__ float wred[4][kS2Waves];
    __shared__ u32x4 stage[kS2Waves][32 * kChunks];  // per wave: 32 rows, swizzled 16-byte chunks
    __shared__ float wd2[kS2Waves][32];               // per wave: |k - kbar|^2 of its 32 rows
    // the block's per-key outputs (d_E, khat.mu, a), written out once at the end:
    // a few long stores instead of three 128-byte stores per 32 keys, which
    // interleave with the read stream at a high price
    __shared__ __attribute__((aligned(16))) float outs[3][KEYS];
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row_base = blockIdx.x * KEYS;
    if (row_base >= T) return;
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, kl = lane & 31;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const int64_t obase = unit_out_base(a, un);
    __shared__ __attribute__((aligned(16))) float sanc[2 * kD + 2 * ECOKV_MAX_ROWS];
    const float *anc = unit_anchors(a, un, u, T, sanc);
    const float sc = a.inv_sqrt_d * kLog2e;
    constexpr int kAnc = 32 - 2;

    // A operand: window rows (zero beyond R), rows 30, 31 mu high / remainder
    bf16x8 aq[1][8];
    load_query_operands<1>(a, un, lane, aq);
    if (kl >= kAnc) mu_operand(anc + kD, kl - kAnc, h, aq[0]);
    // kbar at the 8 dimensions of chunk lane % 16, the chunk this lane loads
    float kbc[8];
    {
        const float4 *src = reinterpret_cast<const float4 *>(anc + 8 * (lane & 15));
        const float4 x = src[0], y = src[1];
        kbc[0] = x.x; kbc[1] = x.y; kbc[2] = x.z; kbc[3] = x.w;
        kbc[4] = y.x; kbc[5] = y.y; kbc[6] = y.z; kbc[7] = y.w;
    }
    // per-lane row shifts M'_m for the rows m = 8(r/4) + 4h + r%4 of accumulator r
    float rsh[16];
    {
        float mv[16], sv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int m = min(8 * (r >> 2) + 4 * h + (r & 3), a.R - 1);
            mv[r] = anc[2 * kD + m];
            sv[r] = anc[2 * kD + a.R + m];
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int m = 8 * (r >> 2) + 4 * h + (r & 3);
            rsh[r] = m < a.R ? mv[r] + __log2f(sv[r]) : INFINITY;
        }
    }

    // this wave's keys [wbase, wbase + 32 kS2Groups) only: loads past them read zero, no traffic
    const int wbase = row_base + wv * (32 * kS2Groups);
    const int wkeys = __builtin_amdgcn_readfirstlane(max(0, min(32 * kS2Groups, T - wbase)));
    const __amdgpu_buffer_rsrc_t rs = key_rows_rsrc(krow0 + (int64_t)wbase * kD, wkeys);
    float dsum = 0.f, dsq = 0.f, dmn = INFINITY, dmx = -INFINITY;
    const float inv_r = 1.f / (float)a.R;

    u32x4 *wst = stage[wv];
    float *wd = wd2[wv];
    auto group = [&](const u32x4 (&ld)[8], int key0, bool valid) {
        // |k - kbar|^2 in the load layout (lane l: chunk l % 16 of rows 4i + l / 16):
        // the differences in fp32, summed over the lane's 8 dimensions, then
        // over the 16 lanes of a row by DPP; one lane per row parks the sum
        {
            float dp[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                float s0 = 0.f, s1 = 0.f;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float d0 = __uint_as_float(ld[i][e] << 16) - kbc[2 * e];
                    const float d1 = __uint_as_float(ld[i][e] & 0xffff0000u) - kbc[2 * e + 1];
                    s0 = fmaf(d0, d0, s0);
                    s1 = fmaf(d1, d1, s1);
                }
                dp[i] = row_sum<16>(s0 + s1);
            }
            if ((lane & 15) == 0) {
#pragma unroll
                for (int i = 0; i < 8; ++i) wd[4 * i + (lane >> 4)] = dp[i];
            }
        }
        // through this wave's LDS stage into the B-operand layout (lane l: key
        // l % 32, chunks 2s + l / 32); a wave's own LDS accesses are ordered
#pragma unroll
        for (int i = 0; i < 8; ++i) wst[sw(4 * i + (lane >> 4), lane & 15)] = ld[i];
        u32x4 b[8];
#pragma unroll
        for (int st = 0; st < 8; ++st) b[st] = wst[sw(kl, 2 * st + h)];
        f32x16 acc = (f32x16){};
        float n2 = 0.f;
#pragma unroll
        for (int st = 0; st < 8; ++st) {
            n2 = dot2sq(b[st][0], dot2sq(b[st][1], dot2sq(b[st][2], dot2sq(b[st][3], n2))));
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[0][st], __builtin_bit_cast(bf16x8, b[st]), acc, 0, 0, 0);
        }
        float att = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) att += fast_exp2(fmaf(acc[r], sc, -rsh[r]));
        float kmu = h ? acc[14] + acc[15] : 0.f;
        n2 += __shfl_xor(n2, 32, kWave);
        att += __shfl_xor(att, 32, kWave);
        kmu += __shfl_xor(kmu, 32, kWave);
        const float dE = __builtin_amdgcn_sqrtf(wd[kl]);
        const float cm = kmu * __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
        const int gi = key0 + kl;
        if (valid && h == 0) {
            if (gi < T) {
                dsum += dE;
                dsq += dE * dE;
            }
            if (gi < P) {
                dmn = fminf(dmn, dE);
                dmx = fmaxf(dmx, dE);
            }
            outs[0][gi - row_base] = dE;
            outs[1][gi - row_base] = cm;
            outs[2][gi - row_base] = att * inv_r;
        }
    };

    // Four register buffers in a ring: three groups (24 KiB per wave) stay in
    // flight while one is used.  Every load is unconditional (the descriptor
    // zero-fills past the wave's keys), so the outstanding-load count is the
    // same on every path and each wait covers only the group about to be used.
    const int ng = (wkeys + 31) >> 5;
    // Waves start at different groups of their range (rotation rot), so that
    // at any moment they read different offsets rather than the same offset
    // of equally sized, equally aligned ranges (which would crowd the same
    // memory channels).  Slot g >= ng reads past the range: zeros, skipped.
    const int rot = ng > 0 ? __builtin_amdgcn_readfirstlane(
                                 (int)(((unsigned)(blockIdx.x * kS2Waves + wv) * 2654435761u + blockIdx.y * 40503u) % (unsigned)ng))
                           : 0;
    auto goff = [&](int g) { return g < ng ? 32 * (g + rot < ng ? g + rot : g + rot - ng) : 32 * ng; };
    u32x4 b0[8], b1[8], b2[8], b3[8];
    group_load(b0, rs, goff(0), lane);
    group_load(b1, rs, goff(1), lane);
    group_load(b2, rs, goff(2), lane);
#pragma unroll 1
    for (int g = 0; g < ng; g += 4) {
        group_load(b3, rs, goff(g + 3), lane);
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the use
        group(b0, wbase + goff(g), g < ng);
        group_load(b0, rs, goff(g + 4), lane);
        __builtin_amdgcn_sched_barrier(0);
        group(b1, wbase + goff(g + 1), g + 1 < ng);
        group_load(b1, rs, goff(g + 5), lane);
        __builtin_amdgcn_sched_barrier(0);
        group(b2, wbase + goff(g + 2), g + 2 < ng);
        group_load(b2, rs, goff(g + 6), lane);
        __builtin_amdgcn_sched_barrier(0);
        group(b3, wbase + goff(g + 3), g + 3 < ng);
    }

    dsum = wave_sum(dsum);
    dsq = wave_sum(dsq);
    dmn = wave_min(dmn);
    dmx = wave_max(dmx);
    if (lane == 0) {
        wred[0][wv] = dsum;
        wred[1][wv] = dmn;
        wred[2][wv] = dmx;
        wred[3][wv] = dsq;
    }
    __syncthreads();
    {
        // keys row_base .. of the unit's P non-window keys; the descriptors end at P
        float *const dst[3] = {a.bufA + obase, a.bufB + obase, a.bufC + obase};
        typedef float f32x4v __attribute__((ext_vector_type(4)));
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            const __amdgpu_buffer_rsrc_t ro =
                __builtin_amdgcn_make_buffer_rsrc(dst[t], (short)0, P * 4, 0x00020000);
            // cache policy sc1 (system scope): the outputs are written through
            // instead of lingering dirty in the caches while K streams in
            // (28-layer stack, sweep 2: default policy 173 us, nt 170, sc1 163;
            // sc0 175, nt + sc1 172)
#pragma unroll
            for (int i = 4 * tid; i < KEYS; i += 4 * 256) {
                const f32x4v v = *reinterpret_cast<const f32x4v *>(&outs[t][i]);
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), ro, (row_base + i) * 4, 0, 16);
            }
        }
    }
    if (tid == 0) {
        float s = 0.f, s2 = 0.f, mn = INFINITY, mx = -INFINITY;
        for (int k = 0; k < kS2Waves; ++k) {
            s += wred[0][k];
            mn = fminf(mn, wred[1][k]);
            mx = fmaxf(mx, wred[2][k]);
            s2 += wred[3][k];
        }
        float *pp = a.part2 + ((int64_t)u * a.nch2 + blockIdx.x) * 4;
        pp[0] = s;
        pp[1] = mn;
        pp[2] = mx;
        pp[3] = s2;
    }
}

// Sweep 1, streaming form (bf16, head_dim 128, G*w <= 32): like the streaming
// sweep 2, each wave streams its own 512 keys in 32-key groups (coalesced
// loads, three register buffers in flight, a wave-private LDS stage) and no
// barrier is needed until the final merge of the four waves.
//  * window logits: v_mfma_f32_32x32x16_bf16 with the keys as the A operand and
//    the window rows as B, so each lane holds one window row against 16 keys
//    and keeps that row's running softmax maximum and sum on its own (the
//    reference moves only when a group exceeds it by more than 2^16);
//  * column sums of k and of k/|k|: v_mfma_f32_16x16x32_bf16 per 16-dimension
//    block with rows (1, 1/|k| high, remainder, 0...) over the wave's 32 keys
//    as A, and the keys transposed out of the stage with ds_read_b64_tr_b16
//    as B.
constexpr float kRebase1 = 16.f;  // log2 headroom of the lazily moved row reference

//
// With CACHE (the KV-cache write of ecokv_prefill_write), each key row is read
// from the token-major new rows a.Ksrc and the loaded registers are written to
// the head-major cache a.K on arrival, before the group is used: one read and
// one write of K, and the sweep rides on them.
template <int KEYS, bool CACHE>
__global__ __launch_bounds__(256, 2) void k_fs1s(ScoreArgs a)
{
    constexpr int kS2Groups = KEYS / (32 * kS2Waves);  // 32-key groups per wave
    __shared__ u32x4 stage[kS2Waves][32 * kChunks];
    __shared__ __attribute__((aligned(16))) uint16_t wts[kS2Waves][4][32];  // 1, 1/|k| hi, remainder, 0
    __shared__ float wcs[kS2Waves][2][kD];                                 // per-wave column sums
    __shared__ float wm[kS2Waves][32], wsm[kS2Waves][32];                  // per-wave row max / sum

    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row_base = blockIdx.x * KEYS;
    if (row_base >= T) return;
    const int tid = threadIdx.x, lane = tid & 63, h = lane >> 5, kl = lane & 31;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const float sc = a.inv_sqrt_d * kLog2e;
    const int lim = a.causal ? P + kl % a.w : T - 1;  // last key visible to window row kl

    bf16x8 aq[1][8];
    load_query_operands<1>(a, un, lane, aq);
    if (lane < 32) {
        wts[wv][0][lane] = 0x3f80;
        wts[wv][3][lane] = 0;
    }

    const int wbase = row_base + wv * (32 * kS2Groups);
    const int wkeys = __builtin_amdgcn_readfirstlane(max(0, min(32 * kS2Groups, T - wbase)));
    // CACHE: key i of the unit at row (l Ttot + cu[s] + i) Hkv + h of the new rows
    const int src_row_bytes = CACHE ? a.Hkv * kD * 2 : kD * 2;
    const __amdgpu_buffer_rsrc_t rs =
        CACHE ? __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<uint16_t *>(uniform_ptr(static_cast<const uint16_t *>(a.Ksrc) +
                                                       (((int64_t)un.l * a.Ttot + a.seq.cu[un.s] + wbase) * a.Hkv +
                                                        un.h) * kD)),
                    (short)0, wkeys * src_row_bytes, 0x00020000)
              : key_rows_rsrc(krow0 + (int64_t)wbase * kD, wkeys);
    const __amdgpu_buffer_rsrc_t rdst = key_rows_rsrc(krow0 + (int64_t)wbase * kD, CACHE ? wkeys : 0);
    u32x4 *wst = stage[wv];

    float ms = -INFINITY, ss = 0.f;  // window row kl over this lane's keys
    typedef float f32x4v __attribute__((ext_vector_type(4)));
    f32x4v cs[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) cs[b] = (f32x4v){0.f, 0.f, 0.f, 0.f};
    // transposed-read addressing: lane 16G + 4a + b reads key row 8G + a (+4),
    // dimensions 16 blk + 4b .. +3; the read returns dimension 16 blk + lane % 16
    // of keys 8G + 0..3 (then 4..7)
    const int tr_row = 8 * (lane >> 4) + ((lane & 15) >> 2), tr_b = lane & 3;
    const int w_row = (lane & 15) < 3 ? (lane & 15) : 3;

    auto group = [&](const u32x4 (&ld)[8], int key0, bool valid) {
        if constexpr (CACHE) group_store(ld, rdst, key0 - wbase, lane);  // (rows past the wave's end are dropped)
#pragma unroll
        for (int i = 0; i < 8; ++i) wst[sw(4 * i + (lane >> 4), lane & 15)] = ld[i];
        u32x4 b[8];
#pragma unroll
        for (int st = 0; st < 8; ++st) b[st] = wst[sw(kl, 2 * st + h)];
        f32x16 acc = (f32x16){};
        float n2 = 0.f;
#pragma unroll
        for (int st = 0; st < 8; ++st) {
            n2 = dot2sq(b[st][0], dot2sq(b[st][1], dot2sq(b[st][2], dot2sq(b[st][3], n2))));
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, b[st]), aq[0][st], acc, 0, 0, 0);
        }
        n2 += __shfl_xor(n2, 32, kWave);
        const float inv = __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
        if (h == 0) {
            const unsigned hi = bf16_rne(inv);
            wts[wv][1][kl] = (uint16_t)hi;
            wts[wv][2][kl] = (uint16_t)bf16_rne(inv - __uint_as_float(hi << 16));
        }
        // softmax statistics of row kl over keys key0 + 8(r/4) + 4h + r%4
        if (valid) {
            float x[16];
            float mx = -INFINITY;
            if (key0 + 32 <= P) {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    x[r] = acc[r] * sc;
                    mx = fmaxf(mx, x[r]);
                }
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gk = key0 + 8 * (r >> 2) + 4 * h + (r & 3);
                    x[r] = (gk < T && gk <= lim) ? acc[r] * sc : -INFINITY;
                    mx = fmaxf(mx, x[r]);
                }
            }
            const bool move = mx > ms + kRebase1 || (ms == -INFINITY && mx != -INFINITY);
            const float nm = move ? mx : ms;
            if (nm != -INFINITY) {
                float add = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) add += fast_exp2(x[r] - nm);
                ss = (move ? ss * fast_exp2(ms - nm) : ss) + add;
                ms = nm;
            }
        }
        // column sums over the wave's 32 keys (zero rows past T add nothing)
        const bf16x8 wa = *reinterpret_cast<const bf16x8 *>(&wts[wv][w_row][8 * (lane >> 4)]);
        typedef short s16x4 __attribute__((ext_vector_type(4)));
        const uint16_t *st16 = reinterpret_cast<const uint16_t *>(wst);
#pragma unroll
        for (int blk = 0; blk < 8; ++blk) {
            const int c = 2 * blk + (tr_b >> 1), off = (tr_b & 1) * 4;
            const uint16_t *p0 = st16 + tr_row * kD + ((c ^ (tr_row & 15)) << 3) + off;
            const uint16_t *p1 = st16 + (tr_row + 4) * kD + ((c ^ ((tr_row + 4) & 15)) << 3) + off;
            const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p0)));
            const s16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p1)));
            const short __attribute__((ext_vector_type(8))) kb8 = {lo[0], lo[1], lo[2], lo[3],
                                                                    hi4[0], hi4[1], hi4[2], hi4[3]};
            cs[blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, __builtin_bit_cast(bf16x8, kb8), cs[blk], 0, 0, 0);
        }
    };

    const int ng = (wkeys + 31) >> 5;
    const int rot = ng > 0 ? __builtin_amdgcn_readfirstlane(
                                 (int)(((unsigned)(blockIdx.x * kS2Waves + wv) * 2654435761u + blockIdx.y * 40503u) % (unsigned)ng))
                           : 0;
    auto goff = [&](int g) { return g < ng ? 32 * (g + rot < ng ? g + rot : g + rot - ng) : 32 * ng; };
    u32x4 b0[8], b1[8], b2[8];
    group_load_rows(b0, rs, goff(0), lane, src_row_bytes);
    group_load_rows(b1, rs, goff(1), lane, src_row_bytes);
#pragma unroll 1
    for (int g = 0; g < ng; g += 3) {
        group_load_rows(b2, rs, goff(g + 2), lane, src_row_bytes);
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the use
        group(b0, wbase + goff(g), g < ng);
        group_load_rows(b0, rs, goff(g + 3), lane, src_row_bytes);
        __builtin_amdgcn_sched_barrier(0);
        group(b1, wbase + goff(g + 1), g + 1 < ng);
        group_load_rows(b1, rs, goff(g + 4), lane, src_row_bytes);
        __builtin_amdgcn_sched_barrier(0);
        group(b2, wbase + goff(g + 2), g + 2 < ng);
    }

    // merge: halves of a row, then the four waves (fixed order)
    {
        const float m2 = __shfl_xor(ms, 32, kWave), s2 = __shfl_xor(ss, 32, kWave);
        softmax_merge2(ms, ss, m2, s2);
    }
    if (lane < 32) {
        wm[wv][lane] = ms;
        wsm[wv][lane] = ss;
    }
    if (lane < 16) {
#pragma unroll
        for (int blk = 0; blk < 8; ++blk) {
            wcs[wv][0][16 * blk + lane] = cs[blk][0];
            wcs[wv][1][16 * blk + lane] = cs[blk][1] + cs[blk][2];
        }
    }
    __syncthreads();
    const int stride = 2 * kD + 2 * a.R;
    float *part = a.part1 + ((int64_t)u * a.nch1 + blockIdx.x) * stride;
    for (int i = tid; i < 2 * kD; i += blockDim.x) {
        const int which = i / kD, d = i % kD;
        float s = 0.f;
        for (int w2 = 0; w2 < kS2Waves; ++w2) s += wcs[w2][which][d];
        part[i] = s;
    }
    if (tid < a.R) {
        float m = wm[0][tid], s = wsm[0][tid];
        for (int w2 = 1; w2 < kS2Waves; ++w2) softmax_merge2(m, s, wm[w2][tid], wsm[w2][tid]);
        part[2 * kD + tid] = m;
        part[2 * kD + a.R + tid] = s;
    }
}

}  // namespace fast

// ---------------------------------------------------------------------------
// Per-unit reduction of the sweep-1 partials.
// ---------------------------------------------------------------------------
// Columns of a unit's partial rows: sum k (D), sum k/|k| (D), the R window
// rows' (max, normaliser) pairs.  `lanes` lanes per column, each over every
// lanes-th block partial with its loads in flight together, then combined by
// butterflies of commutative steps, so every lane ends with the same value.
// Up to 16 partials per unit: 4 lanes, one block per unit looping over the
// columns; more (64 for a 32 Ki-token unit in 512-key blocks): 16 lanes, grid
// (unit, column group of 64), so that no lane waits on a chain of loads
// (one layer: 9 -> 7 us; the 28-layer stack in 2048-key blocks is 0.7 us
// faster with one block per unit).
constexpr int kReduceThreads = 1024;
inline int reduce1_lanes(int nch1) { return nch1 > 16 ? 16 : 4; }

// With PRE (ecokv_prefill_write) the unit's sums are written to a.pre_out in
// the layout ecokv_score_pre takes: plain sums, and the row maxima in natural
// units (max q.k / sqrt(D)).
// op over an aligned group of 4 or 16 lanes (a quad, a DPP row), every lane
// getting the result.
template <int LANES, class Op>
__device__ __forceinline__ float lane_group_reduce(float x, Op op)
{
    static_assert(LANES == 4 || LANES == 16, "a quad or a 16-lane row");
    if constexpr (LANES == 16) return row_reduce<16>(x, op);
    x = op(x, dpp_row<0xB1>(x));  // quad_perm [1, 0, 3, 2]
    return op(x, dpp_row<0x4E>(x));  // quad_perm [2, 3, 0, 1]
}

// Columns cg, cg + ncg, ... (in groups of blockDim.x / LANES) of unit u's
// partials, LANES lanes per column; the calling block's threads all take part.
template <int LANES, bool PRE>
__device__ __forceinline__ void reduce1_columns(const ScoreArgs &a, int u, int cg, int ncg)
{
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int nb = (T + a.rpb1 - 1) / a.rpb1;
    const int stride = 2 * a.D + 2 * a.R;
    const float *p = a.part1 + (int64_t)u * a.nch1 * stride;
    float *anc = (PRE ? a.pre_out : a.anchors) + (int64_t)u * stride;
    constexpr int lanes = LANES;
    const int cpb = blockDim.x / lanes;  // columns per block per step
    const int q = threadIdx.x & (lanes - 1);
    // (every lane of a column takes the same path: the butterflies stay within it)
    for (int c = cg * cpb + threadIdx.x / lanes; c < 2 * a.D + a.R; c += ncg * cpb) {
        if (c < 2 * a.D) {
            float s = 0.f;
#pragma unroll 4
            for (int b = q; b < nb; b += lanes) s += p[(int64_t)b * stride + c];
            s = lane_group_reduce<lanes>(s, OpAdd{});
            if (q == 0) anc[c] = PRE ? s : c < a.D ? centroid_component(a, un, T, c, s) : s / (float)T;
        } else {
            const int r = c - 2 * a.D;
            float m = -INFINITY, s = 0.f;
#pragma unroll 4
            for (int b = q; b < nb; b += lanes)
                softmax_merge2(m, s, p[(int64_t)b * stride + 2 * a.D + r], p[(int64_t)b * stride + 2 * a.D + a.R + r]);
            // the group's largest reference, each lane's sum moved onto it, summed
            const float mg = lane_group_reduce<lanes>(m, OpMax{});
            s = lane_group_reduce<lanes>(m == -INFINITY ? 0.f : s * __builtin_amdgcn_exp2f(m - mg), OpAdd{});
            m = mg;
            if (q == 0) {
                anc[2 * a.D + r] = PRE ? m * (1.f / kLog2e) : m;
                anc[2 * a.D + a.R + r] = s;
            }
        }
    }
}

template <int LANES, bool PRE>
__global__ __launch_bounds__(kReduceThreads) void k_reduce1(ScoreArgs a)
{
    reduce1_columns<LANES, PRE>(a, blockIdx.x, blockIdx.y, gridDim.y);
}

// ---------------------------------------------------------------------------
// Epilogue, two launches over (key blocks, units):
//   epi1: pooled S_imp and S_div of each non-window key; block sums/extrema.
//   epi2: every block derives the unit constants from the partials (same
//         order in every block) and writes S; block 0 writes the statistics.
// Each thread takes 16 consecutive keys with 16-byte buffer loads; the
// descriptors span exactly the unit's P non-window keys, so the pooling halo
// reads zero outside [0, P) (the zero padding of the average pool).
// ---------------------------------------------------------------------------
constexpr int kEpiThreads = 256;
constexpr int kEpiPer = 16;                      // consecutive keys per thread
constexpr int kEpiKeys = kEpiThreads * kEpiPer;  // keys per block
constexpr int kPoolHalfMax = 4;                  // vector pooling for kernels up to 9

struct Red4 {
    float s0, s1, mn, mx;
};

__device__ Red4 block_red4(Red4 v, Red4 *lds)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v.s0 = wave_sum(v.s0);
    v.s1 = wave_sum(v.s1);
    v.mn = wave_min(v.mn);
    v.mx = wave_max(v.mx);
    if (lane == 0) lds[wv] = v;
    __syncthreads();
    Red4 r = lds[0];
    for (int k = 1; k < nw; ++k) {
        r.s0 += lds[k].s0;
        r.s1 += lds[k].s1;
        r.mn = fminf(r.mn, lds[k].mn);
        r.mx = fmaxf(r.mx, lds[k].mx);
    }
    __syncthreads();
    return r;
}

__device__ __forceinline__ float pooled(const float *abuf, int i, int P, int half)
{
    float acc = 0.f;
    for (int t = -half; t <= half; ++t) {
        const int k = i + t;
        if (k >= 0 && k < P) acc += abuf[k];
    }
    return acc * (1.f / (float)(2 * half + 1));
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t float_rsrc(const float *p, int n)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(p), (short)0, n * 4, 0x00020000);
}

// d_E and khat.mu of keys i0 .. i0+PER-1 (zero past P).
template <int PER>
__device__ __forceinline__ void load_dc(const float *dbuf, const float *cbuf, int P, int i0, float (&d)[PER],
                                        float (&c)[PER])
{
    const __amdgpu_buffer_rsrc_t rd = float_rsrc(dbuf, P), rc = float_rsrc(cbuf, P);
#pragma unroll
    for (int q = 0; q < PER / 4; ++q) {
        const f32x4 x = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rd, (i0 + 4 * q) * 4, 0, 0));
        const f32x4 y = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rc, (i0 + 4 * q) * 4, 0, 0));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            d[4 * q + e] = x[e];
            c[4 * q + e] = y[e];
        }
    }
}

// Pooled window attention S_imp of keys i0 .. i0+PER-1 (zero past P).
template <int PER>
__device__ __forceinline__ void load_imp(const ScoreArgs &a, const float *abuf, int P, int i0, float (&imp)[PER])
{
    const __amdgpu_buffer_rsrc_t ra = float_rsrc(abuf, P);
    const int half = a.pool_half;
    const float inv_k = 1.f / (float)(2 * half + 1);
    if (half <= kPoolHalfMax) {
        // av[j] = a[i0 - 4 + j]; a negative offset wraps past the range and reads zero
        float av[PER + 2 * kPoolHalfMax];
#pragma unroll
        for (int q = 0; q < (PER + 2 * kPoolHalfMax) / 4; ++q) {
            const f32x4 x = __builtin_bit_cast(
                f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, (unsigned)(i0 - kPoolHalfMax + 4 * q) * 4u, 0, 0));
#pragma unroll
            for (int e = 0; e < 4; ++e) av[4 * q + e] = x[e];
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            float acc = 0.f;
#pragma unroll
            for (int t = -kPoolHalfMax; t <= kPoolHalfMax; ++t)
                if (t >= -half && t <= half) acc += av[j + kPoolHalfMax + t];
            imp[j] = acc * inv_k;
        }
    } else {
#pragma unroll
        for (int j = 0; j < PER; ++j) imp[j] = i0 + j < P ? pooled(abuf, i0 + j, P, half) : 0.f;
    }
}

// d_E, khat.mu and pooled window attention of keys i0 .. i0+15 (zero past P).
__device__ __forceinline__ void epi_keys(const ScoreArgs &a, const float *dbuf, const float *cbuf, const float *abuf,
                                         int P, int i0, float (&d)[kEpiPer], float (&c)[kEpiPer],
                                         float (&imp)[kEpiPer])
{
    load_dc<kEpiPer>(dbuf, cbuf, P, i0, d, c);
    load_imp<kEpiPer>(a, abuf, P, i0, imp);
}

// s_E of a distance (the Eq. (2) step): min-max over the unit's non-window
// keys; or, after clipping to the q and 1 - q quantiles, min-max between
// them (winsorised); or a sigmoid of the deviation from the median in units
// of the median absolute deviation (MAD) (Sec. 6.3, Table 4).  The quantile
// pair of a unit comes from k_dquant.
struct DNorm {
    float lo, hi, g;
    int sig;
};

__device__ __forceinline__ DNorm d_norm(const ScoreArgs &a, int u, const Red4 &dst)
{
    DNorm n;
    n.sig = 0;
    if (a.norm_mode == ECOKV_NORM_MINMAX) {
        n.lo = dst.mn;
        n.hi = dst.mx;
        n.g = 1.f / (dst.mx - dst.mn + a.eps);
    } else if (a.norm_mode == ECOKV_NORM_WINSOR) {
        n.lo = a.dq[2 * (int64_t)u];
        n.hi = a.dq[2 * (int64_t)u + 1];
        n.g = 1.f / (n.hi - n.lo + a.eps);
    } else {
        n.lo = a.dq[2 * (int64_t)u];
        n.hi = INFINITY;
        n.g = 1.f / (a.mad_tau * a.dq[2 * (int64_t)u + 1] + a.eps);
        n.sig = 1;
    }
    return n;
}

__device__ __forceinline__ float s_euclid(float d, const DNorm &n)
{
    if (n.sig) return 1.f / (1.f + expf(-(d - n.lo) * n.g));
    return (fminf(fmaxf(d, n.lo), n.hi) - n.lo) * n.g;
}

// The per-unit constants of Eq. (3)-(7) from the unit's reductions: d_E
// (sum and sum of squares over T, min / max over P), S_div (sum, min, max over
// P) and S_imp (sum over P), and |mu|^2.
struct EpiConsts {
    float lam, rE, rC, DE, smin, sden, impmean, sbarmean, scale;
};

__device__ __forceinline__ EpiConsts epi_consts(const ScoreArgs &a, const Red4 &dst, const Red4 &sd, float mu2, int T,
                                                int P)
{
    EpiConsts k;
    k.DE = dst.s0 / (float)T;
    if (a.red_std)  // r_std = 1 - sigmoid(D_std / tau), D_std = sqrt(mean_T d_E^2) (Appendix D)
        k.rE = 1.f - 1.f / (1.f + expf(-sqrtf(dst.s1 / (float)T) / a.tau));
    else
        k.rE = 2.f - 2.f / (1.f + expf(-k.DE / a.tau));
    k.rC = ((float)T * mu2 - 1.f) / ((float)T - 1.f);
    k.lam = a.use_override ? a.lambda_override : a.beta * k.rE + (1.f - a.beta) * k.rC;
    if (sd.s0 != sd.s0) k.lam = NAN;  // the split epilogue's wait gave up (or NaN inputs)
    k.smin = sd.mn;
    k.sden = sd.mx - sd.mn + a.eps;
    k.impmean = sd.s1 / (float)P;
    k.sbarmean = (sd.s0 / (float)P - k.smin) / k.sden;
    k.scale = k.impmean / (k.sbarmean + a.eps);
    return k;
}

__device__ __forceinline__ void epi_write_stats(const ScoreArgs &a, int u, const EpiConsts &k, const Red4 &dst,
                                                const Red4 &sd, float mu2)
{
    float st[ECOKV_NSTATS];
    st[ECOKV_STAT_LAMBDA] = k.lam;
    st[ECOKV_STAT_RC] = k.rC;
    st[ECOKV_STAT_RE] = k.rE;
    st[ECOKV_STAT_DE] = k.DE;
    st[ECOKV_STAT_DMIN] = dst.mn;
    st[ECOKV_STAT_DMAX] = dst.mx;
    st[ECOKV_STAT_SDIV_MIN] = sd.mn;
    st[ECOKV_STAT_SDIV_MAX] = sd.mx;
    st[ECOKV_STAT_IMP_MEAN] = k.impmean;
    st[ECOKV_STAT_SBAR_MEAN] = k.sbarmean;
    st[ECOKV_STAT_MU_NORM2] = mu2;
    st[ECOKV_STAT_SCALE] = k.scale;
    if (a.stats)
        for (int q = 0; q < ECOKV_NSTATS; ++q) a.stats[(int64_t)u * ECOKV_NSTATS + q] = st[q];
    if (a.lambda) a.lambda[u] = k.lam;
}

// Sum, sum of squares, min and max of d_E over the unit, from the sweep-2 partials.
__device__ Red4 unit_distance_stats(const ScoreArgs &a, int u, int T, Red4 *lds)
{
    const int nb = (T + a.rpb2 - 1) / a.rpb2;
    Red4 v{0.f, 0.f, INFINITY, -INFINITY};
    for (int b = threadIdx.x; b < nb; b += blockDim.x) {
        const float *pp = a.part2 + ((int64_t)u * a.nch2 + b) * 4;
        v.s0 += pp[0];
        v.s1 += pp[3];
        v.mn = fminf(v.mn, pp[1]);
        v.mx = fmaxf(v.mx, pp[2]);
    }
    return block_red4(v, lds);
}

__global__ __launch_bounds__(kEpiThreads) void k_epi1(ScoreArgs a)
{
    __shared__ Red4 lds[kEpiThreads / kWave];
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int i0 = blockIdx.x * kEpiKeys;
    if (i0 >= P) return;
    const int i1 = min(i0 + kEpiKeys, P);
    const int64_t ob = unit_out_base(a, un);
    const float *dbuf = a.bufA + ob, *cbuf = a.bufB + ob, *abuf = a.bufC + ob;
    const Red4 dst = unit_distance_stats(a, u, T, lds);
    const DNorm dn = d_norm(a, u, dst);

    Red4 w{0.f, 0.f, INFINITY, -INFINITY};
    {
        const int k0 = i0 + kEpiPer * threadIdx.x;
        float d[kEpiPer], c[kEpiPer], imp[kEpiPer];
        epi_keys(a, dbuf, cbuf, abuf, P, k0, d, c, imp);
#pragma unroll
        for (int j = 0; j < kEpiPer; ++j)
            if (k0 + j < i1) {
                const float sE = s_euclid(d[j], dn);
                const float sC = (1.f - c[j]) * 0.5f;
                const float sdiv = a.alpha * sE + (1.f - a.alpha) * sC;
                w.s0 += sdiv;
                w.s1 += imp[j];
                w.mn = fminf(w.mn, sdiv);
                w.mx = fmaxf(w.mx, sdiv);
            }
    }
    const Red4 r = block_red4(w, lds);
    if (threadIdx.x == 0) {
        float *pp = a.part3 + ((int64_t)u * a.nch3 + blockIdx.x) * 4;
        pp[0] = r.s0;
        pp[1] = r.s1;
        pp[2] = r.mn;
        pp[3] = r.mx;
    }
}

__global__ __launch_bounds__(kEpiThreads) void k_epi2(ScoreArgs a)
{
    __shared__ Red4 lds[kEpiThreads / kWave];
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int i0 = blockIdx.x * kEpiKeys;
    if (i0 >= P) return;
    const int i1 = min(i0 + kEpiKeys, P);
    const int64_t ob = unit_out_base(a, un);
    const float *dbuf = a.bufA + ob, *cbuf = a.bufB + ob, *abuf = a.bufC + ob;


    const Red4 dst = unit_distance_stats(a, u, T, lds);
    Red4 v{0.f, 0.f, INFINITY, -INFINITY};
    const int nb3 = (P + kEpiKeys - 1) / kEpiKeys;
    for (int b = threadIdx.x; b < nb3; b += blockDim.x) {
        const float *pp = a.part3 + ((int64_t)u * a.nch3 + b) * 4;
        v.s0 += pp[0];
        v.s1 += pp[1];
        v.mn = fminf(v.mn, pp[2]);
        v.mx = fmaxf(v.mx, pp[3]);
    }
    const Red4 sd = block_red4(v, lds);
    Red4 m2{0.f, 0.f, 0.f, 0.f};
    for (int d = threadIdx.x; d < a.D; d += blockDim.x) {
        const float mv = anchor_value(a, un, u, T, a.D + d);
        m2.s0 += mv * mv;
    }
    const float mu2 = block_red4(m2, lds).s0;
    const EpiConsts k = epi_consts(a, dst, sd, mu2, T, P);
    const float lam = k.lam, smin = k.smin, sden = k.sden, scale = k.scale;
    const DNorm dn = d_norm(a, u, dst);

    float *out = a.scores + ob;
    {
        const int k0 = i0 + kEpiPer * threadIdx.x;
        float d[kEpiPer], c[kEpiPer], imp[kEpiPer], sv[kEpiPer];
        epi_keys(a, dbuf, cbuf, abuf, P, k0, d, c, imp);
#pragma unroll
        for (int j = 0; j < kEpiPer; ++j) {
            const float sE = s_euclid(d[j], dn);
            const float sC = (1.f - c[j]) * 0.5f;
            const float sdiv = a.alpha * sE + (1.f - a.alpha) * sC;
            sv[j] = lam * (((sdiv - smin) / sden) * scale) + (1.f - lam) * imp[j];
        }
        if (k0 + kEpiPer <= i1) {
            const __amdgpu_buffer_rsrc_t ro = float_rsrc(out, P);
#pragma unroll
            for (int q = 0; q < kEpiPer / 4; ++q) {
                const f32x4 x = {sv[4 * q], sv[4 * q + 1], sv[4 * q + 2], sv[4 * q + 3]};
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), ro, (k0 + 4 * q) * 4, 0, 0);
            }
        } else {
#pragma unroll
            for (int j = 0; j < kEpiPer; ++j)
                if (k0 + j < i1) out[k0 + j] = sv[j];
        }
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) epi_write_stats(a, u, k, dst, sd, mu2);
}

// Epilogue in one launch: each unit's P non-window keys in SPLIT blocks
// (1, 2, 4 or 8) of 4096 KVEC keys (KVEC 1, 2, 4 or 8; at most 65536 keys per
// unit), the host choosing the most blocks per unit that fill at most half
// the device (else two per unit if it holds them; one block of 32768 keys
// when the caller allows no waits).  Every per-unit reduction is
// block-local, except that with SPLIT > 1 the parts of a unit exchange their
// S_div / S_imp sums and extrema once (tagged 64-bit relaxed atomics; the
// parts are combined in a fixed order, so all compute the same constants).
// The wait for the other parts is bounded: if it gives up, the unit's lambda
// and scores come out NaN and the workspace status word records the call's
// tag.  Each key's d_E, khat.mu and attention is read once.  Wave w holds
// KVEC chunks of 256 consecutive keys; lane l of chunk j holds keys
// 256 j + 4 l .. +3 of the wave's range, so each load instruction covers
// 1 KiB of consecutive keys.
// The pooling window (up to 4 keys on each side) comes from the neighbouring
// lanes' registers (or the neighbouring chunk's end lane); the wave's
// outermost neighbours come from the neighbouring waves through LDS, and at
// the ends of a block's range from memory.
constexpr int kUThreads = 1024;
constexpr int kUW = kUThreads / kWave;
constexpr int kUKeys = kUThreads * 32;  // 32768 keys: one block of the one-launch epilogue at most
constexpr int kEpiSplitMax = 8;         // blocks per unit at most
constexpr int kEpiUnitMax = 2 * kUKeys; // keys per unit at most (65536)

// Block sum / min / max whose barriers order LDS only, so that global loads
// issued before it stay in flight.
__device__ Red4 block_red4_lds(Red4 v, Red4 *lds)
{
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v.s0 = wave_sum(v.s0);
    v.s1 = wave_sum(v.s1);
    v.mn = wave_min(v.mn);
    v.mx = wave_max(v.mx);
    if (lane == 0) lds[wv] = v;
    lds_barrier();
    Red4 r = lds[0];
    for (int k = 1; k < nw; ++k) {
        r.s0 += lds[k].s0;
        r.s1 += lds[k].s1;
        r.mn = fminf(r.mn, lds[k].mn);
        r.mx = fmaxf(r.mx, lds[k].mx);
    }
    lds_barrier();
    return r;
}

// Whole-wave shifts by one lane (DPP wave_shr:1 / wave_shl:1): lane l gets
// lane l - 1's (resp. l + 1's) value; the lane shifted in gets zero.
__device__ __forceinline__ f32x4 from_prev_lane(f32x4 x)
{
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x[e]), 0x138, 0xF, 0xF, false));
    return r;
}
__device__ __forceinline__ f32x4 from_next_lane(f32x4 x)
{
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x[e]), 0x130, 0xF, 0xF, false));
    return r;
}
__device__ __forceinline__ f32x4 lane_value(f32x4 x, int l)
{
    f32x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x[e]), l));
    return r;
}

__device__ __forceinline__ void epi_tag_store(unsigned long long *p, float v, unsigned tag)
{
    __hip_atomic_store(p, ((unsigned long long)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

template <int SPLIT, int KVEC>
__global__ __launch_bounds__(kUThreads) void k_epi_unit(ScoreArgs a)
{
    static_assert((SPLIT == 1 || SPLIT == 2 || SPLIT == 4 || SPLIT == 8) &&
                      (KVEC == 1 || KVEC == 2 || KVEC == 4 || KVEC == 8) && SPLIT * KVEC * 4096 <= kEpiUnitMax,
                  "1 to 8 blocks of 4096 KVEC keys, at most 65536 keys per unit");
    constexpr int kVec = KVEC;               // chunks (float4 per thread and array)
    constexpr int kWaveKeys = 256 * kVec;    // keys per wave
    constexpr int kPartKeys = kUW * kWaveKeys;
    __shared__ Red4 lds[kUW + 1];
    __shared__ f32x4 svl[kVec][kUThreads];  // S_div of every thread's keys
    __shared__ f32x4 edge[kUW][2];          // per wave: its first and last four attention values
    const int u = blockIdx.x / SPLIT, part = blockIdx.x % SPLIT;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int64_t ob = unit_out_base(a, un);

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int half = a.pool_half;  // <= kPoolHalfMax (checked on the host)
    const int kw = kPartKeys * part + kWaveKeys * wv;

    // every global load first, so that their latencies overlap: the sweep-2
    // partials and mu (d_E sum / extrema and |mu|^2 in one block reduction;
    // one partial and one mu component per thread at most: the host checks
    // that a unit has at most kUThreads sweep-2 blocks, and D <= 128), then
    // d_E, khat.mu and attention of the thread's keys (zero past P), and the
    // attention just outside the block's range (a negative offset wraps past
    // the range and reads zero)
    Red4 v{0.f, 0.f, INFINITY, -INFINITY};
    float dq2 = 0.f;  // this thread's partial sum of d_E^2
    const int nb2 = (T + a.rpb2 - 1) / a.rpb2;
    if ((int)threadIdx.x < nb2) {
        const float *pp = a.part2 + ((int64_t)u * a.nch2 + threadIdx.x) * 4;
        v.s0 = pp[0];
        v.mn = pp[1];
        v.mx = pp[2];
        dq2 = pp[3];
    }
    const float mv = (int)threadIdx.x < a.D ? anchor_value(a, un, u, T, a.D + (int)threadIdx.x) : 0.f;
    const __amdgpu_buffer_rsrc_t rd = float_rsrc(a.bufA + ob, P), rc = float_rsrc(a.bufB + ob, P),
                                 ra = float_rsrc(a.bufC + ob, P);
    f32x4 xd[kVec], xc[kVec], xa[kVec];
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int k4 = kw + 256 * j + 4 * lane;
        xd[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rd, k4 * 4, 0, 0));
        xc[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rc, k4 * 4, 0, 0));
        xa[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, k4 * 4, 0, 0));
    }
    f32x4 bl = {0.f, 0.f, 0.f, 0.f}, br = {0.f, 0.f, 0.f, 0.f};
    if (SPLIT > 1) {
        const int b0 = kPartKeys * part;
        bl = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, (unsigned)(b0 - 4) * 4u, 0, 0));
        br = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ra, (b0 + kPartKeys) * 4, 0, 0));
    }
    __builtin_amdgcn_sched_barrier(0);  // the phases below stay in order (register pressure)

    v.s1 = mv * mv;
    const Red4 dm = block_red4_lds(v, lds);
    const float dsq = a.red_std ? block_red4_lds(Red4{dq2, 0.f, INFINITY, -INFINITY}, lds).s0 : 0.f;
    const Red4 dst{dm.s0, dsq, dm.mn, dm.mx};
    const float mu2 = dm.s1;

    // S_div, kept in LDS (each thread reads back only its own values)
    const DNorm dn = d_norm(a, u, dst);
    Red4 w{0.f, 0.f, INFINITY, -INFINITY};
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const int k4 = kw + 256 * j + 4 * lane;
        f32x4 sv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float sE = s_euclid(xd[j][e], dn);
            const float sC = (1.f - xc[j][e]) * 0.5f;
            sv[e] = a.alpha * sE + (1.f - a.alpha) * sC;
            if (k4 + e < P) {
                w.s0 += sv[e];
                w.mn = fminf(w.mn, sv[e]);
                w.mx = fmaxf(w.mx, sv[e]);
            }
        }
        svl[j][threadIdx.x] = sv;
    }
    // the wave's first and last four attention values for its neighbours
    if (lane == 0) edge[wv][0] = xa[0];
    if (lane == 63) edge[wv][1] = xa[kVec - 1];
    lds_barrier();
    const f32x4 hl = wv > 0 ? edge[wv - 1][1] : bl;       // the four keys before the wave's first
    const f32x4 hr = wv < kUW - 1 ? edge[wv + 1][0] : br;  // the four after its last
    __builtin_amdgcn_sched_barrier(0);
    // pooled S_imp (each chunk's attention registers die as its pooled values are made)
    const float inv_k = 1.f / (float)(2 * half + 1);
    f32x4 im[kVec];
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const f32x4 sl = from_prev_lane(xa[j]), sr = from_next_lane(xa[j]);
        const f32x4 pl = j > 0 ? lane_value(xa[j - 1], 63) : hl;  // lane 0: previous chunk's end
        const f32x4 nr = j < kVec - 1 ? lane_value(xa[j + 1], 0) : hr;  // lane 63: next chunk's start
        const f32x4 left = lane == 0 ? pl : sl;
        const f32x4 right = lane == 63 ? nr : sr;
        float win[12];  // keys k4 - 4 .. k4 + 7
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            win[e] = left[e];
            win[4 + e] = xa[j][e];
            win[8 + e] = right[e];
        }
        const int k4 = kw + 256 * j + 4 * lane;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float acc = 0.f;
#pragma unroll
            for (int t = -kPoolHalfMax; t <= kPoolHalfMax; ++t)
                if (t >= -half && t <= half) acc += win[4 + e + t];
            im[j][e] = acc * inv_k;
            if (k4 + e < P) w.s1 += im[j][e];
        }
    }
    Red4 sd = block_red4_lds(w, lds);
    if (SPLIT > 1) {
        // exchange with the other parts of the unit: publish, then wait for each (bounded)
        if (threadIdx.x == 0) {
            const unsigned tag = *a.tagw;  // this call's (bumped by the second sweep)
            unsigned long long *mine = a.epiT + ((int64_t)u * SPLIT + part) * 4;
            epi_tag_store(mine + 0, sd.s0, tag);
            epi_tag_store(mine + 1, sd.s1, tag);
            epi_tag_store(mine + 2, sd.mn, tag);
            epi_tag_store(mine + 3, sd.mx, tag);
            Red4 c{0.f, 0.f, INFINITY, -INFINITY};
            bool all_ok = true;
            for (int pp = 0; pp < SPLIT; ++pp) {  // in part order, so every part adds in the same order
                Red4 r = sd;
                if (pp != part) {
                    const unsigned long long *other = a.epiT + ((int64_t)u * SPLIT + pp) * 4;
                    unsigned long long o[4] = {0ull, 0ull, 0ull, 0ull};
                    bool ok = false;
                    // a spin limit <= 0 (set by the host to exercise this path) gives up at once
                    for (int tries = 0; tries < a.spin_limit && !ok; ++tries) {
                        ok = true;
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            o[q] = __hip_atomic_load(other + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            ok = ok && (unsigned)(o[q] >> 32) == tag;
                        }
                        if (!ok) __builtin_amdgcn_s_sleep(2);
                    }
                    all_ok = all_ok && ok;
                    r = Red4{__uint_as_float((unsigned)o[0]), __uint_as_float((unsigned)o[1]),
                             __uint_as_float((unsigned)o[2]), __uint_as_float((unsigned)o[3])};
                }
                c = pp == 0 ? r : Red4{c.s0 + r.s0, c.s1 + r.s1, fminf(c.mn, r.mn), fmaxf(c.mx, r.mx)};
            }
            if (!all_ok) {
                __hip_atomic_store(a.status, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                c.s0 = NAN;
            }
            lds[kUW] = c;
        }
        lds_barrier();
        sd = lds[kUW];
    }
    const EpiConsts k = epi_consts(a, dst, sd, mu2, T, P);

    const __amdgpu_buffer_rsrc_t ro = float_rsrc(a.scores + ob, P);
    const float gain = k.lam * k.scale / k.sden, one_m = 1.f - k.lam;
#pragma unroll
    for (int j = 0; j < kVec; ++j) {
        const f32x4 sv = svl[j][threadIdx.x];
        f32x4 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) x[e] = (sv[e] - k.smin) * gain + one_m * im[j][e];
        const int k4 = kw + 256 * j + 4 * lane;
        if (k4 + 4 <= P) {
            // (written through, cache policy sc1: 0.7 us less than the default)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), ro, k4 * 4, 0, 16);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (k4 + e < P) a.scores[ob + k4 + e] = x[e];
        }
    }
    if (part == 0 && threadIdx.x == 0) epi_write_stats(a, u, k, dst, sd, mu2);
}

// Clears the workspace status word (a one-thread kernel rather than a memset,
// so that a captured graph holds no memset node).
__global__ void k_status_clear(unsigned *status) { *status = 0u; }

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

hipError_t status_clear(unsigned *status, hipStream_t st)
{
    hipLaunchKernelGGL(k_status_clear, dim3(1), dim3(1), 0, st, status);
    return hipGetLastError();
}

bool score_fast_path(int D, bool bf16) { return bf16 && D == fast::kD; }

static int rows_per_block(int D, bool bf16) { return score_fast_path(D, bf16) ? fast::kRows : kCh; }

// Key rows per block of the block sweeps for a call: 256-key blocks when
// 1024-key ones would be fewer than 1024 (one 8192-token layer: 32 blocks
// on 256 compute units).
static int block_sweep_rows(int D, bool bf16, int U, int maxT)
{
    if (!score_fast_path(D, bf16)) return kCh;
    return (int64_t)U * ((maxT + fast::kRows - 1) / fast::kRows) >= 1024 ? fast::kRows : fast::kSmallRows;
}

// ---------------------------------------------------------------------------
// Value-norm importance (ECOKV_IMP_ATTN_VNORM, Sec. 5.2): S_imp(i) =
// pool(a)(i) * |v_i|_2 for the non-window keys, in one coalesced pass over V.
// A wave takes 64 consecutive rows; its load instruction q covers the 16-byte
// pieces 64q .. 64q+63 of those rows (SEGS pieces per row), so consecutive
// lanes read consecutive bytes.  The SEGS partial sums of squares of a row
// are combined by DPP butterflies and parked in LDS; lane r then pools the window
// attention around row r (zero padding, fixed divisor, as the epilogue) and
// writes the product.  Rows at or past P read as zero (buffer range).
// ---------------------------------------------------------------------------
constexpr int kVnThreads = 256;

template <bool BF16, int SEGS>
__global__ __launch_bounds__(kVnThreads) void k_vnorm(ScoreArgs a)
{
    __shared__ float n2s[kVnThreads];
    constexpr int kRowBytes = SEGS * 16;
    const int u = blockIdx.y;
    const Unit un = unit_of(u, a.Hkv, a.B);
    const int T = a.seq.cu[un.s + 1] - a.seq.cu[un.s];
    const int P = T - a.w;
    const int row0 = blockIdx.x * kVnThreads;
    if (row0 >= P) return;
    const int lane = threadIdx.x & 63, wv = uniform_i32(threadIdx.x >> 6);
    const int wrow = row0 + 64 * wv;                      // the wave's first row
    const int nrows = max(0, min(64, P - wrow));          // rows of the wave below P
    const char *vw = static_cast<const char *>(a.V) + (unit_row0(a, un) + wrow) * kRowBytes;
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<char *>(uniform_ptr(vw)), (short)0, uniform_i32(nrows * kRowBytes), 0x00020000);
    u32x4 x[SEGS];  // (nontemporal: V is read once)
#pragma unroll
    for (int q = 0; q < SEGS; ++q)
        x[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, (64 * q + lane) * 16, 0, 2));
#pragma unroll
    for (int q = 0; q < SEGS; ++q) {
        float s2 = 0.f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if (BF16) {
                const float lo = __uint_as_float(x[q][c] << 16), hi = __uint_as_float(x[q][c] & 0xffff0000u);
                s2 += lo * lo + hi * hi;
            } else {
                const float v = __uint_as_float(x[q][c]);
                s2 += v * v;
            }
        }
        s2 = row_sum<SEGS>(s2);
        if (lane % SEGS == 0) n2s[64 * wv + (64 / SEGS) * q + lane / SEGS] = s2;
    }
    __syncthreads();
    const int i = wrow + lane;
    if (i < P) {
        const int64_t ob = unit_out_base(a, un);
        const float *att = a.bufC + ob;
        float acc = 0.f;
        for (int t = -a.pool_half; t <= a.pool_half; ++t)
            if (i + t >= 0 && i + t < P) acc += att[i + t];
        a.bufV[ob + i] = acc * (1.f / (float)(2 * a.pool_half + 1)) * sqrtf(n2s[threadIdx.x]);
    }
}

static void launch_vnorm(const ScoreArgs &a, dim3 grid, hipStream_t st, bool bf16)
{
    if (bf16 && a.D == 64) hipLaunchKernelGGL((k_vnorm<true, 8>), grid, dim3(kVnThreads), 0, st, a);
    else if (bf16) hipLaunchKernelGGL((k_vnorm<true, 16>), grid, dim3(kVnThreads), 0, st, a);
    else if (a.D == 64) hipLaunchKernelGGL((k_vnorm<false, 16>), grid, dim3(kVnThreads), 0, st, a);
    else hipLaunchKernelGGL((k_vnorm<false, 32>), grid, dim3(kVnThreads), 0, st, a);
}

WsLayout score_ws_layout(int L, int Hkv, int B, int D, int R, int64_t Ptot, int maxT, bool bf16, bool vnorm)
{
    WsLayout w{};
    const int64_t U = (int64_t)L * Hkv * B;
    // the smallest key block of any sweep: the block sweeps' small blocks
    // (the streaming sweeps' are larger)
    const int rpb = min(rows_per_block(D, bf16), fast::kSmallRows);
    const int64_t nch1 = (maxT + rpb - 1) / rpb;
    const int64_t nch2 = nch1;
    const int64_t nch3 = (maxT + kEpiKeys - 1) / kEpiKeys;
    const int64_t stride = 2 * D + 2 * R;
    size_t o = 0;
    w.status = o;  // first: a fixed offset for the status query
    w.tagw = o + sizeof(unsigned);  // then the call tag (any initial value)
    o = align256(o + 2 * sizeof(unsigned));
    w.part1 = o; o = align256(o + sizeof(float) * U * nch1 * stride);
    w.anchors = o; o = align256(o + sizeof(float) * U * stride);
    w.part2 = o; o = align256(o + sizeof(float) * U * nch2 * 4);
    w.part3 = o; o = align256(o + sizeof(float) * U * nch3 * 4);
    w.bufA = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.bufB = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.bufC = o; o = align256(o + sizeof(float) * (int64_t)L * Hkv * Ptot);
    w.bufV = o; o = align256(o + (vnorm ? sizeof(float) * (int64_t)L * Hkv * Ptot : 0));
    w.dq = o; o = align256(o + sizeof(float) * U * 2);
    w.epiT = o; o = align256(o + sizeof(unsigned long long) * U * kEpiSplitMax * 4);
    w.total = o;
    return w;
}

template <int MT1, int MT2>
static void launch_fast_sweep(int pass, const ScoreArgs &a, dim3 grid, hipStream_t st)
{
    if (pass == 1)
        hipLaunchKernelGGL((fast::k_fs1<MT1>), grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL((fast::k_fs2<MT2>), grid, dim3(256), 0, st, a);
}

static void launch_sweep(int pass, const ScoreArgs &a, dim3 grid, hipStream_t st, bool bf16)
{
    if (score_fast_path(a.D, bf16)) {
        // MT1 = ceil(R / 32) tiles of window rows; MT2 also holds the 2 rows of mu.
        const int mt1 = (a.R + 31) / 32, mt2 = (a.R + 2 + 31) / 32;
        if (pass == 1) {
            if (mt1 == 1) launch_fast_sweep<1, 1>(1, a, grid, st);
            else launch_fast_sweep<2, 1>(1, a, grid, st);
        } else {
            if (mt2 == 1) launch_fast_sweep<1, 1>(2, a, grid, st);
            else if (mt2 == 2) launch_fast_sweep<1, 2>(2, a, grid, st);
            else launch_fast_sweep<1, 3>(2, a, grid, st);
        }
        return;
    }
    if (pass == 1) {
        if (bf16) hipLaunchKernelGGL((k_pass1<64, true>), grid, dim3(kThreads), 0, st, a);
        else if (a.D == 128) hipLaunchKernelGGL((k_pass1<128, false>), grid, dim3(kThreads), 0, st, a);
        else hipLaunchKernelGGL((k_pass1<64, false>), grid, dim3(kThreads), 0, st, a);
    } else {
        if (bf16) hipLaunchKernelGGL((k_pass2<64, true>), grid, dim3(kThreads), 0, st, a);
        else if (a.D == 128) hipLaunchKernelGGL((k_pass2<128, false>), grid, dim3(kThreads), 0, st, a);
        else hipLaunchKernelGGL((k_pass2<64, false>), grid, dim3(kThreads), 0, st, a);
    }
}

// Blocks of k_epi_unit<SPLIT, KVEC> that the current device holds at once (cached per device).
template <int SPLIT, int KVEC>
static int64_t epi_split_capacity()
{
    static int64_t cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    if (cache[dev] == 0) {
        int ncu = 0, nb = 0;
        if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, k_epi_unit<SPLIT, KVEC>, kUThreads, 0) != hipSuccess)
            return 0;
        cache[dev] = (int64_t)ncu * nb;
    }
    return cache[dev];
}

// Launches k_epi_unit<SPLIT, KVEC> over U units if its SPLIT U blocks fit
// the device at once (with half: half of it); returns false (nothing
// launched) otherwise.
template <int SPLIT, int KVEC>
static bool try_epi_unit(ScoreArgs &a, char *ws, const WsLayout &lay, int U, hipStream_t st, bool half)
{
    const int64_t cap = epi_split_capacity<SPLIT, KVEC>();
    if ((int64_t)SPLIT * U > (half ? cap / 2 : cap)) return false;
    a.epiT = reinterpret_cast<unsigned long long *>(ws + lay.epiT);
    ECOKV_TIMED("epilogue", st, hipLaunchKernelGGL((k_epi_unit<SPLIT, KVEC>), dim3(SPLIT * U), dim3(kUThreads), 0, st, a));
    return true;
}

hipError_t score_launch(ScoreArgs a, char *ws, const WsLayout &lay, int maxT, hipStream_t st, bool bf16)
{
    const int U = a.L * a.Hkv * a.B;
    a.part1 = reinterpret_cast<float *>(ws + lay.part1);
    a.anchors = reinterpret_cast<float *>(ws + lay.anchors);
    a.part2 = reinterpret_cast<float *>(ws + lay.part2);
    a.part3 = reinterpret_cast<float *>(ws + lay.part3);
    a.bufA = reinterpret_cast<float *>(ws + lay.bufA);
    a.bufB = reinterpret_cast<float *>(ws + lay.bufB);
    a.bufC = reinterpret_cast<float *>(ws + lay.bufC);
    a.nch3 = (maxT + kEpiKeys - 1) / kEpiKeys;
    a.status = reinterpret_cast<unsigned *>(ws + lay.status);
    a.tagw = reinterpret_cast<unsigned *>(ws + lay.tagw);
    const dim3 grid_e(a.nch3, U);
    hipError_t e;

    // streaming sweeps: 2048-key blocks; 1024-key ones when those would be
    // fewer than four per compute unit (1024 blocks) and the 1024-key ones at
    // least two (one layer over 8 sequences of 4k-32k tokens: the pass
    // 186 -> 174 us against 512-key blocks); else 512-key ones
    auto work_blocks = [&](int keys) {
        int64_t nb = 0;
        for (int s = 0; s < a.B; ++s) nb += (a.seq.cu[s + 1] - a.seq.cu[s] + keys - 1) / keys;
        return nb * a.L * a.Hkv;
    };
    const int sblock = work_blocks(fast::kS2Keys) >= 1024  ? fast::kS2Keys
                       : work_blocks(fast::kS2KeysMid) >= 512 ? fast::kS2KeysMid
                                                              : fast::kS2KeysSmall;
    {
        a.rpb1 = block_sweep_rows(a.D, bf16, U, maxT);
        a.nch1 = (maxT + a.rpb1 - 1) / a.rpb1;
        const dim3 grid(a.nch1, U);
        if (a.pre) {
            // the first sweep's sums come from the caller: K is read once (the
            // sweep-2 blocks and the epilogue convert them as they read them)
        } else {
            if (score_fast_path(a.D, bf16) && a.R <= 32) {
                // streaming sweep 1: one 32-row window operand
                a.rpb1 = sblock;
                a.nch1 = (maxT + a.rpb1 - 1) / a.rpb1;
                if (sblock == fast::kS2Keys)
                    ECOKV_TIMED("sweep1_stream", st,
                                hipLaunchKernelGGL((fast::k_fs1s<fast::kS2Keys, false>), dim3(a.nch1, U), dim3(256), 0, st, a));
                else if (sblock == fast::kS2KeysMid)
                    ECOKV_TIMED("sweep1_stream", st,
                                hipLaunchKernelGGL((fast::k_fs1s<fast::kS2KeysMid, false>), dim3(a.nch1, U), dim3(256), 0, st, a));
                else
                    ECOKV_TIMED("sweep1_stream", st,
                                hipLaunchKernelGGL((fast::k_fs1s<fast::kS2KeysSmall, false>), dim3(a.nch1, U), dim3(256), 0, st, a));
            } else {
                ECOKV_TIMED("sweep1_block", st, launch_sweep(1, a, grid, st, bf16));
            }
            if ((e = hipGetLastError()) != hipSuccess) return e;
            if (reduce1_lanes(a.nch1) == 4)
                ECOKV_TIMED("reduce1", st, hipLaunchKernelGGL((k_reduce1<4, false>), dim3(U), dim3(kReduceThreads), 0, st, a));
            else
                ECOKV_TIMED("reduce1", st,
                            hipLaunchKernelGGL((k_reduce1<16, false>), dim3(U, (2 * a.D + a.R + 63) / 64), dim3(kReduceThreads),
                                               0, st, a));
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (score_fast_path(a.D, bf16) && a.R <= kStreamMaxRows) {
            // streaming sweep 2: window rows and the four anchor rows in one operand
            a.rpb2 = sblock;
            a.nch2 = (maxT + a.rpb2 - 1) / a.rpb2;
            if (sblock == fast::kS2Keys)
                ECOKV_TIMED("sweep2_stream", st,
                            hipLaunchKernelGGL(fast::k_fs2s<fast::kS2Keys>, dim3(a.nch2, U), dim3(256), 0, st, a));
            else if (sblock == fast::kS2KeysMid)
                ECOKV_TIMED("sweep2_stream", st,
                            hipLaunchKernelGGL(fast::k_fs2s<fast::kS2KeysMid>, dim3(a.nch2, U), dim3(256), 0, st, a));
            else
                ECOKV_TIMED("sweep2_stream", st,
                            hipLaunchKernelGGL(fast::k_fs2s<fast::kS2KeysSmall>, dim3(a.nch2, U), dim3(256), 0, st, a));
        } else {
            // block sweep 2: the chunking of the block sweeps (grid)
            a.rpb2 = block_sweep_rows(a.D, bf16, U, maxT);
            a.nch2 = (maxT + a.rpb2 - 1) / a.rpb2;
            ECOKV_TIMED("sweep2_block", st, launch_sweep(2, a, grid, st, bf16));
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.vnorm) {
        // the importance with the value norm; the epilogue then reads it as
        // its (already pooled) importance
        a.bufV = reinterpret_cast<float *>(ws + lay.bufV);
        const dim3 gv((maxT - a.w + kVnThreads - 1) / kVnThreads, U);
        ECOKV_TIMED("vnorm", st, launch_vnorm(a, gv, st, bf16));
        if ((e = hipGetLastError()) != hipSuccess) return e;
        a.bufC = a.bufV;
        a.pool_half = 0;
    }
    if (a.norm_mode != ECOKV_NORM_MINMAX) {
        // quantiles of d_E for the winsorised or MAD normalisation
        DQuantArgs qa;
        memset(&qa, 0, sizeof qa);
        qa.d = a.bufA;
        qa.out = reinterpret_cast<float *>(ws + lay.dq);
        qa.L = a.L;
        qa.Hkv = a.Hkv;
        qa.B = a.B;
        qa.w = a.w;
        qa.Ptot = a.Ptot;
        qa.mode = a.norm_mode;
        qa.q = a.winsor_q;
        qa.seq = a.seq;
        if ((e = dquant_launch(qa, st)) != hipSuccess) return e;
        a.dq = qa.out;
    }
    const bool epi_one = a.pool_half <= kPoolHalfMax && (maxT + a.rpb2 - 1) / a.rpb2 <= kUThreads && a.D <= kUThreads;
    const int64_t maxP = maxT - a.w;
    if (epi_one && !a.no_wait && maxP <= kEpiUnitMax) {
        // The one-launch epilogue with the most blocks per unit (4096 KVEC
        // keys each, KVEC = 1, 2, 4) whose blocks fill at most half the
        // device: the parts of a unit wait for each other, and half the
        // device leaves room for a concurrent call on another stream to be
        // resident at once too.  Past that, two blocks per unit when the
        // device holds all of them (a wait across calls is still bounded).
        bool done = false;
        auto fits = [&](int kvec, int split) { return maxP <= (int64_t)4096 * kvec * split; };
        if (fits(1, 1)) {
            ECOKV_TIMED("epilogue", st, hipLaunchKernelGGL((k_epi_unit<1, 1>), dim3(U), dim3(kUThreads), 0, st, a));
            done = true;
        }
        if (!done && fits(1, 8)) {
            if (fits(1, 2)) done = try_epi_unit<2, 1>(a, ws, lay, U, st, true);
            else if (fits(1, 4)) done = try_epi_unit<4, 1>(a, ws, lay, U, st, true);
            else done = try_epi_unit<8, 1>(a, ws, lay, U, st, true);
        }
        if (!done && fits(2, 8)) {
            if (fits(2, 2)) done = try_epi_unit<2, 2>(a, ws, lay, U, st, true);
            else if (fits(2, 4)) done = try_epi_unit<4, 2>(a, ws, lay, U, st, true);
            else done = try_epi_unit<8, 2>(a, ws, lay, U, st, true);
        }
        if (!done && fits(4, 4)) {
            if (fits(4, 2)) done = try_epi_unit<2, 4>(a, ws, lay, U, st, true) || try_epi_unit<2, 4>(a, ws, lay, U, st, false);
            else done = try_epi_unit<4, 4>(a, ws, lay, U, st, true);
        }
        if (done) return hipGetLastError();
    }
    if (epi_one && maxP <= kUKeys) {
        // one block per unit, no waits
        ECOKV_TIMED("epilogue", st, hipLaunchKernelGGL((k_epi_unit<1, 8>), dim3(U), dim3(kUThreads), 0, st, a));
        return hipGetLastError();
    }
    ECOKV_TIMED("epilogue1", st, hipLaunchKernelGGL(k_epi1, grid_e, dim3(kEpiThreads), 0, st, a));
    if ((e = hipGetLastError()) != hipSuccess) return e;
    ECOKV_TIMED("epilogue2", st, hipLaunchKernelGGL(k_epi2, grid_e, dim3(kEpiThreads), 0, st, a));
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// ecokv_prefill_write: the KV-cache write of a prefill with the first sweep.
// ---------------------------------------------------------------------------

// Copy of unit u's rows x * kCopyRows .. x * kCopyRows + 63 from the
// token-major new rows ([L][Ttot][Hkv] rows of rowb bytes) to the head-major
// cache ([L][Hkv][Ttot] rows), 16 bytes per thread and step, streamed past
// the caches.
constexpr int kCopyRows = 64;
__device__ __forceinline__ void copy_unit_rows(const char *src, char *dst, int rowb, int Hkv, int B, int64_t Ttot,
                                               const SeqTab &seq, int u, int x)
{
    const Unit un = unit_of(u, Hkv, B);
    const int T = seq.cu[un.s + 1] - seq.cu[un.s];
    const int r0 = x * kCopyRows;
    if (r0 >= T) return;
    const int rows = min(kCopyRows, T - r0);
    const int pr = rowb / 16;  // 16-byte pieces per row
    const int64_t t0 = (int64_t)seq.cu[un.s] + r0;
    const char *s0 = src + (((int64_t)un.l * Ttot + t0) * Hkv + un.h) * rowb;
    char *d0 = dst + (((int64_t)un.l * Hkv + un.h) * Ttot + t0) * rowb;
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    for (int p = threadIdx.x; p < rows * pr; p += blockDim.x) {
        const int r = p / pr, c = p - r * pr;
        const v4u v = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(s0 + (int64_t)r * Hkv * rowb) + c);
        __builtin_nontemporal_store(v, reinterpret_cast<v4u *>(d0 + (int64_t)r * rowb) + c);
    }
}

__global__ __launch_bounds__(256) void k_rows_copy(const char *src, char *dst, int rowb, int L, int Hkv, int B,
                                                   int64_t Ttot, SeqTab seq)
{
    copy_unit_rows(src, dst, rowb, Hkv, B, Ttot, seq, blockIdx.y, blockIdx.x);  // block (x, u)
}

// The V rows' copy and the reduction of the K sweep's block partials into
// `pre` in one launch: blocks [0, nred) reduce (unit, group of 16 columns),
// 16 lanes per column, and the rest copy V rows as k_rows_copy does, ncx
// blocks per unit; the reduction's few loads then hide under the copy's
// stream instead of taking a launch of their own.
__global__ __launch_bounds__(256) void k_copy_reduce_pre(ScoreArgs a, const char *src, char *dst, int rowb, int ncg,
                                                         int ncx)
{
    const int nred = a.L * a.Hkv * a.B * ncg;
    if ((int)blockIdx.x < nred) {
        reduce1_columns<16, true>(a, blockIdx.x / ncg, blockIdx.x % ncg, ncg);
        return;
    }
    const int cb = blockIdx.x - nred;
    copy_unit_rows(src, dst, rowb, a.Hkv, a.B, a.Ttot, a.seq, cb / ncx, cb % ncx);
}

size_t prefill_ws_bytes(int L, int Hkv, int B, int D, int R, int maxT, bool bf16)
{
    // the block partials of sweep 1 (part1), for its smallest key block (as
    // in the score's layout)
    const int rpb = min(rows_per_block(D, bf16), fast::kSmallRows);
    const size_t nch1 = (size_t)((maxT + rpb - 1) / rpb);
    return align256(sizeof(float) * (size_t)L * Hkv * B * nch1 * (size_t)(2 * D + 2 * R));
}

hipError_t prefill_launch(ScoreArgs a, const void *Vsrc, void *Vdst, char *ws, int maxT, hipStream_t st, bool bf16)
{
    const int U = a.L * a.Hkv * a.B;
    const int es = bf16 ? 2 : 4;
    a.part1 = reinterpret_cast<float *>(ws);
    hipError_t e;
    const dim3 gc((maxT + kCopyRows - 1) / kCopyRows, U);
    if (score_fast_path(a.D, bf16) && a.R <= 32) {
        // bf16, head_dim 128: the streaming sweep reads the new rows and writes
        // the cache, in 512-key blocks (28-layer stack, 32768 tokens: the sweep
        // with the copy takes 326 us with them, as long as a plain copy of the
        // same rows, against 367 us with 2048-key blocks, whose 1792 blocks
        // leave the last of their 3.5 rounds half empty)
        const int sblock = fast::kS2KeysSmall;
        a.rpb1 = sblock;
        a.nch1 = (maxT + a.rpb1 - 1) / a.rpb1;
        if (sblock == fast::kS2Keys)
            ECOKV_TIMED("prefill_sweep", st,
                        hipLaunchKernelGGL((fast::k_fs1s<fast::kS2Keys, true>), dim3(a.nch1, U), dim3(256), 0, st, a));
        else
            ECOKV_TIMED("prefill_sweep", st,
                        hipLaunchKernelGGL((fast::k_fs1s<fast::kS2KeysSmall, true>), dim3(a.nch1, U), dim3(256), 0, st,
                                           a));
    } else {
        // other shapes: copy the rows, then the first sweep over the cache
        ECOKV_TIMED("prefill_copy", st,
                    hipLaunchKernelGGL(k_rows_copy, gc, dim3(256), 0, st, static_cast<const char *>(a.Ksrc),
                                       static_cast<char *>(const_cast<void *>(a.K)), a.D * es, a.L, a.Hkv, a.B, a.Ttot,
                                       a.seq));
        if ((e = hipGetLastError()) != hipSuccess) return e;
        a.rpb1 = block_sweep_rows(a.D, bf16, U, maxT);
        a.nch1 = (maxT + a.rpb1 - 1) / a.rpb1;
        ECOKV_TIMED("prefill_sweep", st, launch_sweep(1, a, dim3(a.nch1, U), st, bf16));
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (Vsrc) {
        // V's copy with the reduction into pre riding on it
        const int ncg = (2 * a.D + a.R + 15) / 16;
        const int64_t blocks = (int64_t)U * ncg + (int64_t)gc.x * U;
        if (blocks > INT32_MAX) return hipErrorInvalidConfiguration;
        ECOKV_TIMED("prefill_copy_v", st,
                    hipLaunchKernelGGL(k_copy_reduce_pre, dim3((unsigned)blocks), dim3(256), 0, st, a,
                                       static_cast<const char *>(Vsrc), static_cast<char *>(Vdst), a.D * es, ncg,
                                       (int)gc.x));
    } else if (reduce1_lanes(a.nch1) == 4) {
        ECOKV_TIMED("prefill_reduce", st,
                    hipLaunchKernelGGL((k_reduce1<4, true>), dim3(U), dim3(kReduceThreads), 0, st, a));
    } else {
        ECOKV_TIMED("prefill_reduce", st,
                    hipLaunchKernelGGL((k_reduce1<16, true>), dim3(U, (2 * a.D + a.R + 63) / 64),
                                       dim3(kReduceThreads), 0, st, a));
    }
    return hipGetLastError();
}

}  // namespace ecokv
