// ecokv_score, single-read path (gfx950; bf16 keys, head_dim 128, G*w <= 28).
//
// The two-sweep path reads K twice: sweep 2 needs per-unit constants (kbar
// and mu, Eq. (1) / Appendix A.1; the window softmax maximum and normaliser,
// Sec. 3) that only exist once sweep 1 has seen every key.  Here one
// persistent kernel reads every key from HBM once and keeps it on chip until
// the constants of its unit are known:
//
//   * work item = 256 consecutive keys of one (layer, KV head, sequence)
//     unit; block b takes items b, b + G, b + 2G, ... (G = grid size, one
//     block per CU, all co-resident);
//   * 4 loader waves stream the next item's keys and window rows from HBM
//     into registers and swap them into LDS once per iteration;
//   * 8 compute waves run sweep 1 on the item in LDS (window logits on the
//     matrix cores with the keys as the A operand, so each lane holds one
//     window row and the softmax statistics need no cross-lane work; |k|; the
//     column sums of k and k/|k| on the matrix cores from transposed LDS
//     reads) and keep each wave's 32 keys as MFMA operands in registers;
//   * two iterations later, once the unit's constants are published, they
//     run sweep 2 on those registers (window attention a_i, d_E, khat.mu).
//
// Publication between blocks.  Item partials (column sums, softmax max and
// sum per window row) and unit constants are 64-bit words (launch tag << 32 |
// float bits), written and read as relaxed device-scope atomics.  A reader
// accepts a word only if it carries this launch's tag, so no release/acquire
// fence (an L2 write-back / invalidate on this GPU) is ever needed.  Every
// block that holds an item of a unit reduces a fixed slice of the unit's
// columns over all of the unit's items (in item order: deterministic), and
// every block then reads the whole record.  Per iteration k of a block:
//   phase 0   issue loads: partial slices of item k-1's unit, constants of
//             item k-2's unit; loaders issue item k+1.  Sweep 1 logits.
//   phase 1-2 sweep 1 column sums; item partial assembled in LDS.
//   phase 3   check the loads of phase 0 (retry until tagged), publish the
//             item partial, reduce and publish the column slice, stage the
//             constants for sweep 2.
//   phase 4   sweep 2 of item k-2; keep item k's keys in registers.
//   phase 5   loaders swap item k+1 into LDS; item k-2's d_E extrema out.
// Deadlock freedom: a block waits only for partials of a unit whose items
// are all claimed by steps <= k (a unit has at most G items, so it spans at
// most two steps) and for slices reduced by blocks that only wait on older
// units; the block furthest behind never waits on a later one.  Every wait
// is bounded; a timeout marks the launch failed (status = tag) and the
// epilogue then writes NaN.
#include "ecokv_fast.h"

#include <atomic>

namespace ecokv {
namespace fast {

constexpr int kItem = kFusedItem;                  // 256 keys
constexpr int kCWaves = 8;                         // compute waves (32 keys each)
constexpr int kLWaves = 4;                         // loader waves
constexpr int kPWaves = kCWaves;                   // waves that run the publication protocol
constexpr int kFThreads = (kCWaves + kLWaves) * kWave;
constexpr int kPThreads = kPWaves * kWave;         // 512
constexpr int kLThreads = kLWaves * kWave;         // 256
constexpr int kCols = 2 * kD + 2 * kFusedMaxRows;  // record width for the largest R
constexpr int kChunkPerLane = 2;                   // tagged loads per protocol lane for one column slice
constexpr int kQSlots = 4;                         // window-row tiles of items k+1, k, k-1, k-2
constexpr int kChunkMax = kChunkPerLane * kPThreads;
constexpr int kSpinLimit = 1 << 14;                // retries of a wait (each at least one memory round trip)

struct Item {
    int valid;
    int u, j, n;  // unit, index of the item in the unit, items of the unit
    int T, P;     // keys and non-window keys of the unit
    int base;     // first key of the item in the unit
};

// Items of one block in order (b, b + G, b + 2G, ...) as (lh, rem): lh the
// (layer, head) group, rem the item within it; one step adds G with 32-bit
// arithmetic only (the division of G by the group size happens once).
struct ItemGen {
    int lh, rem, qG, rG;
};

__device__ __forceinline__ ItemGen item_gen(const ScoreArgs &a, int first, int G)
{
    ItemGen g;
    g.lh = first / a.slices_per_lh;
    g.rem = first - g.lh * a.slices_per_lh;
    g.qG = G / a.slices_per_lh;
    g.rG = G - g.qG * a.slices_per_lh;
    return g;
}

__device__ __forceinline__ void item_next(const ScoreArgs &a, ItemGen &g)
{
    g.lh += g.qG;
    g.rem += g.rG;
    if (g.rem >= a.slices_per_lh) {
        g.rem -= a.slices_per_lh;
        ++g.lh;
    }
}

__device__ __forceinline__ Item item_of(const ScoreArgs &a, const ItemGen &g)
{
    Item r{};
    if (g.lh >= a.L * a.Hkv) return r;
    int lo = 0, hi = a.seq.nseq - 1;  // last sequence s with spre[s] <= rem
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.seq.spre[mid] <= g.rem) lo = mid;
        else hi = mid - 1;
    }
    r.valid = 1;
    r.u = g.lh * a.B + lo;
    r.j = g.rem - a.seq.spre[lo];
    r.n = a.seq.spre[lo + 1] - a.seq.spre[lo];
    r.T = a.seq.cu[lo + 1] - a.seq.cu[lo];
    r.P = r.T - a.w;
    r.base = r.j * kItem;
    return r;
}

// The column slice reduced by item j of a unit with n items: logical columns
// [j*Cc/n, (j+1)*Cc/n) of Cc = 2D + R (2D sums, then R (max, normaliser)
// pairs).  Its load list: ns sum columns, then np max columns, then np
// normaliser columns, each over the unit's n items.
struct Chunk {
    int cs0, ns, r0, np, nl;
};

__device__ __forceinline__ Chunk chunk_of(int j, int n, int R)
{
    constexpr int D2 = 2 * kD;
    const int Cc = D2 + R;
    const int c0 = j * Cc / n, c1 = (j + 1) * Cc / n;  // j < 2^16, Cc < 2^10
    Chunk c;
    c.cs0 = min(c0, D2);
    c.ns = min(c1, D2) - c.cs0;
    c.r0 = max(c0, D2) - D2;
    c.np = max(c1, D2) - D2 - c.r0;
    c.nl = (c.ns + 2 * c.np) * n;
    return c;
}

__device__ __forceinline__ int chunk_col(const Chunk &c, int i, int R)
{
    constexpr int D2 = 2 * kD;
    if (i < c.ns) return c.cs0 + i;
    i -= c.ns;
    if (i < c.np) return D2 + c.r0 + i;
    return D2 + R + c.r0 + (i - c.np);
}

__device__ __forceinline__ void tag_store(unsigned long long *p, float v, unsigned tag)
{
    __hip_atomic_store(p, ((unsigned long long)tag << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long tag_load(const unsigned long long *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool tag_ok(unsigned long long x, unsigned tag) { return (unsigned)(x >> 32) == tag; }
__device__ __forceinline__ float tag_val(unsigned long long x) { return __uint_as_float((unsigned)x); }

struct __attribute__((aligned(16))) FusedLds {
    u32x4 kt[kItem * kChunks];            // keys of the item in sweep 1 (swizzled 16-byte chunks)
    u32x4 qs[kQSlots][32 * kChunks];      // window rows of item k in slot k % 4 (rows >= R zero); rows
                                          // 28..31 take mu and kbar before the item's sweep 2
    uint16_t aw[2][4][kTile];             // per 128-key tile: 1, 1/|k| high, 1/|k| remainder, 0
    float sm[kCWaves][2][32], ss[kCWaves][2][32];  // per wave and half: row max and sum of 2^(x - max)
    float cx[4][2][32];                   // column sums of the second tile
    float part[kCols];                    // partial record of the sweep-1 item
    float anc[kCols];                     // constants of the sweep-2 item's unit
    float cv[kChunkMax];                  // validated partial values of the column slice
    float rowM[32], rowIS[32];
    float kb2;
    float dred[kCWaves][3];
    int flag[2][2][kPWaves];              // [retry parity][slice, constants][wave]
    int dead;                             // a wait of this block timed out: skip the remaining waits
};

// Loader: one item's keys (16 lanes per 256-byte row) and window rows.
__device__ __forceinline__ void issue_keys(const ScoreArgs &a, const Item &it, int ltid, u32x4 (&lk)[16])
{
    if (!it.valid) return;
    const Unit un = unit_of(it.u, a.Hkv, a.B);
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const __amdgpu_buffer_rsrc_t rs = key_rows_rsrc(krow0, it.T);
    const int c = ltid & 15, g = ltid >> 4;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj)
        lk[jj] = __builtin_amdgcn_raw_buffer_load_b128(rs, (it.base + g + 16 * jj) * (kD * 2) + c * 16, 0, 0);
}

// Loader: the window rows of an item straight into a row tile (no
// registers).  Each direct-to-LDS 16-byte load of a wave fills 64 consecutive
// chunks, i.e. rows 4i .. 4i+3 of the swizzled tile; lane l takes physical
// chunk l % 16 of row 4i + l / 16, which holds logical chunk (l % 16) ^ row.
__device__ __forceinline__ void dma_rows(const ScoreArgs &a, const Item &it, int lw, int lane, u32x4 *q)
{
    if (!it.valid) return;
    const Unit un = unit_of(it.u, a.Hkv, a.B);
    const int ninst = (a.R + 3) >> 2;
    for (int i = lw; i < ninst; i += kLWaves) {
        const int r = 4 * i + (lane >> 4), c = (lane & 15) ^ (r & 15);
        if (r < a.R)
            __builtin_amdgcn_global_load_lds(
                static_cast<const uint16_t *>(a.Q) + window_row(a, un, r) * kD + c * 8,
                (__attribute__((address_space(3))) void *)(q + 64 * i), 16, 0, 0);
    }
}

__device__ __forceinline__ void wait_all_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Barrier for the loader waves between their load issue and their LDS
// writes: they write no LDS in that span, so no release fence (which would
// wait for the in-flight direct-to-LDS loads); the acquire side still orders
// their later LDS reads (the publication flags) after the barrier.
__device__ __forceinline__ void loader_barrier()
{
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Protocol loads: the column slice of item `ic` (partials of its unit) and
// the constants of item `i2`'s unit.
__device__ __forceinline__ void issue_chunk(const ScoreArgs &a, const Item &ic, const Chunk &ch, int C, int ptid,
                                            unsigned long long (&cl)[kChunkPerLane])
{
    if (!ic.valid) return;
#pragma unroll
    for (int q = 0; q < kChunkPerLane; ++q) {
        const int t = ptid + kPThreads * q;
        if (t < ch.nl) {
            const int i = t / ic.n, jj = t - i * ic.n;
            const int col = chunk_col(ch, i, a.R);
            cl[q] = tag_load(&a.partT[((long long)ic.u * C + col) * a.nch1 + jj]);
        }
    }
}

__device__ __forceinline__ bool chunk_ok(const ScoreArgs &a, const Item &ic, const Chunk &ch, int ptid,
                                         const unsigned long long (&cl)[kChunkPerLane])
{
    bool ok = true;
    if (ic.valid) {
#pragma unroll
        for (int q = 0; q < kChunkPerLane; ++q)
            if (ptid + kPThreads * q < ch.nl) ok = ok && tag_ok(cl[q], a.tag);
    }
    return ok;
}

__device__ __forceinline__ void issue_consts(const ScoreArgs &a, const Item &i2, int C, int ptid,
                                             unsigned long long &al)
{
    if (i2.valid && ptid < C) al = tag_load(&a.ancT[(long long)i2.u * C + ptid]);
}

__device__ __forceinline__ bool consts_ok(const ScoreArgs &a, const Item &i2, int C, int ptid,
                                          unsigned long long al)
{
    return !(i2.valid && ptid < C) || tag_ok(al, a.tag);
}

__device__ __forceinline__ bool all_flags(const FusedLds &S, int par, int kind)
{
    int ok = 1;
#pragma unroll
    for (int w = 0; w < kPWaves; ++w) ok &= S.flag[par][kind][w];
    return ok != 0;
}

// Barrier skeleton of a publication wait for the loader waves, which take no
// part in it: the same flag reads (so the same number of iterations) and
// barriers.
__device__ __forceinline__ void follow_flags(const FusedLds &S, int kind)
{
    if (S.dead) return;
    int par = 0, tries = 0;
    while (!all_flags(S, par, kind)) {
        if (++tries > kSpinLimit) break;
        par ^= 1;
        loader_barrier();
    }
}

// Reduce the validated column slice (S.cv) of item ic and publish it: sums /
// T as kbar and mu, merged (max, normaliser) pairs as they are.  The order of
// every sum depends only on (n, j): the result is the same in any block.
__device__ __forceinline__ void reduce_chunk(const ScoreArgs &a, const Item &ic, const Chunk &ch, int C, int ptid,
                                             const FusedLds &S)
{
    const int n = ic.n, ncl = ch.ns + ch.np;
    const float invT = 1.f / (float)ic.T;
    unsigned long long *outT = a.ancT + (long long)ic.u * C;
    float *outP = a.anchors + (long long)ic.u * C;
    if (n >= 16) {
        for (int t = ptid; t < ncl * 16; t += kPThreads) {  // 16 lanes per column; groups stay whole
            const int lc = t >> 4, q = t & 15;
            if (lc < ch.ns) {
                float s = 0.f;
                for (int jj = q; jj < n; jj += 16) s += S.cv[lc * n + jj];
                s += __shfl_xor(s, 8, 16);
                s += __shfl_xor(s, 4, 16);
                s += __shfl_xor(s, 2, 16);
                s += __shfl_xor(s, 1, 16);
                if (q == 0) {
                    const int col = ch.cs0 + lc;
                    tag_store(outT + col, s * invT, a.tag);
                    outP[col] = s * invT;
                }
            } else {
                const int pr = lc - ch.ns;
                const float *mv = S.cv + (ch.ns + pr) * n, *sv = S.cv + (ch.ns + ch.np + pr) * n;
                float m = -INFINITY, s = 0.f;
                for (int jj = q; jj < n; jj += 16) softmax_merge2(m, s, mv[jj], sv[jj]);
#pragma unroll
                for (int x = 8; x >= 1; x >>= 1) {
                    const float m2 = __shfl_xor(m, x, 16), s2 = __shfl_xor(s, x, 16);
                    softmax_merge2(m, s, m2, s2);
                }
                if (q == 0) {
                    const int r = ch.r0 + pr;
                    tag_store(outT + 2 * kD + r, m, a.tag);
                    tag_store(outT + 2 * kD + a.R + r, s, a.tag);
                    outP[2 * kD + r] = m;
                    outP[2 * kD + a.R + r] = s;
                }
            }
        }
    } else {
        for (int lc = ptid; lc < ncl; lc += kPThreads) {
            if (lc < ch.ns) {
                float s = 0.f;
                for (int jj = 0; jj < n; ++jj) s += S.cv[lc * n + jj];
                const int col = ch.cs0 + lc;
                tag_store(outT + col, s * invT, a.tag);
                outP[col] = s * invT;
            } else {
                const int pr = lc - ch.ns;
                const float *mv = S.cv + (ch.ns + pr) * n, *sv = S.cv + (ch.ns + ch.np + pr) * n;
                float m = -INFINITY, s = 0.f;
                for (int jj = 0; jj < n; ++jj) softmax_merge2(m, s, mv[jj], sv[jj]);
                const int r = ch.r0 + pr;
                tag_store(outT + 2 * kD + r, m, a.tag);
                tag_store(outT + 2 * kD + a.R + r, s, a.tag);
                outP[2 * kD + r] = m;
                outP[2 * kD + a.R + r] = s;
            }
        }
    }
}

__global__ __launch_bounds__(kFThreads, 1) void k_fused(ScoreArgs a)
{
    __shared__ FusedLds S;

    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const bool comp = wv < kCWaves, loader = !comp;
    const int G = gridDim.x;
    const int C = 2 * kD + 2 * a.R;
    const float sc = a.inv_sqrt_d * kLog2e;
    const float inv_r = 1.f / (float)a.R;
    const int nsteps = (a.items + G - 1) / G;
    const int niter = nsteps + 2;  // sweep 2 lags two iterations

    // window-row tiles start zero (rows >= R stay zero); tile weights rows 0 and 3
    for (int i = threadIdx.x; i < kQSlots * 32 * kChunks; i += kFThreads)
        (&S.qs[0][0])[i] = (u32x4){0u, 0u, 0u, 0u};
    for (int i = threadIdx.x; i < 2 * kTile; i += kFThreads) {
        S.aw[i / kTile][0][i % kTile] = 0x3f80;
        S.aw[i / kTile][3][i % kTile] = 0;
    }
    if (threadIdx.x == 0) S.dead = 0;

    // One register array serves both roles (the allocator cannot see that the
    // roles are exclusive): loader waves stage the next item's keys in it,
    // compute waves keep the keys of the two items waiting for sweep 2 as MFMA
    // operands (elements 0..7: item k-2, 8..15: item k-1 at iteration k).
    u32x4 lk[16];
    float sn2[2] = {0.f, 0.f}, sinv[2] = {0.f, 0.f};
    unsigned long long cl[kChunkPerLane] = {}, al = 0;
    lds_barrier();  // zero fill done before the first item lands
    // items k+1, k, k-1, k-2 of this block, shifted once per iteration
    ItemGen gen = item_gen(a, blockIdx.x, G);
    Item in = item_of(a, gen), i1{}, ic{}, i2{};
    if (loader) {
        const int ltid = threadIdx.x - kCWaves * kWave;
        const Item &i0 = in;
        dma_rows(a, i0, wv - kCWaves, threadIdx.x & 63, S.qs[0]);
        issue_keys(a, i0, ltid, lk);
        if (i0.valid) {
            const int c = ltid & 15, g = ltid >> 4;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) S.kt[sw(g + 16 * jj, c)] = lk[jj];
        }
        wait_all_loads();
    }

#pragma unroll 1
    for (int k = 0; k < niter; ++k) {
        // lane-derived indices are recomputed every iteration: kept out of the
        // loop-invariant set, which would otherwise pin them in registers
        int tv = threadIdx.x;
        asm volatile("" : "+v"(tv));
        const int tid = tv, lane = tv & 63, h = lane >> 5, qr = lane & 31;
        i2 = ic;  // sweep 2
        ic = i1;  // column slice to reduce
        i1 = in;  // sweep 1
        item_next(a, gen);
        in = item_of(a, gen);  // loaded during this iteration
        const Chunk ch = ic.valid ? chunk_of(ic.j, ic.n, a.R) : Chunk{};
        const u32x4 *q1 = S.qs[k & 3];
        u32x4 *q2 = S.qs[(k + 2) & 3];
        lds_barrier();  // item k in kt and q1; item k-2's rows in q2

        if (loader) {
            // item k+1: window rows into slot (k+1) % 4 (free since the sweep 2
            // of item k-3), keys into registers; the same barrier sequence as
            // the compute waves, with the keys consumed only at its end
            const int ltid = tid - kCWaves * kWave;
            dma_rows(a, in, wv - kCWaves, lane, S.qs[(k + 1) & 3]);
            issue_keys(a, in, ltid, lk);
            loader_barrier();  // phase 0 | 1
            loader_barrier();  // phase 1 | 2
            loader_barrier();  // phase 2 | 3
            loader_barrier();  // publication flags
            follow_flags(S, 0);
            loader_barrier();  // slice values staged
            follow_flags(S, 1);
            loader_barrier();  // constants staged
            loader_barrier();  // phase 3 | 4
            loader_barrier();  // phase 4 | 5
            if (in.valid) {
                const int c = ltid & 15, g = ltid >> 4;
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) S.kt[sw(g + 16 * jj, c)] = lk[jj];
            }
            wait_all_loads();  // the row tile's direct-to-LDS loads too
            continue;
        }
        // ---- phase 0: protocol and loader requests; sweep-1 logits ----
        issue_chunk(a, ic, ch, C, tid, cl);
        issue_consts(a, i2, C, tid, al);
        float n2c = 0.f, invc = 0.f;
        if (i1.valid) {
            const int kr = 32 * wv + qr;
            f32x16 acc = (f32x16){};
            float n2 = 0.f;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const u32x4 kq = S.kt[sw(kr, 2 * s + h)];
                const u32x4 qq = q1[sw(qr, 2 * s + h)];
                n2 = dot2sq(kq[0], dot2sq(kq[1], dot2sq(kq[2], dot2sq(kq[3], n2))));
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kq),
                                                              __builtin_bit_cast(bf16x8, qq), acc, 0, 0, 0);
            }
            n2 += __shfl_xor(n2, 32, kWave);
            const float inv = __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
            n2c = n2;
            invc = inv;
            if (h == 0) {
                const unsigned hi = bf16_rne(inv);
                S.aw[wv >> 2][1][32 * (wv & 3) + lane] = (uint16_t)hi;
                S.aw[wv >> 2][2][32 * (wv & 3) + lane] = (uint16_t)bf16_rne(inv - __uint_as_float(hi << 16));
            }
            // this lane: window row qr against keys 8(r/4) + 4h + r%4 of the wave, r < 16
            float mloc, sloc = 0.f;
            if (i1.base + kItem <= i1.P) {
                float mx = acc[0];
#pragma unroll
                for (int r = 1; r < 16; ++r) mx = fmaxf(mx, acc[r]);
                mloc = mx * sc;
#pragma unroll
                for (int r = 0; r < 16; ++r) sloc += fast_exp2(fmaf(acc[r], sc, -mloc));
            } else {
                const int kb = i1.base + 32 * wv + 4 * h;
                const int lim = a.causal ? i1.P + qr % a.w : i1.T - 1;  // last visible key of row qr
                float x[16];
                mloc = -INFINITY;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gk = kb + 8 * (r >> 2) + (r & 3);
                    x[r] = (gk < i1.T && gk <= lim) ? acc[r] * sc : -INFINITY;
                    mloc = fmaxf(mloc, x[r]);
                }
                if (mloc != -INFINITY)
#pragma unroll
                    for (int r = 0; r < 16; ++r) sloc += fast_exp2(x[r] - mloc);
            }
            S.sm[wv][h][qr] = mloc;
            S.ss[wv][h][qr] = sloc;
        }
        lds_barrier();

        // ---- phase 1: column sums of the two 128-key tiles; softmax fold ----
        f32x16 cs = (f32x16){};
        if (i1.valid) {
            const int ti = wv >> 2, wq = wv & 3;
            const int tr_key = 8 * h + ((lane & 15) >> 2);
            const int tr_dim = 32 * wq + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
            const int aw_row = qr < 3 ? qr : 3;
            typedef short s16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const bf16x8 wa = *reinterpret_cast<const bf16x8 *>(&S.aw[ti][aw_row][16 * ks + 8 * h]);
                const int key0 = kTile * ti + 16 * ks + tr_key;
                const uint16_t *kt16 = reinterpret_cast<const uint16_t *>(S.kt);
                const uint16_t *p0 = kt16 + key0 * kD + (((tr_dim >> 3) ^ (key0 & 15)) << 3) + (tr_dim & 7);
                const uint16_t *p1 =
                    kt16 + (key0 + 4) * kD + (((tr_dim >> 3) ^ ((key0 + 4) & 15)) << 3) + (tr_dim & 7);
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p0)));
                const s16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p1)));
                const short __attribute__((ext_vector_type(8))) kb8 = {lo[0],  lo[1],  lo[2],  lo[3],
                                                                        hi4[0], hi4[1], hi4[2], hi4[3]};
                cs = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa, __builtin_bit_cast(bf16x8, kb8), cs, 0, 0, 0);
            }
            if (ti == 1 && h == 0) {
                S.cx[wq][0][lane] = cs[0];
                S.cx[wq][1][lane] = cs[1] + cs[2];
            }
            if (wv == 0 && lane < a.R) {
                float m = -INFINITY, s = 0.f;
#pragma unroll
                for (int w2 = 0; w2 < kCWaves; ++w2)
#pragma unroll
                    for (int hh = 0; hh < 2; ++hh) softmax_merge2(m, s, S.sm[w2][hh][lane], S.ss[w2][hh][lane]);
                S.part[2 * kD + lane] = m;
                S.part[2 * kD + a.R + lane] = s;
            }
        }
        lds_barrier();

        // ---- phase 2: item partial column sums (tile 0 + tile 1) ----
        if (i1.valid && wv < 4 && h == 0) {
            S.part[32 * wv + lane] = cs[0] + S.cx[wv][0][lane];
            S.part[kD + 32 * wv + lane] = (cs[1] + cs[2]) + S.cx[wv][1][lane];
        }
        lds_barrier();

        // ---- phase 3: publication ----
        {
            const bool okc = __all(chunk_ok(a, ic, ch, tid, cl));
            const bool oka = __all(consts_ok(a, i2, C, tid, al));
            if (lane == 0) {
                S.flag[0][0][wv] = okc;
                S.flag[0][1][wv] = oka;
            }
            if (i1.valid && tid < C) tag_store(&a.partT[((long long)i1.u * C + tid) * a.nch1 + i1.j], S.part[tid], a.tag);
        }
        lds_barrier();
        // column slice: wait until every partial of item ic's unit is published
        if (!S.dead) {
            int par = 0, tries = 0;
            while (!all_flags(S, par, 0)) {
                if (++tries > kSpinLimit) {
                    if (tid == 0) {
                        __hip_atomic_store(a.status, a.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        S.dead = 1;  // read by every wave only after the next barrier
                    }
                    break;
                }
                par ^= 1;
                {
                    __builtin_amdgcn_s_sleep(2);
                    issue_chunk(a, ic, ch, C, tid, cl);
                    const bool okc = __all(chunk_ok(a, ic, ch, tid, cl));
                    if (lane == 0) S.flag[par][0][wv] = okc;
                }
                lds_barrier();
            }
        }
        if (ic.valid) {
#pragma unroll
            for (int q = 0; q < kChunkPerLane; ++q) {
                const int t = tid + kPThreads * q;
                if (t < ch.nl) S.cv[t] = tag_val(cl[q]);
            }
        }
        lds_barrier();
        if (ic.valid) reduce_chunk(a, ic, ch, C, tid, S);
        // constants of item i2's unit
        if (!S.dead) {
            int par = 0, tries = 0;
            while (!all_flags(S, par, 1)) {
                if (++tries > kSpinLimit) {
                    if (tid == 0) {
                        __hip_atomic_store(a.status, a.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        S.dead = 1;  // read by every wave only after the next barrier
                    }
                    break;
                }
                par ^= 1;
                {
                    __builtin_amdgcn_s_sleep(2);
                    issue_consts(a, i2, C, tid, al);
                    const bool oka = __all(consts_ok(a, i2, C, tid, al));
                    if (lane == 0) S.flag[par][1][wv] = oka;
                }
                lds_barrier();
            }
        }
        if (i2.valid && tid < C) S.anc[tid] = tag_val(al);
        lds_barrier();
        if (wv == 0 && i2.valid) {
            if (lane < a.R) {
                S.rowM[lane] = S.anc[2 * kD + lane];
                S.rowIS[lane] = 1.f / S.anc[2 * kD + a.R + lane];
            }
            // |kbar'|^2 of the centroid as the operand rows represent it
            float acc2 = 0.f;
#pragma unroll
            for (int z = 0; z < 2; ++z) {
                const float f = S.anc[2 * lane + z];
                const float fh = __uint_as_float(bf16_rne(f) << 16);
                const float fl = __uint_as_float(bf16_rne(f - fh) << 16);
                acc2 = fmaf(fh + fl, fh + fl, acc2);
            }
            acc2 = wave_sum(acc2);
            if (lane == 0) S.kb2 = acc2;
            // rows 28..31 of the sweep-2 operand: mu high, mu remainder, kbar high, kbar remainder
            const int which = lane >> 4, c = lane & 15;
            const float *src = (which < 2) ? S.anc + kD : S.anc;
            u32x4 q;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                unsigned half2[2];
#pragma unroll
                for (int z = 0; z < 2; ++z) {
                    const float f = src[8 * c + 2 * e + z];
                    const unsigned hb = bf16_rne(f);
                    half2[z] = (which & 1) ? bf16_rne(f - __uint_as_float(hb << 16)) : hb;
                }
                q[e] = half2[0] | (half2[1] << 16);
            }
            q2[sw(kFusedMaxRows + which, c)] = q;
        }
        lds_barrier();

        // ---- phase 4: sweep 2 of item k-2 from registers; shift the key slots ----
        if (i2.valid) {
            f32x16 acc = (f32x16){};
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const u32x4 qa = q2[sw(qr, 2 * s + h)];
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, qa),
                                                              __builtin_bit_cast(bf16x8, lk[s]), acc, 0, 0, 0);
            }
            float att = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int m = 8 * (r >> 2) + 4 * h + (r & 3);
                if (m < a.R) att = fmaf(fast_exp2(fmaf(acc[r], sc, -S.rowM[m])), S.rowIS[m], att);
            }
            float kmu = h ? acc[12] + acc[13] : 0.f;
            float kk = h ? acc[14] + acc[15] : 0.f;
            att += __shfl_xor(att, 32, kWave);
            kmu += __shfl_xor(kmu, 32, kWave);
            kk += __shfl_xor(kk, 32, kWave);
            const float dE = __builtin_amdgcn_sqrtf(fmaxf(sn2[0] - 2.f * kk + S.kb2, 0.f));
            const float cm = kmu * sinv[0];
            const int gi = i2.base + 32 * wv + qr;
            float dsum = 0.f, dmn = INFINITY, dmx = -INFINITY;
            if (h == 0) {
                if (gi < i2.T) dsum = dE;
                if (gi < i2.P) {
                    dmn = dE;
                    dmx = dE;
                    const Unit un = unit_of(i2.u, a.Hkv, a.B);
                    const int64_t ob = unit_out_base(a, un);
                    a.bufA[ob + gi] = dE;
                    a.bufB[ob + gi] = cm;
                    a.bufC[ob + gi] = att * inv_r;
                }
            }
            dsum = wave_sum(dsum);
            dmn = wave_min(dmn);
            dmx = wave_max(dmx);
            if (lane == 0) {
                S.dred[wv][0] = dsum;
                S.dred[wv][1] = dmn;
                S.dred[wv][2] = dmx;
            }
        }
        {
            // item k-1 becomes the next sweep-2 item; item k (still in kt) follows it
            const int kr = 32 * wv + qr;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                lk[s] = lk[8 + s];
                lk[8 + s] = S.kt[sw(kr, 2 * s + h)];
            }
            sn2[0] = sn2[1];
            sinv[0] = sinv[1];
            sn2[1] = n2c;
            sinv[1] = invc;
        }
        lds_barrier();

        // ---- phase 5: d_E extrema of item k-2 ----
        if (wv == 0 && i2.valid && lane == 0) {
            float s = 0.f, mn = INFINITY, mx = -INFINITY;
            for (int w2 = 0; w2 < kCWaves; ++w2) {
                s += S.dred[w2][0];
                mn = fminf(mn, S.dred[w2][1]);
                mx = fmaxf(mx, S.dred[w2][2]);
            }
            float *pp = a.part2 + ((int64_t)i2.u * a.nch2 + i2.j) * 4;
            pp[0] = s;
            pp[1] = mn;
            pp[2] = mx;
            pp[3] = 0.f;
        }
    }
}

}  // namespace fast

namespace {

struct DevInfo {
    int ncu = 0, per_cu = 0;
};

bool dev_info(DevInfo *o)
{
    static DevInfo cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return false;
    DevInfo &d = cache[dev];
    if (d.ncu == 0) {
        int ncu = 0, nb = 0;
        if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fast::k_fused, fast::kFThreads, 0) != hipSuccess)
            return false;
        d.per_cu = nb;
        d.ncu = ncu;
    }
    *o = d;
    return d.ncu > 0 && d.per_cu > 0;
}

int chunk_loads_max(int n, int R)
{
    // largest load list of any column slice of a unit with n items
    const int Cc = 2 * fast::kD + R, D2 = 2 * fast::kD;
    int mx = 0;
    for (int j = 0; j < n; ++j) {
        const int c0 = (int)((long long)j * Cc / n), c1 = (int)((long long)(j + 1) * Cc / n);
        const int ns = (c1 < D2 ? c1 : D2) - (c0 < D2 ? c0 : D2);
        const int np = (c1 > D2 ? c1 - D2 : 0) - (c0 > D2 ? c0 - D2 : 0);
        const int nl = (ns + 2 * np) * n;
        if (nl > mx) mx = nl;
    }
    return mx;
}

std::atomic<unsigned> g_tag{0};

}  // namespace

bool fused_eligible(int D, bool bf16, int R, const SeqTab &seq, int L, int Hkv, int *grid)
{
    if (!bf16 || D != fast::kD || R > kFusedMaxRows || R < 1) return false;
    DevInfo di;
    if (!dev_info(&di)) return false;
    long long ns = 0;
    int nmax = 0;
    for (int s = 0; s < seq.nseq; ++s) {
        const int n = (seq.cu[s + 1] - seq.cu[s] + kFusedItem - 1) / kFusedItem;
        ns += n;
        if (n > nmax) nmax = n;
        if (chunk_loads_max(n, R) > fast::kChunkMax) return false;
    }
    const long long items = (long long)L * Hkv * ns;
    if (items < 1 || items > (1LL << 30)) return false;
    const long long g = items < (long long)di.ncu * di.per_cu ? items : (long long)di.ncu * di.per_cu;
    // every unit must span at most G items (two consecutive steps)
    if (nmax > g) return false;
    *grid = (int)g;
    return true;
}

hipError_t fused_launch(ScoreArgs &a, int grid, hipStream_t st)
{
    unsigned t = ++g_tag;
    if (t == 0) t = ++g_tag;
    a.tag = t;
    hipLaunchKernelGGL(fast::k_fused, dim3(grid), dim3(fast::kFThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace ecokv
