// ecokv_score, single-read path (gfx950; bf16 keys, head_dim 128, G*w <= 28).
//
// The two-sweep path reads K twice: sweep 2 needs per-unit constants (kbar
// and mu, Eq. (1) / Appendix A.1; the window softmax maximum and normaliser,
// Sec. 3) that only exist once sweep 1 has seen every key.  Here one
// persistent kernel reads every key from HBM once and keeps it on chip until
// the constants of its unit are known:
//
//   * work item ("slice") = 224 consecutive keys of one (layer, KV head,
//     sequence) unit; block b takes slices b, b + G, b + 2G, ... (G = grid
//     size, two blocks per CU so that one computes while the other waits,
//     all co-resident);
//   * 7 compute waves own 32 keys each.  A wave's keys arrive in its own 32
//     LDS rows by direct-to-LDS buffer loads (rows past the unit read as
//     zero), are read once into MFMA operand registers and stay there until
//     sweep 2; as soon as they are in registers the wave issues the loads of
//     its rows of the next slice, so HBM traffic continues through the
//     publication wait;
//   * sweep 1 in registers: window logits on the matrix cores (keys as the A
//     operand, so each lane holds one window row and its softmax statistics
//     need no cross-lane work), |k|, and the column sums of k and k/|k| on the
//     matrix cores from transposed LDS reads of the wave's rows;
//   * wave 7 runs the publication protocol alone, so that its waits never
//     queue behind the key loads in flight in the compute waves;
//   * sweep 2 from the same registers: window attention a_i, d_E, khat.mu.
//
// Publication between blocks.  Slice partials (column sums, softmax max and
// sum per window row) and unit constants are 64-bit words (launch tag << 32 |
// float bits), written and read as relaxed device-scope atomics.  A reader
// accepts a word only if it carries this launch's tag, so no release/acquire
// fence (an L2 write-back / invalidate on this GPU) is ever needed.  Every
// block that holds a slice of a unit reduces a fixed part of the unit's
// columns over all of the unit's slices (in slice order: deterministic), and
// every block then reads the whole record.
// Deadlock freedom: a block waits only for slices of the unit it holds; a
// unit has at most G slices, so they sit in at most two consecutive steps,
// and the earliest unfinished unit never waits for a later one.  Every wait
// is bounded; a timeout marks the launch failed (status = tag) and the
// epilogue then writes NaN.
#include "ecokv_fast.h"

#include <atomic>

namespace ecokv {
namespace fast {

constexpr int kItem = kFusedItem;                  // keys per slice
constexpr int kCW = kItem / 32;                    // compute waves, 32 keys each
constexpr int kFThreads = (kCW + 1) * kWave;       // plus the protocol wave
constexpr int kFBlocksPerCU = 2;                   // two blocks per CU: one computes while the other waits
// (the second launch bound is the minimum number of waves per SIMD)
constexpr int kCols = 2 * kD + 2 * kFusedMaxRows;  // record width for the largest R
constexpr int kChunkPerLane = 12;                  // tagged loads per protocol lane for one column part
constexpr int kChunkMax = kChunkPerLane * kWave;
constexpr int kSpinLimit = 1 << 14;                // retries of a wait (each at least one memory round trip)
static_assert(kCW * 32 == kItem && kFThreads <= 1024, "slice = 32 keys per compute wave");

struct Item {
    int valid;
    int u, j, n;  // unit, index of the slice in the unit, slices of the unit
    int T, P;     // keys and non-window keys of the unit
    int base;     // first key of the slice in the unit
};

// Slices of one block in order (b, b + G, b + 2G, ...) as (lh, rem): lh the
// (layer, head) group, rem the slice within it; one step adds G with 32-bit
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

// The column part reduced by slice j of a unit with n slices: logical columns
// [j*Cc/n, (j+1)*Cc/n) of Cc = 2D + R (2D sums, then R (max, normaliser)
// pairs).  Its load list: ns sum columns, then np max columns, then np
// normaliser columns, each over the unit's n slices.
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
    u32x4 kt[kItem * kChunks];  // the slice's keys: rows 32w .. 32w+31 belong to compute wave w
                                // (16-byte chunks swizzled by row)
    uint16_t wts[kCW][4][32];   // per wave: 1, 1/|k| high, 1/|k| remainder, 0
    float wcs[kCW][2][kD];      // per wave: column sums of k and of k/|k|; the protocol wave
                                // reuses the space for the values of its column part
    float wm[kCW][32], wsm[kCW][32];  // per wave: row max and sum of 2^(x - max)
    float anc[kCols];           // constants of the slice's unit
    u32x4 arow[4][kChunks];     // operand rows mu high, mu remainder, kbar high, kbar remainder (bf16)
    float rsh[32];              // per window row: max + log2(normaliser); +inf past R
    float kb2;                  // |kbar|^2 as the operand rows represent kbar
    float dred[kCW][3];         // per wave: sum, min, max of d_E
};
static_assert(sizeof(float) * kCW * 2 * kD >= sizeof(float) * kChunkMax, "column part fits the wcs space");

// A compute wave's 32 rows of slice `it` into its LDS rows: 8 direct-to-LDS
// 16-byte buffer loads; instruction i fills rows 4i .. 4i+3, lane l takes
// physical chunk l % 16 of row 4i + l / 16, which holds logical chunk
// (l % 16) ^ row.  The descriptor spans the unit's T rows, so rows past T
// land as zeros.
__device__ __forceinline__ void dma_keys(const ScoreArgs &a, const Item &it, int cw, int lane, u32x4 *dst)
{
    if (!it.valid) return;
    const Unit un = unit_of(it.u, a.Hkv, a.B);
    const uint16_t *krow0 = static_cast<const uint16_t *>(a.K) + unit_row0(a, un) * kD;
    const __amdgpu_buffer_rsrc_t rs = key_rows_rsrc(krow0, it.T);
    const int r0 = it.base + 32 * cw;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = 4 * i + (lane >> 4), c = (lane & 15) ^ (r & 15);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void *)(dst + 64 * i), 16,
                                                 (r0 + r) * (kD * 2) + c * 16, 0, 0, 0);
    }
}

// Window rows of the slice's unit as the 32-row MFMA operand (lane l: row
// l % 32, chunks 2s + l / 32); rows >= R read as zero (offset past the range).
__device__ __forceinline__ void load_window(const ScoreArgs &a, const Item &it, int lane, u32x4 (&aq)[8])
{
    if (!it.valid) return;
    const Unit un = unit_of(it.u, a.Hkv, a.B);
    const int r = lane & 31;
    const int qbytes = (int)((int64_t)a.L * a.Hq * a.B * a.w * kD * 2);
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(a.Q), (short)0, qbytes, 0x00020000);
    const unsigned off = r < a.R ? (unsigned)(window_row(a, un, r) * (kD * 2)) + (lane >> 5) * 16u : 0x80000000u;
#pragma unroll
    for (int s = 0; s < 8; ++s) aq[s] = __builtin_amdgcn_raw_buffer_load_b128(rs, off + 32u * s, 0, 0);
}

// Protocol wave: loads of its column part of slice `ic` (partials of the unit).
__device__ __forceinline__ void issue_chunk(const ScoreArgs &a, const Item &ic, const Chunk &ch, int C, int lane,
                                            unsigned long long (&cl)[kChunkPerLane])
{
#pragma unroll
    for (int q = 0; q < kChunkPerLane; ++q) {
        const int t = lane + kWave * q;
        if (t < ch.nl) {
            const int i = t / ic.n, jj = t - i * ic.n;
            const int col = chunk_col(ch, i, a.R);
            cl[q] = tag_load(&a.partT[((long long)ic.u * C + col) * a.nch1 + jj]);
        }
    }
}

__device__ __forceinline__ bool chunk_ok(const ScoreArgs &a, const Chunk &ch, int lane,
                                         const unsigned long long (&cl)[kChunkPerLane])
{
    bool ok = true;
#pragma unroll
    for (int q = 0; q < kChunkPerLane; ++q)
        if (lane + kWave * q < ch.nl) ok = ok && tag_ok(cl[q], a.tag);
    return ok;
}

constexpr int kConstPerLane = (kCols + kWave - 1) / kWave;

__device__ __forceinline__ void issue_consts(const ScoreArgs &a, const Item &it, int C, int lane,
                                             unsigned long long (&al)[kConstPerLane])
{
#pragma unroll
    for (int q = 0; q < kConstPerLane; ++q) {
        const int c = lane + kWave * q;
        if (c < C) al[q] = tag_load(&a.ancT[(long long)it.u * C + c]);
    }
}

__device__ __forceinline__ bool consts_ok(const ScoreArgs &a, int C, int lane,
                                          const unsigned long long (&al)[kConstPerLane])
{
    bool ok = true;
#pragma unroll
    for (int q = 0; q < kConstPerLane; ++q)
        if (lane + kWave * q < C) ok = ok && tag_ok(al[q], a.tag);
    return ok;
}

// Reduce the validated column part (cv) of slice ic and publish it: sums / T
// as kbar and mu, merged (max, normaliser) pairs as they are.  The order of
// every sum depends only on (n, j): the result is the same in any block.
__device__ __forceinline__ void reduce_chunk(const ScoreArgs &a, const Item &ic, const Chunk &ch, int C, int lane,
                                             const float *cv)
{
    const int n = ic.n, ncl = ch.ns + ch.np;
    const float invT = 1.f / (float)ic.T;
    unsigned long long *outT = a.ancT + (long long)ic.u * C;
    float *outP = a.anchors + (long long)ic.u * C;
    for (int t = lane; t < ncl * 16; t += kWave) {  // 16 lanes per column; groups stay whole
        const int lc = t >> 4, q = t & 15;
        if (lc < ch.ns) {
            float s = 0.f;
            for (int jj = q; jj < n; jj += 16) s += cv[lc * n + jj];
            s = seg16_sum(s);
            if (q == 0) {
                const int col = ch.cs0 + lc;
                tag_store(outT + col, s * invT, a.tag);
                outP[col] = s * invT;
            }
        } else {
            const int pr = lc - ch.ns;
            const float *mv = cv + (ch.ns + pr) * n, *sv = cv + (ch.ns + ch.np + pr) * n;
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
}

// d_E partial of a finished slice (sum over keys < T, extrema over keys < P)
// from the compute waves' records.
__device__ __forceinline__ void write_dstats(const ScoreArgs &a, const Item &it, const FusedLds &S)
{
    float s = 0.f, mn = INFINITY, mx = -INFINITY;
    for (int w2 = 0; w2 < kCW; ++w2) {
        s += S.dred[w2][0];
        mn = fminf(mn, S.dred[w2][1]);
        mx = fmaxf(mx, S.dred[w2][2]);
    }
    float *pp = a.part2 + ((int64_t)it.u * a.nch2 + it.j) * 4;
    pp[0] = s;
    pp[1] = mn;
    pp[2] = mx;
    pp[3] = 0.f;
}

// The protocol wave's part of one slice: the block partial from the compute
// waves' LDS records and its publication, the unit's column part assigned to
// this slice, then the unit's constants into LDS.  Returns false once a wait
// has run out of time (the caller then stops waiting for the rest of the
// launch).
__device__ bool protocol(const ScoreArgs &a, const Item &it, int lane, FusedLds &S, bool live)
{
    const int C = 2 * kD + 2 * a.R;
    // block partial: column sums over the compute waves, softmax merges over them
    for (int c = lane; c < 2 * kD; c += kWave) {
        const int which = c / kD, d = c % kD;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kCW; ++w) s += S.wcs[w][which][d];
        tag_store(&a.partT[((long long)it.u * C + c) * a.nch1 + it.j], s, a.tag);
    }
    if (lane < a.R) {
        float m = -INFINITY, s = 0.f;
#pragma unroll
        for (int w = 0; w < kCW; ++w) softmax_merge2(m, s, S.wm[w][lane], S.wsm[w][lane]);
        tag_store(&a.partT[((long long)it.u * C + 2 * kD + lane) * a.nch1 + it.j], m, a.tag);
        tag_store(&a.partT[((long long)it.u * C + 2 * kD + a.R + lane) * a.nch1 + it.j], s, a.tag);
    }
    // the column part assigned to this slice: wait for every slice's partial
    const Chunk ch = chunk_of(it.j, it.n, a.R);
    unsigned long long cl[kChunkPerLane] = {};
    issue_chunk(a, it, ch, C, lane, cl);
    int tries = 0;
    while (live && !__all(chunk_ok(a, ch, lane, cl))) {
        if (++tries > kSpinLimit) {
            live = false;
            break;
        }
        __builtin_amdgcn_s_sleep(2);
        issue_chunk(a, it, ch, C, lane, cl);
    }
    float *cv = &S.wcs[0][0][0];  // the wave records were read above
#pragma unroll
    for (int q = 0; q < kChunkPerLane; ++q) {
        const int t = lane + kWave * q;
        if (t < ch.nl) cv[t] = tag_val(cl[q]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    reduce_chunk(a, it, ch, C, lane, cv);
    // the unit's constants
    unsigned long long al[kConstPerLane] = {};
    issue_consts(a, it, C, lane, al);
    tries = 0;
    while (live && !__all(consts_ok(a, C, lane, al))) {
        if (++tries > kSpinLimit) {
            live = false;
            break;
        }
        __builtin_amdgcn_s_sleep(2);
        issue_consts(a, it, C, lane, al);
    }
#pragma unroll
    for (int q = 0; q < kConstPerLane; ++q) {
        const int c = lane + kWave * q;
        if (c < C) S.anc[c] = tag_val(al[q]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    if (lane < 32) {
        const bool r_ok = lane < a.R;
        const float M = r_ok ? S.anc[2 * kD + lane] : 0.f, Sn = r_ok ? S.anc[2 * kD + a.R + lane] : 1.f;
        S.rsh[lane] = r_ok ? M + __log2f(Sn) : INFINITY;
    }
    // |kbar|^2 of the centroid as the operand rows represent it (bf16 high + remainder)
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
    // the anchor rows of the sweep-2 operand: lane 16q + c builds chunk c of row q
    {
        const int which = lane >> 4, c = lane & 15;
        const float *src = ((which < 2) ? S.anc + kD : S.anc) + 8 * c;
        u32x4 q;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            unsigned half2[2];
#pragma unroll
            for (int z = 0; z < 2; ++z) {
                const float f = src[2 * e + z];
                const unsigned hb = bf16_rne(f);
                half2[z] = (which & 1) ? bf16_rne(f - __uint_as_float(hb << 16)) : hb;
            }
            q[e] = half2[0] | (half2[1] << 16);
        }
        S.arow[which][c] = q;
    }
    return live;
}

__global__ __launch_bounds__(kFThreads, kFBlocksPerCU * kFThreads / kWave / 4) void k_fused(ScoreArgs a)
{
    __shared__ FusedLds S;

    const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const bool comp = wv < kCW;
    const int G = gridDim.x;
    const float sc = a.inv_sqrt_d * kLog2e;
    const float inv_r = 1.f / (float)a.R;
    const int nsteps = (a.items + G - 1) / G;
    constexpr int kAnc = kFusedMaxRows;

    ItemGen gen = item_gen(a, blockIdx.x, G);
    Item it = item_of(a, gen);
    Item prev{};

    if (!comp) {
        // the protocol wave: the same barrier sequence as the compute waves
        bool live = true;
#pragma unroll 1
        for (int k = 0; k < nsteps; ++k) {
            item_next(a, gen);
            const Item nx = item_of(a, gen);
            lds_barrier();  // B1: the slice's wave records (and the last slice's d_E records) are in
            if (prev.valid && lane == 0) write_dstats(a, prev, S);
            if (it.valid) {
                const bool ok = protocol(a, it, lane, S, live);
                if (live && !ok && lane == 0)
                    __hip_atomic_store(a.status, a.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                live = ok;
            }
            lds_barrier();  // B2: the unit's constants are in
            prev = it;
            it = nx;
        }
        lds_barrier();
        if (prev.valid && lane == 0) write_dstats(a, prev, S);
        return;
    }

    u32x4 *wkt = S.kt + 32 * kChunks * wv;
    u32x4 aq[8];  // window operand; rows kAnc .. kAnc+3 take mu and kbar before sweep 2
    if (lane < 32) {
        S.wts[wv][0][lane] = 0x3f80;  // 1.0
        S.wts[wv][3][lane] = 0;
    }
    dma_keys(a, it, wv, lane, wkt);
    load_window(a, it, lane, aq);

#pragma unroll 1
    for (int k = 0; k < nsteps; ++k) {
        // lane-derived indices are recomputed every iteration: kept out of the
        // loop-invariant set, which would otherwise pin them in registers
        int tv = threadIdx.x;
        asm volatile("" : "+v"(tv));
        const int lane = tv & 63, h = lane >> 5, kl = lane & 31;
        const int tr_row = 8 * (lane >> 4) + ((lane & 15) >> 2), tr_b = lane & 3;
        const int w_row = (lane & 15) < 3 ? (lane & 15) : 3;
        item_next(a, gen);
        const Item nx = item_of(a, gen);
        u32x4 kb[8];
        float n2 = 0.f, inv = 0.f;
        if (it.valid) {
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's rows and window operand are in
            // keys into the operand layout (lane l: key l % 32, chunks 2s + l / 32)
#pragma unroll
            for (int st = 0; st < 8; ++st) kb[st] = wkt[sw(kl, 2 * st + h)];
#pragma unroll
            for (int st = 0; st < 8; ++st)
                n2 = dot2sq(kb[st][0], dot2sq(kb[st][1], dot2sq(kb[st][2], dot2sq(kb[st][3], n2))));
            n2 += __shfl_xor(n2, 32, kWave);
            inv = __builtin_amdgcn_rsqf(fmaxf(n2, 1e-24f));
            if (h == 0) {
                const unsigned hi = bf16_rne(inv);
                S.wts[wv][1][kl] = (uint16_t)hi;
                S.wts[wv][2][kl] = (uint16_t)bf16_rne(inv - __uint_as_float(hi << 16));
            }
            // column sums over the wave's 32 keys (zero rows past T add nothing); a
            // wave's own LDS accesses are ordered.  Transposed reads: lane 16G + 4a + b
            // reads key row 8G + a (+4), dimensions 16 blk + 4b .. +3; the read returns
            // dimension 16 blk + lane % 16 of keys 8G + 0..3 (then 4..7)
            typedef float f32x4v __attribute__((ext_vector_type(4)));
            typedef short s16x4 __attribute__((ext_vector_type(4)));
            const bf16x8 wa = *reinterpret_cast<const bf16x8 *>(&S.wts[wv][w_row][8 * (lane >> 4)]);
            const uint16_t *st16 = reinterpret_cast<const uint16_t *>(wkt);
#pragma unroll
            for (int blk = 0; blk < 8; ++blk) {
                const int c = 2 * blk + (tr_b >> 1), off = (tr_b & 1) * 4;
                const uint16_t *p0 = st16 + tr_row * kD + ((c ^ (tr_row & 15)) << 3) + off;
                const uint16_t *p1 = st16 + (tr_row + 4) * kD + ((c ^ ((tr_row + 4) & 15)) << 3) + off;
                const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p0)));
                const s16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4 *)(const_cast<uint16_t *>(p1)));
                const short __attribute__((ext_vector_type(8))) kb8 = {lo[0],  lo[1],  lo[2],  lo[3],
                                                                        hi4[0], hi4[1], hi4[2], hi4[3]};
                const f32x4v cs = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    wa, __builtin_bit_cast(bf16x8, kb8), (f32x4v){0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                if (lane < 16) {
                    S.wcs[wv][0][16 * blk + lane] = cs[0];
                    S.wcs[wv][1][16 * blk + lane] = cs[1] + cs[2];
                }
            }
        }
        // every read of this wave's rows has completed: its rows of the next slice may land
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __builtin_amdgcn_sched_barrier(0);
        dma_keys(a, nx, wv, lane, wkt);
        __builtin_amdgcn_sched_barrier(0);
        if (it.valid) {
            // window logits: keys as A, window rows as B; lane holds row kl against
            // keys 8(r/4) + 4h + r%4 of the wave
            f32x16 acc = (f32x16){};
#pragma unroll
            for (int st = 0; st < 8; ++st)
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, kb[st]),
                                                              __builtin_bit_cast(bf16x8, aq[st]), acc, 0, 0, 0);
            float mx = -INFINITY;
            if (it.base + 32 * (wv + 1) <= it.P) {
                // every key of the wave precedes the window: visible to every row
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    acc[r] *= sc;
                    mx = fmaxf(mx, acc[r]);
                }
            } else {
                const int kb0 = it.base + 32 * wv + 4 * h;
                const int lim = a.causal ? it.P + kl % a.w : it.T - 1;  // last key visible to row kl
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int gk = kb0 + 8 * (r >> 2) + (r & 3);
                    acc[r] = (gk < it.T && gk <= lim) ? acc[r] * sc : -INFINITY;
                    mx = fmaxf(mx, acc[r]);
                }
            }
            float s = 0.f;
            if (mx != -INFINITY)
#pragma unroll
                for (int r = 0; r < 16; ++r) s += fast_exp2(acc[r] - mx);
            const float m2 = __shfl_xor(mx, 32, kWave), s2 = __shfl_xor(s, 32, kWave);
            softmax_merge2(mx, s, m2, s2);
            if (h == 0) {
                S.wm[wv][kl] = mx;
                S.wsm[wv][kl] = s;
            }
        }
        lds_barrier();  // B1
        lds_barrier();  // B2: the unit's constants are in
        if (it.valid) {
            // rows kAnc .. kAnc+3 of the operand: mu high, mu remainder, kbar high, kbar remainder
            if (kl >= kAnc) {
#pragma unroll
                for (int st = 0; st < 8; ++st) aq[st] = S.arow[kl - kAnc][2 * st + h];
            }
            // sweep 2: window rows and anchors as A, keys as B; lane holds key kl
            // against rows 8(r/4) + 4h + r%4
            f32x16 acc = (f32x16){};
#pragma unroll
            for (int st = 0; st < 8; ++st)
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, aq[st]),
                                                              __builtin_bit_cast(bf16x8, kb[st]), acc, 0, 0, 0);
            float att = 0.f;
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                typedef float f32x4v __attribute__((ext_vector_type(4)));
                const f32x4v sh = *reinterpret_cast<const f32x4v *>(&S.rsh[8 * g4 + 4 * h]);
#pragma unroll
                for (int e = 0; e < 4; ++e) att += fast_exp2(fmaf(acc[4 * g4 + e], sc, -sh[e]));
            }
            float kmu = h ? acc[12] + acc[13] : 0.f;
            float kk = h ? acc[14] + acc[15] : 0.f;
            att += __shfl_xor(att, 32, kWave);
            kmu += __shfl_xor(kmu, 32, kWave);
            kk += __shfl_xor(kk, 32, kWave);
            const float dE = __builtin_amdgcn_sqrtf(fmaxf(n2 - 2.f * kk + S.kb2, 0.f));
            const float cm = kmu * inv;
            const int gi = it.base + 32 * wv + kl;
            float dsum = 0.f, dmn = INFINITY, dmx = -INFINITY;
            if (h == 0) {
                if (gi < it.T) dsum = dE;
                if (gi < it.P) {
                    dmn = dE;
                    dmx = dE;
                    const Unit un = unit_of(it.u, a.Hkv, a.B);
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
        load_window(a, nx, lane, aq);  // the next slice's window operand
        it = nx;
    }
    lds_barrier();
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
    // largest load list of any column part of a unit with n slices
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

bool fused_eligible(int D, bool bf16, int R, const SeqTab &seq, int L, int Hkv, int Hq, int w, int *grid)
{
    if (!bf16 || D != fast::kD || R > kFusedMaxRows || R < 1) return false;
    // window rows are addressed through one 32-bit buffer range
    if ((long long)L * Hq * seq.nseq * w * D * 2 >= (1LL << 31)) return false;
    DevInfo di;
    if (!dev_info(&di)) return false;
    long long ns = 0;
    int nmax = 0;
    for (int s = 0; s < seq.nseq; ++s) {
        const int T = seq.cu[s + 1] - seq.cu[s];
        if ((long long)(T + kFusedItem) * D * 2 >= (1LL << 31)) return false;  // 32-bit key offsets
        const int n = (T + kFusedItem - 1) / kFusedItem;
        ns += n;
        if (n > nmax) nmax = n;
        if (chunk_loads_max(n, R) > fast::kChunkMax) return false;
    }
    const long long items = (long long)L * Hkv * ns;
    if (items < 1 || items > (1LL << 30)) return false;
    const long long g = items < (long long)di.ncu * di.per_cu ? items : (long long)di.ncu * di.per_cu;
    // every unit must span at most G slices (two consecutive steps)
    if (nmax > g) return false;
    *grid = (int)g;
    return true;
}

unsigned launch_tag()
{
    unsigned t = ++g_tag;
    if (t == 0) t = ++g_tag;
    return t;
}

hipError_t fused_launch(ScoreArgs &a, int grid, hipStream_t st)
{
    a.tag = launch_tag();
    hipLaunchKernelGGL(fast::k_fused, dim3(grid), dim3(fast::kFThreads), 0, st, a);
    return hipGetLastError();
}

}  // namespace ecokv
