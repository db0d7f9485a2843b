// Internal definitions of libecokv (gfx950).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ecokv.h"

namespace ecokv {

constexpr int kWave = 64;

// Per-call table of sequence boundaries and budgets, passed by value as a
// kernel argument so that no device copy of host arrays is needed.
struct SeqTab {
    int nseq;
    int cu[ECOKV_MAX_SEQS + 1];    // token offsets (prefix of T_s)
    int beff[ECOKV_MAX_SEQS];      // min(b_s, T_s)
    int boff[ECOKV_MAX_SEQS + 1];  // prefix of beff
};

// Decode unit u = (l*Hkv + h)*B + s.
struct Unit {
    int l, h, s;
};
__device__ __forceinline__ Unit unit_of(int u, int Hkv, int B)
{
    Unit r;
    r.s = u % B;
    const int lh = u / B;
    r.h = lh % Hkv;
    r.l = lh / Hkv;
    return r;
}

struct ScoreArgs {
    const void *K;
    const void *V;   // values, read only with the value-norm importance (vnorm)
    const void *Q;
    float *scores;
    float *lambda;
    float *stats;
    // workspace regions
    float *part1;    // [U][nch1][2D + 2R]  column sums, row max / sum-exp per block
    float *anchors;  // [U][2D + 2R]        kbar, mu, row max, row normaliser
    float *part2;    // [U][nch2][4]        sum d_E, min d_E, max d_E, sum d_E^2 per block
    float *part3;    // [U][nch3][4]        sum S_div, sum S_imp, min/max S_div per block
    float *bufA;     // [L][Hkv][Ptot]      d_E
    float *bufB;     // [L][Hkv][Ptot]      khat.mu
    float *bufC;     // [L][Hkv][Ptot]      window-mean attention a
    float *bufV;     // [L][Hkv][Ptot]      pool(a) * |v| (vnorm only)
    // values the two blocks of a unit's split epilogue exchange, each a 64-bit
    // word (launch tag << 32 | float bits) so that a reader can tell a value of
    // this launch from anything older without ordering fences
    unsigned long long *epiT;   // [U][4][4]           per-part S_div / S_imp sums and extrema
    unsigned *status;           // workspace status word: set to the call's tag if a wait ran out of time
    unsigned *tagw;             // workspace word: the call's tag (bumped by the second sweep, never 0)
    int spin_limit;             // polls of a bounded wait before it gives up (<= 0: give up at once)
    int no_wait;                // no waits between blocks (the final step one block per unit)
    int L, Hq, Hkv, G, D, w, R, B;
    int64_t Ttot, Ptot;
    int nch1;        // sweep blocks per unit (for the longest sequence)
    int nch3;        // epilogue blocks per unit
    int rpb1;        // key rows per sweep-1 block
    int nch2;        // sweep-2 blocks per unit (d_E partials in part2)
    int rpb2;        // key rows per sweep-2 block
    float alpha, beta, eps, tau, inv_sqrt_d, lambda_override;
    int use_override, pool_half, causal;
    int vnorm;       // S_imp = pool(a) * |v_i|_2
    int kbf16;       // K holds bf16 (else fp32)
    int norm_mode;   // ECOKV_NORM_*: how d_E becomes s_E
    float mad_tau, winsor_q;
    const float *dq; // [U][2] quantile pair of d_E per unit (winsorised or MAD norm)
    int red_std;     // lambda uses r_std (Appendix D) instead of r_E
    int centroid_prefix;  // kbar over the non-window keys (Appendix B.6)
    const float *pre;     // [U][2D + 2R] caller-supplied first-sweep sums (ecokv_score_pre), or null
    // the KV-cache write with the first sweep (ecokv_prefill_write): K rows are
    // read from Ksrc (token-major, [L][Ttot][Hkv][D]) and written to K (the
    // head-major cache) while sweep 1 runs over them; the reduction writes
    // pre_out in the layout of `pre`
    const void *Ksrc;
    float *pre_out;
    SeqTab seq;
};

// Budgets of up to kLhChunk (layer, KV head) pairs, passed by value to one
// launch (ECOKV_HEAD_BUDGETS): pair lh0 + j keeps min(b[j], T_s) tokens of
// sequence s, and its entries start at idx offset start[j] (start[n] = end).
constexpr int kLhChunk = 256;
struct LhTab {
    int lh0, n;
    int b[kLhChunk];
    int start[kLhChunk + 1];
};

// Entries of pair j of `t` before sequence s, and min(b, T_s).
__device__ __forceinline__ int lh_seq_offset(const LhTab &t, const SeqTab &q, int j, int s)
{
    int o = 0;
    for (int r = 0; r < s; ++r) o += min(t.b[j], q.cu[r + 1] - q.cu[r]);
    return o;
}

struct SelectArgs {
    const float *scores;
    int32_t *idx;
    int32_t *counts;
    int32_t *offsets;
    int L, Hkv, B, w;
    int64_t Ptot;
    int64_t per_lh;  // sum over s of min(b_s, T_s) (not ECOKV_HEAD_BUDGETS)
    int flat;
    int heads;       // ECOKV_HEAD_BUDGETS: budgets and starts from lht
    // the caller's workspace (select_ws_layout(mb_groups, mb_maxn)), filled by select_launch
    uint4 *mb_state;     // [3][mb_groups]           selection state after each digit
    uint32_t *mb_hist;   // [mb_groups][5120]        global digit histograms
    uint32_t *mb_head;   // [mb_groups][256][2]      per-head keys above / equal to the threshold
    uint32_t *mb_cnt;    // [mb_groups][slices][2]   per-slice keys above / equal to the threshold
    int64_t mb_groups;   // groups of the largest launch of the call
    int64_t mb_maxn;     // keys of the largest group of the call
    int mb_slices;       // slices per group of this launch
    // two-stage selection of long single-head groups with small budgets:
    // each slice's own top keys, then the group's among them
    int32_t *c_pos;      // [mb_groups][c_slices][slice keys] candidate positions, ascending per slice
    uint32_t *c_key;     // the same layout: their order-preserving keys
    int c_slices;        // slices per group of this launch
    SeqTab seq;
    LhTab lht;
};

// Workspace of ecokv_select.
struct SelWsLayout {
    size_t state, hist, head, cnt, cand, total;
};
// per_head: every group is a single head (ECOKV_PER_HEAD, ECOKV_HEAD_BUDGETS)
SelWsLayout select_ws_layout(int64_t groups, int64_t maxn, bool per_head);

struct CompactArgs {
    const char *K;
    const char *V;
    char *Kc;
    char *Vc;
    const int32_t *idx;
    const int32_t *offsets;
    int L, Hkv, B, flat;
    int heads;         // ECOKV_HEAD_BUDGETS: entries [e0, total) of the pairs in lht
    int64_t Ttot;
    int row_bytes;
    int segs;          // row_bytes / 16
    int64_t e0;        // first entry of this launch
    int64_t total;     // one past its last entry
    int64_t per_lh;
    SeqTab seq;
    LhTab lht;
};

// Workspace layout, shared by the size query and the launcher.
struct WsLayout {
    size_t status, tagw, part1, anchors, part2, part3, bufA, bufB, bufC, bufV, dq, epiT, total;
};

// Order statistics of d_E per unit for the winsorised and MAD normalisations:
// out[u] = (quantile q, quantile 1 - q), or (median, median of |d - median|).
struct DQuantArgs {
    const float *d;  // [L][Hkv][Ptot] d_E of the non-window keys
    float *out;      // [U][2]
    int L, Hkv, B, w;
    int64_t Ptot;
    int mode;        // ECOKV_NORM_WINSOR or ECOKV_NORM_MAD
    float q;
    SeqTab seq;
};
hipError_t dquant_launch(const DQuantArgs &a, hipStream_t st);

// Decode attention over the compressed cache (one query per query head).
struct DecodeArgs {
    const void *Q;        // [L][Hq][B][D]
    const void *Kc;       // [entries][D]
    const void *Vc;
    const int32_t *counts;   // [L][Hkv][B]
    const int32_t *offsets;  // [L][Hkv][B]
    float *O;             // [L][Hq][B][D]
    float *lse;           // [L][Hq][B] or null
    float *part;          // [L][Hq][B][nparts][D + 2]: max, sum, acc per row chunk
    int L, Hq, Hkv, G, B, D;
    int max_count, nparts;  // nparts: chunks per query row in part (decode_parts(max_count))
    int wave_rows;        // rows per wave; a chunk is the rows of a block's waves
    float qscale;         // log2(e) / sqrt(D)
};
int decode_parts(int max_count);
// Sets a.nparts and a.wave_rows, then launches the decode and merge kernels.
hipError_t decode_launch(DecodeArgs a, bool bf16, hipStream_t st);

WsLayout score_ws_layout(int L, int Hkv, int B, int D, int R, int64_t Ptot, int maxT, bool bf16, bool vnorm);
hipError_t score_launch(ScoreArgs a, char *ws, const WsLayout &lay, int maxT, hipStream_t st, bool bf16);

// A launch tag (never 0), distinct for every launch of the process: values a
// launch publishes between its blocks carry it.

// ecokv_prefill_write: workspace bytes, and the launches (a.K = the cache,
// a.Ksrc = the new rows, a.pre_out = pre; Vsrc / Vdst may be null).
size_t prefill_ws_bytes(int L, int Hkv, int B, int D, int R, int maxT, bool bf16);
hipError_t prefill_launch(ScoreArgs a, const void *Vsrc, void *Vdst, char *ws, int maxT, hipStream_t st, bool bf16);
// Clears the workspace status word (stream-ordered, by a one-thread kernel).
hipError_t status_clear(unsigned *status, hipStream_t st);
constexpr int kStreamMaxRows = 30;     // window rows of the streaming sweep 2; 2 more rows carry mu
hipError_t select_launch(SelectArgs a, char *ws, hipStream_t st);
int select_max_flat_heads();
hipError_t compact_launch(const CompactArgs &a, hipStream_t st);

// Optional per-kernel timing (ECOKV_STAGE_TIMING=1): every launch site calls
// stage_begin before and stage_end after its launch; both are no-ops unless
// the variable is set.
bool stage_timing_on();
void stage_begin(const char *name, hipStream_t st);
void stage_end(hipStream_t st);
#define ECOKV_TIMED(name, st, ...)          \
    do {                                    \
        ::ecokv::stage_begin((name), (st)); \
        __VA_ARGS__;                        \
        ::ecokv::stage_end((st));           \
    } while (0)

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// orders global memory, which makes every barrier wait for all outstanding
// global loads; this one leaves prefetched loads in flight.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float bf16_to_f32(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }

// Lane moves within 16-lane rows (DPP, no LDS round trip): quad permutes, the
// mirrored lane within each 8 and within each 16.
template <int CTRL>
__device__ __forceinline__ float dpp_row(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// op over the S lanes of an aligned group (S = 16, 32 or 64), every lane
// getting the result: butterflies by DPP within each 16-lane row (lane ^ 1,
// lane ^ 2 by quad permutes, then the mirrored lane within 8 and, for groups
// of 16 or more, within 16, each pairing a lane with the other half), and one
// cross-lane move for each further doubling (lane ^ 16, lane ^ 32).  The same operations in every lane,
// so all hold the same value.
template <int S, class Op>
__device__ __forceinline__ float row_reduce(float x, Op op)
{
    static_assert(S == 8 || S == 16 || S == 32 || S == 64, "group of 8, 16, 32 or 64 lanes");
    x = op(x, dpp_row<0xB1>(x));   // quad_perm [1, 0, 3, 2]
    x = op(x, dpp_row<0x4E>(x));   // quad_perm [2, 3, 0, 1]
    x = op(x, dpp_row<0x141>(x));  // row_half_mirror
    if constexpr (S >= 16) x = op(x, dpp_row<0x140>(x));  // row_mirror
    if constexpr (S >= 32) x = op(x, __shfl_xor(x, 16, kWave));
    if constexpr (S == 64) x = op(x, __shfl_xor(x, 32, kWave));
    return x;
}
struct OpAdd {
    __device__ float operator()(float x, float y) const { return x + y; }
};
struct OpMin {
    __device__ float operator()(float x, float y) const { return fminf(x, y); }
};
struct OpMax {
    __device__ float operator()(float x, float y) const { return fmaxf(x, y); }
};

// The same on 32-bit unsigned values, and a DPP move with row / bank masks
// (lanes outside them, or without a source lane, take 0).
template <int CTRL, int ROWS = 0xF, int BANKS = 0xF>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, BANKS, false);
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x)
{
    x = min(x, dpp_u32<0xB1>(x));
    x = min(x, dpp_u32<0x4E>(x));
    x = min(x, dpp_u32<0x141>(x));
    x = min(x, dpp_u32<0x140>(x));
    x = min(x, (uint32_t)__shfl_xor(x, 16, kWave));
    return min(x, (uint32_t)__shfl_xor(x, 32, kWave));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x)
{
    x = max(x, dpp_u32<0xB1>(x));
    x = max(x, dpp_u32<0x4E>(x));
    x = max(x, dpp_u32<0x141>(x));
    x = max(x, dpp_u32<0x140>(x));
    x = max(x, (uint32_t)__shfl_xor(x, 16, kWave));
    return max(x, (uint32_t)__shfl_xor(x, 32, kWave));
}

// Inclusive prefix sum over the 64 lanes of a wave (lane i: x_0 + ... + x_i)
// by DPP, with no LDS round trip: within each 16-lane row the inputs shifted
// by 1, 2 and 3 lanes give sums of 4, the partial sums shifted by 4 (lanes
// 4..15) and by 8 (lanes 8..15) sums of 8 and 16; then rows 1 and 3 add the
// last lane of rows 0 and 2 (row broadcast 15) and rows 2 and 3 the last lane
// of row 1 (row broadcast 31).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x)
{
    uint32_t v = x + dpp_u32<0x111>(x);  // row_shr:1
    v += dpp_u32<0x112>(x);              // row_shr:2
    v += dpp_u32<0x113>(x);              // row_shr:3
    v += dpp_u32<0x114, 0xF, 0xE>(v);    // row_shr:4, banks 1-3
    v += dpp_u32<0x118, 0xF, 0xC>(v);    // row_shr:8, banks 2-3
    v += dpp_u32<0x142, 0xA, 0xF>(v);    // row_bcast:15 into rows 1, 3
    v += dpp_u32<0x143, 0xC, 0xF>(v);    // row_bcast:31 into rows 2, 3
    return v;
}

// Sum over the wave (the last lane of the inclusive scan, read as a scalar).
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(x), kWave - 1);
}

// Sum over the 16 lanes of an aligned 16-lane segment; every lane gets the total.
__device__ __forceinline__ float seg16_sum(float x) { return row_reduce<16>(x, OpAdd{}); }

__device__ __forceinline__ float wave_sum(float x) { return row_reduce<64>(x, OpAdd{}); }
__device__ __forceinline__ float wave_min(float x) { return row_reduce<64>(x, OpMin{}); }
__device__ __forceinline__ float wave_max(float x) { return row_reduce<64>(x, OpMax{}); }

// Load the VEC = D/16 elements of segment c of a key row as float.
template <int D, bool BF>
__device__ __forceinline__ void load_seg(const void *row, int c, float *v)
{
    constexpr int VEC = D / 16;
    if constexpr (BF) {
        const uint16_t *p = static_cast<const uint16_t *>(row) + c * VEC;
        if constexpr (VEC == 8) {
            const uint4 q = *reinterpret_cast<const uint4 *>(p);
            const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[2 * e] = __uint_as_float(w4[e] << 16);
                v[2 * e + 1] = __uint_as_float(w4[e] & 0xffff0000u);
            }
        } else {
            const uint2 q = *reinterpret_cast<const uint2 *>(p);
            v[0] = __uint_as_float(q.x << 16);
            v[1] = __uint_as_float(q.x & 0xffff0000u);
            v[2] = __uint_as_float(q.y << 16);
            v[3] = __uint_as_float(q.y & 0xffff0000u);
        }
    } else {
        const float *p = static_cast<const float *>(row) + c * VEC;
        if constexpr (VEC == 8) {
            const float4 a = reinterpret_cast<const float4 *>(p)[0];
            const float4 b = reinterpret_cast<const float4 *>(p)[1];
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
            const float4 a = reinterpret_cast<const float4 *>(p)[0];
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        }
    }
}

// A value the caller knows to be equal in every lane of the wave, made
// visibly so to the compiler (read from the first active lane): buffer
// descriptors built from it then live in scalar registers, instead of every
// buffer access being repeated for each distinct descriptor value.
__device__ __forceinline__ int uniform_i32(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uniform_i64(int64_t v)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
template <class T>
__device__ __forceinline__ T *uniform_ptr(T *p)
{
    return reinterpret_cast<T *>(uniform_i64(reinterpret_cast<int64_t>(p)));
}

// Sum over the S lanes of a row group (S = 8, 16 or 32), in every lane.
template <int S>
__device__ __forceinline__ float row_sum(float x)
{
    return row_reduce<S>(x, OpAdd{});
}

// Order-preserving map of a float score to an unsigned radix key: larger
// score -> larger key; -0 maps like +0; NaN maps below every number.
__device__ __forceinline__ uint32_t score_key(float f)
{
    uint32_t b = __float_as_uint(f);
    if (f != f) return 0u;
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

}  // namespace ecokv
