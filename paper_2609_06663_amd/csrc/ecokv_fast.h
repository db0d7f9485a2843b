// Device helpers shared by the score kernels (gfx950): vector types, unit
// addressing, log2-domain softmax merging and the LDS tile geometry of the
// bf16 / head_dim 128 path.  Not part of the ABI.
#pragma once

#include "ecokv_internal.h"

namespace ecokv {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ int64_t unit_out_base(const ScoreArgs &a, const Unit &un)
{
    return ((int64_t)un.l * a.Hkv + un.h) * a.Ptot + (a.seq.cu[un.s] - un.s * a.w);
}

__device__ __forceinline__ int64_t unit_row0(const ScoreArgs &a, const Unit &un)
{
    return ((int64_t)un.l * a.Hkv + un.h) * a.Ttot + a.seq.cu[un.s];
}

// Global row index of window row r = (g, j) of unit `un` in Q_win.
__device__ __forceinline__ int64_t window_row(const ScoreArgs &a, const Unit &un, int r)
{
    const int g = r / a.w, j = r % a.w;
    return (((int64_t)un.l * a.Hq + (int64_t)un.h * a.G + g) * a.B + un.s) * a.w + j;
}

constexpr float kLog2e = 1.4426950408889634f;

// Combine two softmax partials (max, sum of 2^(x - max)), x in log2 units.
__device__ __forceinline__ void softmax_merge2(float &m, float &s, float m2, float s2)
{
    const float nm = fmaxf(m, m2);
    const float a = (m == -INFINITY) ? 0.f : s * __builtin_amdgcn_exp2f(m - nm);
    const float b = (m2 == -INFINITY) ? 0.f : s2 * __builtin_amdgcn_exp2f(m2 - nm);
    m = nm;
    s = a + b;
}

namespace fast {

// Hot-loop transcendentals as single instructions (v_exp_f32, v_rsq_f32,
// v_sqrt_f32, about 1 ulp).  Every exponent argument here is <= 0, so results
// below 2^-126 (flushed to zero) are negligible next to the softmax terms of
// size 1 they are added to.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

constexpr int kD = 128;
constexpr int kChunks = 16;           // 16-byte chunks per key row
constexpr int kTile = 128;            // keys per LDS tile (4 waves x 32 keys)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void unpack8(u32x4 q, float *v)
{
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[2 * e] = __uint_as_float(q[e] << 16);
        v[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
    }
}

// acc + lo*lo + hi*hi of the two bf16 halves of w (v_dot2c_f32_bf16).
__device__ __forceinline__ float dot2sq(unsigned w, float acc)
{
    const bf16x2 v = __builtin_bit_cast(bf16x2, w);
    return __builtin_amdgcn_fdot2_f32_bf16(v, v, acc, false);
}

// Round-to-nearest-even bf16 of a finite float (bit pattern in the low half).
__device__ __forceinline__ unsigned bf16_rne(float f)
{
    unsigned u = __float_as_uint(f);
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// Swizzled position of 16-byte chunk c of tile row r.
__device__ __forceinline__ int sw(int r, int c) { return r * kChunks + (c ^ (r & 15)); }

// Buffer descriptor over the key rows [0, rows) of a unit (raw buffer, no
// stride): loads at or past the end return zero without touching memory.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t key_rows_rsrc(const uint16_t *krow0, int rows)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(krow0), (short)0, rows * (kD * 2), 0x00020000);
}

// group_load over rows `row_bytes` apart (key rows interleaved with other
// heads' rows, as a projection writes them): the same lane layout.
__device__ __forceinline__ void group_load_rows(u32x4 (&b)[8], __amdgpu_buffer_rsrc_t rs, int key0, int lane,
                                                int row_bytes)
{
#pragma unroll
    for (int i = 0; i < 8; ++i)
        b[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (key0 + 4 * i + (lane >> 4)) * row_bytes + (lane & 15) * 16, 0,
                                                     2);
}

// Store of 32 key rows held in the load layout of group_load to consecutive
// 256-byte rows (stores at or past the descriptor's end are dropped).
__device__ __forceinline__ void group_store(const u32x4 (&b)[8], __amdgpu_buffer_rsrc_t rs, int key0, int lane)
{
#pragma unroll
    for (int i = 0; i < 8; ++i)
        __builtin_amdgcn_raw_buffer_store_b128(b[i], rs, (key0 + 4 * i + (lane >> 4)) * (kD * 2) + (lane & 15) * 16, 0,
                                               2);
}

// Lane layout of a 32-key B operand of v_mfma_f32_32x32x16_bf16 (and of the
// window-row A operands): lane l holds, for k-step s = 0..7, the 16-byte chunk
// 2s + l/32 of its row, i.e. dimensions 8(2s + h) .. +7 with h = l/32.

// MFMA operand row `which` (0: bf16 high part, 1: bf16 remainder) of the
// fp32 vector v [kD] in that layout.
__device__ __forceinline__ void mu_operand(const float *v, int which, int h, bf16x8 (&op)[8])
{
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        const float4 *src = reinterpret_cast<const float4 *>(v + 8 * (2 * s + h));
        const float4 x = src[0], y = src[1];
        const float f8[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
        u32x4 q;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            unsigned half2[2];
#pragma unroll
            for (int z = 0; z < 2; ++z) {
                const float f = f8[2 * e + z];
                const unsigned hb = bf16_rne(f);
                half2[z] = which ? bf16_rne(f - __uint_as_float(hb << 16)) : hb;
            }
            q[e] = half2[0] | (half2[1] << 16);
        }
        op[s] = __builtin_bit_cast(bf16x8, q);
    }
}

// The centroid's components at the 64 dimensions a lane holds in that layout.
__device__ __forceinline__ void centroid_lane(const float *kbar, int h, float (&kb)[8][8])
{
#pragma unroll
    for (int s = 0; s < 8; ++s) {
        const float4 *src = reinterpret_cast<const float4 *>(kbar + 8 * (2 * s + h));
        const float4 x = src[0], y = src[1];
        kb[s][0] = x.x; kb[s][1] = x.y; kb[s][2] = x.z; kb[s][3] = x.w;
        kb[s][4] = y.x; kb[s][5] = y.y; kb[s][6] = y.z; kb[s][7] = y.w;
    }
}

// Sum over the lane's 64 dimensions of (k_d - kbar_d)^2, the differences
// formed in fp32 (exact for bf16 keys near the centroid); two partial sums.
__device__ __forceinline__ float dist2_lane(const u32x4 (&b)[8], const float (&kb)[8][8])
{
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float d0 = __uint_as_float(b[s][e] << 16) - kb[s][2 * e];
            const float d1 = __uint_as_float(b[s][e] & 0xffff0000u) - kb[s][2 * e + 1];
            s0 = fmaf(d0, d0, s0);
            s1 = fmaf(d1, d1, s1);
        }
    return s0 + s1;
}

}  // namespace fast
}  // namespace ecokv
