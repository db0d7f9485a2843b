// ecokv_compact kernel (gfx950): gather of the kept K/V rows (Sec. 3).
//
// A flat grid over (entry, 16-byte segment): consecutive threads copy
// consecutive 16-byte pieces of one row, so both the row read and the
// compacted write are coalesced streams.  The unit of an entry follows from
// the documented idx layout (PER_HEAD: arithmetic; LAYER_FLAT: the group by
// arithmetic, the head from the offsets written by ecokv_select;
// HEAD_BUDGETS: the (layer, head) pair by a binary search of the launch's
// table of pair starts).  Entries whose position lies outside [0, T_s) are
// skipped.
#include "ecokv_internal.h"

namespace ecokv {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCompactThreads = 256;

__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a)
{
    const int64_t t = (int64_t)blockIdx.x * kCompactThreads + threadIdx.x;
    const int64_t e = a.e0 + t / a.segs;
    if (e >= a.total) return;
    const int seg = (int)(t - (e - a.e0) * a.segs);
    int l, h, s;
    if (a.heads) {
        // the pair j with start[j] <= e < start[j + 1]: a binary search for the
        // wave's first entry (wave-uniform, scalar loads), then each lane steps
        // forward (a wave covers a few rows, nearly always of one pair)
        const int64_t ew = a.e0 + ((int64_t)blockIdx.x * kCompactThreads +
                                   64 * __builtin_amdgcn_readfirstlane(threadIdx.x >> 6)) / a.segs;
        int lo = 0, hi = a.lht.n - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (a.lht.start[mid] <= ew) lo = mid;
            else hi = mid - 1;
        }
        while (lo + 1 < a.lht.n && a.lht.start[lo + 1] <= e) ++lo;
        const int lh = a.lht.lh0 + lo;
        l = lh / a.Hkv;
        h = lh - l * a.Hkv;
        int r = (int)(e - a.lht.start[lo]);
        s = 0;
        for (int c; s + 1 < a.B && r >= (c = min(a.lht.b[lo], a.seq.cu[s + 1] - a.seq.cu[s])); ++s) r -= c;
    } else if (!a.flat) {
        const int64_t lh = e / a.per_lh;
        const int64_t r = e - lh * a.per_lh;
        s = 0;
        while (s + 1 < a.B && a.seq.boff[s + 1] <= r) ++s;
        l = (int)(lh / a.Hkv);
        h = (int)(lh - (int64_t)l * a.Hkv);
    } else {
        const int64_t gl = (int64_t)a.Hkv * a.per_lh;
        l = (int)(e / gl);
        const int64_t r = e - (int64_t)l * gl;
        s = 0;
        while (s + 1 < a.B && (int64_t)a.Hkv * a.seq.boff[s + 1] <= r) ++s;
        h = 0;
        while (h + 1 < a.Hkv && a.offsets[((int64_t)l * a.Hkv + h + 1) * a.B + s] <= e) ++h;
    }
    const int T = a.seq.cu[s + 1] - a.seq.cu[s];
    const int32_t pos = a.idx[e];
    if (pos < 0 || pos >= T) return;
    const int64_t src = ((int64_t)l * a.Hkv + h) * a.Ttot + a.seq.cu[s] + pos;
    const int64_t so = src * a.row_bytes + (int64_t)seg * 16;
    const int64_t d = e * a.row_bytes + (int64_t)seg * 16;
    // Nontemporal in both directions: the rows are read once here, and the
    // compacted copy is not read again by this pass.  Without the streaming
    // hint the written lines stay dirty in the caches and are written back
    // while the next pass streams K, taking bandwidth from it.
    const u32x4 kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.K + so));
    const u32x4 vv = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.V + so));
    __builtin_nontemporal_store(kv, reinterpret_cast<u32x4 *>(a.Kc + d));
    __builtin_nontemporal_store(vv, reinterpret_cast<u32x4 *>(a.Vc + d));
}

hipError_t compact_launch(const CompactArgs &a, hipStream_t st)
{
    const int64_t threads = (a.total - a.e0) * a.segs;
    if (threads == 0) return hipSuccess;
    const int64_t blocks = (threads + kCompactThreads - 1) / kCompactThreads;
    ECOKV_TIMED("compact", st, hipLaunchKernelGGL(k_compact, dim3((unsigned)blocks), dim3(kCompactThreads), 0, st, a));
    return hipGetLastError();
}

}  // namespace ecokv
