// Gather-compaction of the retained K/V rows into the ragged per-layer cache.
//
// After eviction every layer keeps b_l tokens (Eq. (10)); the cache of Sec. 3.1
// holds only those rows, in ascending position, followed by decode_reserve free
// slots that decode (Eq. (3)-(4)) fills.  The work is a pure HBM stream: read
// and write each retained row once.  The grid runs over the flat list of
// retained rows (known on the host: B * B_tot per KV head), so it is sized by
// the bytes moved, not by the largest layer; a row finds its (sequence, layer)
// by binary search in the offsets.  A row of head_dim bf16 is moved by
// head_dim/8 lanes with 16-byte loads and stores.
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kRowsPerBlock = 64;

template <int D>
__global__ __launch_bounds__(kThreads) void compact_kernel(Shape s, const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ budgets,
                                                           const int64_t* __restrict__ idx_off,
                                                           const int64_t* __restrict__ seg_off, int reserve,
                                                           long long rows_total, uint16_t* __restrict__ kc,
                                                           uint16_t* __restrict__ vc) {
    constexpr int CPR = D / 8;             // lanes per row
    constexpr int RPP = kThreads / CPR;    // rows per pass
    const int kvh = blockIdx.y;
    const int g = s.ngroups;
    const int nbl = s.B * s.L;
    const int cc = threadIdx.x % CPR;
    const long long r0 = (long long)blockIdx.x * kRowsPerBlock;
#pragma unroll
    for (int pass = 0; pass < kRowsPerBlock / RPP; ++pass) {
        const long long f = r0 + pass * RPP + threadIdx.x / CPR;
        if (f >= rows_total) break;
        // largest bl with idx_off[bl] / g <= f (per-group flat row numbering)
        int lo = 0, hi = nbl - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (idx_off[mid] / g <= f) lo = mid;
            else hi = mid - 1;
        }
        const int bl = lo;
        const int bsz = budgets[bl];
        const long long n = f - idx_off[bl] / g;
        // positions come from tgvkv_select; clamp so a corrupt index can never read outside the slice
        const int p = min(max(idx[idx_off[bl] + (s.head_mode == 0 ? 0 : (long long)kvh * bsz) + n], 0), s.N - 1);
        const size_t src = (((size_t)bl * s.Hkv + kvh) * (size_t)s.N + p) * D + cc * 8;
        const size_t dst = ((size_t)seg_off[bl] * s.Hkv + (size_t)kvh * (bsz + reserve) + n) * D + cc * 8;
        store16(kc + dst, load16(k + src));
        store16(vc + dst, load16(v + src));
    }
}

}  // namespace

hipError_t launch_compact(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                          const int32_t* budgets, const int64_t* idx_off, const int64_t* seg_off, int32_t reserve,
                          int64_t rows_total, uint16_t* kc, uint16_t* vc, hipStream_t st) {
    if (rows_total <= 0 || s.B * s.L == 0) return hipSuccess;
    dim3 grid((unsigned)((rows_total + kRowsPerBlock - 1) / kRowsPerBlock), (unsigned)s.Hkv);
    if (s.D == 128)
        hipLaunchKernelGGL(compact_kernel<128>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, (long long)rows_total, kc, vc);
    else
        hipLaunchKernelGGL(compact_kernel<64>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, (long long)rows_total, kc, vc);
    return hipGetLastError();
}

}  // namespace tgvkv
