// Gather-compaction of the retained K/V rows into the ragged per-layer cache.
//
// After eviction every layer keeps b_l tokens (Eq. (10)); the cache of Sec. 3.1
// holds only those rows, in ascending position, followed by decode_reserve free
// slots that decode (Eq. (3)-(4)) fills.  The work is a pure HBM stream: read
// and write each retained row once.  One workgroup moves the rows of one
// (sequence, layer, KV head), or a contiguous share of them when there are too
// few such units to fill the GPU, so its metadata is three independent loads and
// no search.  A row of head_dim bf16 is moved by head_dim/8 lanes with 16-byte
// accesses (non-temporal loads); each thread keeps kPasses rows in flight, and
// the positions of the next rows are fetched while the current ones are moved.
#include <algorithm>

#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kPasses = 8;

template <int D>
__global__ __launch_bounds__(kThreads) void compact_kernel(Shape s, const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ budgets,
                                                           const int64_t* __restrict__ idx_off,
                                                           const int64_t* __restrict__ seg_off, int reserve,
                                                           int nsplit, uint16_t* __restrict__ kc,
                                                           uint16_t* __restrict__ vc) {
    constexpr int CPR = D / 8;             // lanes per row
    constexpr int RPP = kThreads / CPR;    // rows per pass
    constexpr int ROWS = RPP * kPasses;    // rows per iteration
    const int kvh = blockIdx.y;
    const int split = blockIdx.x % nsplit;
    const int bl = blockIdx.x / nsplit;
    const int bsz = budgets[bl];
    const long long ioff = idx_off[bl] + (s.head_mode == 0 ? 0 : (long long)kvh * bsz);
    const long long soff = seg_off[bl];
    const int per = (bsz + nsplit - 1) / nsplit;
    const int r_beg = min(split * per, bsz), r_end = min(r_beg + per, bsz);
    const int cc = threadIdx.x % CPR, rl = threadIdx.x / CPR;
    const size_t src0 = ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D + cc * 8;
    const size_t dst0 = ((size_t)soff * s.Hkv + (size_t)kvh * (bsz + reserve)) * D + cc * 8;

    // positions come from tgvkv_select; clamp so a corrupt index can never read outside the slice
    int pos[kPasses];
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        const int r = r_beg + i * RPP + rl;
        pos[i] = r < r_end ? min(max(idx[ioff + r], 0), s.N - 1) : -1;
    }
    for (int r0 = r_beg; r0 < r_end; r0 += ROWS) {
        u32x4 kr[kPasses], vr[kPasses];
#pragma unroll
        for (int i = 0; i < kPasses; ++i) {
            if (pos[i] >= 0) {
                kr[i] = load16_stream(k + src0 + (size_t)pos[i] * D);
                vr[i] = load16_stream(v + src0 + (size_t)pos[i] * D);
            }
        }
        int cur[kPasses];
#pragma unroll
        for (int i = 0; i < kPasses; ++i) {
            cur[i] = pos[i];
            const int r = r0 + ROWS + i * RPP + rl;
            pos[i] = r < r_end ? min(max(idx[ioff + r], 0), s.N - 1) : -1;
        }
#pragma unroll
        for (int i = 0; i < kPasses; ++i) {
            if (cur[i] >= 0) {
                const size_t dst = dst0 + (size_t)(r0 + i * RPP + rl) * D;
                store16(kc + dst, kr[i]);
                store16(vc + dst, vr[i]);
            }
        }
    }
}

// Workgroups per (sequence, layer, KV head): enough units to fill the GPU, but
// not fewer than about 64 rows per workgroup on average.
int compact_splits(const Shape& s, int64_t rows_total) {
    const long long units = (long long)s.B * s.L * s.Hkv;
    if (units <= 0 || rows_total <= 0) return 1;
    const long long avg_rows = rows_total / ((long long)s.B * s.L);  // retained rows per (sequence, layer)
    long long n = std::min<long long>(2048 / units, avg_rows / 64);
    return (int)std::max<long long>(1, std::min<long long>(n, 16));
}

}  // namespace

hipError_t launch_compact(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                          const int32_t* budgets, const int64_t* idx_off, const int64_t* seg_off, int32_t reserve,
                          int64_t rows_total, uint16_t* kc, uint16_t* vc, hipStream_t st) {
    if (rows_total <= 0 || s.B * s.L == 0) return hipSuccess;
    const int nsplit = compact_splits(s, rows_total);
    dim3 grid((unsigned)((long long)s.B * s.L * nsplit), (unsigned)s.Hkv);
    if (s.D == 128)
        hipLaunchKernelGGL(compact_kernel<128>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, nsplit, kc, vc);
    else
        hipLaunchKernelGGL(compact_kernel<64>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, nsplit, kc, vc);
    return hipGetLastError();
}

}  // namespace tgvkv
