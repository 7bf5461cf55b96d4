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
// The destination is either a contiguous segment per (sequence, layer) or the
// pages that a block table names (paged cache); only the row addressing differs.
// Budgets differ across layers (TVB), so an optional unit order (the budget
// call's, longest first) sets which (sequence, layer) the i-th group of
// workgroups moves: the long units start first instead of forming the tail.
#include <algorithm>
#include <climits>

#include "tgvkv_device.h"
#include "tgvkv_rows.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kPasses = 8;

template <int D, class Rows>
__global__ __launch_bounds__(kThreads) void compact_kernel(Shape s, Rows rows, const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ budgets,
                                                           const int64_t* __restrict__ idx_off, int nsplit,
                                                           const int32_t* __restrict__ unit_order,
                                                           uint16_t* __restrict__ kc, uint16_t* __restrict__ vc) {
    extern __shared__ int lds_pages[];  // paged layout: the unit's page ids
    constexpr int CPR = D / 8;             // lanes per row
    constexpr int RPP = kThreads / CPR;    // rows per pass
    constexpr int ROWS = RPP * kPasses;    // rows per iteration
    // workgroup id = (unit rank * H_kv + KV head) * nsplit + split: a unit's heads and shares are adjacent
    int bid = blockIdx.x;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int kvh = bid % s.Hkv;
    const int bl = unit_order != nullptr ? min(max(unit_order[bid / s.Hkv], 0), s.B * s.L - 1) : bid / s.Hkv;
    const int bsz = budgets[bl];
    const long long ioff = idx_off[bl] + (s.head_mode == 0 ? 0 : (long long)kvh * bsz);
    const int per = (bsz + nsplit - 1) / nsplit;
    const int r_beg = min(split * per, bsz), r_end = min(r_beg + per, bsz);
    const int cc = threadIdx.x % CPR, rl = threadIdx.x / CPR;
    const size_t src0 = ((size_t)bl * s.Hkv + kvh) * (size_t)s.N * D + cc * 8;

    // positions come from tgvkv_select; clamp so a corrupt index can never read outside the slice
    int pos[kPasses];
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        const int r = r_beg + i * RPP + rl;
        pos[i] = r < r_end ? min(max(idx[ioff + r], 0), s.N - 1) : -1;
    }
    // destination rows (the paged layout's table is read while the positions are in flight)
    rows.init(s, bl, kvh, bsz, bsz, lds_pages);
    __syncthreads();
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
                const size_t dst = rows.row(r0 + i * RPP + rl) + cc * 8;
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

template <int D, class Rows>
hipError_t launch_compact_d(const Shape& s, const Rows& rows, size_t lds, const uint16_t* k, const uint16_t* v,
                            const int32_t* idx, const int32_t* budgets, const int64_t* idx_off, int64_t rows_total,
                            const int32_t* unit_order, uint16_t* kc, uint16_t* vc, hipStream_t st) {
    const int nsplit = compact_splits(s, rows_total);
    dim3 grid((unsigned)((long long)s.B * s.L * s.Hkv * nsplit));
    hipLaunchKernelGGL((compact_kernel<D, Rows>), grid, dim3(kThreads), lds, st, s, rows, k, v, idx, budgets, idx_off,
                       nsplit, unit_order, kc, vc);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_compact(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                          const int32_t* budgets, const int64_t* idx_off, const int64_t* seg_off, int32_t reserve,
                          int64_t rows_total, const int32_t* unit_order, uint16_t* kc, uint16_t* vc, hipStream_t st) {
    if (rows_total <= 0 || s.B * s.L == 0) return hipSuccess;
    if (s.D == 128)
        return launch_compact_d<128>(s, ContigRows<128>{seg_off, reserve, 0}, 0, k, v, idx, budgets, idx_off,
                                     rows_total, unit_order, kc, vc, st);
    return launch_compact_d<64>(s, ContigRows<64>{seg_off, reserve, 0}, 0, k, v, idx, budgets, idx_off, rows_total,
                                unit_order, kc, vc, st);
}

hipError_t launch_compact_paged(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                                const int32_t* budgets, const int64_t* idx_off, int64_t rows_total,
                                const int32_t* block_table, int32_t max_pages, int32_t page_shift, int64_t n_pages,
                                const int32_t* unit_order, uint16_t* k_pool, uint16_t* v_pool, hipStream_t st) {
    if (rows_total <= 0 || s.B * s.L == 0) return hipSuccess;
    const int np = (int)std::min<int64_t>(n_pages, INT32_MAX);
    const size_t lds = PagedRows<128>::lds_bytes(max_pages);
    if (s.D == 128)
        return launch_compact_d<128>(s, PagedRows<128>{block_table, max_pages, page_shift, np, 0, 0, nullptr}, lds, k,
                                     v, idx, budgets, idx_off, rows_total, unit_order, k_pool, v_pool, st);
    return launch_compact_d<64>(s, PagedRows<64>{block_table, max_pages, page_shift, np, 0, 0, nullptr}, lds, k, v,
                                idx, budgets, idx_off, rows_total, unit_order, k_pool, v_pool, st);
}

}  // namespace tgvkv
