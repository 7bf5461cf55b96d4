// Page assignment for the paged compacted cache.
//
// In the paged layout each (sequence, layer) holds its b_l retained rows
// (Eq. (10)) and its decode_reserve appended rows in pages of P rows taken from a
// shared pool, so a serving loop can retire and admit sequences without
// re-packing the cache.  Segment i of a batch needs ceil((b_i + reserve) / P)
// pages; they are taken, in (sequence, layer) order, from the caller's list of
// free page ids.  Workgroup w owns a contiguous range of segments: it sums the
// page counts of all segments before its range (a block reduction over at most
// a few thousand L2-resident budgets), scans its own range, 1024 segments at a
// time, and writes those table rows (unused entries -1); the last workgroup also
// writes the number of pages consumed.  With the range sizes below the redundant
// reductions stay far below the table writes for any batch.
#include <algorithm>

#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxGroups = 256;
constexpr int kMinRowsPerGroup = 8;

__device__ __forceinline__ int pages_of(const int32_t* budgets, int u, int reserve, int shift, int max_pages) {
    const long long need = ((long long)max(budgets[u], 0) + reserve + (1 << shift) - 1) >> shift;
    return (int)min(need, (long long)max_pages);
}

__global__ __launch_bounds__(kThreads) void page_table_kernel(int units, int per_group,
                                                              const int32_t* __restrict__ budgets, int reserve,
                                                              int shift, const int32_t* __restrict__ free_pages,
                                                              int64_t n_free, int32_t* __restrict__ table,
                                                              int max_pages, int64_t* __restrict__ used) {
    __shared__ long long red[kWaves];
    __shared__ int wsum[kWaves];
    __shared__ long long start[kThreads];
    __shared__ int count[kThreads];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u_beg = blockIdx.x * per_group;
    const int u_end = min(u_beg + per_group, units);

    // pages of every segment before this group's range
    long long before = 0;
    for (int u = tid; u < u_beg; u += kThreads) before += pages_of(budgets, u, reserve, shift, max_pages);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) before += __shfl_xor(before, off, 64);
    if (lane == 0) red[wave] = before;
    __syncthreads();
    long long carry = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) carry += red[w];

    for (int c0 = u_beg; c0 < u_end; c0 += kThreads) {
        const int u = c0 + tid;
        // a segment needs at most max_pages pages (checked on the host; clamped here all the
        // same), so the sums within a chunk fit in int
        const int np = u < u_end ? pages_of(budgets, u, reserve, shift, max_pages) : 0;
        int x = np;  // inclusive scan within the wave
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (lane == 63) wsum[wave] = x;
        __syncthreads();
        if (wave == 0) {
            int w = lane < kWaves ? wsum[lane] : 0;
#pragma unroll
            for (int off = 1; off < kWaves; off <<= 1) {
                const int y = __shfl_up(w, off, 64);
                if (lane >= off) w += y;
            }
            if (lane < kWaves) wsum[lane] = w;
        }
        __syncthreads();
        start[tid] = carry + (x - np) + (wave > 0 ? wsum[wave - 1] : 0);
        count[tid] = np;
        const int chunk_total = wsum[kWaves - 1];
        __syncthreads();
        const int nu = min(kThreads, u_end - c0);
        const int n_entries = nu * max_pages;  // <= 1024 * 4096
#pragma unroll 4
        for (int e = tid; e < n_entries; e += kThreads) {
            const int ul = e / max_pages, j = e - ul * max_pages;
            const long long p = start[ul] + j;
            table[(size_t)(c0 + ul) * max_pages + j] = (j < count[ul] && p < n_free) ? free_pages[p] : -1;
        }
        carry += chunk_total;
        __syncthreads();  // start/count/wsum are rewritten by the next chunk
    }
    if (blockIdx.x == gridDim.x - 1 && tid == 0) *used = carry;
}

}  // namespace

hipError_t launch_page_table(const Shape& s, const int32_t* budgets, int32_t reserve, int32_t page_shift,
                             const int32_t* free_pages, int64_t n_free, int32_t* block_table, int32_t max_pages,
                             int64_t* pages_used, hipStream_t st) {
    const int units = s.B * s.L;
    int groups = std::min(kMaxGroups, std::max(1, units / kMinRowsPerGroup));
    const int per_group = (units + groups - 1) / groups;
    groups = (units + per_group - 1) / per_group;  // every group non-empty; the last one writes the count
    hipLaunchKernelGGL(page_table_kernel, dim3(groups), dim3(kThreads), 0, st, units, per_group, budgets, reserve,
                       page_shift, free_pages, n_free, block_table, max_pages, pages_used);
    return hipGetLastError();
}

}  // namespace tgvkv
