// Page assignment for the paged compacted cache.
//
// In the paged layout each (sequence, layer) holds its b_l retained rows
// (Eq. (10)) and its decode_reserve appended rows in pages of P rows taken from a
// shared pool, so a serving loop can retire and admit sequences without
// re-packing the cache.  Segment i of a batch needs ceil((b_i + reserve) / P)
// pages; they are taken, in (sequence, layer) order, from the caller's list of
// free page ids.  One workgroup does the whole batch: a block-wide exclusive scan
// of the page counts, 1024 segments at a time, then a cooperative write of the
// table rows (unused entries -1) and of the number of pages consumed.
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__global__ __launch_bounds__(kThreads) void page_table_kernel(int units, const int32_t* __restrict__ budgets,
                                                              int reserve, int shift,
                                                              const int32_t* __restrict__ free_pages, int64_t n_free,
                                                              int32_t* __restrict__ table, int max_pages,
                                                              int64_t* __restrict__ used) {
    __shared__ int wsum[kWaves];
    __shared__ long long start[kThreads];
    __shared__ int count[kThreads];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    long long carry = 0;
    for (int c0 = 0; c0 < units; c0 += kThreads) {
        const int u = c0 + tid;
        // a segment needs at most max_pages pages (checked on the host; clamped here all the
        // same), so the sums within a chunk fit in int
        const long long need = ((long long)max(budgets[u < units ? u : 0], 0) + reserve + (1 << shift) - 1) >> shift;
        const int np = u < units ? (int)min(need, (long long)max_pages) : 0;
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
        const int nu = min(kThreads, units - c0);
        for (long long e = tid; e < (long long)nu * max_pages; e += kThreads) {
            const int ul = (int)(e / max_pages), j = (int)(e % max_pages);
            const long long p = start[ul] + j;
            table[(size_t)(c0 + ul) * max_pages + j] = (j < count[ul] && p < n_free) ? free_pages[p] : -1;
        }
        carry += chunk_total;
        __syncthreads();  // start/count/wsum are rewritten by the next chunk
    }
    if (tid == 0) *used = carry;
}

}  // namespace

hipError_t launch_page_table(const Shape& s, const int32_t* budgets, int32_t reserve, int32_t page_shift,
                             const int32_t* free_pages, int64_t n_free, int32_t* block_table, int32_t max_pages,
                             int64_t* pages_used, hipStream_t st) {
    hipLaunchKernelGGL(page_table_kernel, dim3(1), dim3(kThreads), 0, st, s.B * s.L, budgets, reserve, page_shift,
                       free_pages, n_free, block_table, max_pages, pages_used);
    return hipGetLastError();
}

}  // namespace tgvkv
