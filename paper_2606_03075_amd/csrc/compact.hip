// Gather-compaction of the retained K/V rows into the ragged per-layer cache.
//
// After eviction every layer keeps b_l tokens (Eq. (10)); the cache of Sec. 3.1
// holds only those rows, in ascending position, followed by decode_reserve free
// slots that decode (Eq. (3)-(4)) fills.  The work is a pure HBM stream: read
// and write each retained row once.  The grid runs over the flat list of
// retained rows (known on the host: B * B_tot per KV head), so it is sized by
// the bytes moved, not by the largest layer.  A row of head_dim bf16 is moved
// by head_dim/8 lanes with 16-byte accesses; each thread moves kPasses rows and
// issues every load (index, K, V) before any store.  The (sequence, layer) of
// the workgroup's first row is found once by binary search over the offsets;
// the other rows advance from it through an LDS copy of the following offsets.
#include "tgvkv_device.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kPasses = 4;
constexpr int kWindow = 128;  // offsets cached in LDS after the first row's block

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
    constexpr int ROWS = RPP * kPasses;    // rows per workgroup
    __shared__ long long win[kWindow + 1];  // per-group row offsets of blocks bl0 .. bl0 + kWindow
    __shared__ int sh_bl0;
    const int kvh = blockIdx.y;
    const long long g = s.ngroups;
    const int nbl = s.B * s.L;
    const int cc = threadIdx.x % CPR;
    const long long r0 = (long long)blockIdx.x * ROWS;

    if (threadIdx.x == 0) {
        int lo = 0, hi = nbl - 1;  // largest bl with idx_off[bl] / g <= r0
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (idx_off[mid] / g <= r0) lo = mid;
            else hi = mid - 1;
        }
        sh_bl0 = lo;
    }
    __syncthreads();
    const int bl0 = sh_bl0;
    for (int i = threadIdx.x; i <= kWindow; i += kThreads) {
        const int bl = min(bl0 + i, nbl);
        win[i] = idx_off[bl] / g;
    }
    __syncthreads();

    long long f[kPasses];
    int blk[kPasses], pos[kPasses];
    bool ok[kPasses];
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        f[i] = r0 + i * RPP + threadIdx.x / CPR;
        ok[i] = f[i] < rows_total;
        int w = 0;
        while (w < kWindow && bl0 + w + 1 < nbl && win[w + 1] <= f[i]) ++w;
        int bl = bl0 + w;
        if (w == kWindow) {  // beyond the cached window (many empty blocks): search
            int lo = bl, hi = nbl - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (idx_off[mid] / g <= f[i]) lo = mid;
                else hi = mid - 1;
            }
            bl = lo;
        }
        blk[i] = bl;
    }
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        pos[i] = 0;
        if (ok[i]) {
            const int bl = blk[i];
            const long long n = f[i] - idx_off[bl] / g;
            const int bsz = budgets[bl];
            // positions come from tgvkv_select; clamp so a corrupt index can never read outside the slice
            pos[i] = min(max(idx[idx_off[bl] + (s.head_mode == 0 ? 0 : (long long)kvh * bsz) + n], 0), s.N - 1);
        }
    }
    u32x4 kr[kPasses], vr[kPasses];
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        if (ok[i]) {
            const size_t src = (((size_t)blk[i] * s.Hkv + kvh) * (size_t)s.N + pos[i]) * D + cc * 8;
            kr[i] = load16_stream(k + src);
            vr[i] = load16_stream(v + src);
        }
    }
#pragma unroll
    for (int i = 0; i < kPasses; ++i) {
        if (ok[i]) {
            const int bl = blk[i];
            const long long n = f[i] - idx_off[bl] / g;
            const size_t dst = ((size_t)seg_off[bl] * s.Hkv + (size_t)kvh * (budgets[bl] + reserve) + n) * D + cc * 8;
            store16(kc + dst, kr[i]);
            store16(vc + dst, vr[i]);
        }
    }
}

}  // namespace

hipError_t launch_compact(const Shape& s, const uint16_t* k, const uint16_t* v, const int32_t* idx,
                          const int32_t* budgets, const int64_t* idx_off, const int64_t* seg_off, int32_t reserve,
                          int64_t rows_total, uint16_t* kc, uint16_t* vc, hipStream_t st) {
    if (rows_total <= 0 || s.B * s.L == 0) return hipSuccess;
    const int rows_per_block = (kThreads / (s.D / 8)) * kPasses;
    dim3 grid((unsigned)((rows_total + rows_per_block - 1) / rows_per_block), (unsigned)s.Hkv);
    if (s.D == 128)
        hipLaunchKernelGGL(compact_kernel<128>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, (long long)rows_total, kc, vc);
    else
        hipLaunchKernelGGL(compact_kernel<64>, grid, dim3(kThreads), 0, st, s, k, v, idx, budgets, idx_off, seg_off,
                           reserve, (long long)rows_total, kc, vc);
    return hipGetLastError();
}

}  // namespace tgvkv
