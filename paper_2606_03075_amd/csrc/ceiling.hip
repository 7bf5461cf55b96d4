// Measurement kernels: the achievable HBM and matrix-core rates of the chip the
// eviction pass runs on, so that each kernel's rate can be set against what the
// hardware delivers in the same process, next to the vendor peaks.  They compute
// nothing of the method.
//
//   ceiling_read   streams a buffer once with the same 16-byte non-temporal loads
//                  the key sweeps, compaction and decode use (8 in flight per lane,
//                  one contiguous chunk per workgroup);
//   ceiling_copy   the same stream, each 16 bytes also stored to a second buffer;
//   ceiling_mfma   back-to-back v_mfma_f32_16x16x32_bf16 on 8 independent
//                  accumulators per wave, 2 waves per SIMD on every SIMD.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "tgvkv_ceiling.h"
#include "tgvkv_device.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
constexpr int kInFlight = 8;                                   // 16-byte loads in flight per lane
constexpr long long kStepBytes = 16LL * kThreads * kInFlight;  // one round of a workgroup: 32 KiB
constexpr long long kChunkBytes = 4 * kStepBytes;               // contiguous bytes per workgroup: 128 KiB

// One round: every lane's 8 loads are issued before any is used.  GUARD: the round
// reaches past `bytes` (only the buffer's last round), so each vector is checked.
template <bool COPY, bool GUARD>
__device__ __forceinline__ void stream_round(const char* src, char* dst, long long base, long long bytes,
                                             u32x4& acc) {
    u32x4 r[kInFlight];
#pragma unroll
    for (int i = 0; i < kInFlight; ++i) {
        const long long off = base + ((long long)i * kThreads + threadIdx.x) * 16;
        if (!GUARD || off < bytes) r[i] = load16_stream(src + off);
        else r[i] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int i = 0; i < kInFlight; ++i) {
        const long long off = base + ((long long)i * kThreads + threadIdx.x) * 16;
        if (COPY) {
            if (!GUARD || off < bytes) store16_stream(dst + off, r[i]);
        } else {
            acc ^= r[i];
        }
    }
}

template <bool COPY>
__global__ __launch_bounds__(kThreads) void ceiling_stream_kernel(const char* __restrict__ src,
                                                                  char* __restrict__ dst, long long bytes,
                                                                  unsigned* __restrict__ sink) {
    const long long c0 = (long long)blockIdx.x * kChunkBytes;
    const long long c1 = std::min(c0 + kChunkBytes, bytes);
    u32x4 acc = {0u, 0u, 0u, 0u};
    long long base = c0;
    for (; base + kStepBytes <= c1; base += kStepBytes) stream_round<COPY, false>(src, dst, base, bytes, acc);
    if (base < c1) stream_round<COPY, true>(src, dst, base, bytes, acc);
    if (!COPY) {
        // keeps the loads live; the word is written only for one pattern of the data
        const unsigned x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
        if (x == 0x9E3779B9u) sink[0] = x;
    }
}

constexpr int kChains = 8;  // independent accumulators per wave

__global__ __launch_bounds__(kThreads) void ceiling_mfma_kernel(int iters, float seed, float* __restrict__ out) {
    // operands depend on the lane and on a run-time seed, so nothing folds
    const float a0 = seed + (float)(threadIdx.x & 63) * 0.001f;
    bf16x8 a, b;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        a[j] = (__bf16)(a0 + 0.01f * j);
        b[j] = (__bf16)(a0 - 0.02f * j);
    }
    f32x4 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) acc[c] = mfma16x16x32(a, b, acc[c]);
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c) s += (acc[c][0] + acc[c][1]) + (acc[c][2] + acc[c][3]);
    out[(size_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

}  // namespace
}  // namespace tgvkv

extern "C" {

long long tgvkv_ceiling_mfma_flops(int32_t workgroups, int32_t iters) {
    if (workgroups < 1 || iters < 1) return 0;
    return (long long)workgroups * (tgvkv::kThreads / 64) * iters * tgvkv::kChains * (2LL * 16 * 16 * 32);
}

int32_t tgvkv_ceiling_read(const void* src, int64_t bytes, uint32_t* sink, hipStream_t stream) {
    if (src == nullptr || sink == nullptr || bytes <= 0 || (bytes & 15) != 0 ||
        (reinterpret_cast<uintptr_t>(src) & 15u) != 0)
        return -1;
    const long long blocks = (bytes + tgvkv::kChunkBytes - 1) / tgvkv::kChunkBytes;
    if (blocks > 0x7FFFFFFFLL) return -2;
    hipLaunchKernelGGL(tgvkv::ceiling_stream_kernel<false>, dim3((unsigned)blocks), dim3(tgvkv::kThreads), 0, stream,
                       static_cast<const char*>(src), nullptr, (long long)bytes, sink);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int32_t tgvkv_ceiling_copy(const void* src, void* dst, int64_t bytes, hipStream_t stream) {
    if (src == nullptr || dst == nullptr || bytes <= 0 || (bytes & 15) != 0 ||
        (reinterpret_cast<uintptr_t>(src) & 15u) != 0 || (reinterpret_cast<uintptr_t>(dst) & 15u) != 0)
        return -1;
    const long long blocks = (bytes + tgvkv::kChunkBytes - 1) / tgvkv::kChunkBytes;
    if (blocks > 0x7FFFFFFFLL) return -2;
    hipLaunchKernelGGL(tgvkv::ceiling_stream_kernel<true>, dim3((unsigned)blocks), dim3(tgvkv::kThreads), 0, stream,
                       static_cast<const char*>(src), static_cast<char*>(dst), (long long)bytes, nullptr);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

int32_t tgvkv_ceiling_mfma(int32_t workgroups, int32_t iters, float* out, hipStream_t stream) {
    if (out == nullptr || workgroups < 1 || iters < 1) return -1;
    hipLaunchKernelGGL(tgvkv::ceiling_mfma_kernel, dim3((unsigned)workgroups), dim3(tgvkv::kThreads), 0, stream,
                       iters, 0.5f, out);
    return hipGetLastError() == hipSuccess ? 0 : -5;
}

}  // extern "C"
