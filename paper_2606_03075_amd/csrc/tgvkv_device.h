// Device-side primitives shared by the gfx950 kernels of libtgvkv.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tgvkv {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kNegInf = -__builtin_inff();

// Wave64 lane id.
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ float bf16_bits_to_float(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// 16 bytes of bf16 (8 elements) as an MFMA operand fragment.
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ u32x4 load16(const void* p) {
    return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ void store16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// 16-byte load with the non-temporal hint, for data streamed once per kernel (K/V
// rows).  On gfx950 it lifts a pure HBM read stream from about 5.9 to 6.8 TB/s.
__device__ __forceinline__ u32x4 load16_stream(const void* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ void store16_stream(void* p, u32x4 v) {
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// Waits here for the load that produced v.  Values loaded before a loop and read
// inside it otherwise get their wait inside the loop, where the compiler cannot
// tell them apart from loads issued by earlier iterations and waits for every
// outstanding load (vmcnt(0)), which would stall each iteration on its own
// prefetch.
template <typename T>
__device__ __forceinline__ void settle(const T& v) {
    asm volatile("" ::"v"(v));
}

// s_waitcnt vmcnt(0) (expcnt and lgkmcnt left at their maxima, gfx9 encoding):
// waits for every vector memory access of the wave, stores included.
__device__ __forceinline__ void wait_vmem_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// v_exp_f32: 2^x, exp2(-inf) = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// One 16x16x32 bf16 MFMA: C[m][n] += sum_k A[m][k] B[k][n].  Lane l holds A row
// l%16 and B column l%16, each with 8 consecutive k of the lane's quarter l/16;
// the accumulator element j of lane l is C[4*(l/16) + j][l%16].
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

// One 16x16x16 bf16 MFMA, same lane layout with 4 consecutive k per quarter: lane l
// holds A row l%16 and B column l%16 at k = 4*(l/16) .. +3; the accumulator element j
// of lane l is C[4*(l/16) + j][l%16].
__device__ __forceinline__ f32x4 mfma16x16x16(bf16x4 a, bf16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a), __builtin_bit_cast(s16x4, b), c,
                                                     0, 0, 0);
}

template <typename T>
__device__ __forceinline__ T shfl_xor(T v, int mask) {
    return __shfl_xor(v, mask, 64);
}

// Cross-lane sums on the VALU (no LDS crossbar traffic, unlike ds_bpermute).
// DPP row controls: quad_perm [1,0,3,2] (lane ^ 1), quad_perm [2,3,0,1] (lane ^ 2),
// row_half_mirror (7 - i within 8 lanes), row_mirror (15 - i within 16 lanes).
template <int CTRL>
__device__ __forceinline__ float dpp_read(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over each aligned group of W lanes (W = 8 or 16), left in every lane of the group.
// Each step adds the value of a partner lane that holds the same partial set, so the
// two lanes of a pair compute the same sum.
template <int W>
__device__ __forceinline__ float group_sum(float x) {
    static_assert(W == 8 || W == 16, "group width");
    x += dpp_read<0xB1>(x);   // lane ^ 1
    x += dpp_read<0x4E>(x);   // lane ^ 2
    x += dpp_read<0x141>(x);  // the other quad of the 8
    if (W == 16) x += dpp_read<0x140>(x);  // the other 8 of the 16
    return x;
}

// x + x of lane (l ^ 16), and x + x of lane (l ^ 32): v_permlane16_swap / v_permlane32_swap
// exchange rows between two registers; passing x twice yields both partners, in the same
// order in both lanes of a pair.
__device__ __forceinline__ float sum_xor16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// max(x, x of lane l ^ 16) and max(x, x of lane l ^ 32), by the same row swaps.
__device__ __forceinline__ float max_xor16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Combine two online-softmax partials (max m in log2 units, sum l, extra sum v
// that shares the normaliser).
__device__ __forceinline__ void merge_stats(float& m, float& l, float& v, float m2, float l2, float v2) {
    float mn = fmaxf(m, m2);
    if (mn == kNegInf) {
        m = kNegInf;
        l = 0.f;
        v = 0.f;
        return;
    }
    float s1 = fast_exp2(m - mn), s2 = fast_exp2(m2 - mn);
    l = l * s1 + l2 * s2;
    v = v * s1 + v2 * s2;
    m = mn;
}

// Map a float to an unsigned key with the same order (-0.0 treated as +0.0).
__device__ __forceinline__ uint32_t ordered_key(float f) {
    uint32_t b = __float_as_uint(f);
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

}  // namespace tgvkv
