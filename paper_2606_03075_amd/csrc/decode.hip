// Single-query decode attention over the pruned, ragged per-layer cache.
//
// Each decode step appends the new token's key and value to every layer's cache
// (Sec. 3.1, Eq. (3)-(4)) and attends over the b_l retained plus the step + 1
// appended tokens.  This is a pure HBM stream of the cache (one read per step),
// so the kernel is organised for bytes in flight, not for math:
//   * one workgroup per (sequence, layer, KV head[, split]): the KV head's rows
//     are read once and serve all query heads that share it (GQA);
//   * a token row of head_dim bf16 is read by head_dim/8 lanes with 16-byte
//     non-temporal loads; each lane group works on blocks of 4 tokens from two
//     register buffers, issuing the next block's K and V loads before consuming
//     the current one (a trip count that is uniform over the workgroup and even,
//     with every load unconditional, so the compiler's waits stay per block);
//   * online softmax per lane group, merged across groups with wave shuffles and
//     across the 4 waves through LDS; when the (sequence, layer, KV head) count is
//     too small to fill the GPU the token range is split and a second kernel
//     combines the partial (max, sum, weighted sum) triples.
// The step's new token is read from the k_new / v_new inputs (the cache slot it
// is written to is not re-read in the same launch).  The cache is either one
// contiguous segment per (sequence, layer) or fixed-size pages found through a
// block table (staged in LDS); with per-sequence steps (continuous batching) a
// sequence whose step is outside [0, reserve) is skipped.  An optional unit order
// (from the budget call: longest segments first) sets which (sequence, layer) each
// workgroup serves, so the long segments do not all start last.
#include <algorithm>
#include <climits>

#include "tgvkv_device.h"
#include "tgvkv_rows.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ void unpack8(u32x4 r, float (&f)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(r[i] << 16);
        f[2 * i + 1] = __uint_as_float(r[i] & 0xFFFF0000u);
    }
}

template <int D, int GMAX, class Rows>
__global__ __launch_bounds__(kThreads) void decode_kernel(Shape s, Rows rows, uint16_t* __restrict__ kc,
                                                          uint16_t* __restrict__ vc,
                                                          const int32_t* __restrict__ budgets, int reserve, int step,
                                                          const int32_t* __restrict__ steps,
                                                          const uint16_t* __restrict__ q,
                                                          const uint16_t* __restrict__ k_new,
                                                          const uint16_t* __restrict__ v_new, float* __restrict__ out,
                                                          float* __restrict__ ws_part, int nsplit,
                                                          const int32_t* __restrict__ unit_order) {
    constexpr int LPR = D / 8;         // lanes per token row
    constexpr int GPW = 64 / LPR;      // lane groups per wave
    constexpr int NGRP = 4 * GPW;      // lane groups per workgroup
    constexpr int kUnroll = 4;  // tokens per lane group in each of the two register buffers
    __shared__ float wm[4][GMAX], wl[4][GMAX];
    __shared__ float wacc[4][GMAX][D];
    extern __shared__ int lds_pages[];  // paged layout: the unit's page ids

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int sub = lane % LPR;
    const int grp = wave * GPW + lane / LPR;
    int bid = blockIdx.x;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int kvh = bid % s.Hkv;
    // dispatch order: unit_order[i] is the (sequence, layer) the i-th group of workgroups serves
    // (clamped, so a wrong order can never address outside the batch)
    const int bl = unit_order != nullptr ? min(max(unit_order[bid / s.Hkv], 0), s.B * s.L - 1) : bid / s.Hkv;
    const int G = s.G;

    // continuous batching: each sequence at its own step, outside [0, reserve) = not decoding
    const int st = steps != nullptr ? steps[bl / s.L] : step;
    if (st < 0 || st >= reserve) return;  // uniform over the workgroup, before any barrier
    const int bsz = budgets[bl];
    const int len = bsz + st + 1;
    rows.init(s, bl, kvh, bsz, len, lds_pages);
    __syncthreads();
    const uint16_t* knew = k_new + ((size_t)bl * s.Hkv + kvh) * D;
    const uint16_t* vnew = v_new + ((size_t)bl * s.Hkv + kvh) * D;

    if (split == 0 && tid < LPR) {
        const size_t r = rows.row(bsz + st);
        store16(kc + r + tid * 8, load16(knew + tid * 8));
        store16(vc + r + tid * 8, load16(vnew + tid * 8));
    }

    float qv[GMAX][8];
#pragma unroll
    for (int h = 0; h < GMAX; ++h) {
        if (h < G) {
            unpack8(load16(q + ((size_t)bl * s.H + kvh * G + h) * D + sub * 8), qv[h]);
#pragma unroll
            for (int e = 0; e < 8; ++e) qv[h][e] *= s.scale2;
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) qv[h][e] = 0.f;
        }
    }

    const int per = (len + nsplit - 1) / nsplit;
    const int t0 = min(split * per, len), t1 = min(t0 + per, len);

    float m[GMAX], l[GMAX], acc[GMAX][8];
#pragma unroll
    for (int h = 0; h < GMAX; ++h) {
        m[h] = kNegInf;
        l[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    }

    constexpr int S = NGRP * kUnroll;
    // loads of one block of kUnroll tokens per lane group; rows past t1 (and the step's own
    // token) read the fresh k_new / v_new row, so every load is unconditional
    auto issue = [&](u32x4 (&kr)[kUnroll], u32x4 (&vr)[kUnroll], int n0) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int n = n0 + u * NGRP;
            const bool fresh = n >= len - 1 || n >= t1;
            const size_t r = fresh ? 0 : rows.row(n);
            kr[u] = load16_stream((fresh ? knew : kc + r) + sub * 8);
            vr[u] = load16_stream((fresh ? vnew : vc + r) + sub * 8);
        }
    };
    auto consume = [&](const u32x4 (&kr)[kUnroll], const u32x4 (&vr)[kUnroll], int n0) {
        bool ok[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) ok[u] = n0 + u * NGRP < t1;
#pragma unroll
        for (int h = 0; h < GMAX; ++h) {
            if (h >= G) continue;
            float z[kUnroll];
            float mx = kNegInf;
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                float kf[8];
                unpack8(kr[u], kf);
                float d = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) d += qv[h][e] * kf[e];
                d = group_sum<LPR>(d);
                z[u] = ok[u] ? d : kNegInf;
                mx = fmaxf(mx, z[u]);
            }
            if (mx > m[h]) {
                const float sc = fast_exp2(m[h] - mx);
                l[h] *= sc;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] *= sc;
                m[h] = mx;
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                if (!ok[u]) continue;
                const float p = fast_exp2(z[u] - m[h]);
                float vf[8];
                unpack8(vr[u], vf);
                l[h] += p;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] += p * vf[e];
            }
        }
    };
    // two register buffers: the next block's loads are in flight while this block is consumed;
    // the trip count is uniform over the workgroup and even (the extra half only masks)
    const int pairs = (t1 - t0 + 2 * S - 1) / (2 * S);
    u32x4 ka[kUnroll], va[kUnroll], kb[kUnroll], vb[kUnroll];
    int n0 = t0 + grp;
    issue(ka, va, n0);
    for (int pi = 0; pi < pairs; ++pi) {
        issue(kb, vb, n0 + S);
        consume(ka, va, n0);
        issue(ka, va, n0 + 2 * S);
        consume(kb, vb, n0 + S);
        n0 += 2 * S;
    }

    // merge the lane groups of the wave
#pragma unroll
    for (int h = 0; h < GMAX; ++h) {
        if (h >= G) continue;
#pragma unroll
        for (int off = LPR; off < 64; off <<= 1) {
            const float m2 = shfl_xor(m[h], off), l2 = shfl_xor(l[h], off);
            float a2[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) a2[e] = shfl_xor(acc[h][e], off);
            const float mn = fmaxf(m[h], m2);
            if (mn != kNegInf) {
                const float s1 = fast_exp2(m[h] - mn), s2 = fast_exp2(m2 - mn);
                l[h] = l[h] * s1 + l2 * s2;
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[h][e] = acc[h][e] * s1 + a2[e] * s2;
                m[h] = mn;
            }
        }
        if (lane < LPR) {
            if (lane == 0) {
                wm[wave][h] = m[h];
                wl[wave][h] = l[h];
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) wacc[wave][h][sub * 8 + e] = acc[h][e];
        }
    }
    __syncthreads();
    for (int x = tid; x < G * D; x += kThreads) {
        const int h = x / D, dd = x % D;
        float M = kNegInf;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w][h]);
        float num = 0.f, den = 0.f;
        if (M != kNegInf) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const float sc = fast_exp2(wm[w][h] - M);
                num += sc * wacc[w][h][dd];
                den += sc * wl[w][h];
            }
        }
        const size_t bh = (size_t)bl * s.H + kvh * G + h;
        if (nsplit == 1) {
            out[bh * D + dd] = num / den;
        } else {
            float* p = ws_part + (bh * nsplit + split) * (size_t)(D + 2);
            p[2 + dd] = num;
            if (dd == 0) {
                p[0] = M;
                p[1] = den;
            }
        }
    }
}

template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(Shape s, const float* __restrict__ ws_part, int nsplit,
                                                           float* __restrict__ out, const int32_t* __restrict__ steps,
                                                           int reserve) {
    const size_t bh = blockIdx.x;
    if (steps != nullptr) {
        const int st = steps[(int)(bh / ((size_t)s.L * s.H))];
        if (st < 0 || st >= reserve) return;  // this sequence is not decoding
    }
    const int dd = threadIdx.x;
    const float* p = ws_part + bh * nsplit * (size_t)(D + 2);
    float M = kNegInf;
    for (int i = 0; i < nsplit; ++i) M = fmaxf(M, p[i * (D + 2)]);
    float num = 0.f, den = 0.f;
    for (int i = 0; i < nsplit; ++i) {
        const float sc = fast_exp2(p[i * (D + 2)] - M);
        num += sc * p[i * (D + 2) + 2 + dd];
        den += sc * p[i * (D + 2) + 1];
    }
    out[bh * D + dd] = num / den;
}

template <int D, class Rows>
hipError_t launch_decode_d(const Shape& s, const Rows& rows, size_t lds_bytes, uint16_t* kc, uint16_t* vc,
                           const int32_t* budgets, int32_t reserve, int32_t step, const int32_t* steps,
                           const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new, float* out, float* ws_part,
                           int nsplit, const int32_t* unit_order, hipStream_t st) {
    dim3 grid((unsigned)((long long)s.B * s.L * s.Hkv * nsplit)), block(kThreads);
#define TGVKV_DECODE_LAUNCH(GM)                                                                                   \
    hipLaunchKernelGGL((decode_kernel<D, GM, Rows>), grid, block, lds_bytes, st, s, rows, kc, vc, budgets, reserve, \
                       step, steps, q, k_new, v_new, out, ws_part, nsplit, unit_order)
    if (s.G <= 1) TGVKV_DECODE_LAUNCH(1);
    else if (s.G <= 2) TGVKV_DECODE_LAUNCH(2);
    else if (s.G <= 4) TGVKV_DECODE_LAUNCH(4);
    else if (s.G <= 8) TGVKV_DECODE_LAUNCH(8);
    else TGVKV_DECODE_LAUNCH(16);
#undef TGVKV_DECODE_LAUNCH
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || nsplit == 1) return e;
    hipLaunchKernelGGL(decode_combine_kernel<D>, dim3((unsigned)((long long)s.B * s.L * s.H)), dim3(D), 0, st, s,
                       ws_part, nsplit, out, steps, reserve);
    return hipGetLastError();
}

}  // namespace

int decode_splits(const Shape& s) {
    const long long units = (long long)s.B * s.L * s.Hkv;
    if (units <= 0) return 1;
    long long n = 2048 / units;
    if (n < 1) n = 1;
    if (n > 8) n = 8;
    return (int)n;
}

hipError_t launch_decode(const Shape& s, uint16_t* kc, uint16_t* vc, const int32_t* budgets, const int64_t* seg_off,
                         int32_t reserve, int32_t step, const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                         float* out, float* ws_part, const int32_t* unit_order, hipStream_t st) {
    if ((long long)s.B * s.L == 0) return hipSuccess;
    const int nsplit = decode_splits(s);
    if (s.D == 128) {
        ContigRows<128> rows{seg_off, reserve, 0};
        return launch_decode_d<128>(s, rows, 0, kc, vc, budgets, reserve, step, nullptr, q, k_new, v_new, out,
                                    ws_part, nsplit, unit_order, st);
    }
    ContigRows<64> rows{seg_off, reserve, 0};
    return launch_decode_d<64>(s, rows, 0, kc, vc, budgets, reserve, step, nullptr, q, k_new, v_new, out, ws_part,
                               nsplit, unit_order, st);
}

hipError_t launch_decode_paged(const Shape& s, uint16_t* k_pool, uint16_t* v_pool, int64_t n_pages,
                               const int32_t* block_table, int32_t max_pages, int32_t page_shift,
                               const int32_t* budgets, int32_t reserve, const int32_t* steps, const uint16_t* q,
                               const uint16_t* k_new, const uint16_t* v_new, float* out, float* ws_part,
                               const int32_t* unit_order, hipStream_t st) {
    if ((long long)s.B * s.L == 0) return hipSuccess;
    const int nsplit = decode_splits(s);
    const size_t lds = PagedRows<128>::lds_bytes(max_pages);
    const int np = (int)std::min<int64_t>(n_pages, INT32_MAX);
    if (s.D == 128) {
        PagedRows<128> rows{block_table, max_pages, page_shift, np, 0, 0, nullptr};
        return launch_decode_d<128>(s, rows, lds, k_pool, v_pool, budgets, reserve, 0, steps, q, k_new, v_new, out,
                                    ws_part, nsplit, unit_order, st);
    }
    PagedRows<64> rows{block_table, max_pages, page_shift, np, 0, 0, nullptr};
    return launch_decode_d<64>(s, rows, lds, k_pool, v_pool, budgets, reserve, 0, steps, q, k_new, v_new, out,
                               ws_part, nsplit, unit_order, st);
}

}  // namespace tgvkv
