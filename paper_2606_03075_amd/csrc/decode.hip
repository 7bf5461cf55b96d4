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
#include <mutex>

#include "tgvkv_device.h"
#include "tgvkv_rows.h"
#include "tgvkv_shape.h"

namespace tgvkv {
namespace {

constexpr int kThreads = 256;
// query heads per KV head from which decode runs on the matrix cores
constexpr int kMfmaMinGroup = 3;

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

    float qv[GMAX][8];  // the scaled query heads, set once the first block's loads are in flight

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
    {
        // the query's latency overlaps the first block's: wait for it (and only it) here
        u32x4 qr[GMAX];
#pragma unroll
        for (int h = 0; h < GMAX; ++h) {
            const u32x4 z = {0u, 0u, 0u, 0u};
            qr[h] = h < G ? load16(q + ((size_t)bl * s.H + kvh * G + h) * D + sub * 8) : z;
            settle(qr[h]);
        }
#pragma unroll
        for (int h = 0; h < GMAX; ++h) {
            unpack8(qr[h], qv[h]);
#pragma unroll
            for (int e = 0; e < 8; ++e) qv[h][e] *= s.scale2;
        }
    }
    for (int pi = 0; pi < pairs; ++pi) {
        issue(kb, vb, n0 + S);
        consume(ka, va, n0);
        issue(ka, va, n0 + 2 * S);
        consume(kb, vb, n0 + S);
        n0 += 2 * S;
    }
    // the step's token into its cache slot (this launch reads it from k_new / v_new)
    if (split == 0 && tid < LPR) {
        const size_t r = rows.row(bsz + st);
        store16(kc + r + tid * 8, load16(knew + tid * 8));
        store16(vc + r + tid * 8, load16(vnew + tid * 8));
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

// Grouped-query decode on the matrix cores, for several query heads per KV head.
// The VALU kernel above spends each lane group's instructions on one token and
// one head at a time, replicated over the 16 lanes of a row: with G heads its
// work per cached byte grows G-fold and it stops being bound by HBM.  Here a
// 16-token block and all G heads (padded to 16) are one MFMA tile:
//   * the block's K and V rows are loaded whole (16 lanes per 256-byte row) and
//     staged in a per-wave LDS area; read straight into MFMA layout, each quarter
//     wave of a K load would touch 16 rows, 8x the L1 lookups of a row-wise load;
//   * S^T = K Q^T on v_mfma_f32_16x16x32_bf16, keys on the M side: lane l then
//     holds the scores of head l%16 for tokens 4*(l/16) .. +3;
//   * the block max of each head is taken over the lane's 4 values and across
//     the lane quarters, so the 16 lanes of a head share one running max; the
//     output rows are rescaled only when some head's max grew;
//   * O += P V on v_mfma_f32_16x16x16_bf16: the A operand P[head][token] is
//     exactly the lane's 4 probabilities, split into a bf16 high part and a bf16
//     remainder (two MFMAs, about 16 significant bits); the B operand needs
//     V[token][dim] with tokens along k, which the V stage gives: rows padded to
//     272 bytes, so the four lane quarters read rows 4 apart from disjoint banks,
//     and each lane reads one dword (two dims) per token, feeding two 16-dim
//     output blocks;
//   * the 4 waves of a workgroup take alternate 16-token blocks of the split.  One
//     register buffer per wave: as soon as a block's rows are in LDS the next
//     block's loads are issued (unconditional, clamped to the fresh row past the
//     end), so they stream in during the block's softmax and P V.  That keeps the
//     kernel at 122 VGPRs, 4 waves per SIMD; a second buffer cost a wave per SIMD
//     and measured slower.  The waves then merge through LDS as the VALU kernel does.
template <int D, int GMAX, class Rows>
__global__ __launch_bounds__(kThreads) void decode_mfma_kernel(Shape s, Rows rows, uint16_t* __restrict__ kc,
                                                               uint16_t* __restrict__ vc,
                                                               const int32_t* __restrict__ budgets, int reserve,
                                                               int step, const int32_t* __restrict__ steps,
                                                               const uint16_t* __restrict__ q,
                                                               const uint16_t* __restrict__ k_new,
                                                               const uint16_t* __restrict__ v_new,
                                                               float* __restrict__ out, float* __restrict__ ws_part,
                                                               int nsplit, const int32_t* __restrict__ unit_order) {
    constexpr int KSTEPS = D / 32;          // k-steps of S^T = K Q^T over the head dim
    constexpr int NB2 = D / 32;             // pairs of 16-dim output blocks
    constexpr int VROWB = D * 2 + 16;       // padded LDS row of the V stage, bytes
    constexpr int VCH = D / 8;              // 16-byte chunks per row
    constexpr int VLOADS = 16 * VCH / 64;   // 16-byte V loads per lane per block
    constexpr int STAGE = 4 * 16 * VROWB * 2;  // per wave: the block's V rows, then its K rows
    constexpr int MERGE = 4 * GMAX * (D + 2) * (int)sizeof(float);
    __shared__ __align__(16) char smem[STAGE > MERGE ? STAGE : MERGE];
    extern __shared__ int lds_pages[];  // paged layout: the unit's page ids

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = lane & 15, qq = lane >> 4;
    int bid = blockIdx.x;
    const int split = bid % nsplit;
    bid /= nsplit;
    const int kvh = bid % s.Hkv;
    const int bl = unit_order != nullptr ? min(max(unit_order[bid / s.Hkv], 0), s.B * s.L - 1) : bid / s.Hkv;
    const int G = s.G;

    const int st = steps != nullptr ? steps[bl / s.L] : step;
    if (st < 0 || st >= reserve) return;  // uniform over the workgroup, before any barrier
    const int bsz = budgets[bl];
    const int len = bsz + st + 1;
    rows.init(s, bl, kvh, bsz, len, lds_pages);
    __syncthreads();
    const uint16_t* knew = k_new + ((size_t)bl * s.Hkv + kvh) * D;
    const uint16_t* vnew = v_new + ((size_t)bl * s.Hkv + kvh) * D;

    // B operand of S^T: query head c (zero for the padding heads), 8 dims of the lane's quarter per k-step
    bf16x8 qf[KSTEPS];
    {
        const bool hv = c < G;
        const uint16_t* qp = q + ((size_t)bl * s.H + kvh * G + (hv ? c : 0)) * D + qq * 8;
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) {
            u32x4 z = {0u, 0u, 0u, 0u};
            qf[ks] = as_bf16x8(hv ? load16(qp + ks * 32) : z);
        }
    }

    const int per = (len + nsplit - 1) / nsplit;
    const int t0 = min(split * per, len), t1 = min(t0 + per, len);
    const int nblk = (t1 - t0 + 15) >> 4;
    const int wblk = (nblk + 3) >> 2;  // blocks per wave, uniform over the workgroup

    float m_run = kNegInf, l_run = 0.f;
    f32x4 o[2 * NB2];
#pragma unroll
    for (int nb = 0; nb < 2 * NB2; ++nb) o[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    char* vst = smem + wave * 16 * VROWB;
    char* kst = smem + (4 + wave) * 16 * VROWB;

    // loads of the block at token n0: its K and V rows, 16 lanes per row; rows past t1
    // (and the step's own token) read the fresh k_new / v_new row, so every load is issued
    auto settle_qf = [&]() {
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks) settle(qf[ks]);
    };
    auto issue = [&](u32x4 (&kr)[VLOADS], u32x4 (&vr)[VLOADS], int n0) {
#pragma unroll
        for (int i = 0; i < VLOADS; ++i) {
            const int ch = i * 64 + lane;
            const int n = n0 + ch / VCH;
            const bool fresh = n >= len - 1 || n >= t1;
            const size_t r = fresh ? 0 : rows.row(n);
            kr[i] = load16_stream((fresh ? knew : kc + r) + (ch % VCH) * 8);
            vr[i] = load16_stream((fresh ? vnew : vc + r) + (ch % VCH) * 8);
        }
    };
    // rows into the wave's LDS stages, then S^T from the staged K (lane: row c, its k-step columns)
    auto stage = [&](const u32x4 (&kr)[VLOADS], const u32x4 (&vr)[VLOADS]) {
        // the stages are free: this wave's reads of the previous block were issued before
        asm volatile("" ::: "memory");
#pragma unroll
        for (int i = 0; i < VLOADS; ++i) {
            const int ch = i * 64 + lane;
            store16(vst + (ch / VCH) * VROWB + (ch % VCH) * 16, vr[i]);
            store16(kst + (ch / VCH) * VROWB + (ch % VCH) * 16, kr[i]);
        }
        asm volatile("" ::: "memory");
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KSTEPS; ++ks)
            acc = mfma16x16x32(as_bf16x8(*reinterpret_cast<const u32x4*>(kst + c * VROWB + (ks * 32 + qq * 8) * 2)),
                               qf[ks], acc);
        return acc;
    };
    auto consume = [&](f32x4 acc, int n0) {
        float z[4], mb = kNegInf;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            z[j] = n0 + 4 * qq + j < t1 ? acc[j] * s.scale2 : kNegInf;
            mb = fmaxf(mb, z[j]);
        }
        mb = max_xor32(max_xor16(mb));
        const float m_new = fmaxf(m_run, mb);
        if (__builtin_amdgcn_ballot_w64(m_new > m_run) != 0) {  // some head's max grew (uniform branch)
            const float sc = m_new == kNegInf ? 1.f : fast_exp2(m_run - m_new);
            l_run *= sc;
            float scr[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) scr[j] = __shfl(sc, 4 * qq + j, 64);  // output row 4*qq + j's head
#pragma unroll
            for (int nb = 0; nb < 2 * NB2; ++nb)
#pragma unroll
                for (int j = 0; j < 4; ++j) o[nb][j] *= scr[j];
            m_run = m_new;
        }
        const float mu = m_run == kNegInf ? 0.f : m_run;
        bf16x4 ph, pl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float p = fast_exp2(z[j] - mu);
            l_run += p;
            ph[j] = (__bf16)p;
            pl[j] = (__bf16)(p - (float)ph[j]);
        }
        asm volatile("" ::: "memory");
        // B operand: tokens 4*qq .. +3 of dims 32*nb2 + 2c (even block) and + 1 (odd block)
#pragma unroll
        for (int nb2 = 0; nb2 < NB2; ++nb2) {
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = *reinterpret_cast<const uint32_t*>(vst + (4 * qq + i) * VROWB + (32 * nb2 + 2 * c) * 2);
            typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
            const u32x2 ev = {(w[0] & 0xFFFFu) | (w[1] << 16), (w[2] & 0xFFFFu) | (w[3] << 16)};
            const u32x2 od = {(w[0] >> 16) | (w[1] & 0xFFFF0000u), (w[2] >> 16) | (w[3] & 0xFFFF0000u)};
            const bf16x4 be = __builtin_bit_cast(bf16x4, ev), bo = __builtin_bit_cast(bf16x4, od);
            o[2 * nb2] = mfma16x16x16(ph, be, o[2 * nb2]);
            o[2 * nb2] = mfma16x16x16(pl, be, o[2 * nb2]);
            o[2 * nb2 + 1] = mfma16x16x16(ph, bo, o[2 * nb2 + 1]);
            o[2 * nb2 + 1] = mfma16x16x16(pl, bo, o[2 * nb2 + 1]);
        }
    };

    u32x4 ka[VLOADS], va[VLOADS];
    int n0 = t0 + 16 * wave;  // this wave's blocks: wave, wave + 4, ... of the split
    issue(ka, va, n0);
    settle_qf();
    for (int bi = 0; bi < wblk; ++bi) {
        const f32x4 acc = stage(ka, va);
        issue(ka, va, n0 + 64);
        consume(acc, n0);
        n0 += 64;
    }

    // the step's token into its cache slot (this launch reads it from k_new / v_new)
    if (split == 0 && tid < VCH) {
        const size_t r = rows.row(bsz + st);
        store16(kc + r + tid * 8, load16(knew + tid * 8));
        store16(vc + r + tid * 8, load16(vnew + tid * 8));
    }
    // the four lane quarters summed different tokens of each head
    l_run = sum_xor32(sum_xor16(l_run));
    __syncthreads();  // every wave is done with its stage: the merge reuses it
    float* wm = reinterpret_cast<float*>(smem);  // [4][GMAX]
    float* wl = wm + 4 * GMAX;                   // [4][GMAX]
    float* wacc = wl + 4 * GMAX;                 // [4][GMAX][D]
    if (qq == 0 && c < G) {
        wm[wave * GMAX + c] = m_run;
        wl[wave * GMAX + c] = l_run;
    }
#pragma unroll
    for (int nb2 = 0; nb2 < NB2; ++nb2)
#pragma unroll
        for (int e = 0; e < 2; ++e)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int h = 4 * qq + j;
                if (h < G) wacc[(wave * GMAX + h) * D + 32 * nb2 + 2 * c + e] = o[2 * nb2 + e][j];
            }
    __syncthreads();
    for (int x = tid; x < G * D; x += kThreads) {
        const int h = x / D, dd = x % D;
        float M = kNegInf;
#pragma unroll
        for (int w = 0; w < 4; ++w) M = fmaxf(M, wm[w * GMAX + h]);
        float num = 0.f, den = 0.f;
        if (M != kNegInf) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const float sc = fast_exp2(wm[w * GMAX + h] - M);
                num += sc * wacc[(w * GMAX + h) * D + dd];
                den += sc * wl[w * GMAX + h];
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
#define TGVKV_DECODE_MFMA_LAUNCH(GM)                                                                           \
    hipLaunchKernelGGL((decode_mfma_kernel<D, GM, Rows>), grid, block, lds_bytes, st, s, rows, kc, vc, budgets,     \
                       reserve, step, steps, q, k_new, v_new, out, ws_part, nsplit, unit_order)
    if (s.G >= kMfmaMinGroup) {
        if (s.G <= 4) TGVKV_DECODE_MFMA_LAUNCH(4);
        else if (s.G <= 8) TGVKV_DECODE_MFMA_LAUNCH(8);
        else TGVKV_DECODE_MFMA_LAUNCH(16);
    } else if (s.G <= 1) TGVKV_DECODE_LAUNCH(1);
    else if (s.G <= 2) TGVKV_DECODE_LAUNCH(2);
    else if (s.G <= 4) TGVKV_DECODE_LAUNCH(4);
    else if (s.G <= 8) TGVKV_DECODE_LAUNCH(8);
    else TGVKV_DECODE_LAUNCH(16);
#undef TGVKV_DECODE_LAUNCH
#undef TGVKV_DECODE_MFMA_LAUNCH
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || nsplit == 1) return e;
    hipLaunchKernelGGL(decode_combine_kernel<D>, dim3((unsigned)((long long)s.B * s.L * s.H)), dim3(D), 0, st, s,
                       ws_part, nsplit, out, steps, reserve);
    return hipGetLastError();
}

}  // namespace

// Split partials of decode for callers that cannot allocate (tgvkv_decode_attn_noalloc):
// one buffer per GPU, living as long as the process.  Host code must not pass the array's
// name to a kernel (it is a host-side stand-in there); decode_scratch() gives its device
// address, looked up once per device with that device current.
static __device__ __align__(256) float scratch[kDecodeScratchBytes / sizeof(float)];

hipError_t decode_scratch(float** ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static float* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = static_cast<float*>(p);
    }
    *ptr = addr[dev];
    return hipSuccess;
}

int decode_splits(const Shape& s) {
    const long long units = (long long)s.B * s.L * s.Hkv;
    if (units <= 0) return 1;
    // split a unit's tokens only up to about 1024 workgroups (one round of 4 workgroups per
    // CU): a split costs partial writes and the combine launch (at the Qwen2-VL shape, 896
    // units: 40.8 us unsplit against 46.3 us in two splits; at the LLaVA-1.5 shape, 1024 units
    // at 5 %: 10.0 us per step replayed from a HIP graph unsplit against 17.2 us in two splits)
    long long n = 1024 / units;
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
